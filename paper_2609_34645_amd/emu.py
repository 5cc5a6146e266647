"""Python binding of libemu.so (the EMU Split/Merge reshard, C ABI in include/emu.h).

Argument marshalling only: every step of the reshard and of bucket pack/unpack runs in the library's
HIP kernels. PyTorch provides device memory, pointer tables and streams. There is no fallback: if the
library is not built, :func:`load` raises.

Typical use::

    src = Layout(model, tp=2, pp=2)
    dst = Layout(model, tp=4, pp=1)
    plan = Plan(src, dst)
    ws = plan.workspace()                      # uploads the plan tables to a fresh device buffer
    S = plan.alloc(0); D = plan.alloc(1)       # one buffer per rank, tensors as views
    plan.reshard(ws, S.ptrs, D.ptrs)           # enqueued on torch's current stream
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libemu.so")

BF16, FP32 = 0, 1
QKV_HEAD_INTERLEAVED, QKV_SEPARATE = 0, 1
GATE_UP_BLOCK, GATE_UP_SEPARATE = 0, 1
DTYPES = {"bf16": BF16, "fp32": FP32}
ESIZE = {BF16: 2, FP32: 4}

(OPT_TILE_VECS, OPT_XCD_REMAP, OPT_NONTEMPORAL, OPT_LDS_STAGING, OPT_BUCKET_WG_PER_CU, OPT_BUCKET_TILES,
 OPT_WG_PER_CU, OPT_ROW_WRAP) = range(8)

KINDS = ["embed", "attn_norm", "qkv", "q", "k", "v", "o", "mlp_norm", "gate_up", "gate", "up", "down",
         "final_norm", "lm_head", "bucket"]

STATUS = {0: "EMU_OK", -1: "EMU_ERR_NULL", -2: "EMU_ERR_LAYOUT", -3: "EMU_ERR_MISMATCH",
          -4: "EMU_ERR_UNSUPPORTED", -5: "EMU_ERR_WORKSPACE", -6: "EMU_ERR_BUCKET", -7: "EMU_ERR_ALIGN",
          -8: "EMU_ERR_HIP", -9: "EMU_ERR_HANDLE", -10: "EMU_ERR_RANGE", -11: "EMU_ERR_ARG",
          -12: "EMU_ERR_INFEASIBLE", -13: "EMU_ERR_OVERLAP"}
STATUS_CODE = {v: k for k, v in STATUS.items()}
ERR_INFEASIBLE = -12
ERR_OVERLAP = -13


class c_model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("num_layers", "hidden", "num_heads", "num_kv_heads", "head_dim", "ffn_hidden", "vocab")]


class c_layout(ctypes.Structure):
    _fields_ = [("model", c_model)] + [(n, ctypes.c_int32) for n in
                                       ("tp", "pp", "vocab_pad_multiple", "dtype", "qkv_format", "mlp_format")]


class c_plan_info(ctypes.Structure):
    _fields_ = [("n_src_ranks", ctypes.c_int32), ("n_dst_ranks", ctypes.c_int32),
                ("n_src_tensors", ctypes.c_int32), ("n_dst_tensors", ctypes.c_int32),
                ("n_segments", ctypes.c_int64), ("n_zero_segments", ctypes.c_int64),
                ("n_tiles", ctypes.c_int64), ("tile_bytes", ctypes.c_uint64),
                ("bytes_read", ctypes.c_uint64), ("bytes_written", ctypes.c_uint64),
                ("zero_fill_bytes", ctypes.c_uint64), ("src_bytes", ctypes.c_uint64),
                ("dst_bytes", ctypes.c_uint64), ("workspace_bytes", ctypes.c_uint64),
                ("src_vocab_padded", ctypes.c_int32), ("dst_vocab_padded", ctypes.c_int32),
                ("n_general_segments", ctypes.c_int32), ("converts", ctypes.c_int32),
                ("n_alias_tensors", ctypes.c_int32), ("aliased", ctypes.c_int32), ("alias_bytes", ctypes.c_uint64)]


class c_tensor_desc(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("kind", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("ndim", ctypes.c_int32), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("bytes", ctypes.c_uint64), ("stream_offset", ctypes.c_uint64), ("alias", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class c_bucket_desc(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("reserved", ctypes.c_int32), ("index", ctypes.c_uint64),
                ("stream_offset", ctypes.c_uint64), ("bytes", ctypes.c_uint64)]


class c_segment(ctypes.Structure):
    _fields_ = [("src_tensor", ctypes.c_int32), ("dst_tensor", ctypes.c_int32),
                ("src_offset", ctypes.c_uint64), ("dst_offset", ctypes.c_uint64),
                ("src_stride", ctypes.c_uint64), ("dst_stride", ctypes.c_uint64),
                ("rows", ctypes.c_uint64), ("run", ctypes.c_uint64), ("src_run", ctypes.c_uint64)]


class c_stage_transition(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("tp", ctypes.c_int32), ("pp", ctypes.c_int32), ("dp", ctypes.c_int32),
                ("tgt_tp", ctypes.c_int32), ("tgt_pp", ctypes.c_int32), ("tgt_dp", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("gpus", ctypes.POINTER(ctypes.c_int32)),
                ("tgt_gpus", ctypes.POINTER(ctypes.c_int32)), ("state_bytes", ctypes.c_double)]


class c_link_model(ctypes.Structure):
    _fields_ = [("gpus_per_node", ctypes.c_int32), ("reserved", ctypes.c_int32), ("intra_bw", ctypes.c_double),
                ("inter_bw", ctypes.c_double), ("hbm_bw", ctypes.c_double), ("setup_s", ctypes.c_double)]


class c_dag_node(ctypes.Structure):
    _fields_ = [("prim", ctypes.c_int32), ("stage", ctypes.c_int32), ("unit", ctypes.c_int32), ("src", ctypes.c_int32),
                ("gpu_first", ctypes.c_int32), ("n_gpus", ctypes.c_int32), ("cost_s", ctypes.c_double),
                ("start_s", ctypes.c_double), ("finish_s", ctypes.c_double)]


class c_dag_edge(ctypes.Structure):
    _fields_ = [("from_", ctypes.c_int32), ("to", ctypes.c_int32), ("resource", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class c_dag_info(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32), ("n_resource_edges", ctypes.c_int32),
                ("n_gpu_entries", ctypes.c_int32), ("l_tran_s", ctypes.c_double), ("plan_ms", ctypes.c_double)]


class EmuError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


_lib = None


def load(path: str = LIB_PATH):
    """Load libemu.so (once). Raises if it has not been built: there is no other implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_34645_amd.build`")
    # torch ships its own HIP runtime, with the same soname as the system one libemu.so links against, but
    # its libraries ask for it by the unversioned name. Loaded first, torch's copy satisfies libemu.so's
    # dependency; loaded after libemu.so, torch would bring in a second HIP runtime in the same process,
    # and the first one to lose the device reports none. The binding's buffers and streams are torch's, so
    # torch's runtime is the one to share.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, V, I32, I64, U64 = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "emu_version": ([], ctypes.c_int),
        "emu_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "emu_last_error": ([], ctypes.c_char_p),
        "emu_set_option": ([I32, I64], ctypes.c_int),
        "emu_get_option": ([I32, ctypes.POINTER(I64)], ctypes.c_int),
        "emu_layout_check": ([ctypes.POINTER(c_layout)], ctypes.c_int),
        "emu_plan": ([ctypes.POINTER(c_layout), ctypes.POINTER(c_layout), ctypes.POINTER(P)], ctypes.c_int),
        "emu_plan_ex": ([ctypes.POINTER(c_layout), ctypes.POINTER(c_layout), ctypes.c_uint32, ctypes.POINTER(P)],
                        ctypes.c_int),
        "emu_plan_to_buckets": ([ctypes.POINTER(c_layout), ctypes.POINTER(c_layout), U64, ctypes.POINTER(P)],
                                ctypes.c_int),
        "emu_plan_from_buckets": ([ctypes.POINTER(c_layout), ctypes.POINTER(c_layout), U64, ctypes.POINTER(P)],
                                  ctypes.c_int),
        "emu_plan_free": ([P], ctypes.c_int),
        "emu_plan_info": ([P, ctypes.POINTER(c_plan_info)], ctypes.c_int),
        "emu_tensor_info": ([P, I32, I32, ctypes.POINTER(c_tensor_desc)], ctypes.c_int),
        "emu_plan_segments": ([P, I64, I64, ctypes.POINTER(c_segment)], ctypes.c_int),
        "emu_plan_upload": ([P, V, U64, V], ctypes.c_int),
        "emu_plan_workspace_image": ([P, V, U64], ctypes.c_int),
        "emu_reshard": ([P, V, V, V, V], ctypes.c_int),
        "emu_reshard_noalloc": ([P, V, V, V], ctypes.c_int),
        "emu_reshard_groups": ([P, V, I32, V, V, V], ctypes.c_int),
        "emu_bucket_info": ([P, I32, U64, U64, U64, ctypes.POINTER(c_bucket_desc)], ctypes.c_int),
        "emu_bucket_layout": ([P, I32, U64, I32, ctypes.POINTER(U64), ctypes.POINTER(U64)], ctypes.c_int),
        "emu_pack_buckets": ([P, V, I32, U64, V, V, V], ctypes.c_int),
        "emu_unpack_buckets": ([P, V, I32, U64, V, V, V], ctypes.c_int),
        "emu_check_tables": ([P, ctypes.POINTER(U64), ctypes.POINTER(U64)], ctypes.c_int),
        "emu_check_bucket_tables": ([P, I32, U64, ctypes.POINTER(U64), ctypes.POINTER(U64)], ctypes.c_int),
        "emu_dag_plan": ([ctypes.POINTER(c_stage_transition), I32, ctypes.POINTER(c_link_model), ctypes.POINTER(P)],
                         ctypes.c_int),
        "emu_dag_free": ([P], ctypes.c_int),
        "emu_dag_info": ([P, ctypes.POINTER(c_dag_info)], ctypes.c_int),
        "emu_dag_nodes": ([P, I32, I32, ctypes.POINTER(c_dag_node)], ctypes.c_int),
        "emu_dag_edges": ([P, I32, I32, ctypes.POINTER(c_dag_edge)], ctypes.c_int),
        "emu_dag_gpus": ([P, I32, I32, ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
        "emu_dag_target_unit": ([P, I32, I32, ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def check(rc: int) -> None:
    if rc != 0:
        raise EmuError(rc, load().emu_last_error().decode())


def set_option(key: int, value: int) -> None:
    check(load().emu_set_option(key, value))


def get_option(key: int) -> int:
    v = ctypes.c_int64()
    check(load().emu_get_option(key, ctypes.byref(v)))
    return v.value


@dataclass(frozen=True)
class Model:
    num_layers: int
    hidden: int
    num_heads: int
    head_dim: int
    num_kv_heads: int
    ffn_hidden: int
    vocab: int

    @classmethod
    def from_tuple(cls, t):
        """(L, H, nH, hd, G, I, V)."""
        return cls(*t)


@dataclass(frozen=True)
class Layout:
    model: Model
    tp: int
    pp: int
    pad: int = 0
    dtype: str = "bf16"
    qkv: str = "interleaved"
    mlp: str = "block"

    def __post_init__(self):
        if self.dtype not in DTYPES:
            raise ValueError(f"dtype must be one of {sorted(DTYPES)}, not {self.dtype!r}")
        if self.qkv not in ("interleaved", "separate"):
            raise ValueError(f"qkv must be 'interleaved' or 'separate', not {self.qkv!r}")
        if self.mlp not in ("block", "separate"):
            raise ValueError(f"mlp must be 'block' or 'separate', not {self.mlp!r}")

    def c(self) -> c_layout:
        m = self.model
        return c_layout(c_model(m.num_layers, m.hidden, m.num_heads, m.num_kv_heads, m.head_dim, m.ffn_hidden,
                                m.vocab), self.tp, self.pp, self.pad, DTYPES[self.dtype],
                        QKV_HEAD_INTERLEAVED if self.qkv == "interleaved" else QKV_SEPARATE,
                        GATE_UP_BLOCK if self.mlp == "block" else GATE_UP_SEPARATE)


def layout_check(lay: Layout) -> int:
    c = lay.c()
    return load().emu_layout_check(ctypes.byref(c))


def _stream_handle(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class ShardSet:
    """One side's tensors on the device: the backing buffers, the tensors and their pointer table.

    ``tensors[i]`` is a uint8 view of tensor i's bytes, ``ptrs`` the device pointer table (int64) in
    global tensor order. ``Plan.alloc`` makes one buffer per rank with 256-byte aligned views; the
    library itself needs only 16-byte aligned tensors.
    """

    def __init__(self, bufs, tensors, ptrs):
        self.bufs = bufs
        self.tensors = tensors
        self.ptrs = ptrs


class Plan:
    """A compiled copy map between two layouts (``emu_plan``)."""

    def __init__(self, src: Layout, dst: Layout, bucket_bytes: int = 0, alias: bool = False,
                 src_bucket_bytes: int = 0):
        """bucket_bytes > 0 compiles the fused map (``emu_plan_to_buckets``): its destination side is
        the destination ranks' buckets of that size. src_bucket_bytes > 0 compiles the receiver's map
        (``emu_plan_from_buckets``): its source side is the source ranks' buckets of that size. alias=True
        leaves destination tensors that are byte copies of a whole source tensor out of the map
        (``emu_plan_ex`` with EMU_PLAN_ALIAS_RESIDENT); ``alloc(1, alias=S)`` makes them views of the
        source set S."""
        lib = load()
        self.src, self.dst, self.bucket_bytes, self.src_bucket_bytes = src, dst, bucket_bytes, src_bucket_bytes
        self._uploads = {}  # data_ptr -> workspace tensor this plan uploaded to (kept alive)
        cs, cd = src.c(), dst.c()
        h = ctypes.c_void_p()
        if (bucket_bytes or src_bucket_bytes) and alias:
            raise ValueError("a bucket plan has buckets on one side: nothing to alias")
        if bucket_bytes and src_bucket_bytes:
            raise ValueError("give bucket_bytes (destination buckets) or src_bucket_bytes (source buckets), not both")
        if bucket_bytes:
            check(lib.emu_plan_to_buckets(ctypes.byref(cs), ctypes.byref(cd), bucket_bytes, ctypes.byref(h)))
        elif src_bucket_bytes:
            check(lib.emu_plan_from_buckets(ctypes.byref(cs), ctypes.byref(cd), src_bucket_bytes, ctypes.byref(h)))
        else:
            check(lib.emu_plan_ex(ctypes.byref(cs), ctypes.byref(cd), 1 if alias else 0, ctypes.byref(h)))
        self._h = h
        info = c_plan_info()
        check(lib.emu_plan_info(h, ctypes.byref(info)))
        self.info = {f: getattr(info, f) for f, _ in c_plan_info._fields_}
        self._descs = [None, None]
        self._n = (self.info["n_src_tensors"], self.info["n_dst_tensors"])
        self._nbuckets = {}  # (side, bucket_bytes) -> bucket count of the side (a plan never changes)

    # -- host queries ------------------------------------------------------------------------
    def tensors(self, side: int) -> list:
        """Per tensor of one side (0 = source, 1 = destination): dict(rank, kind, layer, shape, bytes,
        stream_offset)."""
        if self._descs[side] is None:
            lib = load()
            n = self.info["n_src_tensors" if side == 0 else "n_dst_tensors"]
            out = []
            d = c_tensor_desc()
            for i in range(n):
                check(lib.emu_tensor_info(self._h, side, i, ctypes.byref(d)))
                shape = (d.cols,) if d.ndim == 1 else (d.rows, d.cols)
                if d.kind == 14:
                    shape = (d.bytes,)
                out.append(dict(rank=d.rank, kind=KINDS[d.kind], layer=d.layer, shape=shape, bytes=d.bytes,
                                stream_offset=d.stream_offset, alias=d.alias))
            self._descs[side] = out
        return self._descs[side]

    def segments(self) -> list:
        n = self.info["n_segments"]
        arr = (c_segment * max(1, n))()
        check(load().emu_plan_segments(self._h, 0, n, arr))
        return [{f: getattr(arr[i], f) for f, _ in c_segment._fields_} for i in range(n)]

    def bucket_layout(self, side: int, bucket_bytes: int, rank: int = -1):
        nb, sb = ctypes.c_uint64(), ctypes.c_uint64()
        check(load().emu_bucket_layout(self._h, side, bucket_bytes, rank, ctypes.byref(nb), ctypes.byref(sb)))
        return nb.value, sb.value

    def bucket_info(self, side: int, bucket_bytes: int) -> list:
        """Every bucket of one side (``emu_bucket_info``), in pointer-table order: dict(rank, index,
        stream_offset, bytes)."""
        n = self.bucket_layout(side, bucket_bytes, -1)[0]
        arr = (c_bucket_desc * max(1, n))()
        check(load().emu_bucket_info(self._h, side, bucket_bytes, 0, n, arr))
        return [dict(rank=b.rank, index=b.index, stream_offset=b.stream_offset, bytes=b.bytes) for b in arr[:n]]

    def workspace_image(self) -> bytes:
        """The workspace bytes the upload produces, computed on the host (zero between tables)."""
        n = self.info["workspace_bytes"]
        buf = ctypes.create_string_buffer(max(n, 1))
        check(load().emu_plan_workspace_image(self._h, buf, n))
        return buf.raw[:n]

    # -- device helpers (plumbing) -------------------------------------------------------------
    def workspace(self, device=None, stream=None):
        """Allocate a workspace tensor and enqueue the plan upload into it."""
        import torch

        n = self.info["workspace_bytes"]
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device=device or "cuda")
        self.upload(ws, stream)
        return ws

    def upload(self, ws, stream=None):
        """Upload the plan tables into `ws`. The plan keeps `ws` alive, so its address cannot be handed to
        another buffer while the plan may still name it; execute calls accept only workspaces this plan
        uploaded to (the library also refuses one that another plan has overwritten since)."""
        check(load().emu_plan_upload(self._h, ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream_handle(stream)))
        self._uploads[ws.data_ptr()] = ws

    def alloc(self, side: int, device=None, fill=None, guard: int = 0, alias: ShardSet = None) -> ShardSet:
        """Allocate one side's shard set (one buffer per rank, 256-byte aligned tensor views). With
        guard > 0, at least that many bytes separate consecutive views and precede the first and follow
        the last, so that bytes a call must not touch surround every tensor (tests prefill them). With
        alias=S (destination side of an alias plan), every alias tensor is S's source tensor itself and
        gets no bytes of its own."""
        import torch

        descs = self.tensors(side)
        if alias is not None and (side != 1 or not self.info["aliased"]):
            raise ValueError("alias= needs the destination side of a plan made with alias=True")
        own = [alias is None or d["alias"] < 0 for d in descs]
        nranks = self.info["n_src_ranks" if side == 0 else "n_dst_ranks"]
        offs, sizes = [], [0] * nranks
        for d, mine in zip(descs, own):
            o = (sizes[d["rank"]] + guard + 255) // 256 * 256 if mine else -1
            offs.append(o)
            if mine:
                sizes[d["rank"]] = o + d["bytes"]
        bufs = [torch.empty(max(s + guard, 16), dtype=torch.uint8, device=device or "cuda") for s in sizes]
        if fill is not None:
            for b in bufs:
                b.fill_(fill)
        tensors = [bufs[d["rank"]][o:o + d["bytes"]] if mine else alias.tensors[d["alias"]]
                   for d, o, mine in zip(descs, offs, own)]
        return ShardSet(bufs, tensors, ptr_table(tensors, device))

    def region_bytes(self, side: int) -> int:
        """Bytes ``views`` needs to lay out one side's tensors back to back (256-byte aligned)."""
        end = 0
        for d in self.tensors(side):
            end = (end + 255) // 256 * 256 + d["bytes"]
        return end

    def views(self, side: int, region, device=None, alias: ShardSet = None) -> ShardSet:
        """One side's tensors as 256-byte aligned views laid out back to back in a caller-provided uint8
        device tensor of at least ``region_bytes(side)`` bytes (several plans may place their tensors in one
        region, so that their launches touch the same memory pages). alias=S as for ``alloc``."""
        need = self.region_bytes(side)
        if region.numel() < need:
            raise ValueError(f"region of {region.numel()} bytes, the side needs {need}")
        if alias is not None and (side != 1 or not self.info["aliased"]):
            raise ValueError("alias= needs the destination side of a plan made with alias=True")
        tensors, end = [], 0
        for d in self.tensors(side):
            if alias is not None and d["alias"] >= 0:
                tensors.append(alias.tensors[d["alias"]])
                continue
            o = (end + 255) // 256 * 256
            tensors.append(region[o:o + d["bytes"]])
            end = o + d["bytes"]
        return ShardSet([region], tensors, ptr_table(tensors, device))

    def bucket_region_bytes(self, side: int, bucket_bytes: int) -> int:
        """Bytes ``bucket_views`` needs for one side's buckets of size bucket_bytes."""
        end = 0
        for b in self.bucket_info(side, bucket_bytes):
            end = (end + 255) // 256 * 256 + b["bytes"]
        return end

    def bucket_views(self, side: int, bucket_bytes: int, region, device=None):
        """One side's buckets of size bucket_bytes as 256-byte aligned views back to back in `region`
        (as ``views``); returns (buckets, pointer table)."""
        bufs, end = [], 0
        for b in self.bucket_info(side, bucket_bytes):
            o = (end + 255) // 256 * 256
            if o + b["bytes"] > region.numel():
                raise ValueError("region too small for the buckets")
            bufs.append(region[o:o + b["bytes"]])
            end = o + b["bytes"]
        return bufs, ptr_table(bufs, device)

    def alloc_buckets(self, side: int, bucket_bytes: int, device=None, fill=None, guard: int = 0):
        """Bucket buffers for one side (rank 0's first) and their pointer table. The buckets are
        256-byte aligned views of one backing allocation, separated by at least `guard` bytes (as in
        ``alloc``)."""
        import torch

        sizes = [b["bytes"] for b in self.bucket_info(side, bucket_bytes)]
        offs, total = [], 0
        for n in sizes:
            o = (total + guard + 255) // 256 * 256
            offs.append(o)
            total = o + n
        backing = torch.empty(max(total + guard, 256), dtype=torch.uint8, device=device or "cuda")
        if fill is not None:
            backing.fill_(fill)
        bufs = [backing[o:o + n] for o, n in zip(offs, sizes)]
        return bufs, ptr_table(bufs, device)

    # -- execution -----------------------------------------------------------------------------
    def shard_set(self, side: int, tensors, device=None) -> ShardSet:
        """A ShardSet over the caller's own tensors of one side, in the plan's global order (rank 0's
        first, canonical order within a rank; ``tensors(side)`` lists them). Each must be a contiguous
        device tensor of exactly the plan's byte size for it, 16-byte aligned: the kernels trust the
        pointer table, so a tensor of the wrong size would be written past its end. Raises ValueError
        (EmuError -7 for alignment) before anything reaches the library."""
        descs = self.tensors(side)
        tensors = list(tensors)
        if len(tensors) != len(descs):
            raise ValueError(f"side {side} has {len(descs)} tensors, {len(tensors)} given")
        _check_buffers(tensors, [d["bytes"] for d in descs], lambda i: f"{descs[i]['kind']} (rank {descs[i]['rank']})")
        views = [t.view(-1).view(_uint8()) for t in tensors]
        return ShardSet(tensors, views, ptr_table(tensors, device))

    def bucket_set(self, side: int, bucket_bytes: int, buffers, device=None):
        """(views, pointer table) over the caller's own bucket buffers of one side for bucket size
        bucket_bytes, in pointer-table order (``bucket_info``): each a contiguous device tensor of exactly
        its bucket's bytes, 16-byte aligned; checked as in ``shard_set``."""
        info = self.bucket_info(side, bucket_bytes)
        buffers = list(buffers)
        if len(buffers) != len(info):
            raise ValueError(f"side {side} has {len(info)} buckets of {bucket_bytes} bytes, {len(buffers)} given")
        _check_buffers(buffers, [b["bytes"] for b in info], lambda i: f"bucket {info[i]['index']} of rank {info[i]['rank']}")
        return [b.view(-1).view(_uint8()) for b in buffers], ptr_table(buffers, device)

    def reshard(self, ws, src_ptrs, dst_ptrs, stream=None):
        self._tables(ws, (src_ptrs, self._n[0], "src_ptrs"), (dst_ptrs, self._n[1], "dst_ptrs"))
        check(load().emu_reshard(self._h, ctypes.c_void_p(ws.data_ptr()), ctypes.c_void_p(src_ptrs.data_ptr()),
                                 ctypes.c_void_p(dst_ptrs.data_ptr()), _stream_handle(stream)))

    def reshard_groups(self, ws, src_tables, dst_tables, stream=None):
        """``emu_reshard_groups``: one launch over several shard sets of this plan's layouts. src_tables
        and dst_tables are int64 device tensors holding the groups' pointer tables back to back
        (``group_tables``)."""
        ns, nd = self.info["n_src_tensors"], self.info["n_dst_tensors"]
        n = src_tables.numel() // ns if ns else 0
        self._tables(ws, (src_tables, n * ns, "src_tables"), (dst_tables, n * nd, "dst_tables"))
        check(load().emu_reshard_groups(self._h, ctypes.c_void_p(ws.data_ptr()), n,
                                        ctypes.c_void_p(src_tables.data_ptr()), ctypes.c_void_p(dst_tables.data_ptr()),
                                        _stream_handle(stream)))

    def reshard_noalloc(self, src_ptrs, dst_ptrs, stream=None):
        """``emu_reshard_noalloc``: the reshard with the plan tables in the library's static device array
        (no workspace; nothing allocated by the call)."""
        self._tables(None, (src_ptrs, self.info["n_src_tensors"], "src_ptrs"),
                     (dst_ptrs, self.info["n_dst_tensors"], "dst_ptrs"))
        check(load().emu_reshard_noalloc(self._h, ctypes.c_void_p(src_ptrs.data_ptr()),
                                         ctypes.c_void_p(dst_ptrs.data_ptr()), _stream_handle(stream)))

    def _tables(self, ws, *tables):
        """Refuse, before any library call, pointer tables the kernels would read past the end of:
        each must be an int64 device tensor with exactly the entries the plan indexes."""
        for t, n, what in tables:
            if str(getattr(t, "dtype", None)) != "torch.int64":
                raise ValueError(f"{what} must be an int64 tensor (emu.ptr_table), not {type(t).__name__}")
            if t.numel() != n or (n and not t.is_contiguous()):
                raise ValueError(f"{what} has {t.numel()} entries, the plan needs {n} (contiguous)")
        for t, _, what in tables:
            if not t.is_cuda:
                raise ValueError(f"{what} must be a device tensor")
        if ws is not None:
            if not getattr(ws, "is_cuda", False):
                raise ValueError("the workspace must be a device tensor")
            if ws.data_ptr() not in self._uploads:
                raise EmuError(-5, f"workspace at {ws.data_ptr():#x} holds no upload of this plan (Plan.upload)")

    def _bucket_tables(self, ws, side, bucket_bytes, tensor_ptrs, bucket_ptrs):
        if side not in (0, 1):
            raise ValueError("side must be 0 or 1")
        if bucket_bytes < 0:
            raise ValueError("bucket_bytes must be positive")
        nb = self._nbuckets.get((side, bucket_bytes))
        if nb is None:
            es = ESIZE[DTYPES[(self.src if side == 0 else self.dst).dtype]]
            if bucket_bytes == 0 or bucket_bytes % es:
                return  # the library refuses the size (EMU_ERR_BUCKET) before launching anything
            nb = self._nbuckets[(side, bucket_bytes)] = self.bucket_layout(side, bucket_bytes, -1)[0]
        self._tables(ws, (tensor_ptrs, self._n[side], "tensor_ptrs"), (bucket_ptrs, nb, "bucket_ptrs"))

    def pack(self, ws, side, bucket_bytes, tensor_ptrs, bucket_ptrs, stream=None):
        self._bucket_tables(ws, side, bucket_bytes, tensor_ptrs, bucket_ptrs)
        check(load().emu_pack_buckets(self._h, ctypes.c_void_p(ws.data_ptr()), side, bucket_bytes,
                                      ctypes.c_void_p(tensor_ptrs.data_ptr()), ctypes.c_void_p(bucket_ptrs.data_ptr()),
                                      _stream_handle(stream)))

    def unpack(self, ws, side, bucket_bytes, bucket_ptrs, tensor_ptrs, stream=None):
        self._bucket_tables(ws, side, bucket_bytes, tensor_ptrs, bucket_ptrs)
        check(load().emu_unpack_buckets(self._h, ctypes.c_void_p(ws.data_ptr()), side, bucket_bytes,
                                        ctypes.c_void_p(bucket_ptrs.data_ptr()), ctypes.c_void_p(tensor_ptrs.data_ptr()),
                                        _stream_handle(stream)))

    # -- host-side table checks ------------------------------------------------------------------
    def check_tables(self, src_ptrs, dst_ptrs):
        """``emu_check_tables`` on host copies of two pointer tables (int sequences or int64 tensors)."""
        check(load().emu_check_tables(self._h, _u64_array(src_ptrs), _u64_array(dst_ptrs)))

    def check_bucket_tables(self, side, bucket_bytes, tensor_ptrs, bucket_ptrs):
        """``emu_check_bucket_tables`` on host copies of a side's tensor table and its bucket table."""
        check(load().emu_check_bucket_tables(self._h, side, bucket_bytes, _u64_array(tensor_ptrs),
                                             _u64_array(bucket_ptrs)))

    def close(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            check(_lib.emu_plan_free(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _u64_array(ptrs):
    """A ctypes uint64 array from a sequence of ints or an int64 tensor (copied to the host)."""
    if hasattr(ptrs, "cpu"):
        ptrs = ptrs.cpu().tolist()
    vals = [int(x) & 0xFFFFFFFFFFFFFFFF for x in ptrs]
    return (ctypes.c_uint64 * max(1, len(vals)))(*vals)


def _uint8():
    import torch

    return torch.uint8


def _check_buffers(bufs, sizes, name):
    """Each buffer contiguous, of exactly its size in bytes, 16-byte aligned, on the device (in that
    order, so that the host-side conditions are checked before the device one)."""
    for i, (t, n) in enumerate(zip(bufs, sizes)):
        nbytes = t.numel() * t.element_size()
        if nbytes != n:
            raise ValueError(f"{name(i)}: {nbytes} bytes, the plan needs {n}")
        if not t.is_contiguous():
            raise ValueError(f"{name(i)}: not contiguous")
        if t.data_ptr() % 16:
            raise EmuError(-7, f"{name(i)}: address {t.data_ptr():#x} is not 16-byte aligned")
    for i, t in enumerate(bufs):
        if not t.is_cuda:
            raise ValueError(f"{name(i)}: not a device tensor")


def group_tables(sets, device=None):
    """Back-to-back device pointer table of several ShardSets (for ``Plan.reshard_groups``)."""
    import torch

    return torch.cat([s.ptrs for s in sets]).to(device or "cuda")


def ptr_table(tensors, device=None):
    """Device int64 table of the tensors' addresses; every address must be 16-byte aligned."""
    import torch

    addrs = [t.data_ptr() for t in tensors]
    bad = [i for i, a in enumerate(addrs) if a % 16]
    if bad:
        raise EmuError(-7, f"tensors {bad[:4]} are not 16-byte aligned")
    return torch.tensor(addrs, dtype=torch.int64, device=device or "cuda")


# ----------------------------------------------------------------------------------------------------
# transition-DAG planner (host only)
# ----------------------------------------------------------------------------------------------------

PRIMS = ["split", "destroy", "extend", "merge"]


def dag_plan(stages, gpus_per_node=8, intra_bw=300e9, inter_bw=25e9, hbm_bw=5e12, setup_s=0.05):
    """Plan a transition (``emu_dag_plan``). ``stages``: sequence of dicts with kind (0 generation,
    1 inference, 2 training), tp, pp, dp, gpus, tgt_tp, tgt_pp, tgt_dp, tgt_gpus, state_bytes.

    Returns dict(nodes=[dict(prim, stage, unit, src, gpus, cost, start, finish)], edges=[(from, to,
    resource)], target_units=[[gpu list per target unit] per stage], l_tran, n_resource_edges, plan_ms).
    Raises EmuError (code ERR_INFEASIBLE when no deadlock-free DAG exists)."""
    lib = load()
    n = len(stages)
    arr = (c_stage_transition * n)()
    keep = []
    for i, s in enumerate(stages):
        # the C call reads dp*tp*pp (tgt_dp*tgt_tp*tgt_pp) ids; shorter lists would be read past their end
        if len(s["gpus"]) != s["dp"] * s["tp"] * s["pp"] or \
                len(s["tgt_gpus"]) != s["tgt_dp"] * s["tgt_tp"] * s["tgt_pp"]:
            raise EmuError(-11, f"stage {i}: GPU lists must hold dp*tp*pp ids (current and target)")
        g = (ctypes.c_int32 * len(s["gpus"]))(*s["gpus"])
        tg = (ctypes.c_int32 * len(s["tgt_gpus"]))(*s["tgt_gpus"])
        keep += [g, tg]
        arr[i] = c_stage_transition(s["kind"], s["tp"], s["pp"], s["dp"], s["tgt_tp"], s["tgt_pp"], s["tgt_dp"], 0,
                                    g, tg, float(s["state_bytes"]))
    links = c_link_model(gpus_per_node, 0, intra_bw, inter_bw, hbm_bw, setup_s)
    h = ctypes.c_void_p()
    check(lib.emu_dag_plan(arr, n, ctypes.byref(links), ctypes.byref(h)))
    try:
        info = c_dag_info()
        check(lib.emu_dag_info(h, ctypes.byref(info)))
        nodes = (c_dag_node * max(1, info.n_nodes))()
        edges = (c_dag_edge * max(1, info.n_edges))()
        flat = (ctypes.c_int32 * max(1, info.n_gpu_entries))()
        check(lib.emu_dag_nodes(h, 0, info.n_nodes, nodes))
        check(lib.emu_dag_edges(h, 0, info.n_edges, edges))
        check(lib.emu_dag_gpus(h, 0, info.n_gpu_entries, flat))
        out_nodes = [dict(prim=nd.prim, stage=nd.stage, unit=nd.unit, src=nd.src,
                          gpus=list(flat[nd.gpu_first:nd.gpu_first + nd.n_gpus]), cost=nd.cost_s,
                          start=nd.start_s, finish=nd.finish_s) for nd in nodes[:info.n_nodes]]
        out_edges = [(ed.from_, ed.to, ed.resource) for ed in edges[:info.n_edges]]
        units = []
        for i, s in enumerate(stages):
            per = []
            for u in range(s["tgt_dp"]):
                buf = (ctypes.c_int32 * (s["tgt_tp"] * s["tgt_pp"]))()
                check(lib.emu_dag_target_unit(h, i, u, buf))
                per.append(list(buf))
            units.append(per)
        return dict(nodes=out_nodes, edges=out_edges, target_units=units, l_tran=info.l_tran_s,
                    n_resource_edges=info.n_resource_edges, plan_ms=info.plan_ms)
    finally:
        lib.emu_dag_free(h)
