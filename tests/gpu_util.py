"""Helpers for the GPU parity tests: move seeded inputs to the device, run the library, and compare the
results with the oracle, tensor group by tensor group (so multi-GB models stream through host memory).
"""
import sys
import time

import numpy as np

import oracle
from paper_2609_34645_amd import emu
from synthetic import device_fill, host_tensor

NP_DTYPE = {"bf16": np.uint16, "fp32": np.float32}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _backings(views):
    """Group tensor views by the allocation they live in: {storage ptr: (whole-allocation uint8 tensor,
    [(byte offset, bytes) of each view])}."""
    import torch

    out = {}
    for v in views:
        st = v.untyped_storage()
        key = st.data_ptr()
        if key not in out:
            whole = torch.empty(0, dtype=torch.uint8, device=v.device).set_(st)
            out[key] = (whole, [])
        out[key][1].append((v.data_ptr() - key, v.numel() * v.element_size()))
    return out


def fingerprint(whole):
    """(sum of the 8-byte words, sum of word * (index + 1), tail bytes) of a uint8 device tensor, the
    sums modulo 2^64, computed on the device in slices."""
    import torch

    n8 = whole.numel() // 8 * 8
    words = whole[:n8].view(torch.int64)
    acc = torch.zeros(2, dtype=torch.int64, device=whole.device)
    step = 1 << 25
    for a in range(0, words.numel(), step):
        w = words[a:a + step]
        ramp = torch.arange(a + 1, a + 1 + w.numel(), dtype=torch.int64, device=whole.device)
        acc[0] += w.sum()
        acc[1] += (w * ramp).sum()
    return tuple(acc.cpu().tolist()) + (bytes(whole[n8:].cpu().numpy()),)


def _outside(nbytes, spans):
    """Byte ranges of [0, nbytes) that no span covers."""
    gaps, pos = [], 0
    for o, n in sorted(spans):
        if o > pos:
            gaps.append((pos, o))
        pos = max(pos, o + n)
    if pos < nbytes:
        gaps.append((pos, nbytes))
    return gaps


class Guard:
    """The write footprint of one library call, checked around it.

    ``keep``: views the call only reads (its source tensors or buckets). Their whole allocations --
    views, alignment gaps, guard bands, source pad rows -- must be byte-identical afterwards. The
    snapshot is a host copy (``snapshot="host"``), a device copy ("device", full-size tests), or for
    allocations too large to copy twice a device fingerprint ("hash": two 64-bit sums over the 8-byte
    words, one weighted by position, plus the tail bytes), which any changed word alters.
    ``fills``: (views, fill byte) pairs of what the call writes, in allocations prefilled with that byte.
    Every byte of those allocations outside the views must still hold the fill afterwards. Construction
    checks that the fill is there and that there are such bytes (a check on nothing proves nothing).

    Paper section 5.2 (a)/(b): Split and Merge leave the model state unchanged; section 6.2: each shard
    travels as one contiguous buffer, so nothing outside a destination shard or bucket is written."""

    def __init__(self, keep=(), fills=(), snapshot="host", label=""):
        import torch

        assert snapshot in ("host", "device", "hash")
        self.label = label
        self.mode = snapshot
        self.snaps = []
        for whole, _ in _backings(keep).values():
            snap = whole.cpu() if snapshot == "host" else whole.clone() if snapshot == "device" else fingerprint(whole)
            self.snaps.append((whole, snap))
        self.gaps = []
        for views, fill in fills:
            for whole, spans in _backings(views).values():
                ranges = _outside(whole.numel(), spans)
                assert ranges, f"{label}: an allocation of written views has no byte outside them"
                idx = torch.cat([torch.arange(a, b, device=whole.device) for a, b in ranges])
                got = whole[idx]
                assert bool((got == fill).all()), f"{label}: prefill {fill:#x} missing before the call"
                self.gaps.append((whole, idx, fill))

    def check(self):
        import torch

        for whole, snap in self.snaps:
            if self.mode == "hash":
                assert fingerprint(whole) == snap, f"{self.label}: a read-only allocation changed (fingerprint)"
                continue
            now = whole if snap.is_cuda else whole.cpu()
            if not torch.equal(now, snap):
                bad = torch.nonzero(now != snap).flatten()
                raise AssertionError(f"{self.label}: {bad.numel()} bytes of a read-only allocation changed, "
                                     f"first at byte {int(bad[0])}")
        for whole, idx, fill in self.gaps:
            got = whole[idx]
            if not bool((got == fill).all()):
                bad = idx[got != fill]
                raise AssertionError(f"{self.label}: {bad.numel()} bytes outside the written views changed, "
                                     f"first at byte {int(bad[0])} of its allocation")
        n = sum(idx.numel() for _, idx, _ in self.gaps)
        self.snaps = []
        return n


def o_layout(lay: emu.Layout) -> oracle.Layout:
    m = lay.model
    om = oracle.Model(m.num_layers, m.hidden, m.num_heads, m.head_dim, m.num_kv_heads, m.ffn_hidden, m.vocab)
    return oracle.Layout(om, lay.tp, lay.pp, lay.pad, lay.dtype, lay.qkv, lay.mlp)


def group_of(desc):
    if desc["kind"] == "embed":
        return "embed"
    if desc["kind"] in ("final_norm", "lm_head"):
        return "final"
    return desc["layer"]


def rank_first(descs):
    first = {}
    for i, d in enumerate(descs):
        first.setdefault(d["rank"], i)
    return first


def full_model(model: oracle.Model, seed: int, dtype="bf16"):
    full = {}
    for i, (_, key, shape, kind) in enumerate(oracle.logical_tensors(model)):
        full[key] = host_tensor(seed, (2, i), shape, "norm" if kind.endswith("norm") else "weight", dtype)
    return full


def upload_shards(shards, sset, tweak_replicas=True, tp=1):
    """Copy host shard arrays (oracle rank/position order) into a device ShardSet. With tweak_replicas,
    norm replicas on TP ranks > 0 are altered so that reading the wrong replica shows."""
    import torch

    gi = 0
    for r, rank in enumerate(shards):
        for a in rank:
            a = np.ascontiguousarray(a)
            if tweak_replicas and a.ndim == 1 and r % tp:
                a = (a.view(np.uint8) ^ np.uint8(0x3C)).view(a.dtype)
            sset.tensors[gi].copy_(torch.from_numpy(a.reshape(-1).view(np.uint8).copy()))
            gi += 1
    assert gi == len(sset.tensors)


def fill_device(plan, side, sset, seed, dtype="bf16", dist_override=None):
    descs = plan.tensors(side)
    dists = [dist_override or ("norm" if d["kind"].endswith("norm") else "weight") for d in descs]
    device_fill(sset.tensors, seed, dists, dtype, key_base=side)


def host_view(t, desc, dtype):
    a = t.cpu().numpy()
    return a.view(NP_DTYPE[dtype]).reshape(desc["shape"])


def check_reshard(plan, src_set, dst_set, groups=None, label=""):
    """Destination tensors == oracle.reshard_group(source tensors) for every (or the given) group.
    Element by element, compared as integers."""
    src, dst = plan.src, plan.dst
    os_, od = o_layout(src), o_layout(dst)
    sd, dd = plan.tensors(0), plan.tensors(1)
    sf, df = rank_first(sd), rank_first(dd)
    by_group = {}
    for i, d in enumerate(sd):
        by_group.setdefault(group_of(d), []).append(i)
    gl = oracle.groups(os_.model) if groups is None else groups
    t0 = time.time()
    n_checked = 0
    for g in gl:
        if sum(sd[i]["bytes"] for i in by_group[g]) > 1 << 30:
            say(f"  {label}: checking group {g}")
        cache = {i: host_view(src_set.tensors[i], sd[i], src.dtype) for i in by_group[g]}
        want = oracle.reshard_group(lambda r, j: cache[sf[r] + j], os_, od, g)
        for (r, j), w in want.items():
            i = df[r] + j
            got = host_view(dst_set.tensors[i], dd[i], dst.dtype)
            if not np.array_equal(got.view(np.uint8), np.ascontiguousarray(w).view(np.uint8)):
                bad = np.nonzero(got.reshape(-1).view(np.uint8) != np.ascontiguousarray(w).reshape(-1).view(np.uint8))[0]
                raise AssertionError(f"{label} group {g}: dst tensor {i} ({dd[i]['kind']}, rank {r}) differs at "
                                     f"{bad.size} bytes, first at byte {bad[0]}")
            n_checked += w.nbytes
    say(f"  {label}: {n_checked / 1e9:.3f} GB checked against the oracle in {time.time() - t0:.1f} s")
    return n_checked


def check_buckets(plan, side, B, tensor_sets_host, bucket_bufs, label=""):
    """Bucket contents == oracle.pack(rank tensors, B) for every rank. tensor_sets_host[r] is the list of
    the rank's expected tensors (host arrays) in canonical order."""
    import torch

    flat = torch.cat([b.reshape(-1) for b in bucket_bufs]).cpu().numpy() if bucket_bufs else np.zeros(0, np.uint8)
    k, off = 0, 0
    for r, tensors in enumerate(tensor_sets_host):
        for w in oracle.pack(tensors, B):
            got = flat[off:off + w.size]
            assert bucket_bufs[k].numel() == w.size, f"{label} bucket {k} size"
            if not np.array_equal(got, w):
                bad = np.nonzero(got != w)[0]
                raise AssertionError(f"{label} rank {r} bucket {k}: {bad.size} bytes differ, first at {bad[0]}")
            k += 1
            off += w.size
    assert k == len(bucket_bufs)


def check_upload(plan, label=""):
    """Upload `plan` into a zeroed workspace and compare it byte for byte with the host's image of it
    (emu_plan_workspace_image): the tables the upload's kernels derive on the device included."""
    import torch

    n = plan.info["workspace_bytes"]
    ws = torch.zeros(max(n, 256), dtype=torch.uint8, device="cuda")
    plan.upload(ws)
    torch.cuda.synchronize()
    got = ws[:n].cpu().numpy()
    want = np.frombuffer(plan.workspace_image(), np.uint8)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{label}: uploaded workspace differs from the host image at {bad.size} bytes, first {bad[0]}"
    return ws
