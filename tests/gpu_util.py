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
