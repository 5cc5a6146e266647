"""Run hot-path kernels once each, for hardware-counter profiling (rocprofv3 --pmc) and kernel traces.

Every workload starts with a plain elementwise copy of known size (a torch uint8 add of 0: N bytes read
and N written), which calibrates FETCH_SIZE / WRITE_SIZE. Workloads (--workload):

  main     8B decoder bf16 TP2 PP2 -> TP4 PP1: one emu_reshard, one emu_pack_buckets (2^28-byte
           buckets), one emu_unpack_buckets; then the converting reshards fp32 TP4 PP1 -> bf16 TP2 PP2
           (the weight sync) and bf16 TP2 PP2 -> fp32 TP4 PP1.
  shifted  8B decoder bf16, vocabulary padded to TP*128, TP8 PP4 -> TP2 PP2: one emu_reshard, then
           --repeat rounds of pack and unpack at 2^28-byte buckets and at 2^28 - 2 (every bucket at
           another 16-byte phase), the two bucket sets on the same pages: pack B, unpack B, pack B - 2,
           unpack B - 2 per round.
  formats  8B TP2 PP2 -> TP4 PP1 into fused q/k/v and gate/up tensors, then into separate ones, on the
           same source and destination pages, --repeat times each, alternating.
  receiver 8B TP2 PP2 source set packed into 2^28-byte buckets (emu_pack_buckets, source side), then
           the receiver plan (emu_plan_from_buckets) resharding those buckets into TP4 PP1 tensors.

Example (from /tmp with TMPDIR=/tmp):

    rocprofv3 --pmc FETCH_SIZE -d out -o pmc_fetch -- python3 $R/profile_once.py --workload shifted
"""
import argparse
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

EIGHT_B = (32, 4096, 32, 128, 8, 14336, 128256)


def calibrate(torch, a, b):
    """Plain copies of known size: min(len) bytes of a into b per pair."""
    n = 0
    for x, y in zip(a, b):
        k = min(x.numel(), y.numel())
        torch.add(x[:k], 0, out=y[:k])
        n += k
    torch.cuda.synchronize()
    return n


def main_workload(torch, emu, device_fill):
    m = emu.Model(*EIGHT_B)
    plan = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1))
    ws = plan.workspace()
    S, D, R = plan.alloc(0), plan.alloc(1), plan.alloc(1)
    B = 1 << 28
    bufs, bptrs = plan.alloc_buckets(1, B)
    device_fill(S.tensors, 1, ["weight"] * len(S.tensors))
    for b in D.bufs + R.bufs:
        b.zero_()
    torch.cuda.synchronize()
    n = calibrate(torch, S.bufs, R.bufs)
    plan.reshard(ws, S.ptrs, D.ptrs)
    plan.pack(ws, 1, B, D.ptrs, bptrs)
    plan.unpack(ws, 1, B, bptrs, R.ptrs)
    torch.cuda.synchronize()
    print(f"profile_once: reshard {plan.info['bytes_read']} B read + {plan.info['bytes_written']} B written; "
          f"calibration copies {n} B", flush=True)
    del S, D, R, bufs, bptrs
    torch.cuda.empty_cache()
    for s_lay, d_lay in ((emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 2, 2, 0, "bf16")),
                         (emu.Layout(m, 2, 2, 0, "bf16"), emu.Layout(m, 4, 1, 0, "fp32"))):
        cp = emu.Plan(s_lay, d_lay)
        cws = cp.workspace()
        CS, CD = cp.alloc(0), cp.alloc(1)
        device_fill(CS.tensors, 2, ["weight"] * len(CS.tensors), s_lay.dtype)
        torch.cuda.synchronize()
        cp.reshard(cws, CS.ptrs, CD.ptrs)
        torch.cuda.synchronize()
        print(f"profile_once: {s_lay.dtype} -> {d_lay.dtype} reshard {cp.info['bytes_read']} B read + "
              f"{cp.info['bytes_written']} B written", flush=True)
        del CS, CD, cws
        torch.cuda.empty_cache()


def shifted_workload(torch, emu, device_fill, repeat):
    m = emu.Model(*EIGHT_B)
    plan = emu.Plan(emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2, 128))
    ws = plan.workspace()
    S, D, R = plan.alloc(0), plan.alloc(1), plan.alloc(1)
    device_fill(S.tensors, 1, ["weight"] * len(S.tensors))
    for b in R.bufs:
        b.zero_()
    Bs = (1 << 28, (1 << 28) - 2)
    region = torch.empty(max(plan.bucket_region_bytes(1, B) for B in Bs), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    n = calibrate(torch, D.bufs, R.bufs)
    plan.reshard(ws, S.ptrs, D.ptrs)
    tables = {B: plan.bucket_views(1, B, region)[1] for B in Bs}
    for _ in range(repeat):
        for B in Bs:
            plan.pack(ws, 1, B, D.ptrs, tables[B])
            plan.unpack(ws, 1, B, tables[B], R.ptrs)
    torch.cuda.synchronize()
    ok = all(torch.equal(a, b) for a, b in zip(D.tensors, R.tensors))
    for B in Bs:
        print(f"profile_once: {repeat} x pack + unpack at {B}-byte buckets, {2 * plan.bucket_layout(1, B, -1)[1]} B "
              f"each", flush=True)
    print(f"profile_once: unpacked (last: {Bs[-1]}-byte buckets) == resharded: {ok}", flush=True)
    print(f"profile_once: reshard {plan.info['bytes_read']} B read + {plan.info['bytes_written']} B written; "
          f"calibration copies {n} B", flush=True)


def formats_workload(torch, emu, device_fill, repeat):
    m = emu.Model(*EIGHT_B)
    L = lambda tp, pp, **kw: emu.Layout(m, tp, pp, **kw)
    fused, sep = emu.Plan(L(2, 2), L(4, 1)), emu.Plan(L(2, 2), L(4, 1, qkv="separate", mlp="separate"))
    src = torch.empty(fused.region_bytes(0), dtype=torch.uint8, device="cuda")
    dst = torch.empty(max(fused.region_bytes(1), sep.region_bytes(1)), dtype=torch.uint8, device="cuda")
    R = fused.alloc(1)
    S = fused.views(0, src)
    D, DS = fused.views(1, dst), sep.views(1, dst)
    wf, wsp = fused.workspace(), sep.workspace()
    device_fill(S.tensors, 1, ["weight"] * len(S.tensors))
    torch.cuda.synchronize()
    n = calibrate(torch, D.tensors, R.tensors)
    for _ in range(repeat):
        fused.reshard(wf, S.ptrs, D.ptrs)
        sep.reshard(wsp, S.ptrs, DS.ptrs)
    torch.cuda.synchronize()
    print(f"profile_once: {repeat} x (fused -> fused, fused -> separate) reshards of {fused.info['bytes_written']} B "
          f"on shared pages; calibration copies {n} B", flush=True)


def receiver_workload(torch, emu, device_fill):
    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 2, 2), emu.Layout(m, 4, 1)
    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    B = 1 << 28
    recv = emu.Plan(src, dst, src_bucket_bytes=B)
    wr = recv.workspace()
    S, R = plan.alloc(0), plan.alloc(1)
    bufs, bptrs = plan.alloc_buckets(0, B)
    device_fill(S.tensors, 1, ["weight"] * len(S.tensors))
    for b in R.bufs:
        b.zero_()
    torch.cuda.synchronize()
    n = calibrate(torch, S.bufs, R.bufs)
    plan.pack(ws, 0, B, S.ptrs, bptrs)
    recv.reshard(wr, bptrs, R.ptrs)
    torch.cuda.synchronize()
    print(f"profile_once: receiver {recv.info['bytes_read']} B read + {recv.info['bytes_written']} B written; "
          f"calibration copies {n} B", flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", choices=["main", "shifted", "formats", "receiver"], default="main")
    ap.add_argument("--repeat", type=int, default=1)
    args = ap.parse_args()
    import torch

    from paper_2609_34645_amd import emu
    from synthetic import device_fill

    torch.cuda.set_device(0)
    if args.workload == "main":
        main_workload(torch, emu, device_fill)
    elif args.workload == "shifted":
        shifted_workload(torch, emu, device_fill, args.repeat)
    elif args.workload == "receiver":
        receiver_workload(torch, emu, device_fill)
    else:
        formats_workload(torch, emu, device_fill, args.repeat)


if __name__ == "__main__":
    main()
