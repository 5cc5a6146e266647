"""Run each hot-path kernel once on the 8B TP2 PP2 -> TP4 PP1 workload, for hardware-counter profiling.

Launch order: one plain elementwise copy of the destination bytes (torch uint8 add of 0, a kernel of
known traffic: N bytes read + N written, used to calibrate FETCH_SIZE / WRITE_SIZE), one emu_reshard,
one emu_pack_buckets (2^28-byte buckets) and one emu_unpack_buckets; then the two converting
reshards of the same model: fp32 TP4 PP1 -> bf16 TP2 PP2 (the weight sync) and bf16 TP2 PP2 -> fp32
TP4 PP1. Example:

    rocprofv3 --pmc FETCH_SIZE -d out -o pmc_fetch -- python -m paper_2609_34645_amd.profile_once
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def main():
    import torch

    from paper_2609_34645_amd import emu
    from synthetic import device_fill

    torch.cuda.set_device(0)
    m = emu.Model(32, 4096, 32, 128, 8, 14336, 128256)
    plan = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1))
    ws = plan.workspace()
    S, D, R = plan.alloc(0), plan.alloc(1), plan.alloc(1)
    B = 1 << 28
    bufs, bptrs = plan.alloc_buckets(1, B)
    device_fill(S.tensors, 1, ["weight"] * len(S.tensors))
    for b in D.bufs + R.bufs:
        b.zero_()
    torch.cuda.synchronize()
    n = sum(b.numel() for b in D.bufs)
    for a, b in zip(S.bufs, R.bufs):                 # calibration: plain copy of known size
        k = min(a.numel(), b.numel())
        torch.add(a[:k], 0, out=b[:k])
    torch.cuda.synchronize()
    plan.reshard(ws, S.ptrs, D.ptrs)
    plan.pack(ws, 1, B, D.ptrs, bptrs)
    plan.unpack(ws, 1, B, bptrs, R.ptrs)
    torch.cuda.synchronize()
    print(f"profile_once: reshard {plan.info['bytes_read']} B read + {plan.info['bytes_written']} B written; "
          f"calibration copies {sum(min(a.numel(), b.numel()) for a, b in zip(S.bufs, R.bufs))} B; "
          f"destination {n} B", flush=True)
    del D, R, bufs, bptrs
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


if __name__ == "__main__":
    main()
