"""Concurrent use of one plan and one uploaded workspace, as the C ABI allows: a plan is immutable and a
workspace is only read by the kernels, so several host threads, each with its own stream, may reshard,
pack and unpack at once. Every thread's results must equal a single-stream run whose output is checked
against the oracle. One thread also makes failing calls between its launches: its thread-local error
message must be its own, and the other threads' calls must not see it.

Workload: the 1B decoder bf16, TP4 PP1 -> TP2 PP1 (3.0 GB of destination shards), 2^26-byte buckets.
"""
import threading

import pytest

from paper_2609_34645_amd import emu
from tests.gpu_util import check_reshard, fill_device, say
from tests.shapes import ONE_B

pytestmark = pytest.mark.gpu
THREADS = 3
ROUNDS = 4
B = 1 << 26


def test_threads_share_plan_and_workspace(gpu_lib):
    import torch

    m = emu.Model(*ONE_B)
    plan = emu.Plan(emu.Layout(m, 4, 1), emu.Layout(m, 2, 1))
    ws = plan.workspace()
    S = plan.alloc(0)
    fill_device(plan, 0, S, seed=21)
    D0 = plan.alloc(1, fill=0xA5)
    plan.reshard(ws, S.ptrs, D0.ptrs)
    bufs0, bptrs0 = plan.alloc_buckets(1, B, fill=0x77)
    plan.pack(ws, 1, B, D0.ptrs, bptrs0)
    torch.cuda.synchronize()
    # the single-stream reference, checked against the oracle on the embedding and two layers
    check_reshard(plan, S, D0, groups=["embed", 0, m.num_layers - 1], label="single stream")

    sets = []
    for _ in range(THREADS):
        bufs, bptrs = plan.alloc_buckets(1, B, fill=0x33)
        sets.append((plan.alloc(1, fill=0x5A), bufs, bptrs, plan.alloc(1, fill=0x11)))
    torch.cuda.synchronize()
    errors, start = [], threading.Barrier(THREADS)

    def worker(i):
        try:
            D, bufs, bptrs, R = sets[i]
            stream = torch.cuda.Stream()  # default priority
            with torch.cuda.stream(stream):
                start.wait()
                for k in range(ROUNDS):
                    plan.reshard(ws, S.ptrs, D.ptrs)
                    if i == 0:  # failing calls between launches: this thread's message, nobody else's
                        with pytest.raises(emu.EmuError) as e:
                            plan.pack(ws, 1, 3, D.ptrs, bptrs)
                        assert e.value.code == -6 and "bucket size 3" in str(e.value)
                    plan.pack(ws, 1, B, D.ptrs, bptrs)
                    plan.unpack(ws, 1, B, bptrs, R.ptrs)
                    assert emu.load().emu_last_error() == b""
            stream.synchronize()
        except BaseException as exc:  # noqa: BLE001 - re-raised in the main thread
            errors.append((i, exc))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(THREADS)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    if errors:
        raise errors[0][1]
    torch.cuda.synchronize()
    for i, (D, bufs, _, R) in enumerate(sets):
        for j, (a, b, c) in enumerate(zip(D0.tensors, D.tensors, R.tensors)):
            assert torch.equal(a, b), f"thread {i}: destination tensor {j}"
            assert torch.equal(a, c), f"thread {i}: unpacked tensor {j}"
        assert len(bufs) == len(bufs0)
        for k, (a, b) in enumerate(zip(bufs0, bufs)):
            assert torch.equal(a, b), f"thread {i}: bucket {k}"
    say(f"  {THREADS} threads x {ROUNDS} rounds of reshard + pack + unpack on one plan and workspace: exact")
    del sets, S, D0, bufs0, bptrs0, ws
    torch.cuda.empty_cache()


def test_execute_calls_do_not_wait_for_the_stream(gpu_lib):
    """Execute calls only enqueue: with the stream held by a bounded spin kernel (torch.cuda._sleep),
    reshard, pack and unpack return long before the spin ends, and their work then runs after it. (The
    upload, a copy from pageable host memory, is made beforehand: the runtime may wait for the stream.)"""
    import time

    import torch

    from tests.shapes import TINY

    m = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    ws = plan.workspace()
    S = plan.alloc(0)
    fill_device(plan, 0, S, seed=22)
    D, R = plan.alloc(1, fill=0xA5), plan.alloc(1, fill=0x11)
    bufs, bptrs = plan.alloc_buckets(1, 1 << 16, fill=0x77)
    torch.cuda.synchronize()
    # calibrate the spin: about 0.2-2 s whatever the counter's clock
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cycles = 1 << 24
    while True:
        a.record()
        torch.cuda._sleep(cycles)
        b.record()
        b.synchronize()
        spin_ms = a.elapsed_time(b)
        if spin_ms >= 200 or cycles >= 1 << 34:
            break
        cycles *= 4
    assert spin_ms >= 200, f"spin of {cycles} cycles took only {spin_ms:.1f} ms"
    a.record()
    torch.cuda._sleep(cycles)
    t0 = time.perf_counter()
    plan.reshard(ws, S.ptrs, D.ptrs)
    plan.pack(ws, 1, 1 << 16, D.ptrs, bptrs)
    plan.unpack(ws, 1, 1 << 16, bptrs, R.ptrs)
    host_ms = (time.perf_counter() - t0) * 1e3
    b.record()
    still_spinning = not b.query()
    torch.cuda.synchronize()
    total_ms = a.elapsed_time(b)
    say(f"  spin {spin_ms:.0f} ms; three execute calls returned after {host_ms:.2f} ms; stream done after "
        f"{total_ms:.0f} ms")
    assert still_spinning and host_ms < spin_ms / 4
    assert total_ms >= spin_ms * 0.9
    check_reshard(plan, S, D, label="after the spin")
    for x, y in zip(D.tensors, R.tensors):
        assert torch.equal(x, y)
