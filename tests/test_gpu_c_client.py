"""The GPU path driven from a fresh process.

* From plain C, with no Python or torch in the process: tests/c_abi_gpu_client.c (C99, HIP runtime C API +
  libemu.so) reshards the tiny decoder TP1 PP1 -> TP2 PP1, packs 12,288-byte buckets and unpacks them.
* From Python, with the binding loaded before anything imports torch.

The destination tensors and buckets are compared byte for byte with the oracle on the same source
contents, which the test regenerates from the client's fixed hash."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_2609_34645_amd import emu
from tests.gpu_util import say
from tests.shapes import TINY

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = "/opt/rocm"


def source_shards(layout):
    """The client's source contents: element e of global source tensor i is
    ((i * 2654435761) mod 2^32 xor (e * 40503) mod 2^32) mod 2^16, as bf16 bits."""
    out, i = [], 0
    for specs in oracle.rank_inventory(layout):
        rank = []
        for s in specs:
            e = np.arange(s.numel, dtype=np.uint64)
            v = (((i * 2654435761) & 0xFFFFFFFF) ^ ((e * 40503) & 0xFFFFFFFF)) & 0xFFFF
            rank.append(v.astype(np.uint16).reshape(s.shape))
            i += 1
        out.append(rank)
    return out


def test_c_client_reshard_and_buckets(gpu_lib, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc is not available")
    lib_dir = os.path.dirname(emu.LIB_PATH)
    exe = str(tmp_path / "client")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-D__HIP_PLATFORM_AMD__",
                    "-isystem", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi_gpu_client.c"), "-L", lib_dir, "-lemu",
                    "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{lib_dir}",
                    f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe], check=True)
    say("  c client: running")
    res = subprocess.run([exe, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    facts = dict(line.split(" ", 1) for line in res.stdout.strip().splitlines())
    assert facts["not_uploaded"] == "EMU_ERR_WORKSPACE"
    assert facts["upload_image_equal"] == "1"
    assert facts["unpack_equal"] == "1" and facts["done"] == "1"
    assert facts["receiver_equal"] == "1"
    om = oracle.Model(*TINY)
    src, dst = oracle.Layout(om, 1, 1), oracle.Layout(om, 2, 1)
    want = oracle.reshard(source_shards(src), src, dst)
    got = np.fromfile(tmp_path / "dst.bin", dtype=np.uint8)
    expect = np.concatenate([np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in want for a in rank])
    assert got.size == expect.size and np.array_equal(got, expect)
    buckets = [b for rank in want for b in oracle.pack(rank, 12288)]
    assert facts["buckets"] == str(len(buckets))
    assert np.array_equal(np.fromfile(tmp_path / "buckets.bin", dtype=np.uint8), np.concatenate(buckets))


CHILD = r"""
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
from paper_2609_34645_amd import emu
emu.load()  # the first thing the process does: torch is not imported yet
maps = open("/proc/self/maps").read().split("\n")
hip = sorted({l.split()[-1] for l in maps if "libamdhip64" in l})
print("hip_runtimes", len(hip))
import torch
m = emu.Model(2, 256, 4, 64, 2, 688, 1024)
plan = emu.Plan(emu.Layout(m, tp=1, pp=1), emu.Layout(m, tp=2, pp=1))
ws = plan.workspace()
S, D = plan.alloc(0), plan.alloc(1, fill=0xA5)
for i, t in enumerate(S.tensors):
    e = np.arange(t.numel() // 2, dtype=np.uint64)
    v = ((((i * 2654435761) & 0xFFFFFFFF) ^ ((e * 40503) & 0xFFFFFFFF)) & 0xFFFF).astype(np.uint16)
    t.copy_(torch.from_numpy(v.view(np.uint8)))
plan.reshard(ws, S.ptrs, D.ptrs)
torch.cuda.synchronize()
np.concatenate([t.cpu().numpy() for t in D.tensors]).tofile(sys.argv[2])
print("done 1")
"""


def test_binding_loaded_before_torch(gpu_lib, tmp_path):
    """A process whose first act is loading the library through the binding (no torch imported yet) holds
    one HIP runtime, and its reshard of the tiny decoder TP1 PP1 -> TP2 PP1 matches the oracle byte for
    byte. torch ships its own copy of the HIP runtime; had the binding loaded libemu.so before torch, the
    process would hold two, and the one libemu.so uses would see no device."""
    import sys

    out = tmp_path / "dst.bin"
    say("  binding-first child: running")
    res = subprocess.run([sys.executable, "-c", CHILD, ROOT, str(out)], capture_output=True, text=True,
                         timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    facts = dict(line.split(" ", 1) for line in res.stdout.strip().splitlines())
    assert facts["hip_runtimes"] == "1" and facts["done"] == "1"
    om = oracle.Model(*TINY)
    src, dst = oracle.Layout(om, 1, 1), oracle.Layout(om, 2, 1)
    want = oracle.reshard(source_shards(src), src, dst)
    expect = np.concatenate([np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in want for a in rank])
    got = np.fromfile(out, dtype=np.uint8)
    assert got.size == expect.size and np.array_equal(got, expect)
