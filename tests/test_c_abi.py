"""The C ABI used from plain C: tests/c_abi_client.c, compiled with gcc as strict C99 with warnings as
errors against include/emu.h and linked against libemu.so, runs the host-only calls (no GPU) and must
report the same facts the Python binding and the oracle give."""
import os
import shutil
import subprocess

import pytest

import oracle
from paper_2609_34645_amd import emu
from tests.shapes import EIGHT_B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc is not available")
    emu.load()
    lib_dir = os.path.dirname(emu.LIB_PATH)
    exe = str(tmp_path_factory.mktemp("c_abi") / "client")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi_client.c"), "-L", lib_dir, "-lemu", f"-Wl,-rpath,{lib_dir}",
                    "-o", exe], check=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    return dict(line.split(" ", 1) for line in out.strip().splitlines())


def test_header_compiles_as_c99_and_host_calls_work(client):
    assert int(client["version"]) == emu.load().emu_version()
    assert client["bad_layout"] == "EMU_ERR_LAYOUT"                      # tp = 3 divides no KV-head count
    om = oracle.Model(*EIGHT_B)
    src, dst = oracle.Layout(om, 2, 2), oracle.Layout(om, 4, 1)
    n_src = sum(len(r) for r in oracle.rank_inventory(src))
    n_dst = sum(len(r) for r in oracle.rank_inventory(dst))
    assert client["tensors"] == f"{n_src} {n_dst}"
    dst_bytes = sum(s.numel * 2 for r in oracle.rank_inventory(dst) for s in r)
    assert client["bytes"] == f"{dst_bytes} {dst_bytes}"
    spec = oracle.rank_inventory(dst)[0][1]                              # rank 0's second tensor
    assert spec.kind == "attn_norm" and client["dst1"] == f"0 {emu.KINDS.index('attn_norm')} 1 {om.H}"
    assert client["overlap"] == "EMU_ERR_OVERLAP"
    # buckets at 2^28 bytes: the destination streams cut by the oracle's rule
    streams = [sum(s.numel * 2 for s in r) for r in oracle.rank_inventory(dst)]
    nb = sum(-(-n // (1 << 28)) for n in streams)
    last = streams[-1] - (streams[-1] - 1) // (1 << 28) * (1 << 28)
    assert client["buckets"] == f"{nb} {sum(streams)} {len(streams) - 1} {(streams[-1] - 1) // (1 << 28)} {last}"
    assert client["bucket_range"] == "EMU_ERR_RANGE"
    # TP4 PP2 -> TP4 PP1 aliased: every destination tensor is a whole source tensor, nothing is read
    n_dst41 = sum(len(r) for r in oracle.rank_inventory(oracle.Layout(om, 4, 1)))
    assert client["alias"] == f"{n_dst41} 1 {dst_bytes} 0 0"
    assert client["image_short"] == "EMU_ERR_WORKSPACE" and client["image_nonzero"] == "1"
    src_streams = [sum(s.numel * 2 for s in r) for r in oracle.rank_inventory(src)]
    n_src_buckets = sum(-(-n // (1 << 28)) for n in src_streams)
    assert client["receiver"] == f"{n_src_buckets} {n_dst} {n_src_buckets} 1"
    assert client["receiver_odd"] == "EMU_ERR_BUCKET"
    assert client["freed_again"] == "EMU_ERR_HANDLE"
    n_nodes, n_edges, l_tran = client["dag"].split()
    py = emu.dag_plan([dict(kind=2, tp=4, pp=8, dp=1, gpus=list(range(32)), tgt_tp=8, tgt_pp=2, tgt_dp=1,
                            tgt_gpus=list(range(16)), state_bytes=3200.0)],
                      gpus_per_node=8, intra_bw=100.0, inter_bw=10.0, hbm_bw=1000.0, setup_s=0.5)
    assert (int(n_nodes), int(n_edges)) == (len(py["nodes"]), len(py["edges"])) and int(n_nodes) == 4
    # the paper's example: one Split, two Destroys, one Merge; L_tran = Split + Merge (closed form)
    assert abs(float(l_tran) - (0.5 + (3200 / 8 - 3200 / 32) / 10.0 + (3200 / 16) / 1000.0)) < 1e-9
