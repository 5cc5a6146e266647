// Host-side driver for the sanitizer build of the plan compiler and the transition-DAG planner
// (tests/test_host_sanitizers.py compiles it with emu_plan.cpp and emu_transition.cpp under
// AddressSanitizer and UndefinedBehaviorSanitizer; no HIP, no GPU). It walks the C ABI over every
// micro-model layout pair in both element types, the fused and converting plans, the 8B benchmark
// plans, the host-side table checks, the DAG planner on random scenarios and every error path it can
// reach, and prints "ok <calls>" when every status is the expected one.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "emu.h"

namespace {

uint64_t g_calls = 0;
uint64_t g_rng = 0x9e3779b97f4a7c15ull;

uint32_t rnd(uint32_t n) {  // xorshift64*, deterministic
  g_rng ^= g_rng >> 12;
  g_rng ^= g_rng << 25;
  g_rng ^= g_rng >> 27;
  return uint32_t(((g_rng * 2685821657736338717ull) >> 33) % n);
}

bool expect(int got, int want, const char* what) {
  ++g_calls;
  if (got == want) return true;
  std::fprintf(stderr, "%s: got %s, want %s (%s)\n", what, emu_status_str(got), emu_status_str(want), emu_last_error());
  return false;
}

emu_layout_t layout(const emu_model_t& m, int tp, int pp, int pad, int dtype, int qkv, int mlp) {
  emu_layout_t l;
  l.model = m;
  l.tp = tp;
  l.pp = pp;
  l.vocab_pad_multiple = pad;
  l.dtype = dtype;
  l.qkv_format = qkv;
  l.mlp_format = mlp;
  return l;
}

// Every query the ABI offers on a plan, then free it.
bool walk(emu_plan_t p) {
  emu_plan_info_t info;
  if (!expect(emu_plan_info(p, &info), EMU_OK, "info")) return false;
  emu_tensor_desc_t d;
  std::vector<uint64_t> ptrs[2];
  std::vector<int> written;  // destination tensors the map writes (all but an alias plan's aliases)
  for (int side = 0; side < 2; ++side) {
    const int n = side ? info.n_dst_tensors : info.n_src_tensors;
    uint64_t a = (1ull << 36) * uint64_t(side + 1);
    for (int i = 0; i < n; ++i) {
      if (!expect(emu_tensor_info(p, side, i, &d), EMU_OK, "tensor_info")) return false;
      ptrs[side].push_back(a);
      a = (a + d.bytes + 255) / 256 * 256;
      if (side == 1 && !(info.aliased && d.alias >= 0)) written.push_back(i);
    }
    if (!expect(emu_tensor_info(p, side, n, &d), EMU_ERR_RANGE, "tensor_info past the end")) return false;
    uint64_t nb = 0, sb = 0;
    for (uint64_t B : {4ull, 28ull, 4096ull, 1ull << 28}) {  // multiples of either element size
      if (!expect(emu_bucket_layout(p, side, B, -1, &nb, &sb), EMU_OK, "bucket_layout")) return false;
      if (nb > (1u << 16)) continue;  // small buckets of the 8B plans: billions of them
      std::vector<emu_bucket_desc_t> bk(size_t(nb) + 1);
      if (!expect(emu_bucket_info(p, side, B, 0, nb, bk.data()), EMU_OK, "bucket_info") ||
          !expect(emu_bucket_info(p, side, B, nb, 1, bk.data()), EMU_ERR_RANGE, "bucket_info past the end"))
        return false;
    }
  }
  // the workspace image: the host's copy of the tables the upload builds on the device
  std::vector<uint8_t> img(size_t(info.workspace_bytes) + 1);
  if (!expect(emu_plan_workspace_image(p, img.data(), info.workspace_bytes), EMU_OK, "workspace_image") ||
      !expect(emu_plan_workspace_image(p, img.data(), info.workspace_bytes - 1), EMU_ERR_WORKSPACE, "short image"))
    return false;
  std::vector<emu_segment_t> segs(size_t(info.n_segments) + 1);
  if (!expect(emu_plan_segments(p, 0, info.n_segments, segs.data()), EMU_OK, "segments")) return false;
  if (!expect(emu_plan_segments(p, 0, info.n_segments + 1, segs.data()), EMU_ERR_RANGE, "segments past the end"))
    return false;
  if (!expect(emu_check_tables(p, ptrs[0].data(), ptrs[1].data()), EMU_OK, "check_tables")) return false;
  if (written.size() > 1) {
    std::vector<uint64_t> bad = ptrs[1];
    bad[size_t(written[1])] = bad[size_t(written[0])];
    if (!expect(emu_check_tables(p, ptrs[0].data(), bad.data()), EMU_ERR_OVERLAP, "overlap")) return false;
  }
  return expect(emu_plan_free(p), EMU_OK, "free") && expect(emu_plan_free(p), EMU_ERR_HANDLE, "double free");
}

bool plans() {
  const emu_model_t micro = {4, 16, 8, 4, 2, 12, 20};
  const int qkvs[2] = {EMU_QKV_HEAD_INTERLEAVED, EMU_QKV_SEPARATE};
  const int mlps[2] = {EMU_GATE_UP_BLOCK, EMU_GATE_UP_SEPARATE};
  std::vector<emu_layout_t> lays;
  for (int tp : {1, 2, 4})
    for (int pp : {1, 2, 3, 4})
      for (int pad : {0, 2})
        for (int f = 0; f < 4; ++f)
          for (int dt : {EMU_BF16, EMU_FP32})
            lays.push_back(layout(micro, tp, pp, pad, dt, qkvs[f & 1], mlps[f >> 1]));
  for (const emu_layout_t& a : lays)
    for (size_t k = 0; k < 24; ++k) {
      const emu_layout_t& b = lays[rnd(uint32_t(lays.size()))];
      emu_plan_t p = nullptr;
      if (!expect(emu_plan(&a, &b, &p), EMU_OK, "micro plan") || !walk(p)) return false;
      if (!expect(emu_plan_ex(&a, &b, EMU_PLAN_ALIAS_RESIDENT, &p), EMU_OK, "micro alias plan") || !walk(p)) return false;
      if (a.dtype == b.dtype) {
        const uint64_t B = (a.dtype == EMU_FP32 ? 4u : 2u) * (1 + rnd(40));
        if (!expect(emu_plan_to_buckets(&a, &b, B, &p), EMU_OK, "micro fused plan") || !walk(p)) return false;
      }
      const uint64_t Bs = (a.dtype == EMU_FP32 ? 4u : 2u) * (1 + rnd(40));  // whole source elements
      if (!expect(emu_plan_from_buckets(&a, &b, Bs, &p), EMU_OK, "micro receiver plan") || !walk(p)) return false;
    }
  const emu_model_t m8 = {32, 4096, 32, 8, 128, 14336, 128256};
  const emu_layout_t pairs[][2] = {
      {layout(m8, 2, 2, 0, EMU_BF16, 0, 0), layout(m8, 4, 1, 0, EMU_BF16, 0, 0)},
      {layout(m8, 8, 4, 128, EMU_BF16, 0, 0), layout(m8, 2, 2, 0, EMU_BF16, 0, 0)},
      {layout(m8, 4, 1, 0, EMU_FP32, 0, 0), layout(m8, 2, 2, 0, EMU_BF16, 0, 0)},
      {layout(m8, 2, 2, 0, EMU_BF16, 0, 0), layout(m8, 16, 3, 0, EMU_BF16, 1, 1)},
  };
  for (const auto& pr : pairs) {
    emu_plan_t p = nullptr;
    if (!expect(emu_plan(&pr[0], &pr[1], &p), EMU_OK, "8B plan") || !walk(p)) return false;
    if (pr[0].dtype == pr[1].dtype)
      for (uint64_t B : {1ull << 28, (1ull << 28) - 2})
        if (!expect(emu_plan_to_buckets(&pr[0], &pr[1], B, &p), EMU_OK, "8B fused plan") || !walk(p)) return false;
    for (uint64_t B : {1ull << 28, (1ull << 28) - 4})
      if (!expect(emu_plan_from_buckets(&pr[0], &pr[1], B, &p), EMU_OK, "8B receiver plan") || !walk(p)) return false;
  }
  return true;
}

bool errors() {
  const emu_model_t m = {2, 256, 4, 2, 64, 688, 1024};
  emu_layout_t good = layout(m, 1, 1, 0, EMU_BF16, 0, 0), bad = layout(m, 3, 1, 0, EMU_BF16, 0, 0);
  emu_plan_t p = nullptr;
  bool ok = expect(emu_plan(nullptr, &good, &p), EMU_ERR_NULL, "null src") &&
            expect(emu_plan(&good, &bad, &p), EMU_ERR_LAYOUT, "bad layout") &&
            expect(emu_layout_check(&bad), EMU_ERR_LAYOUT, "layout_check") &&
            expect(emu_plan_to_buckets(&good, &good, 0, &p), EMU_ERR_BUCKET, "zero bucket") &&
            expect(emu_plan_info(nullptr, nullptr), EMU_ERR_HANDLE, "null handle") &&
            expect(emu_set_option(0, 3), EMU_ERR_ARG, "bad option value") &&
            expect(emu_set_option(99, 1), EMU_ERR_RANGE, "unknown option");
  emu_layout_t other = good;
  other.model.vocab = 2048;
  ok = ok && expect(emu_plan(&good, &other, &p), EMU_ERR_MISMATCH, "different models");
  ok = ok && expect(emu_plan(&good, &good, &p), EMU_OK, "identity plan");
  uint64_t nb = 0, sb = 0;
  ok = ok && expect(emu_bucket_layout(p, 1, 3, -1, &nb, &sb), EMU_ERR_BUCKET, "odd bucket") &&
       expect(emu_bucket_layout(p, 2, 64, -1, &nb, &sb), EMU_ERR_RANGE, "bad side") &&
       expect(emu_check_tables(p, nullptr, nullptr), EMU_ERR_NULL, "null tables") &&
       expect(emu_plan_free(p), EMU_OK, "free");
  return ok;
}

bool dags() {
  emu_link_model_t links = {8, 0, 100.0, 10.0, 1000.0, 0.5};
  int ok_n = 0, arg_n = 0, inf_n = 0;
  for (int it = 0; it < 400; ++it) {
    const int ns = 1 + int(rnd(3));
    std::vector<emu_stage_transition_t> st(size_t(ns) + 0);
    std::vector<std::vector<int32_t>> g(size_t(2 * ns));
    const int degs[4] = {1, 2, 4, 0};
    for (int i = 0; i < ns; ++i) {
      emu_stage_transition_t& s = st[size_t(i)];
      s.kind = int32_t(rnd(3));
      s.tp = degs[rnd(3)]; s.pp = degs[rnd(3)]; s.dp = 1 + int32_t(rnd(2));
      s.tgt_tp = degs[rnd(3)]; s.tgt_pp = degs[rnd(3)]; s.tgt_dp = 1 + int32_t(rnd(2));
      if (rnd(10) == 0) s.tp = 0;  // malformed now and then
      s.reserved = 0;
      const int64_t n = int64_t(s.dp) * s.tp * s.pp, tn = int64_t(s.tgt_dp) * s.tgt_tp * s.tgt_pp;
      for (int64_t k = 0; k < n; ++k) g[size_t(2 * i)].push_back(int32_t(rnd(rnd(4) == 0 ? 8 : 64)));
      for (int64_t k = 0; k < tn; ++k) g[size_t(2 * i + 1)].push_back(int32_t(rnd(64)));
      g[size_t(2 * i)].push_back(0);  // never empty
      g[size_t(2 * i + 1)].push_back(0);
      s.gpus = g[size_t(2 * i)].data();
      s.tgt_gpus = g[size_t(2 * i + 1)].data();
      s.state_bytes = 1e9;
    }
    emu_dag_t dag = nullptr;
    const int rc = emu_dag_plan(st.data(), ns, &links, &dag);
    ++g_calls;
    if (rc == EMU_OK) {
      ++ok_n;
      emu_dag_info_t info;
      if (!expect(emu_dag_info(dag, &info), EMU_OK, "dag info")) return false;
      std::vector<emu_dag_node_t> nodes(size_t(info.n_nodes) + 1);
      std::vector<emu_dag_edge_t> edges(size_t(info.n_edges) + 1);
      std::vector<int32_t> gp(size_t(info.n_gpu_entries) + 1);
      if (!expect(emu_dag_nodes(dag, 0, info.n_nodes, nodes.data()), EMU_OK, "dag nodes") ||
          !expect(emu_dag_edges(dag, 0, info.n_edges, edges.data()), EMU_OK, "dag edges") ||
          !expect(emu_dag_gpus(dag, 0, info.n_gpu_entries, gp.data()), EMU_OK, "dag gpus") ||
          !expect(emu_dag_free(dag), EMU_OK, "dag free") || !expect(emu_dag_free(dag), EMU_ERR_HANDLE, "dag double free"))
        return false;
    } else if (rc == EMU_ERR_ARG) {
      ++arg_n;
    } else if (rc == EMU_ERR_INFEASIBLE) {
      ++inf_n;
    } else {
      std::fprintf(stderr, "dag plan: unexpected %s\n", emu_status_str(rc));
      return false;
    }
  }
  std::printf("dags %d %d %d\n", ok_n, arg_n, inf_n);
  return ok_n > 0 && arg_n > 0;
}

}  // namespace

int main() {
  if (!plans() || !errors() || !dags()) return 1;
  std::printf("ok %llu\n", (unsigned long long)g_calls);
  return 0;
}
