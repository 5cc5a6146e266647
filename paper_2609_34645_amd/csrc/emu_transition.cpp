// Transition-DAG planner: from a current to a target plan of several model-stages, the primitives that
// carry every model-stage's EMU collection over (Split -> Destroy -> Extend -> Merge through the largest
// common layout T_sub), the resource-dependency edges between model-stages that hand GPUs to each other,
// and the DAG's critical-path cost (paper section 6.1; cost inputs from the section 6 introduction).
// Host only: no GPU calls.
//
// Rules (the paper gives no listing; these are the readings the library implements):
//   * T_sub = (gcd(tp, tp*), gcd(pp, pp*)). Splitting a (tp, pp) unit gives (tp/tps)(pp/pps) sub-units;
//     sub-unit (a, b) holds ranks (a*tps + t', b*pps + p') at its own rank (t', p'); ranks r = p*tp + t.
//   * A sub-unit whose GPUs all lie in the target GPU set is kept (first fit, up to the
//     tgt_dp * (tgt_tp/tps)(tgt_pp/pps) sub-units the target needs); the others are destroyed.
//   * Missing sub-units are extended onto the target GPUs no kept sub-unit occupies (ascending ids,
//     tps*pps per sub-unit). The i-th Extend copies from the first sub-unit, scanning cyclically from i,
//     whose GPUs are disjoint from its own. A destroyed sub-unit is destroyed only after it was copied.
//   * Every k* = (tgt_tp/tps)(tgt_pp/pps) sub-units (kept first, then extended) merge into one target
//     unit; target rank (t*, p*) is rank (t* mod tps, p* mod pps) of sub-unit (t* div tps) +
//     (p* div pps)(tgt_tp/tps).
//   * Model-stages of one stage kind run concurrently and hold disjoint GPUs; an Extend onto a GPU another
//     such model-stage holds waits for the Destroy releasing it (a resource-dependency edge), unless that
//     Destroy depends on the Extend: then no deadlock-free order exists (EMU_ERR_INFEASIBLE). Blocked
//     acquisitions are resolved in generation -> inference -> training order.
//   * Costs: Split = setup + (shard_sub - shard_cur)/bw(unit GPUs); Extend = setup + max over rank pairs
//     of shard_sub/bw(pair); Merge = shard_target/hbm_bw; Destroy = 0. bw is intra-node when every GPU
//     involved sits in one node (id / gpus_per_node), else inter-node. L_tran = longest path.
#include <algorithm>
#include <chrono>
#include <cstring>
#include <mutex>
#include <new>
#include <numeric>
#include <set>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "emu_internal.h"

namespace emu {

namespace {

constexpr uint32_t kDagMagic = 0x454d5544u;  // "EMUD"

struct Node {
  int32_t prim, stage, unit, src;
  std::vector<int32_t> gpus;
  double cost = 0, start = 0, finish = 0;
};

struct Edge {
  int32_t from, to, resource;
  bool operator<(const Edge& o) const {
    if (to != o.to) return to < o.to;
    if (from != o.from) return from < o.from;
    return resource < o.resource;
  }
  bool operator==(const Edge& o) const { return to == o.to && from == o.from && resource == o.resource; }
};

struct Dag {
  uint32_t magic = kDagMagic;
  std::vector<Node> nodes;
  std::vector<Edge> edges;
  std::vector<std::vector<std::vector<int32_t>>> target_units;  // [stage][unit] -> GPU ids in rank order
  std::vector<int32_t> flat_gpus;                                // node GPU lists, concatenated
  std::vector<int32_t> gpu_first;
  int32_t n_resource = 0;
  double l_tran = 0;
  double plan_ms = 0;
};

std::mutex g_dag_mu;
std::unordered_set<const Dag*> g_dags;

bool dag_live(const Dag* d) {
  std::lock_guard<std::mutex> lk(g_dag_mu);
  return d && g_dags.count(d) && d->magic == kDagMagic;
}

int64_t igcd(int64_t a, int64_t b) { return b ? igcd(b, a % b) : a; }

double bw_of(const emu_link_model_t& L, const int32_t* g, size_t n) {
  const int32_t node = g[0] / L.gpus_per_node;
  for (size_t i = 1; i < n; ++i)
    if (g[i] / L.gpus_per_node != node) return L.inter_bw;
  return L.intra_bw;
}

std::vector<std::vector<int32_t>> split_gpus(const int32_t* gpus, int tp, int pp, int tps, int pps) {
  std::vector<std::vector<int32_t>> out;
  for (int b = 0; b < pp / pps; ++b)
    for (int a = 0; a < tp / tps; ++a) {
      std::vector<int32_t> sub;
      for (int pq = 0; pq < pps; ++pq)
        for (int tq = 0; tq < tps; ++tq) sub.push_back(gpus[(b * pps + pq) * tp + (a * tps + tq)]);
      out.push_back(std::move(sub));
    }
  return out;
}

int check_input(const emu_stage_transition_t* S, int32_t n, const emu_link_model_t* L) {
  if (!S || !L) return fail(EMU_ERR_NULL, "NULL argument");
  if (n <= 0) return fail(EMU_ERR_ARG, "need at least one model-stage");
  if (L->gpus_per_node <= 0 || !(L->intra_bw > 0) || !(L->inter_bw > 0) || !(L->hbm_bw > 0) || !(L->setup_s >= 0))
    return fail(EMU_ERR_ARG, "link model needs positive bandwidths, GPUs per node and a non-negative setup time");
  for (int32_t i = 0; i < n; ++i) {
    const emu_stage_transition_t& s = S[i];
    if (s.tp <= 0 || s.pp <= 0 || s.dp <= 0 || s.tgt_tp <= 0 || s.tgt_pp <= 0 || s.tgt_dp <= 0)
      return fail(EMU_ERR_ARG, "stage %d: degrees must be positive", i);
    if (!s.gpus || !s.tgt_gpus) return fail(EMU_ERR_NULL, "stage %d: NULL GPU list", i);
    if (!(s.state_bytes >= 0)) return fail(EMU_ERR_ARG, "stage %d: negative state size", i);
    for (int side = 0; side < 2; ++side) {
      const int32_t* g = side ? s.tgt_gpus : s.gpus;
      const int64_t cnt = side ? int64_t(s.tgt_dp) * s.tgt_tp * s.tgt_pp : int64_t(s.dp) * s.tp * s.pp;
      std::unordered_set<int32_t> seen;
      for (int64_t k = 0; k < cnt; ++k) {
        if (g[k] < 0) return fail(EMU_ERR_ARG, "stage %d: negative GPU id", i);
        if (!seen.insert(g[k]).second) return fail(EMU_ERR_ARG, "stage %d: GPU %d listed twice", i, g[k]);
      }
    }
  }
  for (int32_t i = 0; i < n; ++i)
    for (int32_t j = 0; j < i; ++j) {
      if (S[i].kind != S[j].kind) continue;
      for (int side = 0; side < 2; ++side) {
        const emu_stage_transition_t &a = S[i], &b = S[j];
        const int32_t* ga = side ? a.tgt_gpus : a.gpus;
        const int32_t* gb = side ? b.tgt_gpus : b.gpus;
        const int64_t na = side ? int64_t(a.tgt_dp) * a.tgt_tp * a.tgt_pp : int64_t(a.dp) * a.tp * a.pp;
        const int64_t nb = side ? int64_t(b.tgt_dp) * b.tgt_tp * b.tgt_pp : int64_t(b.dp) * b.tp * b.pp;
        std::unordered_set<int32_t> sb(gb, gb + nb);
        for (int64_t k = 0; k < na; ++k)
          if (sb.count(ga[k])) return fail(EMU_ERR_ARG, "stages %d and %d run concurrently but share GPU %d", j, i, ga[k]);
      }
    }
  return EMU_OK;
}

int build(const emu_stage_transition_t* S, int32_t n, const emu_link_model_t& L, Dag& D) {
  std::set<Edge> edges;
  std::vector<std::unordered_map<int32_t, int32_t>> destroy_of_gpu(n);
  std::vector<std::pair<int32_t, int32_t>> extends;  // (stage, node)
  auto& nodes = D.nodes;

  for (int32_t si = 0; si < n; ++si) {
    const emu_stage_transition_t& s = S[si];
    const int tps = int(igcd(s.tp, s.tgt_tp)), pps = int(igcd(s.pp, s.tgt_pp));
    const int n_sub = tps * pps;
    const int k = (s.tp / tps) * (s.pp / pps), ks = (s.tgt_tp / tps) * (s.tgt_pp / pps);
    const double shard_cur = s.state_bytes / double(s.tp * s.pp), shard_sub = s.state_bytes / double(n_sub);
    const int unit_size = s.tp * s.pp;

    // Split: current units -> T_sub units
    std::vector<std::vector<int32_t>> subs;
    std::vector<int32_t> split_of;
    for (int u = 0; u < s.dp; ++u) {
      const int32_t* ug = s.gpus + int64_t(u) * unit_size;
      auto parts = split_gpus(ug, s.tp, s.pp, tps, pps);
      int32_t sid = -1;
      if (k > 1) {
        sid = int32_t(nodes.size());
        Node nd{EMU_PRIM_SPLIT, si, u, -1, std::vector<int32_t>(ug, ug + unit_size)};
        nd.cost = L.setup_s + (shard_sub - shard_cur) / bw_of(L, ug, unit_size);
        nodes.push_back(std::move(nd));
      }
      for (auto& part : parts) {
        subs.push_back(std::move(part));
        split_of.push_back(sid);
      }
    }

    // keep the sub-units already inside the target GPU set
    const int64_t ntgt = int64_t(s.tgt_dp) * s.tgt_tp * s.tgt_pp;
    std::unordered_set<int32_t> tgt(s.tgt_gpus, s.tgt_gpus + ntgt);
    const int64_t need = int64_t(s.tgt_dp) * ks;
    std::vector<int32_t> kept;
    std::vector<char> is_kept(subs.size(), 0);
    for (size_t j = 0; j < subs.size(); ++j) {
      if (int64_t(kept.size()) >= need) break;
      bool inside = true;
      for (int32_t g : subs[j]) inside = inside && tgt.count(g);
      if (inside) {
        kept.push_back(int32_t(j));
        is_kept[j] = 1;
      }
    }

    // Destroy the rest
    std::unordered_map<int32_t, int32_t> dnode;  // sub-unit -> node
    auto& dmap = destroy_of_gpu[si];
    for (size_t j = 0; j < subs.size(); ++j) {
      if (is_kept[j]) continue;
      const int32_t did = int32_t(nodes.size());
      nodes.push_back(Node{EMU_PRIM_DESTROY, si, int32_t(j), -1, subs[j]});
      dnode[int32_t(j)] = did;
      if (split_of[j] >= 0) edges.insert({split_of[j], did, 0});
      for (int32_t g : subs[j]) dmap[g] = did;
    }

    // Extend the missing sub-units onto the free target GPUs
    std::unordered_set<int32_t> used;
    for (int32_t j : kept)
      for (int32_t g : subs[j]) used.insert(g);
    std::vector<int32_t> free_g;
    for (int32_t g : tgt)
      if (!used.count(g)) free_g.push_back(g);
    std::sort(free_g.begin(), free_g.end());
    std::vector<std::pair<std::vector<int32_t>, int32_t>> slots;  // (GPU list, provider node or -1)
    for (int32_t j : kept) slots.push_back({subs[j], split_of[j]});
    const int64_t n_ext = need - int64_t(kept.size());
    for (int64_t i = 0; i < n_ext; ++i) {
      std::vector<int32_t> slot(free_g.begin() + i * n_sub, free_g.begin() + (i + 1) * n_sub);
      std::unordered_set<int32_t> sl(slot.begin(), slot.end());
      int32_t src = -1;
      for (size_t c = 0; c < subs.size(); ++c) {
        const size_t cand = (size_t(i) + c) % subs.size();
        bool disjoint = true;
        for (int32_t g : subs[cand]) disjoint = disjoint && !sl.count(g);
        if (disjoint) {
          src = int32_t(cand);
          break;
        }
      }
      if (src < 0) return fail(EMU_ERR_INFEASIBLE, "stage %d: no replica disjoint from extend slot %lld", si, (long long)i);
      const int32_t eid = int32_t(nodes.size());
      double worst = 0;
      for (int r = 0; r < n_sub; ++r) {
        const int32_t pair[2] = {subs[src][r], slot[r]};
        worst = std::max(worst, shard_sub / bw_of(L, pair, 2));
      }
      Node nd{EMU_PRIM_EXTEND, si, int32_t(kept.size() + i), src, slot};
      nd.cost = L.setup_s + worst;
      nodes.push_back(std::move(nd));
      if (split_of[src] >= 0) edges.insert({split_of[src], eid, 0});
      auto ds = dnode.find(src);
      if (ds != dnode.end()) edges.insert({eid, ds->second, 0});  // destroyed only after it was copied
      for (int32_t g : slot) {                                     // release before acquire, same stage
        auto it = dmap.find(g);
        if (it != dmap.end() && (ds == dnode.end() || it->second != ds->second)) edges.insert({it->second, eid, 0});
      }
      extends.push_back({si, eid});
      slots.push_back({slot, eid});
    }

    // Merge k* sub-units into each target unit
    D.target_units.emplace_back();
    for (int u = 0; u < s.tgt_dp; ++u) {
      std::vector<int32_t> ug(size_t(s.tgt_tp) * s.tgt_pp);
      for (int p = 0; p < s.tgt_pp; ++p)
        for (int t = 0; t < s.tgt_tp; ++t) {
          const int sub = (p / pps) * (s.tgt_tp / tps) + t / tps;
          ug[size_t(p) * s.tgt_tp + t] = slots[size_t(u) * ks + sub].first[(p % pps) * tps + t % tps];
        }
      if (ks > 1) {
        const int32_t mid = int32_t(nodes.size());
        Node nd{EMU_PRIM_MERGE, si, u, -1, ug};
        nd.cost = (s.state_bytes / double(s.tgt_tp * s.tgt_pp)) / L.hbm_bw;
        nodes.push_back(std::move(nd));
        for (int j = 0; j < ks; ++j) {
          const int32_t prov = slots[size_t(u) * ks + j].second;
          if (prov >= 0) edges.insert({prov, mid, 0});
        }
      }
      D.target_units.back().push_back(std::move(ug));
    }
  }

  // cross-model-stage resource edges
  std::vector<std::vector<int32_t>> succ(nodes.size());
  for (const Edge& e : edges) succ[e.from].push_back(e.to);
  std::vector<int32_t> mark(nodes.size(), -1);
  int32_t epoch = 0;
  auto reaches = [&](int32_t a, int32_t b) {
    ++epoch;
    std::vector<int32_t> stack{a};
    mark[a] = epoch;
    while (!stack.empty()) {
      const int32_t x = stack.back();
      stack.pop_back();
      if (x == b) return true;
      for (int32_t y : succ[x])
        if (mark[y] != epoch) {
          mark[y] = epoch;
          stack.push_back(y);
        }
    }
    return false;
  };
  std::vector<std::unordered_set<int32_t>> cur_gpus(n);
  for (int32_t i = 0; i < n; ++i)
    cur_gpus[i].insert(S[i].gpus, S[i].gpus + int64_t(S[i].dp) * S[i].tp * S[i].pp);
  std::stable_sort(extends.begin(), extends.end(), [&](const auto& a, const auto& b) {
    if (S[a.first].kind != S[b.first].kind) return S[a.first].kind < S[b.first].kind;
    if (a.first != b.first) return a.first < b.first;
    return a.second < b.second;
  });
  for (const auto& ex : extends) {
    const int32_t si = ex.first, eid = ex.second;
    const std::vector<int32_t> gl = nodes[eid].gpus;
    for (int32_t g : gl)
      for (int32_t sj = 0; sj < n; ++sj) {
        if (sj == si || S[sj].kind != S[si].kind || !cur_gpus[sj].count(g)) continue;
        auto it = destroy_of_gpu[sj].find(g);
        if (it == destroy_of_gpu[sj].end())
          return fail(EMU_ERR_INFEASIBLE, "stage %d needs GPU %d, which stage %d keeps", si, g, sj);
        const int32_t did = it->second;
        if (edges.count({did, eid, 1})) continue;
        if (reaches(eid, did))
          return fail(EMU_ERR_INFEASIBLE, "stage %d: the Destroy releasing GPU %d depends on the acquisition", si, g);
        edges.insert({did, eid, 1});
        succ[did].push_back(eid);
        ++D.n_resource;
      }
  }

  D.edges.assign(edges.begin(), edges.end());  // ordered by (to, from, resource)
  // ASAP schedule in a topological order; its makespan is the critical path
  std::vector<int32_t> indeg(nodes.size(), 0);
  std::vector<std::vector<int32_t>> preds(nodes.size());
  for (const Edge& e : D.edges) {
    ++indeg[e.to];
    preds[e.to].push_back(e.from);
  }
  std::set<int32_t> ready;
  for (size_t i = 0; i < nodes.size(); ++i)
    if (!indeg[i]) ready.insert(int32_t(i));
  size_t done = 0;
  D.l_tran = 0;
  while (!ready.empty()) {
    const int32_t x = *ready.begin();
    ready.erase(ready.begin());
    ++done;
    double st = 0;
    for (int32_t p : preds[x]) st = std::max(st, nodes[p].finish);
    nodes[x].start = st;
    nodes[x].finish = st + nodes[x].cost;
    D.l_tran = std::max(D.l_tran, nodes[x].finish);
    for (int32_t y : succ[x])
      if (--indeg[y] == 0) ready.insert(y);
  }
  if (done != nodes.size()) return fail(EMU_ERR_INFEASIBLE, "cycle in the transition DAG");
  for (const Node& nd : nodes) {
    D.gpu_first.push_back(int32_t(D.flat_gpus.size()));
    D.flat_gpus.insert(D.flat_gpus.end(), nd.gpus.begin(), nd.gpus.end());
  }
  return EMU_OK;
}

}  // namespace
}  // namespace emu

using namespace emu;

extern "C" {

int emu_dag_plan(const emu_stage_transition_t* stages, int32_t n_stages, const emu_link_model_t* links,
                 emu_dag_t* out) {
  clear_error();
  if (!out) return fail(EMU_ERR_NULL, "out is NULL");
  *out = nullptr;
  const auto t0 = std::chrono::steady_clock::now();
  int rc = check_input(stages, n_stages, links);
  if (rc) return rc;
  Dag* D = new (std::nothrow) Dag();
  if (!D) return fail(EMU_ERR_ARG, "out of host memory");
  try {
    rc = build(stages, n_stages, *links, *D);
  } catch (const std::bad_alloc&) {
    rc = fail(EMU_ERR_ARG, "out of host memory");
  }
  if (rc) {
    delete D;
    return rc;
  }
  D->plan_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  {
    std::lock_guard<std::mutex> lk(g_dag_mu);
    g_dags.insert(D);
  }
  *out = reinterpret_cast<emu_dag_t>(D);
  return EMU_OK;
}

int emu_dag_free(emu_dag_t dag) {
  clear_error();
  Dag* D = reinterpret_cast<Dag*>(dag);
  {
    std::lock_guard<std::mutex> lk(g_dag_mu);
    if (!D || !g_dags.count(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
    g_dags.erase(D);
  }
  D->magic = 0;
  delete D;
  return EMU_OK;
}

int emu_dag_info(emu_dag_t dag, emu_dag_info_t* out) {
  clear_error();
  const Dag* D = reinterpret_cast<const Dag*>(dag);
  if (!dag_live(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
  if (!out) return fail(EMU_ERR_NULL, "out is NULL");
  *out = emu_dag_info_t{};
  out->n_nodes = int32_t(D->nodes.size());
  out->n_edges = int32_t(D->edges.size());
  out->n_resource_edges = D->n_resource;
  out->n_gpu_entries = int32_t(D->flat_gpus.size());
  out->l_tran_s = D->l_tran;
  out->plan_ms = D->plan_ms;
  return EMU_OK;
}

int emu_dag_nodes(emu_dag_t dag, int32_t first, int32_t count, emu_dag_node_t* out) {
  clear_error();
  const Dag* D = reinterpret_cast<const Dag*>(dag);
  if (!dag_live(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
  if (count > 0 && !out) return fail(EMU_ERR_NULL, "out is NULL");
  if (first < 0 || count < 0 || size_t(first) + size_t(count) > D->nodes.size())
    return fail(EMU_ERR_RANGE, "node range out of bounds");
  for (int32_t i = 0; i < count; ++i) {
    const Node& nd = D->nodes[size_t(first) + i];
    emu_dag_node_t& o = out[i];
    o.prim = nd.prim;
    o.stage = nd.stage;
    o.unit = nd.unit;
    o.src = nd.src;
    o.gpu_first = D->gpu_first[size_t(first) + i];
    o.n_gpus = int32_t(nd.gpus.size());
    o.cost_s = nd.cost;
    o.start_s = nd.start;
    o.finish_s = nd.finish;
  }
  return EMU_OK;
}

int emu_dag_edges(emu_dag_t dag, int32_t first, int32_t count, emu_dag_edge_t* out) {
  clear_error();
  const Dag* D = reinterpret_cast<const Dag*>(dag);
  if (!dag_live(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
  if (count > 0 && !out) return fail(EMU_ERR_NULL, "out is NULL");
  if (first < 0 || count < 0 || size_t(first) + size_t(count) > D->edges.size())
    return fail(EMU_ERR_RANGE, "edge range out of bounds");
  for (int32_t i = 0; i < count; ++i) {
    const Edge& e = D->edges[size_t(first) + i];
    out[i] = emu_dag_edge_t{e.from, e.to, e.resource, 0};
  }
  return EMU_OK;
}

int emu_dag_gpus(emu_dag_t dag, int32_t first, int32_t count, int32_t* out) {
  clear_error();
  const Dag* D = reinterpret_cast<const Dag*>(dag);
  if (!dag_live(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
  if (count > 0 && !out) return fail(EMU_ERR_NULL, "out is NULL");
  if (first < 0 || count < 0 || size_t(first) + size_t(count) > D->flat_gpus.size())
    return fail(EMU_ERR_RANGE, "GPU range out of bounds");
  if (count) std::memcpy(out, D->flat_gpus.data() + first, size_t(count) * sizeof(int32_t));
  return EMU_OK;
}

int emu_dag_target_unit(emu_dag_t dag, int32_t stage, int32_t unit, int32_t* gpus_out) {
  clear_error();
  const Dag* D = reinterpret_cast<const Dag*>(dag);
  if (!dag_live(D)) return fail(EMU_ERR_HANDLE, "not a live DAG");
  if (!gpus_out) return fail(EMU_ERR_NULL, "gpus_out is NULL");
  if (stage < 0 || size_t(stage) >= D->target_units.size() || unit < 0 ||
      size_t(unit) >= D->target_units[stage].size())
    return fail(EMU_ERR_RANGE, "stage or unit out of range");
  const auto& u = D->target_units[stage][unit];
  std::memcpy(gpus_out, u.data(), u.size() * sizeof(int32_t));
  return EMU_OK;
}

}  // extern "C"
