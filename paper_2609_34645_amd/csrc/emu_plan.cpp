// Host side of the EMU reshard library: layout validation, shard inventory, copy-map compilation,
// bucket geometry, plan queries, options and error reporting. No GPU calls in this file.
//
// The copy map is destination-driven. Every shard tensor is described by "blocks": rectangles of one
// logical tensor (row range x column range) placed at a row/column position of the shard. A
// destination block is intersected with the source blocks of the same logical tensor; each non-empty
// intersection is one 2D copy segment (rows x run bytes, with source and destination row strides).
// Destination rows that no block covers (vocabulary padding) become zero-fill segments. This one rule
// covers the column-parallel, row-parallel and vocab-parallel cuts, the fused QKV and gate/up
// permutations, PP regrouping (a layer's blocks live on the stage that owns it) and changes of the
// fused format, for Split, Merge and their compositions (paper section 5.2, primitives (a) and (b)).
#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <unordered_map>
#include <unordered_set>

#include "emu_internal.h"

namespace emu {

// ------------------------------------------------------------------------------------------------
// errors, handles, options
// ------------------------------------------------------------------------------------------------

static thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_err[0] = 0; }

static std::mutex g_plans_mu;
static std::unordered_set<const Plan*> g_plans;

bool plan_live(const Plan* p) {
  if (!p) return false;
  std::lock_guard<std::mutex> lk(g_plans_mu);
  return g_plans.count(p) && p->magic == kPlanMagic;
}

static std::mutex g_ws_mu;
static std::unordered_map<const void*, const Plan*> g_ws;

void ws_register(const void* ws, const Plan* p) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  g_ws[ws] = p;
}

bool ws_current(const void* ws, const Plan* p) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  const auto it = g_ws.find(ws);
  return it != g_ws.end() && it->second == p;
}

void ws_forget(const Plan* p) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  for (auto it = g_ws.begin(); it != g_ws.end();) it = it->second == p ? g_ws.erase(it) : std::next(it);
}

uint64_t next_plan_id() {
  static std::atomic<uint64_t> next{1};
  return next.fetch_add(1, std::memory_order_relaxed);
}

static std::atomic<int64_t> g_opt[8] = {{0}, {1}, {1}, {0}, {32}, {1}, {-1}, {1}};

int64_t option(int32_t key) { return g_opt[key].load(std::memory_order_relaxed); }

// ------------------------------------------------------------------------------------------------
// layouts and inventory
// ------------------------------------------------------------------------------------------------

// Logical tensor ids: 0 = embedding; 1 + 9*l + k for layer l (k: 0 attn_norm, 1 q, 2 k, 3 v, 4 o,
// 5 mlp_norm, 6 gate, 7 up, 8 down); 1 + 9*L = final norm; 2 + 9*L = LM head.
enum { LK_ATTN_NORM = 0, LK_Q, LK_K, LK_V, LK_O, LK_MLP_NORM, LK_GATE, LK_UP, LK_DOWN };

struct Block {
  int32_t lt;             // logical tensor id
  int64_t lrow0, nrows;   // logical rows covered
  int64_t lcol0, ncols;   // logical columns covered
  int64_t row0, col0;     // position inside the shard tensor
  bool replica = false;   // a copy of data an earlier rank holds too (never used as a source)
};

static int elem_size(int32_t dtype) { return dtype == EMU_BF16 ? 2 : dtype == EMU_FP32 ? 4 : 0; }

static int check_layout(const emu_layout_t* l) {
  if (!l) return fail(EMU_ERR_NULL, "layout is NULL");
  const emu_model_t& m = l->model;
  if (m.num_layers <= 0 || m.hidden <= 0 || m.num_heads <= 0 || m.num_kv_heads <= 0 ||
      m.head_dim <= 0 || m.ffn_hidden <= 0 || m.vocab <= 0)
    return fail(EMU_ERR_LAYOUT, "model dimensions must be positive");
  if (l->tp <= 0 || l->pp <= 0 || l->vocab_pad_multiple < 0)
    return fail(EMU_ERR_LAYOUT, "tp and pp must be positive, the pad multiple non-negative");
  if (!elem_size(l->dtype)) return fail(EMU_ERR_LAYOUT, "unknown dtype %d", l->dtype);
  if (l->qkv_format != EMU_QKV_HEAD_INTERLEAVED && l->qkv_format != EMU_QKV_SEPARATE)
    return fail(EMU_ERR_LAYOUT, "unknown qkv format %d", l->qkv_format);
  if (l->mlp_format != EMU_GATE_UP_BLOCK && l->mlp_format != EMU_GATE_UP_SEPARATE)
    return fail(EMU_ERR_LAYOUT, "unknown mlp format %d", l->mlp_format);
  if (m.num_heads % m.num_kv_heads)
    return fail(EMU_ERR_LAYOUT, "query heads (%d) not a multiple of KV heads (%d)", m.num_heads, m.num_kv_heads);
  if (l->tp <= m.num_kv_heads && m.num_kv_heads % l->tp)
    return fail(EMU_ERR_LAYOUT, "tp=%d does not divide %d KV heads", l->tp, m.num_kv_heads);
  if (l->tp > m.num_kv_heads && (l->tp % m.num_kv_heads || m.num_heads % l->tp))
    return fail(EMU_ERR_LAYOUT, "tp=%d replicates KV heads: it must be a multiple of %d KV heads and divide %d heads",
                l->tp, m.num_kv_heads, m.num_heads);
  if (m.ffn_hidden % l->tp) return fail(EMU_ERR_LAYOUT, "tp=%d does not divide the MLP width %d", l->tp, m.ffn_hidden);
  if (l->pp > m.num_layers) return fail(EMU_ERR_LAYOUT, "pp=%d exceeds %d layers", l->pp, m.num_layers);
  if (l->vocab_pad_multiple == 0 && m.vocab % l->tp)
    return fail(EMU_ERR_LAYOUT, "tp=%d does not divide the unpadded vocabulary %d", l->tp, m.vocab);
  return EMU_OK;
}

static int64_t padded_vocab(const emu_layout_t& l) {
  int64_t V = l.model.vocab;
  if (l.vocab_pad_multiple == 0) return V;
  int64_t q = int64_t(l.tp) * l.vocab_pad_multiple;
  return (V + q - 1) / q * q;
}

// Build one side's tensor list (global, rank-major canonical order) and each tensor's blocks.
static int build_side(const emu_layout_t& lay, SideInfo& s, std::vector<std::vector<Block>>& blocks) {
  int rc = check_layout(&lay);
  if (rc) return rc;
  const emu_model_t& m = lay.model;
  const int tp = lay.tp, pp = lay.pp, es = elem_size(lay.dtype);
  const int64_t H = m.hidden, hd = m.head_dim, G = m.num_kv_heads, nH = m.num_heads, I = m.ffn_hidden;
  const int64_t qpg = nH / G, V = m.vocab;
  const bool kv_rep = tp > G;                 // KV heads replicated over tp / G ranks each
  const int64_t gl = kv_rep ? 1 : G / tp;     // KV heads (groups) held per rank
  const int L = m.num_layers, per_stage = L / pp, extra = L % pp;  // the first `extra` stages hold one more
  s.lay = lay;
  s.vp = padded_vocab(lay);
  s.nranks = tp * pp;
  const int64_t vr = s.vp / tp;
  s.tensors.clear();
  s.rank_first.assign(s.nranks + 1, 0);
  blocks.clear();

  auto add = [&](int r, int kind, int layer, int ndim, int64_t rows, int64_t cols) {
    emu_tensor_desc_t d{};
    d.rank = r; d.kind = kind; d.layer = layer; d.ndim = ndim; d.rows = rows; d.cols = cols;
    d.alias = -1;
    d.bytes = uint64_t(rows) * uint64_t(cols) * uint64_t(es);
    s.tensors.push_back(d);
    blocks.emplace_back();
    return &blocks.back();
  };
  auto lt_layer = [&](int l, int k) { return 1 + 9 * l + k; };
  auto vocab_block = [&](std::vector<Block>* b, int lt, int t) {
    int64_t real = std::max<int64_t>(0, std::min<int64_t>(vr, V - t * vr));
    if (real > 0) b->push_back({lt, t * vr, real, 0, H, 0, 0});
  };

  for (int p = 0; p < pp; ++p) {
    for (int t = 0; t < tp; ++t) {
      const int r = p * tp + t;
      s.rank_first[r] = uint32_t(s.tensors.size());
      const bool norm_rep = t != 0;                              // norms: TP rank 0 is the source
      const int64_t rep = kv_rep ? tp / G : 1;                   // ranks sharing one KV head
      const bool kv_replica = kv_rep && t % rep != 0;            // not the first holder of its KV head
      const int l0 = p * per_stage + std::min(p, extra);
      const int l1 = l0 + per_stage + (p < extra ? 1 : 0);
      if (p == 0) vocab_block(add(r, EMU_T_EMBED, -1, 2, vr, H), 0, t);
      for (int l = l0; l < l1; ++l) {
        add(r, EMU_T_ATTN_NORM, l, 1, 1, H)->push_back({lt_layer(l, LK_ATTN_NORM), 0, 1, 0, H, 0, 0, norm_rep});
        const int64_t nq = nH / tp * hd;                         // query rows of this rank
        if (kv_rep) {
          const int64_t g = t / rep;                             // the KV head this rank holds a copy of
          Block q{lt_layer(l, LK_Q), t * nq, nq, 0, H, 0, 0};
          Block k{lt_layer(l, LK_K), g * hd, hd, 0, H, 0, 0, kv_replica};
          Block v{lt_layer(l, LK_V), g * hd, hd, 0, H, 0, 0, kv_replica};
          if (lay.qkv_format == EMU_QKV_HEAD_INTERLEAVED) {
            auto* b = add(r, EMU_T_QKV, l, 2, nq + 2 * hd, H);
            k.row0 = nq;
            v.row0 = nq + hd;
            b->push_back(q);
            b->push_back(k);
            b->push_back(v);
          } else {
            add(r, EMU_T_Q, l, 2, nq, H)->push_back(q);
            add(r, EMU_T_K, l, 2, hd, H)->push_back(k);
            add(r, EMU_T_V, l, 2, hd, H)->push_back(v);
          }
        } else if (lay.qkv_format == EMU_QKV_HEAD_INTERLEAVED) {
          auto* b = add(r, EMU_T_QKV, l, 2, (nH / tp + 2 * gl) * hd, H);
          for (int64_t j = 0; j < gl; ++j) {
            const int64_t g = t * gl + j, base = j * (qpg + 2) * hd;
            b->push_back({lt_layer(l, LK_Q), g * qpg * hd, qpg * hd, 0, H, base, 0});
            b->push_back({lt_layer(l, LK_K), g * hd, hd, 0, H, base + qpg * hd, 0});
            b->push_back({lt_layer(l, LK_V), g * hd, hd, 0, H, base + (qpg + 1) * hd, 0});
          }
        } else {
          add(r, EMU_T_Q, l, 2, nq, H)->push_back({lt_layer(l, LK_Q), t * nq, nq, 0, H, 0, 0});
          add(r, EMU_T_K, l, 2, gl * hd, H)->push_back({lt_layer(l, LK_K), t * gl * hd, gl * hd, 0, H, 0, 0});
          add(r, EMU_T_V, l, 2, gl * hd, H)->push_back({lt_layer(l, LK_V), t * gl * hd, gl * hd, 0, H, 0, 0});
        }
        const int64_t oc = nH * hd / tp;
        add(r, EMU_T_O, l, 2, H, oc)->push_back({lt_layer(l, LK_O), 0, H, t * oc, oc, 0, 0});
        add(r, EMU_T_MLP_NORM, l, 1, 1, H)->push_back({lt_layer(l, LK_MLP_NORM), 0, 1, 0, H, 0, 0, norm_rep});
        const int64_t il = I / tp;
        if (lay.mlp_format == EMU_GATE_UP_BLOCK) {
          auto* b = add(r, EMU_T_GATE_UP, l, 2, 2 * il, H);
          b->push_back({lt_layer(l, LK_GATE), t * il, il, 0, H, 0, 0});
          b->push_back({lt_layer(l, LK_UP), t * il, il, 0, H, il, 0});
        } else {
          add(r, EMU_T_GATE, l, 2, il, H)->push_back({lt_layer(l, LK_GATE), t * il, il, 0, H, 0, 0});
          add(r, EMU_T_UP, l, 2, il, H)->push_back({lt_layer(l, LK_UP), t * il, il, 0, H, 0, 0});
        }
        add(r, EMU_T_DOWN, l, 2, H, il)->push_back({lt_layer(l, LK_DOWN), 0, H, t * il, il, 0, 0});
      }
      if (p == pp - 1) {
        add(r, EMU_T_FINAL_NORM, -1, 1, 1, H)->push_back({1 + 9 * L, 0, 1, 0, H, 0, 0, norm_rep});
        vocab_block(add(r, EMU_T_LM_HEAD, -1, 2, vr, H), 2 + 9 * L, t);
      }
      if (s.tensors.size() - s.rank_first[r] > size_t(kMaxRankTensors))
        return fail(EMU_ERR_UNSUPPORTED, "rank %d holds more than %d tensors", r, kMaxRankTensors);
    }
  }
  s.rank_first[s.nranks] = uint32_t(s.tensors.size());
  s.rank_bytes.assign(s.nranks, 0);
  s.chunk_first.assign(s.nranks + 1, 0);
  s.total_bytes = 0;
  s.offsets_grid = true;
  for (int r = 0; r < s.nranks; ++r) {
    uint64_t off = 0;
    for (uint32_t i = s.rank_first[r]; i < s.rank_first[r + 1]; ++i) {
      s.tensors[i].stream_offset = off;
      s.offsets_grid = s.offsets_grid && off % kTileChunkBytes == 0;
      off += s.tensors[i].bytes;
    }
    s.rank_bytes[r] = off;
    s.total_bytes += off;
    s.chunk_first[r + 1] = s.chunk_first[r] + (off + kChunkBytes - 1) / kChunkBytes;
  }
  return EMU_OK;
}

// ------------------------------------------------------------------------------------------------
// copy map
// ------------------------------------------------------------------------------------------------

struct SrcRef {
  int32_t tensor;
  Block b;
};

static void push_segment(std::vector<emu_segment_t>& out, const emu_segment_t& s) {
  if (!out.empty()) {
    emu_segment_t& p = out.back();
    // append to the previous run when both are single runs, same tensors, contiguous on both sides
    if (p.rows == 1 && s.rows == 1 && p.src_tensor == s.src_tensor && p.dst_tensor == s.dst_tensor &&
        p.src_tensor >= 0 && p.src_offset + p.src_run == s.src_offset && p.dst_offset + p.run == s.dst_offset) {
      p.run += s.run;
      p.src_run += s.src_run;
      p.src_stride = p.src_run;
      p.dst_stride = p.run;
      return;
    }
  }
  out.push_back(s);
}

static int compile(Plan& P, const std::vector<std::vector<Block>>& sb, const std::vector<std::vector<Block>>& db) {
  const SideInfo& S = P.side[0];
  const SideInfo& D = P.side[1];
  const uint64_t ess = uint64_t(elem_size(S.lay.dtype)), esd = uint64_t(elem_size(D.lay.dtype));
  const int nlt = 3 + 9 * S.lay.model.num_layers;

  // source blocks per logical tensor; replicated data (norms on TP ranks > 0, KV heads past their first
  // holder) is read from its first holder only
  std::vector<std::vector<SrcRef>> by_lt(nlt);
  for (size_t i = 0; i < S.tensors.size(); ++i)
    for (const Block& b : sb[i])
      if (!b.replica) by_lt[b.lt].push_back({int32_t(i), b});
  for (auto& v : by_lt)
    std::sort(v.begin(), v.end(), [](const SrcRef& a, const SrcRef& b) {
      return a.b.lrow0 != b.b.lrow0 ? a.b.lrow0 < b.b.lrow0 : a.b.lcol0 < b.b.lcol0;
    });

  P.segs.clear();
  for (size_t j = 0; j < D.tensors.size(); ++j) {
    const emu_tensor_desc_t& dt = D.tensors[j];
    int64_t covered_rows = 0;
    for (const Block& b : db[j]) {
      for (const SrcRef& sr : by_lt[b.lt]) {
        const Block& s = sr.b;
        const int64_t r0 = std::max(b.lrow0, s.lrow0), r1 = std::min(b.lrow0 + b.nrows, s.lrow0 + s.nrows);
        const int64_t c0 = std::max(b.lcol0, s.lcol0), c1 = std::min(b.lcol0 + b.ncols, s.lcol0 + s.ncols);
        if (r0 >= r1 || c0 >= c1) continue;
        const emu_tensor_desc_t& st = S.tensors[sr.tensor];
        emu_segment_t g{};
        g.src_tensor = sr.tensor;
        g.dst_tensor = int32_t(j);
        g.src_offset = uint64_t((s.row0 + r0 - s.lrow0) * st.cols + (s.col0 + c0 - s.lcol0)) * ess;
        g.dst_offset = uint64_t((b.row0 + r0 - b.lrow0) * dt.cols + (b.col0 + c0 - b.lcol0)) * esd;
        g.src_stride = uint64_t(st.cols) * ess;
        g.dst_stride = uint64_t(dt.cols) * esd;
        g.rows = uint64_t(r1 - r0);
        g.run = uint64_t(c1 - c0) * esd;
        g.src_run = uint64_t(c1 - c0) * ess;
        if (g.rows == 1 || (g.src_run == g.src_stride && g.run == g.dst_stride)) {
          g.run *= g.rows;
          g.src_run *= g.rows;
          g.rows = 1;
          g.src_stride = g.src_run;
          g.dst_stride = g.run;
        }
        push_segment(P.segs, g);
      }
      covered_rows += b.nrows * (b.ncols == dt.cols ? 1 : 0);
    }
    if ((dt.kind == EMU_T_EMBED || dt.kind == EMU_T_LM_HEAD) && covered_rows < dt.rows) {
      // destination vocabulary pad rows: no source, written with zeros
      emu_segment_t z{};
      z.src_tensor = -1;
      z.dst_tensor = int32_t(j);
      z.dst_offset = uint64_t(covered_rows) * dt.cols * esd;
      z.run = uint64_t(dt.rows - covered_rows) * dt.cols * esd;
      z.src_run = 0;
      z.rows = 1;
      z.src_stride = z.dst_stride = z.run;
      P.segs.push_back(z);
    }
  }
  return EMU_OK;
}

// Destination tensors that are byte copies of one whole source tensor: exactly one segment covers them,
// from offset 0 of a source tensor of the same size, as one run, without conversion. These are the shards
// a transition finds already in place (a PP-only change: every tensor; a TP change: the replicated norms,
// and tensors whose TP slicing the two layouts share). With `drop`, their segments leave the map.
static void find_aliases(Plan& P, bool drop) {
  SideInfo& D = P.side[1];
  const SideInfo& S = P.side[0];
  std::vector<int32_t> nseg(D.tensors.size(), 0);
  for (const emu_segment_t& g : P.segs) ++nseg[g.dst_tensor];
  for (const emu_segment_t& g : P.segs) {
    emu_tensor_desc_t& d = D.tensors[g.dst_tensor];
    if (nseg[g.dst_tensor] == 1 && g.src_tensor >= 0 && P.cvt == CVT_NONE && g.rows == 1 && g.src_offset == 0 &&
        g.dst_offset == 0 && g.run == d.bytes && S.tensors[g.src_tensor].bytes == d.bytes)
      d.alias = g.src_tensor;
  }
  P.aliased = drop;
  if (drop)
    P.segs.erase(std::remove_if(P.segs.begin(), P.segs.end(),
                                [&](const emu_segment_t& g) { return D.tensors[g.dst_tensor].alias >= 0; }),
                 P.segs.end());
}

// The bucket list of one side for bucket size B: per rank its stream cut every B bytes, each bucket a
// 1D tensor whose stream offset is k * B.
static SideInfo bucket_side(const SideInfo& X, uint64_t B) {
  const uint64_t es = uint64_t(elem_size(X.lay.dtype));
  SideInfo bk;
  bk.lay = X.lay;
  bk.vp = X.vp;
  bk.nranks = X.nranks;
  bk.total_bytes = X.total_bytes;
  bk.offsets_grid = B % kTileChunkBytes == 0 || X.nranks == 0;
  bk.rank_first.assign(X.nranks + 1, 0);
  bk.rank_bytes = X.rank_bytes;
  bk.chunk_first.assign(X.nranks + 1, 0);
  for (int r = 0; r < X.nranks; ++r) {
    bk.rank_first[r] = uint32_t(bk.tensors.size());
    for (uint64_t k = 0; k * B < X.rank_bytes[r]; ++k) {
      emu_tensor_desc_t d{};
      d.rank = r;
      d.kind = EMU_T_BUCKET;
      d.layer = -1;
      d.ndim = 1;
      d.bytes = std::min<uint64_t>(B, X.rank_bytes[r] - k * B);
      d.alias = -1;
      d.rows = 1;
      d.cols = int64_t(d.bytes / es);
      d.stream_offset = k * B;
      bk.tensors.push_back(d);
    }
    bk.chunk_first[r + 1] = bk.chunk_first[r] + (X.rank_bytes[r] + kChunkBytes - 1) / kChunkBytes;
  }
  bk.rank_first[X.nranks] = uint32_t(bk.tensors.size());
  return bk;
}

// Rewrite a destination-driven copy map so that it writes the destination ranks' bucket streams
// instead of the destination tensors: tensor j's byte o lands at stream position
// stream_offset(j) + o of its rank, i.e. in bucket (pos / B) at offset (pos % B). Rows that stay inside
// one bucket keep their 2D shape; a row that crosses a bucket boundary is cut into 1D pieces there.
// The destination side becomes the list of buckets (rank 0's first), so the result runs on the
// ordinary reshard kernel with the bucket pointer table as its destination table.
static int to_buckets(Plan& P, uint64_t B) {
  SideInfo& D = P.side[1];
  const uint64_t es = uint64_t(elem_size(D.lay.dtype));
  const uint64_t ess = uint64_t(elem_size(P.side[0].lay.dtype));  // source bytes per destination element
  if (B == 0 || B % es)
    return fail(EMU_ERR_BUCKET, "bucket size %llu is not a positive multiple of %llu", (unsigned long long)B,
                (unsigned long long)es);
  std::vector<uint64_t> base(D.nranks + 1, 0);
  for (int r = 0; r < D.nranks; ++r) base[r + 1] = base[r] + (D.rank_bytes[r] + B - 1) / B;
  if (base[D.nranks] > 0x7fffffffull) return fail(EMU_ERR_UNSUPPORTED, "too many buckets");
  std::vector<emu_segment_t> out;
  out.reserve(P.segs.size() + 64);
  auto emit = [&](const emu_segment_t& g, uint64_t src_off, int64_t bucket, uint64_t dst_off, uint64_t rows,
                  uint64_t run, bool one_d) {
    emu_segment_t s = g;
    s.src_offset = src_off;
    s.dst_tensor = int32_t(bucket);
    s.dst_offset = dst_off;
    s.rows = rows;
    s.run = run;
    s.src_run = g.src_tensor >= 0 ? run / es * ess : 0;
    if (one_d) {
      s.src_stride = s.src_run;
      s.dst_stride = run;
    }
    push_segment(out, s);
  };
  for (const emu_segment_t& g : P.segs) {
    const emu_tensor_desc_t& t = D.tensors[g.dst_tensor];
    const uint64_t s0 = t.stream_offset + g.dst_offset;
    uint64_t i = 0;
    while (i < g.rows) {
      const uint64_t si = s0 + i * g.dst_stride;
      const uint64_t k = si / B, bend = (k + 1) * B;
      const uint64_t so = g.src_offset + i * g.src_stride;
      if (si + g.run <= bend) {
        // rows i .. i+n-1 end inside bucket k
        uint64_t n = 1;
        if (g.rows > 1) n = std::min<uint64_t>(g.rows - i, (bend - si - g.run) / g.dst_stride + 1);
        emit(g, so, int64_t(base[t.rank] + k), si - k * B, n, g.run, g.rows == 1);
        i += n;
      } else {
        // row i crosses at least one bucket boundary: cut it there
        for (uint64_t pos = 0; pos < g.run;) {
          const uint64_t sp = si + pos, kk = sp / B;
          const uint64_t e = std::min<uint64_t>(g.run, (kk + 1) * B - si);
          emit(g, so + (g.src_tensor >= 0 ? pos / es * ess : 0), int64_t(base[t.rank] + kk), sp - kk * B, 1, e - pos,
               true);
          pos = e;
        }
        i += 1;
      }
    }
  }
  P.segs.swap(out);
  P.side[1] = bucket_side(D, B);  // the destination side is now the bucket list
  return EMU_OK;
}

// Rewrite a copy map so that it reads the source ranks' bucket streams instead of the source tensors:
// source tensor i's byte o sits at stream position stream_offset(i) + o of its rank, in bucket (pos / B)
// at offset (pos % B). Rows whose source bytes stay inside one bucket keep their 2D shape; a row whose
// source bytes cross a bucket boundary is cut there, on an element boundary (B and every stream offset
// are multiples of the source element size), and its destination bytes with it. The source side
// becomes the list of buckets (rank 0's first), so that the receiver of a transfer restores -- or
// reshards -- its tensors straight from the contiguous buffers on the ordinary reshard kernel.
static int from_buckets(Plan& P, uint64_t B) {
  SideInfo& S = P.side[0];
  const uint64_t ess = uint64_t(elem_size(S.lay.dtype));          // source bytes per element
  const uint64_t esd = uint64_t(elem_size(P.side[1].lay.dtype));  // destination bytes per element
  if (B == 0 || B % ess)
    return fail(EMU_ERR_BUCKET, "bucket size %llu is not a positive multiple of %llu", (unsigned long long)B,
                (unsigned long long)ess);
  std::vector<uint64_t> base(S.nranks + 1, 0);
  for (int r = 0; r < S.nranks; ++r) base[r + 1] = base[r] + (S.rank_bytes[r] + B - 1) / B;
  if (base[S.nranks] > 0x7fffffffull) return fail(EMU_ERR_UNSUPPORTED, "too many buckets");
  std::vector<emu_segment_t> out;
  out.reserve(P.segs.size() + 64);
  auto emit = [&](const emu_segment_t& g, int64_t bucket, uint64_t src_off, uint64_t dst_off, uint64_t rows,
                  uint64_t run, uint64_t src_run, bool one_d) {
    emu_segment_t s = g;
    s.src_tensor = int32_t(bucket);
    s.src_offset = src_off;
    s.dst_offset = dst_off;
    s.rows = rows;
    s.run = run;
    s.src_run = src_run;
    if (one_d) {
      s.src_stride = src_run;
      s.dst_stride = run;
    }
    push_segment(out, s);
  };
  for (const emu_segment_t& g : P.segs) {
    if (g.src_tensor < 0) {  // zero fill: no source bytes
      push_segment(out, g);
      continue;
    }
    const emu_tensor_desc_t& t = S.tensors[g.src_tensor];
    const uint64_t s0 = t.stream_offset + g.src_offset;
    uint64_t i = 0;
    while (i < g.rows) {
      const uint64_t si = s0 + i * g.src_stride;
      const uint64_t k = si / B, bend = (k + 1) * B;
      const uint64_t di = g.dst_offset + i * g.dst_stride;
      if (si + g.src_run <= bend) {
        // rows i .. i+n-1 read inside bucket k
        uint64_t n = 1;
        if (g.rows > 1)
          n = g.src_stride ? std::min<uint64_t>(g.rows - i, (bend - si - g.src_run) / g.src_stride + 1) : g.rows - i;
        emit(g, int64_t(base[t.rank] + k), si - k * B, di, n, g.run, g.src_run, g.rows == 1);
        i += n;
      } else {
        // row i's source bytes cross at least one bucket boundary: cut them there
        for (uint64_t pos = 0; pos < g.src_run;) {
          const uint64_t sp = si + pos, kk = sp / B;
          const uint64_t e = std::min<uint64_t>(g.src_run, (kk + 1) * B - si);
          emit(g, int64_t(base[t.rank] + kk), sp - kk * B, di + pos / ess * esd, 1, (e - pos) / ess * esd, e - pos,
               true);
          pos = e;
        }
        i += 1;
      }
    }
  }
  P.segs.swap(out);
  P.side[0] = bucket_side(S, B);  // the source side is now the bucket list
  for (emu_tensor_desc_t& d : P.side[1].tensors) d.alias = -1;  // no destination tensor is a source tensor
  return EMU_OK;
}

// The tables the upload's kernels build on the device, written into a workspace image of w.total bytes:
// the tile map (each segment's tiles from its first map index; kNoSeg padding), and per side: per tensor its stream offset (exclusive prefix sum of the rank's
// tensor sizes), per rank {first 4 KB chunk, stream bytes, end of its tensor range, 0}, and per 4 KB
// chunk the rank and the global index of the tensor holding its first byte (chunk j of a rank starts in
// the last tensor whose stream offset is <= j * 4 KB), padded with kNoSeg.
static void device_tables(const Plan& P, uint8_t* h) {
  const WsLayout& w = P.ws;
  uint32_t* tm = reinterpret_cast<uint32_t*>(h + w.off_tilemap);
  for (size_t i = 0; i < P.dsegs.size(); ++i) std::fill_n(tm + P.dsegs[i].tile0, P.seg_tiles[i], uint32_t(i));
  std::fill(tm + P.ntiles_copy, tm + P.zero_tile0, kNoSeg);  // the two sections' padding
  std::fill(tm + P.zero_tile0 + P.ntiles_zero, tm + w.n_map, kNoSeg);
  for (int sd = 0; sd < 2; ++sd) {
    const SideInfo& s = P.side[sd];
    uint64_t* so = reinterpret_cast<uint64_t*>(h + w.side[sd].off_stream);
    for (size_t i = 0; i < s.tensors.size(); ++i) so[i] = s.tensors[i].stream_offset;
    uint64_t* ri = reinterpret_cast<uint64_t*>(h + w.side[sd].off_rank_info);
    uint32_t* cm = reinterpret_cast<uint32_t*>(h + w.side[sd].off_tile_map);
    uint64_t first = 0;
    for (int r = 0; r < s.nranks; ++r) {
      const uint32_t t0 = s.rank_first[r], t1 = s.rank_first[r + 1];
      const uint64_t nch = (s.rank_bytes[r] + kTileChunkBytes - 1) / kTileChunkBytes;
      ri[4 * r + 0] = first;
      ri[4 * r + 1] = s.rank_bytes[r];
      ri[4 * r + 2] = t1;
      ri[4 * r + 3] = 0;
      if (w.side[sd].n_tiles)
        for (uint32_t g = t0; g < t1; ++g) {
          const uint64_t j0 = (s.tensors[g].stream_offset + kTileChunkBytes - 1) / kTileChunkBytes;
          const uint64_t j1 = g + 1 < t1 ? (s.tensors[g + 1].stream_offset + kTileChunkBytes - 1) / kTileChunkBytes : nch;
          if (j1 > j0) std::fill(cm + first + j0, cm + first + j1, (uint32_t(r) << kMapTensorBits) | g);
        }
      first += nch;
    }
    if (w.side[sd].n_tiles) std::fill(cm + first, cm + w.side[sd].n_tiles, kNoSeg);
  }
}

// Device segments, tiles and the workspace layout.
// Whether a 2D vector segment can run as SEG_VEC_FLAT with tiles of TV vectors: the kernel finds the
// row of vector n (n below rows * rv) as umulhi(n, ceil(2^32 / rv)), exact while n * rv < 2^32, and
// keeps in-tile byte offsets in 31 bits: a tile spans at most 2 + TV / rv rows.
static bool flat_ok(const emu_segment_t& g, uint64_t TV) {
  const uint64_t rv = g.run / 16;
  if (g.rows < 2 || rv == 0 || g.rows > 0xffffffffull) return false;
  if (rv > 0xffffffffull / rv || g.rows > 0xffffffffull / (rv * rv)) return false;  // rows * rv * rv < 2^32
  const uint64_t stride = std::max(g.src_stride, g.dst_stride);
  return stride < (1ull << 31) / (2 + TV / rv);
}

static int finalize(Plan& P) {
  const int U = P.tile_vecs;
  const uint64_t TV = uint64_t(kReshardThreads) * U;  // vectors per tile
  const uint64_t TB = TV * 16;                 // bytes per tile
  P.tile_bytes = TB;
  P.dsegs.clear();
  std::vector<uint64_t> segtiles;  // tiles of each segment
  uint64_t tiles = 0, zero_bytes = 0, written = 0, read = 0;
  int64_t nzero = 0;
  // source alignment the vector paths need: 16 bytes when each destination vector reads one or two
  // whole source vectors, 8 bytes when it reads half of one (bf16 -> fp32)
  const uint64_t salign = P.cvt == CVT_BF16_F32 ? 8 : 16;
  int32_t ngeneral = 0;
  const bool row_wrap = option(EMU_OPT_ROW_WRAP) != 0;
  for (size_t i = 0; i < P.segs.size(); ++i) {
    const emu_segment_t& g = P.segs[i];
    DevSeg d{};
    d.src_off = g.src_offset; d.dst_off = g.dst_offset;
    d.src_stride = g.src_stride; d.dst_stride = g.dst_stride;
    d.rows = g.rows; d.run = g.run;
    d.src_idx = g.src_tensor; d.dst_idx = g.dst_tensor;
    const bool zero = g.src_tensor < 0;
    const bool vec = ((g.dst_offset | g.run) % 16 == 0) && (g.rows == 1 || g.dst_stride % 16 == 0) &&
                     (zero || (g.src_offset % salign == 0 && (g.rows == 1 || g.src_stride % salign == 0)));
    uint64_t nt;
    if (!vec) {
      d.mode = SEG_GENERAL;
      const uint64_t tpr = (g.run + TB - 1) / TB;
      if (tpr > 0xffffffffull) return fail(EMU_ERR_UNSUPPORTED, "row of %llu bytes too long", (unsigned long long)g.run);
      d.param = uint32_t(tpr);
      nt = g.rows * tpr;
      ++ngeneral;
    } else if (g.rows == 1) {
      d.mode = SEG_VEC_1D;
      nt = (g.run + TB - 1) / TB;
    } else if (row_wrap && flat_ok(g, TV)) {
      d.mode = SEG_VEC_FLAT;
      d.rv = uint32_t(g.run / 16);
      d.param = uint32_t(g.rows * d.rv);
      d.magic = d.rv > 1 ? uint32_t(((1ull << 32) + d.rv - 1) / d.rv) : 0u;
      nt = (d.param + TV - 1) / TV;
    } else if (g.run <= TB) {
      d.mode = SEG_VEC_ROWS;
      d.rv = uint32_t(g.run / 16);
      // whole rows per tile, few enough that every in-tile byte offset stays below 2^31
      const uint64_t stride = std::max(g.src_stride, g.dst_stride);
      const uint64_t by_offset = stride < (1ull << 31) ? ((1ull << 31) - g.run) / stride + 1 : 1;
      d.param = uint32_t(std::max<uint64_t>(1, std::min<uint64_t>(TB / g.run, by_offset)));
      d.magic = d.rv > 1 ? uint32_t(((1ull << 32) + d.rv - 1) / d.rv) : 0u;
      nt = (g.rows + d.param - 1) / d.param;
    } else {
      d.mode = SEG_VEC_ROWCHUNK;
      const uint64_t tpr = (g.run + TB - 1) / TB;
      d.param = uint32_t(tpr);
      nt = g.rows * tpr;
    }
    if (zero) {
      d.mode |= SEG_ZERO;
      zero_bytes += g.rows * g.run;
      ++nzero;
    }
    written += g.rows * g.run;
    read += g.rows * g.src_run;
    if (tiles + nt > 0xfffffff0ull) return fail(EMU_ERR_UNSUPPORTED, "too many tiles");
    tiles += nt;
    segtiles.push_back(nt);
    P.dsegs.push_back(d);
  }
  P.ntiles = tiles;
  // Tile map: the copy segments' tiles, then the zero-fill segments' tiles, which run on their own
  // kernel instance. Each section is padded with kNoSeg to a whole number of XCD groups, so that every
  // workgroup of a grid (a multiple of kXcdCount) reads an entry of its own section and the kernel
  // needs no bounds check before its first load. Here each segment gets its first map index; the
  // upload's k_tile_map writes the map on the device from those indices and the tile counts.
  uint64_t nmap = 0;
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1) P.zero_tile0 = nmap;
    for (size_t i = 0; i < P.dsegs.size(); ++i) {
      if (((P.dsegs[i].mode & SEG_ZERO) != 0) != (pass == 1)) continue;
      P.dsegs[i].tile0 = nmap;
      nmap += segtiles[i];
    }
    if (pass == 0) P.ntiles_copy = nmap;
    else P.ntiles_zero = nmap - P.zero_tile0;
    nmap = (nmap + kXcdCount - 1) / kXcdCount * kXcdCount;
  }
  int32_t n_alias = 0;
  uint64_t alias_bytes = 0;
  for (const emu_tensor_desc_t& d : P.side[1].tensors)
    if (d.alias >= 0) {
      ++n_alias;
      alias_bytes += d.bytes;
    }
  if (written + (P.aliased ? alias_bytes : 0) != P.side[1].total_bytes)
    return fail(EMU_ERR_ARG, "internal: copy map covers %llu of %llu destination bytes",
                (unsigned long long)written, (unsigned long long)P.side[1].total_bytes);

  // Per side, for the tile-per-workgroup pack/unpack kernel: a chunk -> (rank, global tensor) map,
  // padded with kNoSeg to a multiple of kXcdCount (the kernel's grid), and per rank {first chunk,
  // stream bytes, end of its tensor range}. A side the map cannot encode gets an empty map.
  uint64_t nchunk[2] = {0, 0};
  for (int sd = 0; sd < 2; ++sd) {
    const SideInfo& s = P.side[sd];
    const bool encodable = s.nranks < (1 << (32 - kMapTensorBits)) && s.tensors.size() <= (1u << kMapTensorBits);
    uint64_t n = 0;
    for (int r = 0; r < s.nranks; ++r) n += (s.rank_bytes[r] + kTileChunkBytes - 1) / kTileChunkBytes;
    nchunk[sd] = encodable && n <= 0x7fffff00ull ? (n + kXcdCount - 1) / kXcdCount * kXcdCount : 0;
  }

  // workspace image (WsLayout): the host fills the segments, their tile counts and the sides' host
  // tables; the upload's kernels derive the tile map and the sides' stream tables (device_tables below
  // gives the host's copy of those, for checking)
  auto align = [](uint64_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; };
  P.seg_tiles.assign(segtiles.begin(), segtiles.end());  // each below 2^32: the map has fewer tiles
  WsLayout& w = P.ws;
  uint64_t off = 0;
  w.off_segs = off; off = align(off + P.dsegs.size() * sizeof(DevSeg));
  w.off_seg_tiles = off; off = align(off + P.dsegs.size() * 4);
  w.off_tilemap = off; off = align(off + nmap * 4);
  w.n_map = nmap;
  w.reshard_bytes = off;
  for (int sd = 0; sd < 2; ++sd) {
    const SideInfo& s = P.side[sd];
    w.side[sd].off_sizes = off; off = align(off + s.tensors.size() * 8);
    w.side[sd].off_rank_first = off; off = align(off + (s.nranks + 1) * 4);
    w.side[sd].off_rank_bytes = off; off = align(off + s.nranks * 8);
    w.side[sd].off_chunk_first = off; off = align(off + (s.nranks + 1) * 8);
  }
  w.host_end = off;
  for (int sd = 0; sd < 2; ++sd) {
    const SideInfo& s = P.side[sd];
    w.side[sd].off_stream = off; off = align(off + s.tensors.size() * 8);
    w.side[sd].off_rank_info = off; off = align(off + size_t(s.nranks) * 4 * 8);
    w.side[sd].off_tile_map = off; off = align(off + nchunk[sd] * 4);
    w.side[sd].n_tiles = nchunk[sd];
  }
  w.total = off;
  const uint64_t head = w.off_tilemap;  // host_ws: workspace [0, head), then [reshard_bytes, host_end)
  P.host_ws.assign(head + (w.host_end - w.reshard_bytes), 0);
  uint8_t* h = P.host_ws.data();
  if (!P.dsegs.empty()) {
    std::memcpy(h + w.off_segs, P.dsegs.data(), P.dsegs.size() * sizeof(DevSeg));
    std::memcpy(h + w.off_seg_tiles, P.seg_tiles.data(), P.seg_tiles.size() * 4);
  }
  uint8_t* hb = h + head - w.reshard_bytes;  // hb + (workspace offset of a side host table)
  for (int sd = 0; sd < 2; ++sd) {
    const SideInfo& s = P.side[sd];
    uint64_t* sz = reinterpret_cast<uint64_t*>(hb + w.side[sd].off_sizes);
    for (size_t i = 0; i < s.tensors.size(); ++i) sz[i] = s.tensors[i].bytes;
    std::memcpy(hb + w.side[sd].off_rank_first, s.rank_first.data(), s.rank_first.size() * 4);
    std::memcpy(hb + w.side[sd].off_rank_bytes, s.rank_bytes.data(), s.rank_bytes.size() * 8);
    std::memcpy(hb + w.side[sd].off_chunk_first, s.chunk_first.data(), s.chunk_first.size() * 8);
  }

  emu_plan_info_t& I = P.info;
  I = emu_plan_info_t{};
  I.n_src_ranks = P.side[0].nranks;
  I.n_dst_ranks = P.side[1].nranks;
  I.n_src_tensors = int32_t(P.side[0].tensors.size());
  I.n_dst_tensors = int32_t(P.side[1].tensors.size());
  I.n_segments = int64_t(P.segs.size());
  I.n_zero_segments = nzero;
  I.n_tiles = int64_t(tiles);
  I.tile_bytes = TB;
  I.bytes_written = written;
  I.zero_fill_bytes = zero_bytes;
  I.bytes_read = read;
  I.converts = P.cvt;
  I.src_bytes = P.side[0].total_bytes;
  I.dst_bytes = P.side[1].total_bytes;
  I.workspace_bytes = w.total;
  I.src_vocab_padded = int32_t(P.side[0].vp);
  I.dst_vocab_padded = int32_t(P.side[1].vp);
  I.n_general_segments = ngeneral;
  I.n_alias_tensors = n_alias;
  I.aliased = P.aliased ? 1 : 0;
  I.alias_bytes = alias_bytes;
  return EMU_OK;
}

}  // namespace emu

using namespace emu;

// ------------------------------------------------------------------------------------------------
// C ABI (host part)
// ------------------------------------------------------------------------------------------------

// ------------------------------------------------------------------------------------------------
// host-side pointer-table checks
// ------------------------------------------------------------------------------------------------

namespace {

struct Range {
  uint64_t lo, hi;  // [lo, hi)
  bool shared;      // may overlap other shared ranges (reshard sources)
  const char* what;
  int64_t index;
};

int add_ranges(std::vector<Range>& out, const uint64_t* ptrs, const std::vector<uint64_t>& sizes, bool shared,
               const char* what, const std::vector<bool>* skip = nullptr) {
  for (size_t i = 0; i < sizes.size(); ++i) {
    if (skip && (*skip)[i]) continue;
    const uint64_t p = ptrs[i];
    if (p == 0) return emu::fail(EMU_ERR_NULL, "%s %zu has a NULL address", what, i);
    if (p % 16) return emu::fail(EMU_ERR_ALIGN, "%s %zu at 0x%llx is not 16-byte aligned", what, i, (unsigned long long)p);
    if (sizes[i] == 0) continue;
    if (p + sizes[i] < p) return emu::fail(EMU_ERR_ARG, "%s %zu wraps the address space", what, i);
    out.push_back(Range{p, p + sizes[i], shared, what, int64_t(i)});
  }
  return EMU_OK;
}

// Sweep in address order: a range conflicts with an earlier one that is still open unless both are
// shared. Holding the furthest-reaching earlier range of each kind is enough to see every conflict.
int sweep(std::vector<Range>& rs) {
  std::sort(rs.begin(), rs.end(), [](const Range& a, const Range& b) { return a.lo < b.lo; });
  const Range* open_shared = nullptr;
  const Range* open_excl = nullptr;
  for (const Range& r : rs) {
    const Range* hit = nullptr;
    if (open_excl && r.lo < open_excl->hi) hit = open_excl;
    else if (!r.shared && open_shared && r.lo < open_shared->hi) hit = open_shared;
    if (hit)
      return emu::fail(EMU_ERR_OVERLAP, "%s %lld [0x%llx, 0x%llx) overlaps %s %lld [0x%llx, 0x%llx)", r.what,
                       (long long)r.index, (unsigned long long)r.lo, (unsigned long long)r.hi, hit->what,
                       (long long)hit->index, (unsigned long long)hit->lo, (unsigned long long)hit->hi);
    const Range*& slot = r.shared ? open_shared : open_excl;
    if (!slot || r.hi > slot->hi) slot = &r;
  }
  return EMU_OK;
}

std::vector<uint64_t> tensor_sizes(const emu::SideInfo& s) {
  std::vector<uint64_t> v(s.tensors.size());
  for (size_t i = 0; i < v.size(); ++i) v[i] = s.tensors[i].bytes;
  return v;
}

}  // namespace

extern "C" {

int emu_version(void) { return EMU_ABI_VERSION; }

const char* emu_status_str(int s) {
  switch (s) {
    case EMU_OK: return "EMU_OK";
    case EMU_ERR_NULL: return "EMU_ERR_NULL";
    case EMU_ERR_LAYOUT: return "EMU_ERR_LAYOUT";
    case EMU_ERR_MISMATCH: return "EMU_ERR_MISMATCH";
    case EMU_ERR_UNSUPPORTED: return "EMU_ERR_UNSUPPORTED";
    case EMU_ERR_WORKSPACE: return "EMU_ERR_WORKSPACE";
    case EMU_ERR_BUCKET: return "EMU_ERR_BUCKET";
    case EMU_ERR_ALIGN: return "EMU_ERR_ALIGN";
    case EMU_ERR_HIP: return "EMU_ERR_HIP";
    case EMU_ERR_HANDLE: return "EMU_ERR_HANDLE";
    case EMU_ERR_RANGE: return "EMU_ERR_RANGE";
    case EMU_ERR_ARG: return "EMU_ERR_ARG";
    case EMU_ERR_INFEASIBLE: return "EMU_ERR_INFEASIBLE";
    case EMU_ERR_OVERLAP: return "EMU_ERR_OVERLAP";
    default: return "EMU_ERR_UNKNOWN";
  }
}

const char* emu_last_error(void) { return g_err; }

int emu_set_option(int32_t key, int64_t value) {
  clear_error();
  switch (key) {
    case EMU_OPT_TILE_VECS:
      if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8 && value != 16)
        return fail(EMU_ERR_ARG, "tile vectors must be 0 (automatic), 1, 2, 4, 8 or 16");
      break;
    case EMU_OPT_WG_PER_CU:
      if (value < -1 || value > 32) return fail(EMU_ERR_ARG, "resident workgroups per CU must be in [-1, 32]");
      break;
    case EMU_OPT_BUCKET_WG_PER_CU:
      if (value < 1 || value > 64) return fail(EMU_ERR_ARG, "workgroups per CU must be in [1, 64]");
      break;
    case EMU_OPT_XCD_REMAP:
    case EMU_OPT_BUCKET_TILES:
    case EMU_OPT_ROW_WRAP:
    case EMU_OPT_NONTEMPORAL:
    case EMU_OPT_LDS_STAGING:
      if (value != 0 && value != 1) return fail(EMU_ERR_ARG, "flag must be 0 or 1");
      break;
    default:
      return fail(EMU_ERR_RANGE, "unknown option %d", key);
  }
  g_opt[key].store(value, std::memory_order_relaxed);
  return EMU_OK;
}

int emu_get_option(int32_t key, int64_t* value) {
  clear_error();
  if (!value) return fail(EMU_ERR_NULL, "value is NULL");
  if (key < 0 || key > EMU_OPT_ROW_WRAP) return fail(EMU_ERR_RANGE, "unknown option %d", key);
  *value = option(key);
  return EMU_OK;
}

int emu_layout_check(const emu_layout_t* layout) {
  clear_error();
  return check_layout(layout);
}

int emu_plan(const emu_layout_t* src, const emu_layout_t* dst, emu_plan_t* out) {
  return emu_plan_ex(src, dst, EMU_PLAN_DEFAULT, out);
}

int emu_plan_ex(const emu_layout_t* src, const emu_layout_t* dst, uint32_t flags, emu_plan_t* out) {
  clear_error();
  if (!src || !dst || !out) return fail(EMU_ERR_NULL, "NULL argument");
  *out = nullptr;
  if (flags & ~uint32_t(EMU_PLAN_ALIAS_RESIDENT)) return fail(EMU_ERR_ARG, "unknown plan flags 0x%x", flags);
  int rc = check_layout(src);
  if (rc) return rc;
  rc = check_layout(dst);
  if (rc) return rc;
  if (std::memcmp(&src->model, &dst->model, sizeof(emu_model_t)) != 0)
    return fail(EMU_ERR_MISMATCH, "source and destination layouts describe different models");
  Plan* P = new (std::nothrow) Plan();
  if (!P) return fail(EMU_ERR_ARG, "out of host memory");
  P->id = next_plan_id();
  try {
    P->cvt = src->dtype == dst->dtype ? CVT_NONE : (src->dtype == EMU_FP32 ? CVT_F32_BF16 : CVT_BF16_F32);
    // automatic tile size: 4 KB (4 vectors per lane of the one-wave workgroup), the size that ran
    // fastest on MI355X for copying and converting plans together with the residency rule of the
    // launch (EMU_OPT_WG_PER_CU)
    const int64_t tv = option(EMU_OPT_TILE_VECS);
    P->tile_vecs = tv > 0 ? int(tv) : 4;
    std::vector<std::vector<Block>> sb, db;
    rc = build_side(*src, P->side[0], sb);
    if (!rc) rc = build_side(*dst, P->side[1], db);
    if (!rc) rc = compile(*P, sb, db);
    if (!rc) find_aliases(*P, (flags & EMU_PLAN_ALIAS_RESIDENT) != 0);
    if (!rc) rc = finalize(*P);
  } catch (const std::bad_alloc&) {
    rc = fail(EMU_ERR_ARG, "out of host memory");
  }
  if (rc) {
    delete P;
    return rc;
  }
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    g_plans.insert(P);
  }
  *out = reinterpret_cast<emu_plan_t>(P);
  return EMU_OK;
}

// emu_plan_to_buckets / emu_plan_from_buckets: the plan of (src, dst) with one side rewritten into
// bucket space, then finalized again.
static int bucket_plan(const emu_layout_t* src, const emu_layout_t* dst, uint64_t bucket_bytes, int side,
                       emu_plan_t* out) {
  clear_error();
  if (!src || !dst || !out) return fail(EMU_ERR_NULL, "NULL argument");
  *out = nullptr;
  emu_plan_t base = nullptr;
  int rc = emu_plan(src, dst, &base);
  if (rc) return rc;
  Plan* P = reinterpret_cast<Plan*>(base);
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    g_plans.erase(P);
  }
  try {
    rc = side == 1 ? to_buckets(*P, bucket_bytes) : from_buckets(*P, bucket_bytes);
    if (!rc) rc = finalize(*P);
  } catch (const std::bad_alloc&) {
    rc = fail(EMU_ERR_ARG, "out of host memory");
  }
  if (rc) {
    delete P;
    return rc;
  }
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    g_plans.insert(P);
  }
  *out = base;
  return EMU_OK;
}

int emu_plan_to_buckets(const emu_layout_t* src, const emu_layout_t* dst, uint64_t bucket_bytes, emu_plan_t* out) {
  return bucket_plan(src, dst, bucket_bytes, 1, out);
}

int emu_plan_from_buckets(const emu_layout_t* src, const emu_layout_t* dst, uint64_t bucket_bytes, emu_plan_t* out) {
  return bucket_plan(src, dst, bucket_bytes, 0, out);
}

int emu_plan_free(emu_plan_t plan) {
  clear_error();
  Plan* P = reinterpret_cast<Plan*>(plan);
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    if (!P || !g_plans.count(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
    g_plans.erase(P);
  }
  ws_forget(P);
  P->magic = 0;
  delete P;
  return EMU_OK;
}

int emu_plan_info(emu_plan_t plan, emu_plan_info_t* out) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!out) return fail(EMU_ERR_NULL, "out is NULL");
  *out = P->info;
  return EMU_OK;
}

int emu_plan_workspace_image(emu_plan_t plan, void* out, uint64_t bytes) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!out) return fail(EMU_ERR_NULL, "out is NULL");
  if (bytes < P->ws.total)
    return fail(EMU_ERR_WORKSPACE, "%llu bytes given, the image takes %llu", (unsigned long long)bytes,
                (unsigned long long)P->ws.total);
  const WsLayout& w = P->ws;
  uint8_t* h = static_cast<uint8_t*>(out);
  std::memset(h, 0, w.total);
  std::memcpy(h, P->host_ws.data(), w.off_tilemap);
  std::memcpy(h + w.reshard_bytes, P->host_ws.data() + w.off_tilemap, w.host_end - w.reshard_bytes);
  device_tables(*P, h);
  return EMU_OK;
}

int emu_tensor_info(emu_plan_t plan, int32_t side, int32_t index, emu_tensor_desc_t* out) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!out) return fail(EMU_ERR_NULL, "out is NULL");
  if (side != 0 && side != 1) return fail(EMU_ERR_RANGE, "side must be 0 (source) or 1 (destination)");
  const auto& t = P->side[side].tensors;
  if (index < 0 || size_t(index) >= t.size()) return fail(EMU_ERR_RANGE, "tensor index %d out of range", index);
  *out = t[index];
  return EMU_OK;
}

int emu_plan_segments(emu_plan_t plan, int64_t first, int64_t count, emu_segment_t* out) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (count > 0 && !out) return fail(EMU_ERR_NULL, "out is NULL");
  if (first < 0 || count < 0 || uint64_t(first) + uint64_t(count) > P->segs.size())
    return fail(EMU_ERR_RANGE, "segment range out of bounds");
  if (count) std::memcpy(out, P->segs.data() + first, size_t(count) * sizeof(emu_segment_t));
  return EMU_OK;
}

int emu_bucket_layout(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, int32_t rank, uint64_t* n_buckets,
                      uint64_t* stream_bytes) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (side != 0 && side != 1) return fail(EMU_ERR_RANGE, "side must be 0 or 1");
  const SideInfo& s = P->side[side];
  const uint64_t es = uint64_t(elem_size(s.lay.dtype));
  if (bucket_bytes == 0 || bucket_bytes % es)
    return fail(EMU_ERR_BUCKET, "bucket size %llu is not a positive multiple of %llu",
                (unsigned long long)bucket_bytes, (unsigned long long)es);
  if (rank < -1 || rank >= s.nranks) return fail(EMU_ERR_RANGE, "rank %d out of range", rank);
  uint64_t nb = 0, sb = 0;
  for (int r = (rank < 0 ? 0 : rank); r < (rank < 0 ? s.nranks : rank + 1); ++r) {
    nb += (s.rank_bytes[r] + bucket_bytes - 1) / bucket_bytes;
    sb += s.rank_bytes[r];
  }
  if (n_buckets) *n_buckets = nb;
  if (stream_bytes) *stream_bytes = sb;
  return EMU_OK;
}



int emu_bucket_info(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, uint64_t first, uint64_t count,
                    emu_bucket_desc_t* out) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (side != 0 && side != 1) return fail(EMU_ERR_RANGE, "side must be 0 or 1");
  if (count > 0 && !out) return fail(EMU_ERR_NULL, "out is NULL");
  const SideInfo& s = P->side[side];
  const uint64_t es = uint64_t(elem_size(s.lay.dtype));
  if (bucket_bytes == 0 || bucket_bytes % es)
    return fail(EMU_ERR_BUCKET, "bucket size %llu is not a positive multiple of %llu",
                (unsigned long long)bucket_bytes, (unsigned long long)es);
  uint64_t total = 0;
  for (int r = 0; r < s.nranks; ++r) total += (s.rank_bytes[r] + bucket_bytes - 1) / bucket_bytes;
  if (first > total || count > total - first)
    return fail(EMU_ERR_RANGE, "buckets [%llu, %llu + %llu) out of %llu", (unsigned long long)first,
                (unsigned long long)first, (unsigned long long)count, (unsigned long long)total);
  uint64_t k0 = 0, i = 0;  // global index of rank r's first bucket
  for (int r = 0; r < s.nranks && i < count; ++r) {
    const uint64_t nb = (s.rank_bytes[r] + bucket_bytes - 1) / bucket_bytes;
    for (uint64_t k = first + i > k0 ? first + i - k0 : 0; k < nb && i < count; ++k, ++i) {
      emu_bucket_desc_t& b = out[i];
      b.rank = r;
      b.reserved = 0;
      b.index = k;
      b.stream_offset = k * bucket_bytes;
      b.bytes = std::min<uint64_t>(bucket_bytes, s.rank_bytes[r] - k * bucket_bytes);
    }
    k0 += nb;
  }
  return EMU_OK;
}

int emu_check_tables(emu_plan_t plan, const uint64_t* src_ptrs, const uint64_t* dst_ptrs) {
  emu::clear_error();
  const emu::Plan* P = reinterpret_cast<const emu::Plan*>(plan);
  if (!emu::plan_live(P)) return emu::fail(EMU_ERR_HANDLE, "not a live plan");
  if (!src_ptrs || !dst_ptrs) return emu::fail(EMU_ERR_NULL, "NULL pointer table");
  try {
    std::vector<Range> rs;
    int rc = add_ranges(rs, src_ptrs, tensor_sizes(P->side[0]), true, "source tensor");
    if (rc) return rc;
    // alias tensors left out of the map are never written: their entries take no part
    std::vector<bool> skip(P->side[1].tensors.size(), false);
    if (P->aliased)
      for (size_t i = 0; i < skip.size(); ++i) skip[i] = P->side[1].tensors[i].alias >= 0;
    rc = add_ranges(rs, dst_ptrs, tensor_sizes(P->side[1]), false, "destination tensor", &skip);
    if (rc) return rc;
    return sweep(rs);
  } catch (const std::bad_alloc&) {
    return emu::fail(EMU_ERR_ARG, "out of host memory");
  }
}

int emu_check_bucket_tables(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, const uint64_t* tensor_ptrs,
                            const uint64_t* bucket_ptrs) {
  emu::clear_error();
  const emu::Plan* P = reinterpret_cast<const emu::Plan*>(plan);
  if (!emu::plan_live(P)) return emu::fail(EMU_ERR_HANDLE, "not a live plan");
  if (side != 0 && side != 1) return emu::fail(EMU_ERR_RANGE, "side must be 0 or 1");
  if (!tensor_ptrs || !bucket_ptrs) return emu::fail(EMU_ERR_NULL, "NULL pointer table");
  if (bucket_bytes == 0) return emu::fail(EMU_ERR_BUCKET, "bucket size is zero");
  try {
    const emu::SideInfo& s = P->side[side];
    std::vector<uint64_t> bsizes;
    for (int r = 0; r < s.nranks; ++r)
      for (uint64_t k = 0; k * bucket_bytes < s.rank_bytes[r]; ++k)
        bsizes.push_back(std::min(bucket_bytes, s.rank_bytes[r] - k * bucket_bytes));
    std::vector<Range> rs;
    int rc = add_ranges(rs, tensor_ptrs, tensor_sizes(s), false, "tensor");
    if (rc) return rc;
    rc = add_ranges(rs, bucket_ptrs, bsizes, false, "bucket");
    if (rc) return rc;
    return sweep(rs);
  } catch (const std::bad_alloc&) {
    return emu::fail(EMU_ERR_ARG, "out of host memory");
  }
}

}  // extern "C"
