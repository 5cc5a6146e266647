// Device side of the EMU reshard library for CDNA4 (gfx950): the reshard kernel that executes a
// compiled copy map, the bucket pack/unpack kernel, and the C ABI entry points that launch them.
//
// Both kernels are pure HBM streams: no arithmetic on the data, integer address math only. Every
// thread moves 16-byte vectors (global_load/store_dwordx4), a tile is kThreads * U vectors, and all U
// loads of a tile are issued before its stores, so that each CU keeps tens of KB of reads in flight.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>

#include "emu_internal.h"

namespace emu {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------------------------------------
// device helpers
// ------------------------------------------------------------------------------------------------

template <bool NT>
__device__ __forceinline__ v4u ld16(const v4u* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ __forceinline__ void st16(v4u* p, v4u v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(x >> 32));
  return (uint64_t(hi) << 32) | lo;
}

// 16 bytes starting `sh` bytes (0 < sh < 16) into the 32-byte pair (lo, hi). Q = sh / 4 is a
// template parameter so that the dword selection is static; the byte shift uses v_alignbyte.
template <int Q>
__device__ __forceinline__ v4u funnel(v4u lo, v4u hi, uint32_t b) {
  const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  v4u o;
  o.x = __builtin_amdgcn_alignbyte(w[Q + 1], w[Q + 0], b);
  o.y = __builtin_amdgcn_alignbyte(w[Q + 2], w[Q + 1], b);
  o.z = __builtin_amdgcn_alignbyte(w[Q + 3], w[Q + 2], b);
  o.w = __builtin_amdgcn_alignbyte(w[Q + 4], w[Q + 3], b);
  return o;
}

// Workgroup-cooperative copy of nv 16-byte vectors, both sides 16-byte aligned (ZERO: store zeros).
template <int U, bool NT, bool ZERO>
__device__ __forceinline__ void wg_vec_copy(const v4u* __restrict__ s, v4u* __restrict__ d, uint64_t nv) {
  const uint32_t tid = threadIdx.x;
  constexpr uint32_t TV = uint32_t(kThreads) * U;
  for (uint64_t base = 0; base < nv; base += TV) {
    const uint64_t cnt = nv - base < TV ? nv - base : TV;
    v4u r[U];
    if (cnt == TV) {
#pragma unroll
      for (int u = 0; u < U; ++u) r[u] = ZERO ? v4u{0, 0, 0, 0} : ld16<NT>(s + base + u * kThreads + tid);
#pragma unroll
      for (int u = 0; u < U; ++u) st16<NT>(d + base + u * kThreads + tid, r[u]);
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = u * kThreads + tid;
        r[u] = (!ZERO && i < cnt) ? ld16<NT>(s + base + i) : v4u{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = u * kThreads + tid;
        if (i < cnt) st16<NT>(d + base + i, r[u]);
      }
    }
  }
}

// Workgroup-cooperative copy of nv destination-aligned vectors whose source starts `sh` bytes past
// the 16-byte aligned address sa (0 < sh < 16): each output vector is cut from two aligned source
// vectors. The second vector of the last output lies in the granule of the last source byte, so no
// read leaves the granules the copy's own bytes occupy.
template <int U, bool NT, int Q>
__device__ __forceinline__ void wg_shift_copy(const v4u* __restrict__ sa, v4u* __restrict__ d, uint64_t nv,
                                              uint32_t b) {
  const uint32_t tid = threadIdx.x;
  constexpr uint32_t TV = uint32_t(kThreads) * U;
  for (uint64_t base = 0; base < nv; base += TV) {
    const uint64_t cnt = nv - base < TV ? nv - base : TV;
    v4u lo[U], hi[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * kThreads + tid;
      if (i < cnt) {
        lo[u] = ld16<NT>(sa + base + i);
        hi[u] = ld16<NT>(sa + base + i + 1);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * kThreads + tid;
      if (i < cnt) st16<NT>(d + base + i, funnel<Q>(lo[u], hi[u], b));
    }
  }
}

// Workgroup-cooperative copy of n bytes at any alignment (ZERO: write n zero bytes).
// The destination drives the split: a head up to the first 16-byte boundary, a vector body and a
// tail, the head and tail moved byte by byte.
template <int U, bool NT, bool ZERO>
__device__ void wg_copy_bytes(const uint8_t* s, uint8_t* d, uint64_t n) {
  const uint32_t tid = threadIdx.x;
  const uint64_t head0 = (16 - (reinterpret_cast<uintptr_t>(d) & 15)) & 15;
  const uint64_t head = head0 < n ? head0 : n;
  const uint64_t nv = (n - head) / 16;
  const uint64_t tail = n - head - nv * 16;
  if (tid < head) d[tid] = ZERO ? 0 : s[tid];
  if (tid < tail) d[head + nv * 16 + tid] = ZERO ? 0 : s[head + nv * 16 + tid];
  if (nv == 0) return;
  v4u* dv = reinterpret_cast<v4u*>(d + head);
  if constexpr (ZERO) {
    wg_vec_copy<U, NT, true>(nullptr, dv, nv);
  } else {
    const uintptr_t sp = reinterpret_cast<uintptr_t>(s + head);
    const uint32_t sh = uint32_t(sp & 15);
    if (sh == 0) {
      wg_vec_copy<U, NT, false>(reinterpret_cast<const v4u*>(sp), dv, nv);
    } else {
      const v4u* sa = reinterpret_cast<const v4u*>(sp - sh);
      switch (sh >> 2) {
        case 0: wg_shift_copy<U, NT, 0>(sa, dv, nv, sh & 3); break;
        case 1: wg_shift_copy<U, NT, 1>(sa, dv, nv, sh & 3); break;
        case 2: wg_shift_copy<U, NT, 2>(sa, dv, nv, sh & 3); break;
        default: wg_shift_copy<U, NT, 3>(sa, dv, nv, sh & 3); break;
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// reshard kernel: one tile = kThreads * U destination vectors of one segment
// ------------------------------------------------------------------------------------------------

template <int U, bool NT, bool ZERO, bool LDS>
__device__ __forceinline__ void tile_rows(const DevSeg& g, uint64_t lt, const uint8_t* sb, uint8_t* db,
                                          v4u* stage) {
  // SEG_VEC_ROWS: `param` whole rows of rv vectors per tile; n -> (row, col) by a multiply-high
  const uint32_t tid = threadIdx.x;
  const uint64_t row0 = lt * g.param;
  const uint64_t nrows = g.rows - row0 < g.param ? g.rows - row0 : g.param;
  const uint32_t cnt = uint32_t(nrows) * g.rv;
  const uint8_t* s = sb + g.src_off + row0 * g.src_stride;
  uint8_t* d = db + g.dst_off + row0 * g.dst_stride;
  v4u r[U];
  uint32_t q[U], c[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t n = u * kThreads + tid;
    q[u] = g.rv > 1 ? __umulhi(n, g.magic) : n;
    c[u] = n - q[u] * g.rv;
    if (!ZERO && n < cnt)
      r[u] = ld16<NT>(reinterpret_cast<const v4u*>(s + q[u] * g.src_stride) + c[u]);
    else
      r[u] = v4u{0, 0, 0, 0};
  }
  if constexpr (LDS) {
#pragma unroll
    for (int u = 0; u < U; ++u) stage[u * kThreads + tid] = r[u];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = stage[u * kThreads + tid];
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t n = u * kThreads + tid;
    if (n < cnt) st16<NT>(reinterpret_cast<v4u*>(d + q[u] * g.dst_stride) + c[u], r[u]);
  }
}

template <int U, bool NT, bool ZERO, bool LDS>
__device__ __forceinline__ void tile_run(const v4u* s, v4u* d, uint64_t cnt, v4u* stage) {
  // a contiguous run of cnt <= kThreads*U vectors on both sides
  const uint32_t tid = threadIdx.x;
  constexpr uint32_t TV = uint32_t(kThreads) * U;
  v4u r[U];
  if (cnt == TV) {
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = ZERO ? v4u{0, 0, 0, 0} : ld16<NT>(s + u * kThreads + tid);
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * kThreads + tid;
      r[u] = (!ZERO && i < cnt) ? ld16<NT>(s + i) : v4u{0, 0, 0, 0};
    }
  }
  if constexpr (LDS) {
#pragma unroll
    for (int u = 0; u < U; ++u) stage[u * kThreads + tid] = r[u];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = stage[u * kThreads + tid];
    __syncthreads();
  }
  if (cnt == TV) {
#pragma unroll
    for (int u = 0; u < U; ++u) st16<NT>(d + u * kThreads + tid, r[u]);
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * kThreads + tid;
      if (i < cnt) st16<NT>(d + i, r[u]);
    }
  }
}

template <int U, bool NT, bool ZERO, bool LDS>
__device__ __forceinline__ void run_tile(const DevSeg& g, uint64_t lt, const uint8_t* sb, uint8_t* db, v4u* stage) {
  constexpr uint64_t TV = uint64_t(kThreads) * U;
  const uint32_t mode = g.mode & SEG_MODE_MASK;
  if (mode == SEG_VEC_1D) {
    const uint64_t nv = g.run / 16, v0 = lt * TV;
    const uint64_t cnt = nv - v0 < TV ? nv - v0 : TV;
    tile_run<U, NT, ZERO, LDS>(reinterpret_cast<const v4u*>(sb + g.src_off) + v0,
                               reinterpret_cast<v4u*>(db + g.dst_off) + v0, cnt, stage);
  } else if (mode == SEG_VEC_ROWS) {
    tile_rows<U, NT, ZERO, LDS>(g, lt, sb, db, stage);
  } else if (mode == SEG_VEC_ROWCHUNK) {
    const uint64_t row = lt / g.param, ch = lt - row * g.param;
    const uint64_t nv = g.run / 16, v0 = ch * TV;
    const uint64_t cnt = nv - v0 < TV ? nv - v0 : TV;
    tile_run<U, NT, ZERO, LDS>(reinterpret_cast<const v4u*>(sb + g.src_off + row * g.src_stride) + v0,
                               reinterpret_cast<v4u*>(db + g.dst_off + row * g.dst_stride) + v0, cnt, stage);
  } else {  // SEG_GENERAL
    const uint64_t row = lt / g.param, ch = lt - row * g.param;
    const uint64_t b0 = ch * TV * 16;
    const uint64_t n = g.run - b0 < TV * 16 ? g.run - b0 : TV * 16;
    wg_copy_bytes<U, NT, ZERO>(sb + g.src_off + row * g.src_stride + b0, db + g.dst_off + row * g.dst_stride + b0, n);
  }
}

template <int U, bool NT, bool LDS>
__global__ __launch_bounds__(kThreads) void k_reshard(const DevSeg* __restrict__ segs,
                                                      const uint32_t* __restrict__ tilemap, uint64_t ntiles,
                                                      const uint64_t* __restrict__ src_ptrs,
                                                      const uint64_t* __restrict__ dst_ptrs) {
  extern __shared__ v4u stage[];
  for (uint64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const uint32_t si = tilemap[tile];
    const DevSeg g = segs[si];
    const uint64_t lt = tile - g.tile0;
    uint8_t* db = reinterpret_cast<uint8_t*>(dst_ptrs[g.dst_idx]);
    if (g.mode & SEG_ZERO) {
      run_tile<U, NT, true, LDS>(g, lt, nullptr, db, stage);
    } else {
      const uint8_t* sb = reinterpret_cast<const uint8_t*>(src_ptrs[g.src_idx]);
      run_tile<U, NT, false, LDS>(g, lt, sb, db, stage);
    }
  }
}

// ------------------------------------------------------------------------------------------------
// bucket pack / unpack kernel
// ------------------------------------------------------------------------------------------------
// Work unit: a chunk of kChunkBytes of one rank's stream. When a workgroup reaches a new rank it
// computes, in LDS, the exclusive prefix sum of that rank's ragged tensor sizes with a wave64 scan
// (wave 0), and the index of the rank's first bucket, sum over earlier ranks of ceil(bytes / B),
// with a wave64 reduction (wave 1). A chunk is then cut at tensor and bucket boundaries into pieces,
// each copied by the whole workgroup.

__device__ __forceinline__ uint64_t wave_incl_scan(uint64_t v, uint32_t lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = __shfl_up(v, d, 64);
    if (lane >= uint32_t(d)) v += y;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

template <bool UNPACK, bool NT, int U>
__global__ __launch_bounds__(kThreads) void k_buckets(const uint64_t* __restrict__ sizes,
                                                      const uint32_t* __restrict__ rank_first,
                                                      const uint64_t* __restrict__ rank_bytes,
                                                      const uint64_t* __restrict__ chunk_first, int32_t nranks,
                                                      uint64_t B, const uint64_t* __restrict__ tensor_ptrs,
                                                      const uint64_t* __restrict__ bucket_ptrs) {
  __shared__ uint64_t offs[kMaxRankTensors + 1];
  __shared__ uint64_t s_bucket0;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t nchunks = chunk_first[nranks];
  int32_t r = 0, cur = -1;
  uint32_t t0 = 0, nt = 0;
  for (uint64_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
    while (chunk_first[r + 1] <= c) ++r;
    if (r != cur) {
      __syncthreads();  // previous rank's offsets no longer read
      t0 = rank_first[r];
      nt = rank_first[r + 1] - t0;
      if (wave == 0) {
        uint64_t carry = 0;
        for (uint32_t base = 0; base < nt; base += 64) {
          const uint32_t i = base + lane;
          const uint64_t incl = wave_incl_scan(i < nt ? sizes[t0 + i] : 0, lane);
          if (i < nt) offs[i + 1] = carry + incl;
          carry += __shfl(incl, 63, 64);
        }
        if (lane == 0) offs[0] = 0;
      } else if (wave == 1) {
        uint64_t acc = 0;
        for (int32_t q = lane; q < r; q += 64) acc += (rank_bytes[q] + B - 1) / B;
        acc = wave_sum(acc);
        if (lane == 0) s_bucket0 = acc;
      }
      __syncthreads();
      cur = r;
    }
    const uint64_t S = offs[nt];
    const uint64_t start = (c - chunk_first[r]) * kChunkBytes;
    const uint64_t end = start + kChunkBytes < S ? start + kChunkBytes : S;
    const uint64_t bucket0 = s_bucket0;
    // last tensor whose offset is <= start
    uint32_t lo = 0, hi = nt;
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (offs[mid] <= start) lo = mid; else hi = mid;
    }
    uint32_t ti = lo;
    uint64_t pos = start;
    while (pos < end) {
      while (offs[ti + 1] <= pos) ++ti;  // skips zero-size tensors too
      const uint64_t toff = offs[ti], tend = offs[ti + 1];
      const uint64_t k = pos / B;
      uint64_t pend = end < tend ? end : tend;
      if ((k + 1) * B < pend) pend = (k + 1) * B;
      uint8_t* tp = reinterpret_cast<uint8_t*>(tensor_ptrs[t0 + ti]) + (pos - toff);
      uint8_t* bp = reinterpret_cast<uint8_t*>(bucket_ptrs[bucket0 + k]) + (pos - k * B);
      const uint64_t n = uniform64(pend - pos);
      if constexpr (UNPACK) wg_copy_bytes<U, NT, false>(bp, tp, n);
      else wg_copy_bytes<U, NT, false>(tp, bp, n);
      pos = uniform64(pend);
    }
  }
}

// ------------------------------------------------------------------------------------------------
// launch helpers
// ------------------------------------------------------------------------------------------------

static int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (dev >= 0 && dev < 64) {
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return -1;
  if (dev >= 0 && dev < 64) cache[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

static int hip_check(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(EMU_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return EMU_OK;
}

template <int U, bool NT, bool LDS>
static void launch_reshard(uint32_t grid, hipStream_t st, const DevSeg* segs, const uint32_t* tm, uint64_t nt,
                           const uint64_t* sp, const uint64_t* dp) {
  const size_t lds = LDS ? size_t(kThreads) * U * 16 : 0;
  hipLaunchKernelGGL((k_reshard<U, NT, LDS>), dim3(grid), dim3(kThreads), lds, st, segs, tm, nt, sp, dp);
}

template <int U>
static void dispatch_reshard(bool nt_hint, bool lds, uint32_t grid, hipStream_t st, const DevSeg* segs,
                             const uint32_t* tm, uint64_t nt, const uint64_t* sp, const uint64_t* dp) {
  if (nt_hint) {
    if (lds) launch_reshard<U, true, true>(grid, st, segs, tm, nt, sp, dp);
    else launch_reshard<U, true, false>(grid, st, segs, tm, nt, sp, dp);
  } else {
    if (lds) launch_reshard<U, false, true>(grid, st, segs, tm, nt, sp, dp);
    else launch_reshard<U, false, false>(grid, st, segs, tm, nt, sp, dp);
  }
}

static bool misaligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

static int bucket_call(emu_plan_t plan, const void* ws, int32_t side, uint64_t B, const uint64_t* tptr,
                       const uint64_t* bptr, void* stream, bool unpack) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!ws || !tptr || !bptr) return fail(EMU_ERR_NULL, "NULL workspace or pointer table");
  if (side != 0 && side != 1) return fail(EMU_ERR_RANGE, "side must be 0 or 1");
  if (misaligned(ws, kWsAlign)) return fail(EMU_ERR_WORKSPACE, "workspace not %llu-byte aligned", (unsigned long long)kWsAlign);
  if (misaligned(tptr, 8) || misaligned(bptr, 8)) return fail(EMU_ERR_ALIGN, "pointer tables must be 8-byte aligned");
  const SideInfo& s = P->side[side];
  const uint64_t es = s.lay.dtype == EMU_BF16 ? 2 : 4;
  if (B == 0 || B % es) return fail(EMU_ERR_BUCKET, "bucket size %llu is not a positive multiple of %llu",
                                    (unsigned long long)B, (unsigned long long)es);
  const uint64_t nchunks = s.chunk_first[s.nranks];
  if (nchunks == 0) return EMU_OK;
  const int cus = device_cus();
  if (cus <= 0) return fail(EMU_ERR_HIP, "cannot query the current device");
  const uint64_t want = uint64_t(cus) * uint64_t(option(EMU_OPT_BUCKET_WG_PER_CU));
  const uint32_t grid = uint32_t(nchunks < want ? nchunks : want);
  const uint8_t* w = static_cast<const uint8_t*>(ws);
  const SideTables& t = P->ws.side[side];
  const uint64_t* sizes = reinterpret_cast<const uint64_t*>(w + t.off_sizes);
  const uint32_t* rf = reinterpret_cast<const uint32_t*>(w + t.off_rank_first);
  const uint64_t* rb = reinterpret_cast<const uint64_t*>(w + t.off_rank_bytes);
  const uint64_t* cf = reinterpret_cast<const uint64_t*>(w + t.off_chunk_first);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool ntm = option(EMU_OPT_NONTEMPORAL) != 0;
  if (unpack) {
    if (ntm) hipLaunchKernelGGL((k_buckets<true, true, 16>), dim3(grid), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
    else hipLaunchKernelGGL((k_buckets<true, false, 16>), dim3(grid), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
  } else {
    if (ntm) hipLaunchKernelGGL((k_buckets<false, true, 16>), dim3(grid), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
    else hipLaunchKernelGGL((k_buckets<false, false, 16>), dim3(grid), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
  }
  return hip_check(unpack ? "emu_unpack_buckets launch" : "emu_pack_buckets launch");
}

}  // namespace emu

using namespace emu;

extern "C" {

int emu_plan_upload(emu_plan_t plan, void* d_workspace, uint64_t workspace_bytes, void* hip_stream) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!d_workspace) return fail(EMU_ERR_NULL, "workspace is NULL");
  if (misaligned(d_workspace, kWsAlign)) return fail(EMU_ERR_WORKSPACE, "workspace not %llu-byte aligned", (unsigned long long)kWsAlign);
  if (workspace_bytes < P->host_ws.size())
    return fail(EMU_ERR_WORKSPACE, "workspace of %llu bytes, plan needs %llu", (unsigned long long)workspace_bytes,
                (unsigned long long)P->host_ws.size());
  const hipError_t e = hipMemcpyAsync(d_workspace, P->host_ws.data(), P->host_ws.size(), hipMemcpyHostToDevice,
                                      static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(EMU_ERR_HIP, "workspace upload: %s", hipGetErrorString(e));
  return EMU_OK;
}

int emu_reshard(emu_plan_t plan, const void* d_workspace, const uint64_t* d_src_ptrs, const uint64_t* d_dst_ptrs,
                void* hip_stream) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!d_workspace || !d_src_ptrs || !d_dst_ptrs) return fail(EMU_ERR_NULL, "NULL workspace or pointer table");
  if (misaligned(d_workspace, kWsAlign)) return fail(EMU_ERR_WORKSPACE, "workspace not %llu-byte aligned", (unsigned long long)kWsAlign);
  if (misaligned(d_src_ptrs, 8) || misaligned(d_dst_ptrs, 8)) return fail(EMU_ERR_ALIGN, "pointer tables must be 8-byte aligned");
  if (P->ntiles == 0) return EMU_OK;
  const int cus = device_cus();
  if (cus <= 0) return fail(EMU_ERR_HIP, "cannot query the current device");
  const int64_t per_cu = option(EMU_OPT_WG_PER_CU);
  uint64_t grid = per_cu == 0 ? P->ntiles : uint64_t(cus) * uint64_t(per_cu);
  if (grid > P->ntiles) grid = P->ntiles;
  if (grid > 0x7fffffffull) grid = 0x7fffffffull;
  const uint8_t* w = static_cast<const uint8_t*>(d_workspace);
  const DevSeg* segs = reinterpret_cast<const DevSeg*>(w + P->ws.off_segs);
  const uint32_t* tm = reinterpret_cast<const uint32_t*>(w + P->ws.off_tilemap);
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  const bool ntm = option(EMU_OPT_NONTEMPORAL) != 0, lds = option(EMU_OPT_LDS_STAGING) != 0;
  switch (P->tile_vecs) {
    case 4: dispatch_reshard<4>(ntm, lds, uint32_t(grid), st, segs, tm, P->ntiles, d_src_ptrs, d_dst_ptrs); break;
    case 16: dispatch_reshard<16>(ntm, lds, uint32_t(grid), st, segs, tm, P->ntiles, d_src_ptrs, d_dst_ptrs); break;
    default: dispatch_reshard<8>(ntm, lds, uint32_t(grid), st, segs, tm, P->ntiles, d_src_ptrs, d_dst_ptrs); break;
  }
  return hip_check("emu_reshard launch");
}

int emu_pack_buckets(emu_plan_t plan, const void* d_workspace, int32_t side, uint64_t bucket_bytes,
                     const uint64_t* d_tensor_ptrs, const uint64_t* d_bucket_ptrs, void* hip_stream) {
  return bucket_call(plan, d_workspace, side, bucket_bytes, d_tensor_ptrs, d_bucket_ptrs, hip_stream, false);
}

int emu_unpack_buckets(emu_plan_t plan, const void* d_workspace, int32_t side, uint64_t bucket_bytes,
                       const uint64_t* d_bucket_ptrs, const uint64_t* d_tensor_ptrs, void* hip_stream) {
  return bucket_call(plan, d_workspace, side, bucket_bytes, d_tensor_ptrs, d_bucket_ptrs, hip_stream, true);
}

}  // extern "C"
