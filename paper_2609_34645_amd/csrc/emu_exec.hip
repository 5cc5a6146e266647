// Device side of the EMU reshard library for CDNA4 (gfx950): the reshard kernel that executes a
// compiled copy map, the bucket pack/unpack kernel, the small kernels that build a plan's tile map and
// bucket stream tables in its workspace at upload, and the C ABI entry points that launch them.
//
// Both kernels are pure HBM streams: no arithmetic on the data (fp32 <-> bf16 conversion aside),
// integer address math only. Every thread moves 16-byte vectors (global_load/store_dwordx4), a tile is
// threads * U vectors, and all U loads of a tile are issued before its stores. How many tiles are
// resident per CU is bounded (EMU_OPT_WG_PER_CU), so that each CU keeps 48-64 KB of loads in flight:
// enough to cover HBM latency, and few enough that the mixed read/write stream does not congest. Both
// tile kernels run one wave64 per workgroup, so that each tile's address computation (map entry,
// descriptor or rank record, pointers) is done once rather than once per wave.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>

#include "emu_internal.h"


namespace emu {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------------------------------------
// device helpers
// ------------------------------------------------------------------------------------------------

// Global-address-space views: table-loaded pointers are generic to the compiler, which would emit
// flat loads; casting to address space 1 gives global_load/store_dwordx4 with a scalar base.
typedef __attribute__((address_space(1))) v4u gv4u;
typedef __attribute__((address_space(1))) uint8_t gu8;

template <bool NT>
__device__ __forceinline__ v4u ld16(const uint8_t* base, uint32_t off) {
  const gv4u* p = (const gv4u*)((const gu8*)base + off);
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ __forceinline__ void st16(uint8_t* base, uint32_t off, v4u v) {
  gv4u* p = (gv4u*)((gu8*)base + off);
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) v2u gv2u;

template <bool NT>
__device__ __forceinline__ v2u ld8(const uint8_t* base, uint32_t off) {
  const gv2u* p = (const gv2u*)((const gu8*)base + off);
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ __forceinline__ void st8(uint8_t* base, uint32_t off, v2u v) {
  gv2u* p = (gv2u*)((gu8*)base + off);
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// fp32 bits -> bf16 bits: round to nearest, ties to even; a NaN keeps its sign and top payload bits and
// gets the quiet bit (so that a NaN whose payload sits in the low half never turns into infinity).
__device__ __forceinline__ uint32_t bf16_rne(uint32_t u) {
  const uint32_t r = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return (u & 0x7fffffffu) > 0x7f800000u ? ((u >> 16) | 0x40u) : r;
}

// Source data behind one 16-byte destination vector, per element conversion of the plan:
// CVT_NONE one 16-byte vector; CVT_F32_BF16 two (8 fp32 -> 8 bf16); CVT_BF16_F32 half of one (4 bf16).
template <int CVT> struct Raw { v4u a; };
template <> struct Raw<CVT_F32_BF16> { v4u a, b; };
template <> struct Raw<CVT_BF16_F32> { v2u a; };

template <int CVT>
constexpr uint32_t kSrcVecBytes = CVT == CVT_F32_BF16 ? 32u : CVT == CVT_BF16_F32 ? 8u : 16u;

template <int CVT, bool NT>
__device__ __forceinline__ Raw<CVT> ld_raw(const uint8_t* s, uint32_t off) {
  Raw<CVT> r;
  if constexpr (CVT == CVT_F32_BF16) {
    r.a = ld16<NT>(s, off);
    r.b = ld16<NT>(s, off + 16u);
  } else if constexpr (CVT == CVT_BF16_F32) {
    r.a = ld8<NT>(s, off);
  } else {
    r.a = ld16<NT>(s, off);
  }
  return r;
}

template <int CVT>
__device__ __forceinline__ v4u cook(const Raw<CVT>& r) {
  if constexpr (CVT == CVT_F32_BF16) {
    v4u o;
    o.x = bf16_rne(r.a.x) | (bf16_rne(r.a.y) << 16);
    o.y = bf16_rne(r.a.z) | (bf16_rne(r.a.w) << 16);
    o.z = bf16_rne(r.b.x) | (bf16_rne(r.b.y) << 16);
    o.w = bf16_rne(r.b.z) | (bf16_rne(r.b.w) << 16);
    return o;
  } else if constexpr (CVT == CVT_BF16_F32) {
    return v4u{r.a.x << 16, r.a.x & 0xffff0000u, r.a.y << 16, r.a.y & 0xffff0000u};
  } else {
    return r.a;
  }
}

// Element-wise conversion of n destination elements (misaligned converting segments; rare).
template <int NTH, int CVT>
__device__ void wg_convert_elems(const uint8_t* s, uint8_t* d, uint32_t n) {
  for (uint32_t i = threadIdx.x; i < n; i += NTH) {
    if constexpr (CVT == CVT_F32_BF16) {
      const uint32_t u = *(const __attribute__((address_space(1))) uint32_t*)((const gu8*)s + 4u * i);
      *(__attribute__((address_space(1))) uint16_t*)((gu8*)d + 2u * i) = uint16_t(bf16_rne(u));
    } else {
      const uint32_t b = *(const __attribute__((address_space(1))) uint16_t*)((const gu8*)s + 2u * i);
      *(__attribute__((address_space(1))) uint32_t*)((gu8*)d + 4u * i) = b << 16;
    }
  }
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
// nv * 16 must fit in 32 bits: offsets are 32-bit from uniform base pointers. Lanes past the end load
// the last valid vector again (so every load is unconditional and all U are in flight together) and
// skip their store.
template <int NTH, int U, bool NT, bool ZERO>
__device__ __forceinline__ void wg_vec_copy(const uint8_t* __restrict__ s, uint8_t* __restrict__ d, uint32_t nv) {
  const uint32_t tid = threadIdx.x;
  constexpr uint32_t TV = uint32_t(NTH) * U;
#pragma nounroll
  for (uint32_t base = 0; base < nv; base += TV) {
    const uint32_t last = umin(nv - base, TV) - 1;
    v4u r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (ZERO) r[u] = v4u{0, 0, 0, 0};
      else r[u] = ld16<NT>(s, (base + umin(u * NTH + tid, last)) * 16u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * NTH + tid;
      if (i <= last) st16<NT>(d, (base + i) * 16u, r[u]);
    }
  }
}

// Workgroup-cooperative copies of nv destination-aligned vectors whose source starts `sh` bytes past the
// 16-byte aligned address sa (0 < sh < 16): output vector i is cut from aligned source vectors i and
// i + 1 (funnel). Each lane loads vector i; vector i + 1 comes from the next lane through DPP
// (wave_shl:1, a VALU operand modifier rather than an LDS permute). The last output's second vector is
// the granule holding the copy's last source byte, so no read leaves the granules the copy's own bytes
// occupy.
//
// One wave per workgroup: lane 63 of a block of 64 vectors takes lane 0 of the next block through
// wave_rol:1, and only lane 63 of a pass's last block loads a vector of its own (one masked load per
// pass). Lanes past the end load vector last + 1, so lane `last` finds its second vector in the next lane.
template <int U, bool NT, int Q>
__device__ __forceinline__ void wave_shift_copy(const uint8_t* __restrict__ sa, uint8_t* __restrict__ d, uint32_t nv,
                                                uint32_t b) {
  const uint32_t lane = threadIdx.x;
  constexpr uint32_t TV = 64u * U;
#pragma nounroll
  for (uint32_t base = 0; base < nv; base += TV) {
    const uint32_t last = umin(nv - base, TV) - 1;
    v4u lo[U + 1];
#pragma unroll
    for (int u = 0; u < U; ++u) lo[u] = ld16<NT>(sa, (base + umin(u * 64u + lane, last + 1)) * 16u);
    lo[U] = v4u{0, 0, 0, 0};
    if (lane == 63u) lo[U] = ld16<NT>(sa, (base + umin(TV - 1, last) + 1u) * 16u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * 64u + lane;
      v4u nx, hi;
      if (u + 1 < U) {
        nx.x = __builtin_amdgcn_update_dpp(0u, lo[u + 1].x, 0x134, 0xf, 0xf, false);  // wave_rol:1
        nx.y = __builtin_amdgcn_update_dpp(0u, lo[u + 1].y, 0x134, 0xf, 0xf, false);
        nx.z = __builtin_amdgcn_update_dpp(0u, lo[u + 1].z, 0x134, 0xf, 0xf, false);
        nx.w = __builtin_amdgcn_update_dpp(0u, lo[u + 1].w, 0x134, 0xf, 0xf, false);
      } else {
        nx = lo[U];
      }
      // wave_shl:1; lane 63 has no source lane and keeps nx
      hi.x = __builtin_amdgcn_update_dpp(nx.x, lo[u].x, 0x130, 0xf, 0xf, false);
      hi.y = __builtin_amdgcn_update_dpp(nx.y, lo[u].y, 0x130, 0xf, 0xf, false);
      hi.z = __builtin_amdgcn_update_dpp(nx.z, lo[u].z, 0x130, 0xf, 0xf, false);
      hi.w = __builtin_amdgcn_update_dpp(nx.w, lo[u].w, 0x130, 0xf, 0xf, false);
      if (i <= last) st16<NT>(d, (base + i) * 16u, funnel<Q>(lo[u], hi, b));
    }
  }
}

// Several waves per workgroup: lane 63 of every wave, and the lanes from the last output on, load their
// second vector themselves.
template <int NTH, int U, bool NT, int Q>
__device__ __forceinline__ void wg_shift_copy(const uint8_t* __restrict__ sa, uint8_t* __restrict__ d, uint32_t nv,
                                              uint32_t b) {
  const uint32_t tid = threadIdx.x, lane = tid & 63u;
  constexpr uint32_t TV = uint32_t(NTH) * U;
#pragma nounroll
  for (uint32_t base = 0; base < nv; base += TV) {
    const uint32_t last = umin(nv - base, TV) - 1;
    v4u lo[U], own[U];
#pragma unroll
    for (int u = 0; u < U; ++u) lo[u] = ld16<NT>(sa, (base + umin(u * NTH + tid, last)) * 16u);
#pragma unroll
    for (int u = 0; u < U; ++u) {  // issued before any wait, next to the loads above
      const uint32_t i = u * NTH + tid;
      own[u] = v4u{0, 0, 0, 0};
      if (lane == 63u || i >= last) own[u] = ld16<NT>(sa, (base + umin(i, last) + 1u) * 16u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = u * NTH + tid;
      v4u hi;
      hi.x = __builtin_amdgcn_update_dpp(0u, lo[u].x, 0x130, 0xf, 0xf, false);  // wave_shl:1
      hi.y = __builtin_amdgcn_update_dpp(0u, lo[u].y, 0x130, 0xf, 0xf, false);
      hi.z = __builtin_amdgcn_update_dpp(0u, lo[u].z, 0x130, 0xf, 0xf, false);
      hi.w = __builtin_amdgcn_update_dpp(0u, lo[u].w, 0x130, 0xf, 0xf, false);
      if (lane == 63u || i >= last) hi = own[u];
      if (i <= last) st16<NT>(d, (base + i) * 16u, funnel<Q>(lo[u], hi, b));
    }
  }
}

// Workgroup-cooperative copy of n bytes (n < 2^32) at any alignment (ZERO: write n zero bytes).
// The destination drives the split: a head up to the first 16-byte boundary, a vector body and a
// tail, the head and tail moved byte by byte. UA is the unroll of the co-aligned body, US that of the
// realigned body (which holds two source vectors per output vector).
template <int NTH, int UA, int US, bool NT, bool ZERO>
__device__ __forceinline__ void wg_copy_bytes(const uint8_t* s, uint8_t* d, uint32_t n) {
  const uint32_t tid = threadIdx.x;
  const uint32_t head0 = (16u - uint32_t(reinterpret_cast<uintptr_t>(d) & 15)) & 15u;
  const uint32_t head = head0 < n ? head0 : n;
  const uint32_t nv = (n - head) / 16u;
  const uint32_t tail = n - head - nv * 16u;
  if (tid < head) d[tid] = ZERO ? 0 : s[tid];
  if (tid < tail) d[head + nv * 16u + tid] = ZERO ? 0 : s[head + nv * 16u + tid];
  if (nv == 0) return;
  if constexpr (ZERO) {
    wg_vec_copy<NTH, UA, NT, true>(nullptr, d + head, nv);
  } else {
    const uint32_t sh = uint32_t(reinterpret_cast<uintptr_t>(s + head) & 15);
    if (sh == 0) {
      wg_vec_copy<NTH, UA, NT, false>(s + head, d + head, nv);
    } else {
      const uint8_t* sa = s + head - sh;
      if constexpr (NTH == 64) {
        switch (sh >> 2) {
          case 0: wave_shift_copy<US, NT, 0>(sa, d + head, nv, sh & 3); break;
          case 1: wave_shift_copy<US, NT, 1>(sa, d + head, nv, sh & 3); break;
          case 2: wave_shift_copy<US, NT, 2>(sa, d + head, nv, sh & 3); break;
          default: wave_shift_copy<US, NT, 3>(sa, d + head, nv, sh & 3); break;
        }
      } else {
        switch (sh >> 2) {
          case 0: wg_shift_copy<NTH, US, NT, 0>(sa, d + head, nv, sh & 3); break;
          case 1: wg_shift_copy<NTH, US, NT, 1>(sa, d + head, nv, sh & 3); break;
          case 2: wg_shift_copy<NTH, US, NT, 2>(sa, d + head, nv, sh & 3); break;
          default: wg_shift_copy<NTH, US, NT, 3>(sa, d + head, nv, sh & 3); break;
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// reshard kernel: one tile = kReshardThreads * U destination vectors of one segment
// ------------------------------------------------------------------------------------------------

#ifndef EMU_RESHARD_WAVES_PER_EU
#define EMU_RESHARD_WAVES_PER_EU 4
#endif
#ifndef EMU_BUCKET_WAVES_PER_EU
#define EMU_BUCKET_WAVES_PER_EU 4
#endif
#ifndef EMU_BUCKET_UNROLL
#define EMU_BUCKET_UNROLL 8
#endif
#ifndef EMU_SHIFT_UNROLL
#define EMU_SHIFT_UNROLL 4
#endif
#ifndef EMU_BUCKET_TILE_VECS
#define EMU_BUCKET_TILE_VECS 4
#endif
#ifndef EMU_BUCKET_TILE_THREADS
#define EMU_BUCKET_TILE_THREADS 64
#endif
constexpr int kXcds = int(kXcdCount);  // workgroups are dealt to the XCDs round-robin
constexpr int kGeneralUnroll = 2;  // byte-granular reshard segments (misaligned runs; rare)
constexpr int kBucketUnroll = EMU_BUCKET_UNROLL;
constexpr int kShiftUnroll = EMU_SHIFT_UNROLL;
constexpr int kBucketTileVecs = EMU_BUCKET_TILE_VECS;  // vectors per thread per pass of k_buckets_tile
constexpr int kBucketTileThreads = EMU_BUCKET_TILE_THREADS;  // workgroup size of k_buckets_tile

template <int U, bool LDS>
__device__ __forceinline__ void stage_through_lds(v4u (&r)[U], v4u* stage) {
  if constexpr (LDS) {
    const uint32_t tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < U; ++u) stage[u * kReshardThreads + tid] = r[u];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = stage[u * kReshardThreads + tid];
    __syncthreads();
  }
}

// Rows of rv vectors at strides ss and ds bytes from s and d, read in row-major vector order: the tile
// holds vectors r0 .. r0 + last of that order. Vector n is in row n / rv (a multiply-high by the host's
// magic number) at column n % rv; the host keeps every in-tile byte offset below 2^31.
template <int U, bool NT, bool ZERO, bool LDS, int CVT>
__device__ __forceinline__ void tile_rows(const uint8_t* s, uint8_t* d, uint32_t r0, uint32_t last, uint32_t rv,
                                          uint32_t mg, uint32_t ss, uint32_t ds, v4u* stage) {
  const uint32_t tid = threadIdx.x;
  v4u r[U];
  if constexpr (ZERO) {
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = v4u{0, 0, 0, 0};
  } else {
    Raw<CVT> raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t n = r0 + umin(u * kReshardThreads + tid, last);
      const uint32_t q = rv > 1 ? __umulhi(n, mg) : n;
      raw[u] = ld_raw<CVT, NT>(s, q * ss + (n - q * rv) * kSrcVecBytes<CVT>);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = cook<CVT>(raw[u]);
  }
  stage_through_lds<U, LDS>(r, stage);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = u * kReshardThreads + tid;
    const uint32_t n = r0 + i;
    const uint32_t q = rv > 1 ? __umulhi(n, mg) : n;
    if (i <= last) st16<NT>(d, q * ds + (n - q * rv) * 16u, r[u]);
  }
}

// A contiguous run of cnt (1 <= cnt <= kReshardThreads * U) destination vectors.
template <int U, bool NT, bool ZERO, bool LDS, int CVT>
__device__ __forceinline__ void tile_run(const uint8_t* s, uint8_t* d, uint32_t cnt, v4u* stage) {
  const uint32_t tid = threadIdx.x;
  const uint32_t last = cnt - 1;
  v4u r[U];
  if constexpr (ZERO) {
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = v4u{0, 0, 0, 0};
  } else {
    Raw<CVT> raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) raw[u] = ld_raw<CVT, NT>(s, umin(u * kReshardThreads + tid, last) * kSrcVecBytes<CVT>);
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = cook<CVT>(raw[u]);
  }
  stage_through_lds<U, LDS>(r, stage);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = u * kReshardThreads + tid;
    if (i <= last) st16<NT>(d, i * 16u, r[u]);
  }
}

// fp32 -> bf16 tiles, in source vectors: a tile of cnt destination vectors reads 2 * cnt source vectors
// of four fp32 each and writes 2 * cnt eight-byte halves. Each lane loads whole source vectors,
// consecutive across the lanes, and stores the four converted elements (8 bytes), so every load and
// every store instruction covers one contiguous span. Reading a destination vector's two source
// vectors in one lane instead makes every load instruction touch twice the cache lines it uses.
__device__ __forceinline__ v2u to_bf16x4(v4u a) {
  return v2u{bf16_rne(a.x) | (bf16_rne(a.y) << 16), bf16_rne(a.z) | (bf16_rne(a.w) << 16)};
}

// At most 8 destination vectors per lane per pass (16 source vectors, 64 VGPRs): larger tiles are moved in
// passes, so that the conversion never spills registers.
template <int U>
constexpr int kCvtPass = U > 8 ? 8 : U;

template <int U, bool NT>
__device__ __forceinline__ void tile_run_f32_bf16(const uint8_t* s, uint8_t* d, uint32_t cnt) {
  constexpr int P = kCvtPass<U>;
  const uint32_t tid = threadIdx.x;
  const uint32_t last = 2 * cnt - 1;
#pragma unroll
  for (int h = 0; h < U / P; ++h) {
    v4u a[2 * P];
#pragma unroll
    for (int k = 0; k < 2 * P; ++k) a[k] = ld16<NT>(s, umin((h * 2 * P + k) * kReshardThreads + tid, last) * 16u);
#pragma unroll
    for (int k = 0; k < 2 * P; ++k) {
      const uint32_t i = (h * 2 * P + k) * kReshardThreads + tid;
      if (i <= last) st8<NT>(d, i * 8u, to_bf16x4(a[k]));
    }
  }
}

// The same rows converted: destination vectors r0 .. r0 + last, moved as halves (four fp32 read, four
// bf16 written). Half n of the tile belongs to destination vector r0 + n / 2, in row (r0 + n / 2) / rv;
// its column in halves is 2 r0 + n less twice the row's first vector.
template <int U, bool NT>
__device__ __forceinline__ void tile_rows_f32_bf16(const uint8_t* s, uint8_t* d, uint32_t r0, uint32_t last,
                                                   uint32_t rv, uint32_t mg, uint32_t ss, uint32_t ds) {
  constexpr int P = kCvtPass<U>;
  const uint32_t tid = threadIdx.x;
  const uint32_t lasth = 2 * last + 1, h = 2 * rv;
#pragma unroll
  for (int p = 0; p < U / P; ++p) {
    v4u a[2 * P];
#pragma unroll
    for (int k = 0; k < 2 * P; ++k) {
      const uint32_t n = 2 * r0 + umin((p * 2 * P + k) * kReshardThreads + tid, lasth);
      const uint32_t q = rv > 1 ? __umulhi(n >> 1, mg) : (n >> 1);
      a[k] = ld16<NT>(s, q * ss + (n - q * h) * 16u);
    }
#pragma unroll
    for (int k = 0; k < 2 * P; ++k) {
      const uint32_t i = (p * 2 * P + k) * kReshardThreads + tid;
      const uint32_t n = 2 * r0 + i;
      const uint32_t q = rv > 1 ? __umulhi(n >> 1, mg) : (n >> 1);
      if (i <= lasth) st8<NT>(d, q * ds + (n - q * h) * 8u, to_bf16x4(a[k]));
    }
  }
}

template <int U, bool NT, bool ZERO, bool LDS, int CVT>
__device__ __forceinline__ void run_tile(const DevSeg& g, uint64_t lt, const uint8_t* sb, uint8_t* db, v4u* stage) {
  constexpr uint64_t TV = uint64_t(kReshardThreads) * U;
  constexpr uint64_t SV = kSrcVecBytes<CVT>;
  const uint32_t mode = g.mode & SEG_MODE_MASK;
  constexpr bool kHalves = CVT == CVT_F32_BF16 && !ZERO;
  if (mode == SEG_VEC_1D) {
    const uint64_t nv = g.run / 16, v0 = lt * TV;
    const uint32_t cnt = uint32_t(nv - v0 < TV ? nv - v0 : TV);
    if constexpr (kHalves) tile_run_f32_bf16<U, NT>(sb + g.src_off + v0 * SV, db + g.dst_off + v0 * 16, cnt);
    else tile_run<U, NT, ZERO, LDS, CVT>(ZERO ? nullptr : sb + g.src_off + v0 * SV, db + g.dst_off + v0 * 16, cnt, stage);
  } else if (mode == SEG_VEC_FLAT || mode == SEG_VEC_ROWS) {
    // FLAT: vectors [lt * TV, lt * TV + TV) of the rows' row-major order, starting in row row0 at
    // column r0. ROWS: `param` whole rows per tile.
    uint64_t row0;
    uint32_t r0, last;
    if (mode == SEG_VEC_FLAT) {
      const uint32_t n0 = uint32_t(lt) * uint32_t(TV);  // below param = rows * rv < 2^32
      const uint32_t q0 = g.rv > 1 ? __umulhi(n0, g.magic) : n0;
      row0 = q0;
      r0 = n0 - q0 * g.rv;
      last = umin(g.param - n0, uint32_t(TV)) - 1;
    } else {
      row0 = lt * g.param;
      r0 = 0;
      last = uint32_t(g.rows - row0 < g.param ? g.rows - row0 : g.param) * g.rv - 1;
    }
    const uint8_t* s = ZERO ? nullptr : sb + g.src_off + row0 * g.src_stride;
    uint8_t* d = db + g.dst_off + row0 * g.dst_stride;
    const uint32_t ss = uint32_t(g.src_stride), ds = uint32_t(g.dst_stride);
    if constexpr (kHalves) tile_rows_f32_bf16<U, NT>(s, d, r0, last, g.rv, g.magic, ss, ds);
    else tile_rows<U, NT, ZERO, LDS, CVT>(s, d, r0, last, g.rv, g.magic, ss, ds, stage);
  } else if (mode == SEG_VEC_ROWCHUNK) {
    const uint64_t row = lt / g.param, ch = lt - row * g.param;
    const uint64_t nv = g.run / 16, v0 = ch * TV;
    const uint32_t cnt = uint32_t(nv - v0 < TV ? nv - v0 : TV);
    const uint8_t* s = ZERO ? nullptr : sb + g.src_off + row * g.src_stride + v0 * SV;
    uint8_t* d = db + g.dst_off + row * g.dst_stride + v0 * 16;
    if constexpr (kHalves) tile_run_f32_bf16<U, NT>(s, d, cnt);
    else tile_run<U, NT, ZERO, LDS, CVT>(s, d, cnt, stage);
  } else {  // SEG_GENERAL: misaligned runs, moved at a small unroll so that this rare path does not set
            // the kernel's register budget
    const uint64_t row = lt / g.param, ch = lt - row * g.param;
    const uint64_t b0 = ch * TV * 16;
    const uint32_t n = uint32_t(g.run - b0 < TV * 16 ? g.run - b0 : TV * 16);
    uint8_t* d = db + g.dst_off + row * g.dst_stride + b0;
    if constexpr (CVT == CVT_NONE || ZERO) {
      wg_copy_bytes<kReshardThreads, kGeneralUnroll, kGeneralUnroll, NT, ZERO>(ZERO ? nullptr : sb + g.src_off + row * g.src_stride + b0,
                                                              d, n);
    } else {
      constexpr uint32_t esd = CVT == CVT_F32_BF16 ? 2u : 4u;  // destination element bytes
      constexpr uint32_t ess = CVT == CVT_F32_BF16 ? 4u : 2u;  // source element bytes
      wg_convert_elems<kReshardThreads, CVT>(sb + g.src_off + row * g.src_stride + b0 / esd * ess, d, n / esd);
    }
  }
}

// One workgroup per tile. With XCD remapping, the round-robin dispatch of workgroups over the 8 XCDs is
// undone: XCD x (workgroups x, x+8, ...) works through one contiguous eighth of the tile range, so each
// XCD's L2 sees one stream instead of every eighth tile of all of them. ZERO instances run the map's
// zero-fill section, the others its copy section.
template <int U, bool NT, bool LDS, bool XCD, int CVT, bool ZERO>
__global__ __launch_bounds__(kReshardThreads, EMU_RESHARD_WAVES_PER_EU) void k_reshard(const DevSeg* __restrict__ segs,
                                                                             const uint32_t* __restrict__ tilemap,
                                                                             uint64_t tile_base,
                                                                             const uint64_t* __restrict__ src_ptrs,
                                                                             const uint64_t* __restrict__ dst_ptrs,
                                                                             uint32_t src_n, uint32_t dst_n) {
  extern __shared__ v4u stage[];
  uint32_t local = blockIdx.x;
  if constexpr (XCD) {
    const uint32_t per = gridDim.x / kXcds;  // the host launches a multiple of kXcds workgroups
    local = (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
  }
  // Each section of the map is padded with kNoSeg to the grid's size, so no bounds check precedes
  // the map load. Every path of a copy instance reads the source pointer, so its load issues together
  // with the destination pointer's, right after the descriptor: the chain before the first data load
  // is kernel arguments, map entry, descriptor, pointers.
  const uint64_t tile = tile_base + local;
  const uint32_t si = tilemap[tile];
  if (si == kNoSeg) return;
  const DevSeg g = segs[si];
  // grid row y runs tensor group y: its pointer tables follow the earlier groups' back to back
  uint8_t* db = reinterpret_cast<uint8_t*>(dst_ptrs[uint64_t(blockIdx.y) * dst_n + g.dst_idx]);
  const uint64_t lt = tile - g.tile0;
  if constexpr (ZERO) {
    run_tile<U, NT, true, LDS, CVT_NONE>(g, lt, nullptr, db, stage);
  } else {
    const uint8_t* sb = reinterpret_cast<const uint8_t*>(src_ptrs[uint64_t(blockIdx.y) * src_n + g.src_idx]);
    run_tile<U, NT, false, LDS, CVT>(g, lt, sb, db, stage);
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
__global__ __launch_bounds__(kThreads, EMU_BUCKET_WAVES_PER_EU) void k_buckets(const uint64_t* __restrict__ sizes,
                                                      const uint32_t* __restrict__ rank_first,
                                                      const uint64_t* __restrict__ rank_bytes,
                                                      const uint64_t* __restrict__ chunk_first, int32_t nranks,
                                                      uint64_t B, const uint64_t* __restrict__ tensor_ptrs,
                                                      const uint64_t* __restrict__ bucket_ptrs) {
  __shared__ uint64_t offs[kMaxRankTensors + 1];
  __shared__ uint64_t s_bucket0;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t nchunks = chunk_first[nranks];
  // XCD-aware chunk order: with a grid that is a multiple of the XCD count, the workgroups of XCD x
  // (x, x+8, ...) stride through the contiguous eighth [x*N/8, (x+1)*N/8) of the chunks.
  uint64_t c_begin = blockIdx.x, c_end = nchunks, c_step = gridDim.x;
  if (gridDim.x % kXcds == 0) {
    const uint32_t x = blockIdx.x % kXcds;
    c_begin = nchunks * x / kXcds + blockIdx.x / kXcds;
    c_end = nchunks * (x + 1) / kXcds;
    c_step = gridDim.x / kXcds;
  }
  int32_t r = 0, cur = -1;
  uint32_t t0 = 0, nt = 0, ti = 0;
  uint64_t bucket0 = 0;
  for (uint64_t c = c_begin; c < c_end; c += c_step) {
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
      ti = 0;
      bucket0 = uniform64(s_bucket0);
    }
    const uint64_t S = uniform64(offs[nt]);
    const uint64_t start = (c - chunk_first[r]) * kChunkBytes;
    const uint64_t end = start + kChunkBytes < S ? start + kChunkBytes : S;
    // tensor holding `start`: chunks of one workgroup move forward through the rank, so walk on from
    // the previous chunk's tensor when it is close, else binary-search the offsets
    if (offs[ti] > start || (ti + 8 < nt && offs[ti + 8] <= start)) {
      uint32_t lo = 0, hi = nt;
      while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (offs[mid] <= start) lo = mid; else hi = mid;
      }
      ti = lo;
    }
    ti = __builtin_amdgcn_readfirstlane(ti);
    uint64_t k = start / B;            // bucket of `start`; advanced incrementally below
    uint64_t kend = (k + 1) * B;
    uint64_t pos = start;
    while (pos < end) {
      while (uniform64(offs[ti + 1]) <= pos) ti = __builtin_amdgcn_readfirstlane(ti + 1);  // skips empty tensors
      const uint64_t toff = uniform64(offs[ti]), tend = uniform64(offs[ti + 1]);
      uint64_t pend = end < tend ? end : tend;
      if (kend < pend) pend = kend;
      uint8_t* tp = reinterpret_cast<uint8_t*>(tensor_ptrs[t0 + ti]) + (pos - toff);
      uint8_t* bp = reinterpret_cast<uint8_t*>(bucket_ptrs[bucket0 + k]) + (pos - k * B);
      const uint32_t n = uint32_t(pend - pos);
      if constexpr (UNPACK) wg_copy_bytes<kThreads, U, kShiftUnroll, NT, false>(bp, tp, n);
      else wg_copy_bytes<kThreads, U, kShiftUnroll, NT, false>(tp, bp, n);
      pos = pend;
      if (pos == kend) {
        ++k;
        kend += B;
      }
    }
  }
}

// Tile-per-workgroup variant: one workgroup per 4 KB chunk (kTileChunkBytes) of one rank's stream, in
// block-cyclic XCD order. The upload-time map gives the chunk's rank and the global index of the tensor
// holding its first byte, so the tensor's stream offset and pointer load in parallel with the rank's
// record; the map is padded to the grid, so no bounds check precedes it. The rank's first bucket, the
// sum over earlier ranks of ceil(bytes / B), comes from the host in a kernel argument for the first
// kArgRanks ranks, else from a wave64 reduction. The chunk is then cut at tensor and bucket boundaries.
//
// Chunk ends sit on the destination's 4 KB grid. For aligned buckets and tensors that is the stream's
// grid. When it is not (pack into buckets whose size is not a multiple of 4 KB, unpack into tensors whose
// stream offsets are not), both ends of every chunk move down to the destination's grid, by the same
// rule on either side of each cut, so consecutive chunks still tile the stream. Every destination cache
// line is then written by one workgroup; cut on the stream's grid, every chunk end would split a line
// between two workgroups, which costs partial-line writes to HBM.
constexpr int kArgRanks = 128;
// Chunks per block of the bucket kernel's XCD order (64 x 4 KB = 256 KB). Contiguous eighths per XCD, the
// reshard's order, put the eight XCD streams exactly one eighth of the streams apart; on a rank set laid out
// in one allocation that ran pack and unpack at 75-80% of HBM peak against 82% in per-rank buffers. Blocks of
// 256 KB ran both layouts at 82%; 64 KB and 128 KB blocks lost 5-12 points, 512 KB to 2 MB blocks 0.3-1.
constexpr uint32_t kBucketBlock = 64;
struct BucketBases {
  uint64_t first[kArgRanks];  // first bucket of each rank, for ranks below kArgRanks
};

template <bool UNPACK, bool NT, int U>
__global__ __launch_bounds__(kBucketTileThreads, EMU_RESHARD_WAVES_PER_EU) void k_buckets_tile(
    const uint64_t* __restrict__ stream_off, const uint64_t* __restrict__ rank_info,
    const uint64_t* __restrict__ rank_bytes, const uint32_t* __restrict__ tile_map, uint64_t B, int32_t b_shift,
    uint32_t realign, const uint64_t* __restrict__ tensor_ptrs, const uint64_t* __restrict__ bucket_ptrs,
    BucketBases bases) {
  // Block-cyclic order: the dispatcher deals workgroups to the XCDs round-robin, and XCD x takes blocks
  // x, x + 8, ... of kBucketBlock consecutive chunks, so the eight XCDs stream through neighbouring
  // 256 KB blocks of one front. The map's tail past the last whole round of blocks keeps plain order
  // (the mapping stays a bijection on the padded map). See kBucketBlock.
  const uint32_t w = blockIdx.x, full = gridDim.x / (kXcds * kBucketBlock) * (kXcds * kBucketBlock);
  const uint32_t j = w / kXcds;
  const uint32_t c = w < full ? ((j / kBucketBlock) * kXcds + w % kXcds) * kBucketBlock + j % kBucketBlock : w;
  const uint32_t m = tile_map[c];
  if (m == kNoSeg) return;
  const uint32_t r = m >> kMapTensorBits;
  uint32_t g = m & ((1u << kMapTensorBits) - 1);
  const uint64_t c0 = rank_info[4 * r], S = rank_info[4 * r + 1];
  const uint32_t gend = uint32_t(rank_info[4 * r + 2]);
  uint64_t bucket0;
  if (r < uint32_t(kArgRanks)) {
    bucket0 = bases.first[r];
  } else {
    const uint32_t lane = threadIdx.x & 63;
    uint64_t acc = 0;
    for (uint32_t q = lane; q < r; q += 64) acc += (rank_bytes[q] + B - 1) / B;
    bucket0 = uniform64(wave_sum(acc));
  }
  uint64_t start = (c - c0) * kTileChunkBytes;
  uint64_t end = start + kTileChunkBytes < S ? start + kTileChunkBytes : S;
  uint64_t k = b_shift >= 0 ? start >> b_shift : start / B;
  if (realign) {
    // pack: bucket k's grid starts at stream byte k*B; unpack: a tensor's grid starts at its stream
    // offset (the tensor holding `end` is the next chunk's map entry). A start never leaves its bucket
    // (pack) or tensor (unpack); it may move back into earlier tensors (pack) or an earlier bucket
    // (unpack). Chunks stay non-empty and below 2 * kTileChunkBytes.
    constexpr uint64_t kGrid = kTileChunkBytes - 1;
    if constexpr (UNPACK) {
      start -= (start - stream_off[g]) & kGrid;
      if (end < S) end -= (end - stream_off[tile_map[c + 1] & ((1u << kMapTensorBits) - 1)]) & kGrid;
      k = b_shift >= 0 ? start >> b_shift : start / B;
    } else {
      start -= (start - k * B) & kGrid;
      if (end < S) end -= (end - end / B * B) & kGrid;
      while (stream_off[g] > start) --g;
    }
  }
  uint64_t kend = (k + 1) * B;
  uint64_t pos = start;
  while (pos < end) {
    const uint64_t toff = stream_off[g];
    const uint64_t tend = g + 1 < gend ? stream_off[g + 1] : S;
    if (tend <= pos) {  // the chunk moves on into the next tensor (or past an empty one)
      ++g;
      continue;
    }
    uint64_t pend = end < tend ? end : tend;
    if (kend < pend) pend = kend;
    uint8_t* tp = reinterpret_cast<uint8_t*>(tensor_ptrs[g]) + (pos - toff);
    uint8_t* bp = reinterpret_cast<uint8_t*>(bucket_ptrs[bucket0 + k]) + (pos - k * B);
    const uint32_t n = uint32_t(pend - pos);
    if constexpr (UNPACK) wg_copy_bytes<kBucketTileThreads, U, kShiftUnroll, NT, false>(bp, tp, n);
    else wg_copy_bytes<kBucketTileThreads, U, kShiftUnroll, NT, false>(tp, bp, n);
    pos = pend;
    if (pos == kend) {
      ++k;
      kend += B;
    }
  }
}

// ------------------------------------------------------------------------------------------------
// upload-time tables
// ------------------------------------------------------------------------------------------------
// emu_plan_upload copies the segments with their tile counts and each side's host tables (tensor sizes,
// each rank's tensor range and stream length), and derives the rest on the device.
//
// k_tile_map: workgroup x < n_seg writes segment x's index into its tiles' map entries, from the
// segment's first map index on (workgroups y = 0, 1, ... stride through a long segment); workgroup n_seg
// fills the padding after each section (copy tiles, zero-fill tiles) with kNoSeg.
__global__ __launch_bounds__(256) void k_tile_map(const DevSeg* __restrict__ segs,
                                                  const uint32_t* __restrict__ seg_tiles, uint32_t n_seg,
                                                  uint32_t* __restrict__ map, uint64_t copy_end, uint64_t zero0,
                                                  uint64_t zero_end, uint64_t n_map) {
  const uint32_t x = blockIdx.x;
  if (x == n_seg) {
    if (blockIdx.y != 0) return;
    for (uint64_t j = copy_end + threadIdx.x; j < zero0; j += blockDim.x) map[j] = kNoSeg;
    for (uint64_t j = zero_end + threadIdx.x; j < n_map; j += blockDim.x) map[j] = kNoSeg;
    return;
  }
  const uint64_t t0 = segs[x].tile0;
  const uint32_t n = seg_tiles[x];
  for (uint64_t j = uint64_t(blockIdx.y) * blockDim.x + threadIdx.x; j < n; j += uint64_t(gridDim.y) * blockDim.x)
    map[t0 + j] = x;
}

// k_stream_tables, one wave64 per rank: the
// exclusive prefix sum of the rank's tensor sizes (each tensor's stream offset), and the rank's record
// {first 4 KB chunk, stream bytes, end of its tensor range, 0}, whose first chunk is the sum over earlier
// ranks of ceil(bytes / 4 KB).
__global__ __launch_bounds__(64) void k_stream_tables(const uint64_t* __restrict__ sizes,
                                                      const uint32_t* __restrict__ rank_first,
                                                      const uint64_t* __restrict__ rank_bytes,
                                                      uint64_t* __restrict__ stream_off,
                                                      uint64_t* __restrict__ rank_info) {
  const uint32_t r = blockIdx.x, lane = threadIdx.x;
  const uint32_t t0 = rank_first[r], t1 = rank_first[r + 1];
  uint64_t carry = 0;
  for (uint32_t base = t0; base < t1; base += 64) {
    const uint32_t i = base + lane;
    const uint64_t v = i < t1 ? sizes[i] : 0;
    const uint64_t incl = wave_incl_scan(v, lane);
    if (i < t1) stream_off[i] = carry + incl - v;
    carry += __shfl(incl, 63, 64);
  }
  uint64_t acc = 0;
  for (uint32_t q = lane; q < r; q += 64) acc += (rank_bytes[q] + kTileChunkBytes - 1) / kTileChunkBytes;
  acc = wave_sum(acc);
  if (lane == 0) {
    rank_info[4 * r + 0] = acc;
    rank_info[4 * r + 1] = rank_bytes[r];
    rank_info[4 * r + 2] = t1;
    rank_info[4 * r + 3] = 0;
  }
}

// The chunk map, after k_stream_tables: workgroup g < n_tensors gives every chunk of g's rank whose first
// byte lies in tensor g the entry rank << 20 | g (chunk j of a rank starts in the last tensor whose stream
// offset is <= j * 4 KB: chunks ceil(offset_g / 4 KB) up to ceil(offset_g+1 / 4 KB), or to the rank's
// chunk count for its last tensor), and workgroup n_tensors fills the map's padding after the last
// rank's chunks with kNoSeg.
__global__ __launch_bounds__(256) void k_chunk_map(const uint32_t* __restrict__ rank_first,
                                                   const uint64_t* __restrict__ rank_bytes, uint32_t nranks,
                                                   uint32_t n_tensors, const uint64_t* __restrict__ stream_off,
                                                   const uint64_t* __restrict__ rank_info,
                                                   uint32_t* __restrict__ map, uint64_t n_map) {
  constexpr uint64_t C = kTileChunkBytes;
  const uint32_t g = blockIdx.x;
  uint64_t first = 0, j0, j1;
  uint32_t v = kNoSeg;
  if (g == n_tensors) {
    j0 = rank_info[4 * (nranks - 1)] + (rank_bytes[nranks - 1] + C - 1) / C;
    j1 = n_map;
  } else {
    uint32_t lo = 0, hi = nranks;  // the rank r with rank_first[r] <= g < rank_first[r + 1]
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (rank_first[mid] <= g) lo = mid; else hi = mid;
    }
    const uint32_t t1 = rank_first[lo + 1];
    first = rank_info[4 * lo];
    j0 = (stream_off[g] + C - 1) / C;
    j1 = g + 1 < t1 ? (stream_off[g + 1] + C - 1) / C : (rank_bytes[lo] + C - 1) / C;
    v = (lo << kMapTensorBits) | g;
  }
  for (uint64_t j = j0 + threadIdx.x; j < j1; j += blockDim.x) map[first + j] = v;
}

// ------------------------------------------------------------------------------------------------
// launch helpers
// ------------------------------------------------------------------------------------------------

// A device attribute of the current device, cached per device (0 when it cannot be read).
static int device_attr(hipDeviceAttribute_t attr, int slot) {
  static std::atomic<int> cache[3][64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  const bool cached = dev >= 0 && dev < 64;
  if (cached) {
    const int v = cache[slot][dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, attr, dev) != hipSuccess || v <= 0) return 0;
  if (cached) cache[slot][dev].store(v, std::memory_order_relaxed);
  return v;
}

static int device_cus() {
  const int v = device_attr(hipDeviceAttributeMultiprocessorCount, 0);
  return v > 0 ? v : -1;
}

// Dynamic LDS for a tile kernel that needs `need` bytes and moves `tile_bytes` per workgroup pass.
// A residency cap of c workgroups per CU (EMU_OPT_WG_PER_CU) is enforced by reserving the CU's LDS
// divided by c, rounded down to whole KB; the kernels never touch the reserved bytes. The CU's LDS is
// allocated in two halves and a workgroup's block lies in one half, so the resident count is
// 2 * floor(c / 2) for c >= 2 (c = 1 keeps one). The cap bounds the bytes in flight per CU: on MI355X
// a copy stream runs fastest with about 24-64 KB in flight per CU and drops by about 8% at 128 KB,
// where the HBM read/write mix degrades. Automatic (-1): flight / tile_bytes workgroups, at least 2,
// and no cap from 32 up, with `flight` in destination bytes. Measured optima at 4 KB tiles: a copying
// reshard 12 tiles (48 KB), fp32 -> bf16 10 (40 KB; each tile reads twice what it writes), bf16 ->
// fp32 16 (64 KB; each reads half), all about 100-120 KB of reads and writes together; the
// pack/unpack kernel, whose per-chunk setup is longer, 16 of its 4 KB chunks (64 KB).
template <int CVT>
constexpr uint64_t kReshardFlightBytes = CVT == CVT_F32_BF16 ? 40 * 1024 : CVT == CVT_BF16_F32 ? 64 * 1024 : 48 * 1024;
constexpr uint64_t kBucketFlightBytes = 64 * 1024;
static size_t occupancy_lds(size_t need, uint64_t tile_bytes, uint64_t flight) {
  int64_t cap = option(EMU_OPT_WG_PER_CU);
  if (cap < 0) {
    cap = int64_t(flight / (tile_bytes ? tile_bytes : 1));
    cap = cap < 2 ? 2 : cap >= 32 ? 0 : cap;
  }
  if (cap == 0) return need;
  const int per_cu = device_attr(hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, 1);
  const int per_wg = device_attr(hipDeviceAttributeMaxSharedMemoryPerBlock, 2);
  if (per_cu <= 0 || per_wg <= 0) return need;
  size_t r = (size_t(per_cu) / size_t(cap)) & ~size_t(1023);
  if (r > size_t(per_wg)) r = size_t(per_wg);
  return r > need ? r : need;
}

// Kernel launches report through the runtime's per-thread last-error state. An error some earlier
// runtime call left there belongs to that call, which has already returned it: it is dropped before the
// library launches, so that hip_check afterwards sees only the library's own launches.
static void drop_pending_error() { (void)hipGetLastError(); }

static int hip_check(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(EMU_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return EMU_OK;
}

// Pointer tables of one reshard launch: `groups` source and destination tables back to back, each group
// src_n source and dst_n destination entries (one group for emu_reshard).
struct Tables {
  const uint64_t* sp;
  const uint64_t* dp;
  uint32_t groups, src_n, dst_n;
};

// Launches k_reshard over the map section [first, first + count) for every group (grid row y = group y);
// first is a multiple of kXcds and the section is padded to one.
template <int U, bool NT, bool LDS, bool XCD, int CVT, bool ZERO>
static void launch_reshard(hipStream_t st, const DevSeg* segs, const uint32_t* tm, uint64_t first, uint64_t count,
                           const Tables& tb) {
  const size_t lds = occupancy_lds(LDS ? size_t(kReshardThreads) * U * 16 : 0, uint64_t(kReshardThreads) * U * 16,
                                   kReshardFlightBytes<CVT>);
  // a multiple of kXcds whose work-items (64 per workgroup) stay below 2^32 in the grid's x dimension
  constexpr uint64_t kMaxGrid = (1ull << 26) - kXcds;
  for (uint64_t done = 0; done < count; done += kMaxGrid) {
    const uint32_t n = uint32_t(count - done < kMaxGrid ? count - done : kMaxGrid);
    const uint32_t grid = XCD ? (n + kXcds - 1) / kXcds * kXcds : n;
    hipLaunchKernelGGL((k_reshard<U, NT, LDS, XCD, CVT, ZERO>), dim3(grid, tb.groups), dim3(kReshardThreads), lds, st,
                       segs, tm, first + done, tb.sp, tb.dp, tb.src_n, tb.dst_n);
  }
}

// The copy section of the map, with the plan's conversion, for every combination of
// the launch options (converting plans: no LDS staging).
template <int U, int CVT>
static void launch_copy(bool nt_hint, bool lds, bool xcd, hipStream_t st, const DevSeg* segs, const uint32_t* tm,
                        uint64_t first, uint64_t count, const Tables& tb) {
  constexpr bool kLds = CVT == CVT_NONE;  // staging instances exist for plain copies only
  const int key = (nt_hint ? 4 : 0) | (lds && kLds ? 2 : 0) | (xcd ? 1 : 0);
  switch (key) {
    case 0: launch_reshard<U, false, false, false, CVT, false>(st, segs, tm, first, count, tb); break;
    case 1: launch_reshard<U, false, false, true, CVT, false>(st, segs, tm, first, count, tb); break;
    case 2: launch_reshard<U, false, kLds, false, CVT, false>(st, segs, tm, first, count, tb); break;
    case 3: launch_reshard<U, false, kLds, true, CVT, false>(st, segs, tm, first, count, tb); break;
    case 4: launch_reshard<U, true, false, false, CVT, false>(st, segs, tm, first, count, tb); break;
    case 5: launch_reshard<U, true, false, true, CVT, false>(st, segs, tm, first, count, tb); break;
    case 6: launch_reshard<U, true, kLds, false, CVT, false>(st, segs, tm, first, count, tb); break;
    default: launch_reshard<U, true, kLds, true, CVT, false>(st, segs, tm, first, count, tb); break;
  }
}

template <int U>
static void dispatch_reshard(const Plan* P, bool nt_hint, bool lds, bool xcd, hipStream_t st, const DevSeg* segs,
                             const uint32_t* tm, const Tables& tb) {
  if (P->ntiles_copy > 0) {
    const uint64_t n = P->ntiles_copy;
    switch (P->cvt) {
      case CVT_F32_BF16: launch_copy<U, CVT_F32_BF16>(nt_hint, lds, xcd, st, segs, tm, 0, n, tb); break;
      case CVT_BF16_F32: launch_copy<U, CVT_BF16_F32>(nt_hint, lds, xcd, st, segs, tm, 0, n, tb); break;
      default: launch_copy<U, CVT_NONE>(nt_hint, lds, xcd, st, segs, tm, 0, n, tb); break;
    }
  }
  if (P->ntiles_zero > 0) {
    const uint64_t z0 = P->zero_tile0, n = P->ntiles_zero;
    const int key = (nt_hint ? 2 : 0) | (xcd ? 1 : 0);
    switch (key) {
      case 0: launch_reshard<U, false, false, false, CVT_NONE, true>(st, segs, tm, z0, n, tb); break;
      case 1: launch_reshard<U, false, false, true, CVT_NONE, true>(st, segs, tm, z0, n, tb); break;
      case 2: launch_reshard<U, true, false, false, CVT_NONE, true>(st, segs, tm, z0, n, tb); break;
      default: launch_reshard<U, true, false, true, CVT_NONE, true>(st, segs, tm, z0, n, tb); break;
    }
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
  for (int r = 0; r < s.nranks; ++r)
    if (s.rank_first[r + 1] - s.rank_first[r] > uint32_t(kMaxRankTensors))
      return fail(EMU_ERR_UNSUPPORTED, "rank %d has more than %d tensors on this side", r, kMaxRankTensors);
  const uint64_t nchunks = s.chunk_first[s.nranks];
  if (nchunks == 0) return EMU_OK;
  if (!ws_current(ws, P))
    return fail(EMU_ERR_WORKSPACE, "workspace %p holds no upload of this plan (fill it with emu_plan_upload)", ws);
  const int cus = device_cus();
  if (cus <= 0) return fail(EMU_ERR_HIP, "cannot query the current device");
  const uint64_t want = uint64_t(cus) * uint64_t(option(EMU_OPT_BUCKET_WG_PER_CU));
  uint64_t grid = nchunks < want ? nchunks : want;
  if (grid > kXcds) grid -= grid % kXcds;  // keep the XCD-aware chunk order available
  const uint8_t* w = static_cast<const uint8_t*>(ws);
  const SideTables& t = P->ws.side[side];
  const uint64_t* sizes = reinterpret_cast<const uint64_t*>(w + t.off_sizes);
  const uint32_t* rf = reinterpret_cast<const uint32_t*>(w + t.off_rank_first);
  const uint64_t* rb = reinterpret_cast<const uint64_t*>(w + t.off_rank_bytes);
  const uint64_t* cf = reinterpret_cast<const uint64_t*>(w + t.off_chunk_first);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool ntm = option(EMU_OPT_NONTEMPORAL) != 0;
  if (option(EMU_OPT_BUCKET_TILES) != 0 && t.n_tiles > 0) {
    const uint64_t* so = reinterpret_cast<const uint64_t*>(w + t.off_stream);
    const uint64_t* ri = reinterpret_cast<const uint64_t*>(w + t.off_rank_info);
    const uint32_t* tm = reinterpret_cast<const uint32_t*>(w + t.off_tile_map);
    BucketBases bases;
    uint64_t acc = 0;
    for (int r = 0; r < s.nranks && r < kArgRanks; ++r) {
      bases.first[r] = acc;
      acc += (s.rank_bytes[r] + B - 1) / B;
    }
    const int32_t b_shift = (B & (B - 1)) == 0 ? __builtin_ctzll(B) : -1;
    // chunks are cut on the stream's 16-byte grid unless the destination's grid differs: buckets whose
    // size is not a multiple of 16 (pack), tensors at stream offsets that are not (unpack)
    const uint32_t realign = unpack ? uint32_t(!s.offsets_grid) : uint32_t(B % kTileChunkBytes != 0);
    const dim3 g(uint32_t(t.n_tiles));  // padded to a multiple of kXcds
    const size_t lds = occupancy_lds(0, kTileChunkBytes, kBucketFlightBytes);
    drop_pending_error();
    if (unpack) {
      if (ntm) hipLaunchKernelGGL((k_buckets_tile<true, true, kBucketTileVecs>), g, dim3(kBucketTileThreads), lds, st, so, ri, rb, tm, B, b_shift, realign, tptr, bptr, bases);
      else hipLaunchKernelGGL((k_buckets_tile<true, false, kBucketTileVecs>), g, dim3(kBucketTileThreads), lds, st, so, ri, rb, tm, B, b_shift, realign, tptr, bptr, bases);
    } else {
      if (ntm) hipLaunchKernelGGL((k_buckets_tile<false, true, kBucketTileVecs>), g, dim3(kBucketTileThreads), lds, st, so, ri, rb, tm, B, b_shift, realign, tptr, bptr, bases);
      else hipLaunchKernelGGL((k_buckets_tile<false, false, kBucketTileVecs>), g, dim3(kBucketTileThreads), lds, st, so, ri, rb, tm, B, b_shift, realign, tptr, bptr, bases);
    }
    return hip_check(unpack ? "emu_unpack_buckets launch" : "emu_pack_buckets launch");
  }
  drop_pending_error();
  if (unpack) {
    if (ntm) hipLaunchKernelGGL((k_buckets<true, true, kBucketUnroll>), dim3(uint32_t(grid)), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
    else hipLaunchKernelGGL((k_buckets<true, false, kBucketUnroll>), dim3(uint32_t(grid)), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
  } else {
    if (ntm) hipLaunchKernelGGL((k_buckets<false, true, kBucketUnroll>), dim3(uint32_t(grid)), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
    else hipLaunchKernelGGL((k_buckets<false, false, kBucketUnroll>), dim3(uint32_t(grid)), dim3(kThreads), 0, st, sizes, rf, rb, cf, s.nranks, B, tptr, bptr);
  }
  return hip_check(unpack ? "emu_unpack_buckets launch" : "emu_pack_buckets launch");
}

// Launches the reshard of plan P, whose tables (segments, tile map) start at device address w, for
// `groups` tensor groups.
static int launch_plan(const Plan* P, const uint8_t* w, const uint64_t* sp, const uint64_t* dp, uint32_t groups,
                       hipStream_t st, const char* what) {
  const DevSeg* segs = reinterpret_cast<const DevSeg*>(w + P->ws.off_segs);
  const uint32_t* tm = reinterpret_cast<const uint32_t*>(w + P->ws.off_tilemap);
  const bool ntm = option(EMU_OPT_NONTEMPORAL) != 0, lds = option(EMU_OPT_LDS_STAGING) != 0;
  const bool xcd = option(EMU_OPT_XCD_REMAP) != 0;
  const Tables tb{sp, dp, groups, uint32_t(P->side[0].tensors.size()), uint32_t(P->side[1].tensors.size())};
  drop_pending_error();
  switch (P->tile_vecs) {
    case 1: dispatch_reshard<1>(P, ntm, lds, xcd, st, segs, tm, tb); break;
    case 2: dispatch_reshard<2>(P, ntm, lds, xcd, st, segs, tm, tb); break;
    case 4: dispatch_reshard<4>(P, ntm, lds, xcd, st, segs, tm, tb); break;
    case 16: dispatch_reshard<16>(P, ntm, lds, xcd, st, segs, tm, tb); break;
    default: dispatch_reshard<8>(P, ntm, lds, xcd, st, segs, tm, tb); break;
  }
  return hip_check(what);
}

// Enqueue on st the plan's tables into device memory at `base` laid out as the workspace: the copies of
// the host-filled parts, then the kernels that derive the tile map and, with `sides`, each side's stream
// tables. Without `sides` only the workspace's first ws.reshard_bytes (all emu_reshard reads) are written.
static int enqueue_tables(const Plan* P, uint8_t* base, bool sides, hipStream_t st, const char* what) {
  const WsLayout& w = P->ws;
  const uint64_t head = w.off_tilemap;
  if (head) {
    const hipError_t e = hipMemcpyAsync(base, P->host_ws.data(), head, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return fail(EMU_ERR_HIP, "%s: segment upload: %s", what, hipGetErrorString(e));
  }
  if (sides && w.host_end > w.reshard_bytes) {
    const hipError_t e = hipMemcpyAsync(base + w.reshard_bytes, P->host_ws.data() + head, w.host_end - w.reshard_bytes,
                                        hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return fail(EMU_ERR_HIP, "%s: table upload: %s", what, hipGetErrorString(e));
  }
  drop_pending_error();
  if (w.n_map) {
    uint32_t longest = 0;
    for (uint32_t n : P->seg_tiles) longest = n > longest ? n : longest;
    const uint32_t gy = uint32_t(std::max<uint64_t>(1, std::min<uint64_t>(64, (uint64_t(longest) + 255) / 256)));
    hipLaunchKernelGGL(k_tile_map, dim3(uint32_t(P->dsegs.size()) + 1, gy), dim3(256), 0, st,
                       reinterpret_cast<const DevSeg*>(base + w.off_segs),
                       reinterpret_cast<const uint32_t*>(base + w.off_seg_tiles), uint32_t(P->dsegs.size()),
                       reinterpret_cast<uint32_t*>(base + w.off_tilemap), P->ntiles_copy, P->zero_tile0,
                       P->zero_tile0 + P->ntiles_zero, w.n_map);
  }
  for (int sd = 0; sides && sd < 2; ++sd) {
    const SideInfo& s = P->side[sd];
    const SideTables& t = w.side[sd];
    if (s.nranks <= 0) continue;
    const uint32_t* rf = reinterpret_cast<const uint32_t*>(base + t.off_rank_first);
    const uint64_t* rb = reinterpret_cast<const uint64_t*>(base + t.off_rank_bytes);
    uint64_t* so = reinterpret_cast<uint64_t*>(base + t.off_stream);
    uint64_t* ri = reinterpret_cast<uint64_t*>(base + t.off_rank_info);
    hipLaunchKernelGGL(k_stream_tables, dim3(uint32_t(s.nranks)), dim3(64), 0, st,
                       reinterpret_cast<const uint64_t*>(base + t.off_sizes), rf, rb, so, ri);
    if (t.n_tiles)  // an encodable side: at most 2^20 tensors
      hipLaunchKernelGGL(k_chunk_map, dim3(uint32_t(s.tensors.size()) + 1), dim3(256), 0, st, rf, rb,
                         uint32_t(s.nranks), uint32_t(s.tensors.size()), so, ri,
                         reinterpret_cast<uint32_t*>(base + t.off_tile_map), t.n_tiles);
  }
  return hip_check(what);
}

// ------------------------------------------------------------------------------------------------
// plan tables without a caller workspace (emu_reshard_noalloc)
// ------------------------------------------------------------------------------------------------
// For callers that cannot allocate device memory, the reshard tables go to a static device array. Each
// device the library runs on holds its own copy of the array, at its own address, until the process
// ends. Host code never uses the array's name as an address (in host code it names a host-side
// stand-in): once per device, with that device current, hipGetSymbolAddress gives the device address,
// which is kept per device and used for the upload and as the kernels' table pointer.
constexpr uint64_t kScratchBytes = 32ull << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
  std::mutex mu;
  void* ptr = nullptr;    // device address of `scratch` on this device
  uint64_t resident = 0;  // id of the plan whose tables the array holds (0: none)
};
static ScratchSlot g_scratch[kMaxDevices];

// The current device's array, holding P's tables: the first call on a device looks the array up, and
// the tables are copied in (on stream st) unless the array already holds them from an earlier call.
static int scratch_tables(const Plan* P, hipStream_t st, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(EMU_ERR_HIP, "cannot query the current device");
  if (dev < 0 || dev >= kMaxDevices) return fail(EMU_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  ScratchSlot& sl = g_scratch[dev];
  std::lock_guard<std::mutex> lk(sl.mu);
  if (!sl.ptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(EMU_ERR_HIP, "scratch address on device %d: %s", dev, hipGetErrorString(e));
    sl.ptr = p;
  }
  if (sl.resident != P->id) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone)
      return fail(EMU_ERR_ARG, "the static scratch does not hold this plan's tables: make one call outside stream "
                  "capture first");
    sl.resident = 0;
    if (int rc = enqueue_tables(P, static_cast<uint8_t*>(sl.ptr), false, st, "emu_reshard_noalloc tables")) return rc;
    sl.resident = P->id;
  }
  *out = sl.ptr;
  return EMU_OK;
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
  if (workspace_bytes < P->ws.total)
    return fail(EMU_ERR_WORKSPACE, "workspace of %llu bytes, plan needs %llu", (unsigned long long)workspace_bytes,
                (unsigned long long)P->ws.total);
  ws_register(d_workspace, nullptr);  // until this upload is enqueued whole, the address holds no plan's tables
  if (int rc = enqueue_tables(P, static_cast<uint8_t*>(d_workspace), true, static_cast<hipStream_t>(hip_stream),
                              "emu_plan_upload"))
    return rc;
  ws_register(d_workspace, P);
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
  if (!ws_current(d_workspace, P))
    return fail(EMU_ERR_WORKSPACE, "workspace %p holds no upload of this plan (fill it with emu_plan_upload)",
                d_workspace);
  return launch_plan(P, static_cast<const uint8_t*>(d_workspace), d_src_ptrs, d_dst_ptrs, 1,
                     static_cast<hipStream_t>(hip_stream), "emu_reshard launch");
}

int emu_reshard_groups(emu_plan_t plan, const void* d_workspace, int32_t n_groups, const uint64_t* d_src_ptrs,
                       const uint64_t* d_dst_ptrs, void* hip_stream) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!d_workspace || !d_src_ptrs || !d_dst_ptrs) return fail(EMU_ERR_NULL, "NULL workspace or pointer table");
  if (n_groups < 1 || n_groups > 65535) return fail(EMU_ERR_RANGE, "n_groups %d not in [1, 65535]", n_groups);
  if (misaligned(d_workspace, kWsAlign)) return fail(EMU_ERR_WORKSPACE, "workspace not %llu-byte aligned", (unsigned long long)kWsAlign);
  if (misaligned(d_src_ptrs, 8) || misaligned(d_dst_ptrs, 8)) return fail(EMU_ERR_ALIGN, "pointer tables must be 8-byte aligned");
  if (P->ntiles == 0) return EMU_OK;
  if (!ws_current(d_workspace, P))
    return fail(EMU_ERR_WORKSPACE, "workspace %p holds no upload of this plan (fill it with emu_plan_upload)",
                d_workspace);
  return launch_plan(P, static_cast<const uint8_t*>(d_workspace), d_src_ptrs, d_dst_ptrs, uint32_t(n_groups),
                     static_cast<hipStream_t>(hip_stream), "emu_reshard_groups launch");
}

int emu_reshard_noalloc(emu_plan_t plan, const uint64_t* d_src_ptrs, const uint64_t* d_dst_ptrs, void* hip_stream) {
  clear_error();
  const Plan* P = reinterpret_cast<const Plan*>(plan);
  if (!plan_live(P)) return fail(EMU_ERR_HANDLE, "not a live plan");
  if (!d_src_ptrs || !d_dst_ptrs) return fail(EMU_ERR_NULL, "NULL pointer table");
  if (misaligned(d_src_ptrs, 8) || misaligned(d_dst_ptrs, 8)) return fail(EMU_ERR_ALIGN, "pointer tables must be 8-byte aligned");
  if (P->ntiles == 0) return EMU_OK;
  if (P->ws.reshard_bytes > kScratchBytes)
    return fail(EMU_ERR_WORKSPACE, "the plan's tables take %llu bytes, the static scratch holds %llu: use emu_reshard "
                "with a workspace", (unsigned long long)P->ws.reshard_bytes, (unsigned long long)kScratchBytes);
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  void* w = nullptr;
  const int rc = scratch_tables(P, st, &w);
  if (rc) return rc;
  return launch_plan(P, static_cast<const uint8_t*>(w), d_src_ptrs, d_dst_ptrs, 1, st, "emu_reshard_noalloc launch");
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
