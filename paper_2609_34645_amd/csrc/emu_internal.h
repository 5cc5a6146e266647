// Internal structures shared by the host plan compiler (emu_plan.cpp) and the HIP executor
// (emu_exec.hip). Not part of the public ABI.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "emu.h"

namespace emu {

constexpr uint32_t kPlanMagic = 0x454d5550u;  // "EMUP"
constexpr int kThreads = 256;                 // workgroup size of the persistent pack/unpack kernel (4 wave64s)
constexpr int kReshardThreads = 64;           // workgroup size of the reshard kernel (one wave64)
constexpr int kMaxRankTensors = 2048;         // per-rank tensor offsets live in LDS during pack/unpack
#ifndef EMU_CHUNK_BYTES
#define EMU_CHUNK_BYTES 32768
#endif
constexpr uint64_t kChunkBytes = EMU_CHUNK_BYTES;  // pack/unpack work unit, in stream bytes
#ifndef EMU_TILE_CHUNK_BYTES
#define EMU_TILE_CHUNK_BYTES 4096
#endif
constexpr uint64_t kTileChunkBytes = EMU_TILE_CHUNK_BYTES;  // unit of the tile-per-workgroup pack/unpack kernel
constexpr uint32_t kMapTensorBits = 20;            // chunk map entry: rank << 20 | global tensor index
constexpr uint64_t kWsAlign = 256;
constexpr uint32_t kXcdCount = 8;          // XCDs of an MI355X; reshard grids are a multiple of this
constexpr uint32_t kNoSeg = 0xffffffffu;   // tile map padding entry: the workgroup has no tile

// Segment execution modes. Every "vec" mode needs src/dst offsets, strides and the run to be
// multiples of 16 bytes (and 16-byte aligned tensor bases, an ABI requirement).
enum SegMode : uint32_t {
  SEG_VEC_1D = 0,        // one contiguous run; a tile is a fixed slice of it
  SEG_VEC_ROWS = 1,      // rows shorter than a tile; a tile is `param` whole rows
  SEG_VEC_ROWCHUNK = 2,  // rows longer than a tile; a tile is one slice of one row
  SEG_GENERAL = 3,       // any byte alignment; a tile is one slice of one row, copied bytewise
  SEG_VEC_FLAT = 4,      // rows of any length; a tile is a fixed slice of the rows' vectors in row-major
                         // order, so rows wrap inside a tile and only a segment's last tile is partial
};
constexpr uint32_t SEG_MODE_MASK = 0xff;
constexpr uint32_t SEG_ZERO = 0x100;  // no source: write zeros

// Element conversion of a plan (all copy segments of one plan share it).
enum Convert : int { CVT_NONE = 0, CVT_F32_BF16 = 1, CVT_BF16_F32 = 2 };

// Device copy of one segment. 80 bytes, read with scalar loads by the reshard kernel.
struct alignas(16) DevSeg {
  uint64_t src_off, dst_off;
  uint64_t src_stride, dst_stride;
  uint64_t rows, run;
  int32_t src_idx, dst_idx;
  uint32_t mode;   // SegMode | SEG_ZERO
  uint32_t param;  // SEG_VEC_ROWS: rows per tile; SEG_VEC_ROWCHUNK / SEG_GENERAL: tiles per row;
                   // SEG_VEC_FLAT: rows * rv, the segment's vectors
  uint32_t rv;     // SEG_VEC_ROWS / SEG_VEC_FLAT: 16-byte vectors per row
  uint32_t magic;  // SEG_VEC_ROWS / SEG_VEC_FLAT: ceil(2^32 / rv) for rv > 1 (n / rv == umulhi(n, magic)
                   // for n * rv < 2^32)
  uint64_t tile0;  // map index of the segment's first tile
};
static_assert(sizeof(DevSeg) == 80, "DevSeg layout");

// Byte offsets of the tables inside the device workspace.
struct SideTables {
  uint64_t off_sizes;        // uint64[n_tensors]   tensor byte sizes, global order
  uint64_t off_rank_first;   // uint32[n_ranks + 1] first global tensor index of each rank
  uint64_t off_rank_bytes;   // uint64[n_ranks]     stream length of each rank
  uint64_t off_chunk_first;  // uint64[n_ranks + 1] first pack/unpack chunk of each rank
  uint64_t off_stream;       // uint64[n_tensors]   stream offset of each tensor inside its rank
  uint64_t off_rank_info;    // uint64[n_ranks][4]  {first chunk (kTileChunkBytes), stream bytes,
                             //                      end of the rank's global tensor range, 0}
  uint64_t off_tile_map;     // uint32[n_tiles]     rank << 20 | global index of the tensor holding the
                             //                      chunk's first byte; padded with kNoSeg to kXcdCount
  uint64_t n_tiles;          // map entries including the padding (0 when the map cannot encode the side)
};

// Workspace order: segments, their tile counts, the tile map, each side's host tables (sizes, rank_first,
// rank_bytes, chunk_first), then each side's device-built tables (stream offsets, rank records, chunk
// map). emu_plan_upload copies the segments with their tile counts and the host tables; its kernels
// derive the tile map and the device-built tables from them. Segments, tile counts and tile map -- all
// emu_reshard reads -- are the workspace's first reshard_bytes.
struct WsLayout {
  uint64_t off_segs;       // DevSeg[n_segments]
  uint64_t off_seg_tiles;  // uint32[n_segments]  tiles of each segment
  uint64_t off_tilemap;    // uint32[n_map]  segment index of every tile: copy tiles, then zero-fill tiles,
                           //                each section padded with kNoSeg to a multiple of kXcdCount
  uint64_t n_map;
  uint64_t reshard_bytes;  // end of the tile map: start of the sides' host tables
  SideTables side[2];
  uint64_t host_end;       // end of the sides' host tables: start of the device-built tables
  uint64_t total;
};

struct SideInfo {
  emu_layout_t lay{};
  int64_t vp = 0;
  int32_t nranks = 0;
  uint64_t total_bytes = 0;
  bool offsets_grid = true;           // every tensor's stream offset is a multiple of kTileChunkBytes
  std::vector<emu_tensor_desc_t> tensors;
  std::vector<uint32_t> rank_first;   // nranks + 1
  std::vector<uint64_t> rank_bytes;   // nranks
  std::vector<uint64_t> chunk_first;  // nranks + 1
};

struct Plan {
  uint32_t magic = kPlanMagic;
  uint64_t id = 0;                  // unique per plan object of the process (never reused)
  SideInfo side[2];
  std::vector<emu_segment_t> segs;  // execution order
  std::vector<DevSeg> dsegs;
  int tile_vecs = 2;                // 16-byte vectors per thread per tile
  int cvt = CVT_NONE;               // element conversion of the whole plan
  bool aliased = false;             // alias destination tensors are left out of the map
  uint64_t tile_bytes = 0;
  uint64_t ntiles = 0;              // copy + zero-fill tiles
  uint64_t ntiles_copy = 0;         // tiles [0, ntiles_copy) of the map: copy segments
  uint64_t zero_tile0 = 0;          // tiles [zero_tile0, zero_tile0 + ntiles_zero): zero-fill segments
  uint64_t ntiles_zero = 0;
  emu_plan_info_t info{};
  WsLayout ws{};
  std::vector<uint32_t> seg_tiles;  // tiles of each segment (dsegs order)
  // The uploaded bytes: workspace [0, ws.off_tilemap) (segments and their tile counts), then workspace
  // [ws.reshard_bytes, ws.host_end) (the sides' host tables), back to back.
  std::vector<uint8_t> host_ws;
};

uint64_t next_plan_id();

// errors.cpp-style helpers (defined in emu_plan.cpp)
int fail(int code, const char* fmt, ...);
void clear_error();
bool plan_live(const Plan* p);
int64_t option(int32_t key);

// Workspace registry (emu_plan.cpp): which plan's tables were last uploaded to each workspace address.
// Execute calls refuse an address that never received an upload of their plan, or whose last upload
// was another plan's. The registry knows addresses, not allocations: a workspace freed after its upload
// and an unrelated buffer later allocated at the same address pass for the upload (the caller must keep
// an uploaded workspace alive while it uses it; the Python binding holds the tensors it uploaded to).
void ws_register(const void* ws, const Plan* p);
bool ws_current(const void* ws, const Plan* p);
void ws_forget(const Plan* p);

}  // namespace emu
