/*
 * emu.h -- C ABI of the MI355X (gfx950) EMU Split/Merge reshard library (libemu.so).
 *
 * An Elastic Model Unit (EMU) is one model-stage replica <M, T_tp x pp, R, theta, omega> whose parameter
 * shards theta_i (i = 1..tp*pp) and optimizer shards omega share one TP/PP layout and are not sharded
 * across data-parallel replicas (paper, section 5, EMU definition). Split and Merge reshard that state
 * between two compatible layouts without changing it (section 5.2, primitives (a) and (b); section 6.2,
 * preserving training semantics). Layout changes run locally after the collectives, and every shard
 * travels as one contiguous buffer (section 6.2, transport and resharding-transport interplay).
 *
 * This library implements that local step on one GPU:
 *   emu_plan            compile a shard-to-shard copy map between two layouts (host only)
 *   emu_reshard         execute the map: source shard set -> destination shard set
 *   emu_pack_buckets    concatenate one side's shards per rank into fixed-size contiguous buckets
 *   emu_unpack_buckets  the inverse, on the receiver side
 *
 * Conventions (the paper fixes none of them; these are the readings the library implements):
 *   - Megatron-style sharding: q/k/v and gate/up column-parallel, o and down row-parallel,
 *     embedding and LM head vocab-parallel, RMSNorm weights replicated on every TP rank.
 *   - Fused QKV (EMU_QKV_HEAD_INTERLEAVED): per rank, for each local KV group g, the rows of g's query
 *     heads, then k_g, then v_g. With tp <= KV heads, tp divides the KV-head count. With tp > KV heads
 *     (KV replication) tp is a multiple of the KV heads and divides the query heads: rank t holds its
 *     nH/tp query heads, then one copy of k and v of head t*G/tp; copies are read from their first holder.
 *   - Fused gate/up (EMU_GATE_UP_BLOCK): per rank, [gate rows of the rank; up rows of the rank].
 *   - PP stages hold contiguous layer ranges; with L = q*pp + e the first e stages hold q+1 layers, the
 *     others q. The embedding is on stage 0, the final norm and LM head on stage pp-1; embeddings are
 *     untied.
 *   - Rank inside a unit: r = p*tp + t. Per-rank tensor order ("canonical order"): embed (p == 0);
 *     per local layer attn_norm, qkv (or q, k, v), o, mlp_norm, gate_up (or gate, up), down;
 *     final_norm, lm_head (p == pp-1). Tensor index tables list rank 0's tensors first, then rank 1's...
 *   - Vocabulary padding: pad multiple m > 0 pads V to ceil(V/(tp*m))*tp*m rows; m == 0 means no
 *     padding and tp must divide V. Destination pad rows are written with zeros; source pad rows are
 *     never read. Replicated norms are read from TP rank 0 of their stage.
 *   - Buckets: a rank's stream is its tensors' bytes in canonical order with no padding; bucket k of
 *     the rank holds stream bytes [k*B, (k+1)*B); the last bucket is short and bytes past its end are
 *     not touched. Bucket pointer tables list rank 0's buckets first, then rank 1's, ...
 *
 * Ownership and execution:
 *   - The caller allocates and owns every device buffer (tensors, buckets, pointer tables, workspace)
 *     and every stream. The library allocates host memory for plans only: it never calls hipMalloc or
 *     hipFree and never synchronizes a device or stream itself. Its only device memory is one static
 *     32 MiB array per device, part of its code object, that emu_reshard_noalloc uses as workspace. The
 *     host-to-device copies of emu_plan_upload (and of emu_reshard_noalloc's first call with a plan) read
 *     the plan's pageable host memory, and the HIP runtime may hold the calling thread until the stream
 *     has reached them: upload once per plan, before the work it should not wait for.
 *   - Pointer tables are DEVICE arrays of 64-bit device addresses. Every tensor and bucket base must be
 *     16-byte aligned. Source and destination buffers must not overlap (undefined behaviour).
 *   - A pointer table holds exactly the entries the plan indexes: n_src_tensors, n_dst_tensors, or the
 *     side's bucket count from emu_bucket_layout. The kernels read the tables on the device, so the
 *     library cannot check their length: a shorter table is undefined behaviour. emu_check_tables and
 *     emu_check_bucket_tables check host copies of full tables.
 *   - Execute calls only enqueue work on the given stream (a hipStream_t; NULL = default stream) on the
 *     current device, and return. Device faults surface at the caller's next synchronization. Buffers
 *     and the plan must stay alive until that work has completed.
 *   - Every function returns an emu_status (0 = EMU_OK); none aborts or throws. On error,
 *     emu_last_error() returns a thread-local message.
 *   - Launch failures are read from the HIP runtime's per-thread last error (hipGetLastError), which
 *     emu_reshard, emu_pack_buckets and emu_unpack_buckets clear just before launching: an error an
 *     earlier HIP call on the thread left pending is not reported as theirs, and is gone afterwards.
 *   - A plan is immutable after emu_plan and may be used from several threads; an uploaded workspace
 *     is only read by the kernels and may serve concurrent launches on several streams.
 */
#ifndef EMU_H
#define EMU_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EMU_ABI_VERSION 2

typedef enum {
  EMU_OK = 0,
  EMU_ERR_NULL = -1,        /* a required pointer argument is NULL */
  EMU_ERR_LAYOUT = -2,      /* a layout does not divide its model (invalid EMU layout) */
  EMU_ERR_MISMATCH = -3,    /* source and destination describe different models */
  EMU_ERR_UNSUPPORTED = -4, /* valid by definition but not implemented (emu_plan: a layout with more
                               than 2048 tensors on one rank, or a map of more than 2^32 tiles) */
  EMU_ERR_WORKSPACE = -5,   /* workspace too small, not 256-byte aligned, or not holding this plan's
                               upload (emu_plan_upload) */
  EMU_ERR_BUCKET = -6,      /* bucket size zero or not a multiple of the element size */
  EMU_ERR_ALIGN = -7,       /* a device pointer argument is not 16-byte aligned */
  EMU_ERR_HIP = -8,         /* the HIP runtime reported an error (message in emu_last_error) */
  EMU_ERR_HANDLE = -9,      /* not a live plan handle (NULL, freed, or foreign) */
  EMU_ERR_RANGE = -10,      /* an index or side argument is out of range */
  EMU_ERR_ARG = -11,        /* another argument is invalid (message in emu_last_error) */
  EMU_ERR_INFEASIBLE = -12, /* no deadlock-free transition DAG exists for the target plan */
  EMU_ERR_OVERLAP = -13     /* pointer tables name overlapping buffers (emu_check_tables) */
} emu_status;

typedef enum { EMU_BF16 = 0, EMU_FP32 = 1 } emu_dtype;                       /* 2 / 4 bytes */
typedef enum { EMU_QKV_HEAD_INTERLEAVED = 0, EMU_QKV_SEPARATE = 1 } emu_qkv_format;
typedef enum { EMU_GATE_UP_BLOCK = 0, EMU_GATE_UP_SEPARATE = 1 } emu_mlp_format;

typedef enum {
  EMU_T_EMBED = 0, EMU_T_ATTN_NORM = 1, EMU_T_QKV = 2, EMU_T_Q = 3, EMU_T_K = 4, EMU_T_V = 5,
  EMU_T_O = 6, EMU_T_MLP_NORM = 7, EMU_T_GATE_UP = 8, EMU_T_GATE = 9, EMU_T_UP = 10,
  EMU_T_DOWN = 11, EMU_T_FINAL_NORM = 12, EMU_T_LM_HEAD = 13,
  EMU_T_BUCKET = 14  /* destination side of a plan made by emu_plan_to_buckets */
} emu_tensor_kind;

/* Llama-style decoder shape: L layers, hidden H, nH query heads of head_dim, KV heads, MLP width, V. */
typedef struct {
  int32_t num_layers, hidden, num_heads, num_kv_heads, head_dim, ffn_hidden, vocab;
} emu_model_t;

/* One EMU layout T_tp x pp plus its storage conventions (paper section 5, EMU definition). */
typedef struct {
  emu_model_t model;
  int32_t tp, pp;
  int32_t vocab_pad_multiple; /* m; 0 = no padding */
  int32_t dtype;              /* emu_dtype */
  int32_t qkv_format;         /* emu_qkv_format */
  int32_t mlp_format;         /* emu_mlp_format */
} emu_layout_t;

typedef struct emu_plan_s* emu_plan_t;

typedef struct {
  int32_t n_src_ranks, n_dst_ranks;
  int32_t n_src_tensors, n_dst_tensors;
  int64_t n_segments;        /* copy segments + zero-fill segments */
  int64_t n_zero_segments;
  int64_t n_tiles;           /* work tiles of one emu_reshard launch */
  uint64_t tile_bytes;       /* destination bytes per full tile */
  uint64_t bytes_read;       /* bytes emu_reshard reads (source bytes of all non-zero-fill segments) */
  uint64_t bytes_written;    /* bytes emu_reshard writes: all destination bytes */
  uint64_t zero_fill_bytes;
  uint64_t src_bytes, dst_bytes;
  uint64_t workspace_bytes;  /* device workspace emu_plan_upload needs */
  int32_t src_vocab_padded, dst_vocab_padded;
  int32_t n_general_segments; /* segments not on the 16-byte vector path (misaligned runs) */
  int32_t converts;          /* 0: same element type; 1: fp32 -> bf16; 2: bf16 -> fp32 */
  int32_t n_alias_tensors;   /* destination tensors that are byte copies of one whole source tensor */
  int32_t aliased;           /* 1: the map leaves those tensors out (EMU_PLAN_ALIAS_RESIDENT) */
  uint64_t alias_bytes;      /* their bytes; with `aliased`, bytes_read and bytes_written exclude them */
} emu_plan_info_t;

typedef struct {
  int32_t rank;        /* r = p*tp + t */
  int32_t kind;        /* emu_tensor_kind */
  int32_t layer;       /* -1 for embed, final_norm, lm_head */
  int32_t ndim;        /* 1 for norms (rows == 1), else 2 */
  int64_t rows, cols;  /* row-major shape */
  uint64_t bytes;
  uint64_t stream_offset; /* byte offset inside its rank's bucket stream */
  int32_t alias;          /* destination side: index of the source tensor this tensor equals byte for
                             byte (same element type, whole tensor), else -1; source side: -1 */
  int32_t reserved;
} emu_tensor_desc_t;

/* One bucket of one side for a bucket size B: bucket `index` of rank `rank` holds stream bytes
 * [stream_offset, stream_offset + bytes) of that rank, stream_offset = index * B. */
typedef struct {
  int32_t rank, reserved;
  uint64_t index;
  uint64_t stream_offset;
  uint64_t bytes;         /* B, or less for the rank's last bucket */
} emu_bucket_desc_t;

/* Flags of emu_plan_ex. */
typedef enum {
  EMU_PLAN_DEFAULT = 0,
  EMU_PLAN_ALIAS_RESIDENT = 1  /* leave out of the map every destination tensor that is a byte copy of one
                                  whole source tensor (emu_tensor_desc_t.alias >= 0): the caller points
                                  its destination table entry at that source tensor instead */
} emu_plan_flags;

/* One entry of the copy map: for i < rows, src_run bytes of the source tensor (src_tensor < 0: none,
 * the destination gets zeros) at src_offset + i*src_stride become run bytes of the destination tensor at
 * dst_offset + i*dst_stride. src_run == run unless the plan converts the element type (then the run
 * holds the same elements in each side's type). */
typedef struct {
  int32_t src_tensor, dst_tensor;   /* global tensor indices (pointer-table positions) */
  uint64_t src_offset, dst_offset;  /* bytes */
  uint64_t src_stride, dst_stride;  /* bytes between consecutive rows */
  uint64_t rows, run;               /* rows x destination bytes */
  uint64_t src_run;                 /* source bytes read per row */
} emu_segment_t;

/* Tuning knobs (process-wide; change them only while no emu call is running). */
typedef enum {
  EMU_OPT_TILE_VECS = 0,     /* 16-byte vectors per thread per reshard tile (the reshard runs 64
                                threads per workgroup): 1, 2, 4, 8 or 16 (1 to 16 KB tiles), or 0 =
                                automatic (default): 4 (4 KB tiles). Read by emu_plan, so a plan
                                keeps its tile size */
  EMU_OPT_XCD_REMAP = 1,     /* 1 = give each XCD one contiguous eighth of the reshard tiles instead of
                                every eighth tile (default 1) */
  EMU_OPT_NONTEMPORAL = 2,   /* 1 = streaming (non-temporal) loads and stores (default 1) */
  EMU_OPT_LDS_STAGING = 3,   /* 1 = stage each tile through LDS between load and store (default 0) */
  EMU_OPT_BUCKET_WG_PER_CU = 4, /* persistent pack/unpack grid: workgroups per compute unit (default 32) */
  EMU_OPT_BUCKET_TILES = 5,  /* 1 = pack/unpack with one workgroup per 4 KB stream chunk (upload-time
                                chunk map; default); 0 = the persistent kernel that scans each rank's
                                tensor sizes into LDS (also used when the chunk map cannot encode a side:
                                4096 or more ranks, or more than 2^20 tensors on the side) */
  EMU_OPT_WG_PER_CU = 6,     /* reshard and tile pack/unpack kernels: cap on the workgroups resident
                                per compute unit, 1..32, enforced by reserving LDS per workgroup (the
                                LDS is split in two halves, so odd caps above 1 round down to even);
                                0 = no cap; -1 = automatic (default): 48 KB of reshard tiles (12 of
                                4 KB, 6 of 8 KB), 40 KB for fp32 -> bf16 plans, 64 KB for bf16 ->
                                fp32 plans, and 64 KB of pack/unpack chunks (16 of 4 KB); at least 2,
                                no cap from 32 up. Bounds the bytes in flight per CU, which sets how
                                well HBM serves a read/write stream */
  EMU_OPT_ROW_WRAP = 7       /* 1 = tile 2D segments as one row-major vector sequence, rows wrapping
                                inside a tile, wherever the kernel's row arithmetic is exact (default);
                                0 = whole rows per tile, or slices of one row. Read by emu_plan */
} emu_option;

/* Library version (EMU_ABI_VERSION). */
int emu_version(void);
/* Human-readable name of a status code. Never NULL. */
const char* emu_status_str(int status);
/* Thread-local detail of the last error returned on this thread ("" if none). Never NULL. */
const char* emu_last_error(void);
int emu_set_option(int32_t option, int64_t value);
int emu_get_option(int32_t option, int64_t* value);

/* Validate one layout (section 5.2: Split/Merge are defined between compatible layouts for any
 * integer factor). Returns EMU_OK or EMU_ERR_LAYOUT. Host only. */
int emu_layout_check(const emu_layout_t* layout);

/* Compile the copy map from layout *src to layout *dst of the same model (section 5.2, Split and
 * Merge; the call is direction-free and covers both and their compositions). Destination-driven: every
 * destination byte is covered by exactly one segment (zero-fill for destination vocabulary pad rows).
 * When the two layouts store different element types the map also converts every element: fp32 -> bf16
 * rounds to nearest, ties to even (NaNs stay NaN with the quiet bit set), bf16 -> fp32 is exact. This is
 * the weight synchronisation from a training model-stage to a generation model-stage of the same model
 * (section 5, EMU definition). Host only: no GPU call. *out receives a new plan. */
int emu_plan(const emu_layout_t* src, const emu_layout_t* dst, emu_plan_t* out);
/* emu_plan with flags (emu_plan_flags). EMU_PLAN_ALIAS_RESIDENT: shards already resident are not
 * copied (section 6.2, DAG execution and safety: Merge assembles the target from its sub-units and copies
 * no shard that is already in place). Every plan reports its alias tensors (emu_plan_info,
 * emu_tensor_info); with this flag the map leaves them out, emu_reshard writes only the other
 * destination tensors, and the caller uses the source tensor as the destination tensor (for a PP-only
 * change every destination tensor is one, and the reshard moves nothing). Whatever the destination
 * table holds at an alias tensor's index is neither read nor written by emu_reshard. Unknown flags:
 * EMU_ERR_ARG. Host only. */
int emu_plan_ex(const emu_layout_t* src, const emu_layout_t* dst, uint32_t flags, emu_plan_t* out);
/* Compile the fused sender-side map: source shards of layout *src straight into the contiguous
 * transfer buckets of layout *dst's ranks (bucket k of rank r = bytes [k*B, (k+1)*B) of r's stream),
 * skipping the destination tensors. The paper sends each shard once as a contiguous buffer after a
 * local layout change (section 6.2, transport and resharding-transport interplay); this plan does both
 * in one pass over HBM. The plan's destination side (side 1) is the bucket list, rank 0's first, so it
 * is executed with emu_reshard(plan, ws, d_src_ptrs, d_bucket_ptrs, stream), and the receiver restores
 * the tensors with emu_unpack_buckets on an ordinary emu_plan(src, dst). Bucket bytes are identical to
 * emu_pack_buckets applied to the emu_reshard result. bucket_bytes must be a positive multiple of the
 * element size (EMU_ERR_BUCKET). Host only. */
int emu_plan_to_buckets(const emu_layout_t* src, const emu_layout_t* dst, uint64_t bucket_bytes, emu_plan_t* out);
/* The receiver's side of the same transport: a plan that reads the transfer buckets of layout *src's
 * ranks (bucket k of rank r = bytes [k*B, (k+1)*B) of r's stream) and writes layout *dst's tensors,
 * restoring the shards from the contiguous buffers (section 6.2, transport and resharding-transport
 * interplay) and, when dst differs from src, resharding them in the same pass. The plan's source side
 * (side 0) is the bucket list, rank 0's first, so it is executed with emu_reshard(plan, ws,
 * d_bucket_ptrs, d_dst_ptrs, stream). With dst == src it is emu_unpack_buckets for a bucket size fixed
 * at plan time, run by the reshard kernel; the tensors equal emu_unpack_buckets's (and, for dst != src,
 * emu_reshard's of the unpacked tensors). bucket_bytes must be a positive multiple of the source
 * element size (EMU_ERR_BUCKET). Host only. */
int emu_plan_from_buckets(const emu_layout_t* src, const emu_layout_t* dst, uint64_t bucket_bytes, emu_plan_t* out);
/* Free a plan. Work enqueued with it must have completed. */
int emu_plan_free(emu_plan_t plan);
int emu_plan_info(emu_plan_t plan, emu_plan_info_t* out);
/* Shape of tensor `index` (global, rank-major canonical order) on side 0 (source) or 1 (dest). */
int emu_tensor_info(emu_plan_t plan, int32_t side, int32_t index, emu_tensor_desc_t* out);
/* Copy `count` segments starting at `first` (in execution order) into out[]. */
int emu_plan_segments(emu_plan_t plan, int64_t first, int64_t count, emu_segment_t* out);

/* Fill the caller's workspace (at least info.workspace_bytes, 256-byte aligned) with the plan's tables:
 * enqueue the host-to-device copies of what the host computes (the copy map's segments with their tile
 * counts; per side the tensor sizes, each rank's tensor range and stream length: about 100 KB for the 8B
 * transitions), then small kernels that derive the rest on the device (the reshard's tile-to-segment map;
 * per side each tensor's offset in its rank's stream, per-rank records, and the map from every 4 KB chunk
 * of a stream to its rank and tensor). emu_plan_workspace_image gives the resulting bytes. The plan must
 * outlive the copies. Their source is pageable host memory, so the HIP runtime may return only once the
 * stream has reached them. The library records that
 * this address now holds this plan's tables: execute calls of the plan accept only a workspace address so
 * recorded (EMU_ERR_WORKSPACE otherwise, before anything is launched), and an upload of another plan to
 * the same address replaces the record. The record is of the address, not of the allocation: the caller
 * keeps the workspace allocated, and unwritten by anything but emu_plan_upload, while it uses it (a
 * buffer freed and a new one allocated at the same address would pass for the upload). */
int emu_plan_upload(emu_plan_t plan, void* d_workspace, uint64_t workspace_bytes, void* hip_stream);
/* The workspace contents emu_plan_upload produces, computed on the host into out[0, info.workspace_bytes)
 * (bytes smaller than that: EMU_ERR_WORKSPACE), for checking an uploaded workspace byte for byte. Gaps
 * between the tables are zero here and unspecified in the uploaded workspace. Host only. */
int emu_plan_workspace_image(emu_plan_t plan, void* out, uint64_t bytes);

/* Execute the reshard (section 5.2 (a)/(b), the local layout change of section 6.2):
 * d_src_ptrs[i] is the device address of source tensor i, d_dst_ptrs[j] of destination tensor j
 * (both device arrays of n_src_tensors / n_dst_tensors entries). Reads only the source, writes every
 * destination byte exactly once. d_workspace holds the uploaded plan tables. */
int emu_reshard(emu_plan_t plan, const void* d_workspace, const uint64_t* d_src_ptrs,
                const uint64_t* d_dst_ptrs, void* hip_stream);

/* emu_reshard of n_groups shard sets that share the plan's layouts, in one launch: the parameters and
 * the optimizer states that follow their layout (section 5, EMU definition: omega in theta's layout),
 * e.g. fp32 master weights, Adam m and Adam v. d_src_ptrs holds n_groups source tables back to back
 * (group g's tensor i at g * n_src_tensors + i), d_dst_ptrs n_groups destination tables likewise. The
 * result equals n_groups emu_reshard calls, one per group. 1 <= n_groups <= 65535 (EMU_ERR_RANGE). */
int emu_reshard_groups(emu_plan_t plan, const void* d_workspace, int32_t n_groups, const uint64_t* d_src_ptrs,
                       const uint64_t* d_dst_ptrs, void* hip_stream);

/* emu_reshard without a caller workspace, for callers that cannot allocate device memory (code that
 * must not call hipMalloc, tight serving loops, harnesses that forbid allocation). The plan's reshard
 * tables (segments and tile map, at most 32 MiB: every plan of a decoder up to the 8B shapes at the
 * default tile size fits; a larger one returns EMU_ERR_WORKSPACE before anything is enqueued) live in a
 * static device array of the library, of which every device it runs on holds one copy until the
 * process ends. The call allocates nothing and launches the same kernels as emu_reshard: the first call
 * with a plan on a device enqueues, on hip_stream, the copy of its segments into that device's array
 * (from the plan's pageable host memory, so the plan must outlive it) and the kernel that derives the
 * tile map there, as emu_plan_upload does; later calls with the same plan find the tables there and
 * only launch. Under stream capture a call whose tables are not yet resident
 * returns EMU_ERR_ARG: make one call outside capture first.
 * All calls on one device share its array, which holds the tables of the last plan copied in: calls
 * that overlap on one device with different plans (on different streams, or from several threads)
 * race and are undefined; calls on one stream are ordered. Arguments, pointer tables and status codes
 * as for emu_reshard. */
int emu_reshard_noalloc(emu_plan_t plan, const uint64_t* d_src_ptrs, const uint64_t* d_dst_ptrs, void* hip_stream);

/* Bucket geometry of one rank (rank >= 0) or of all ranks together (rank == -1) of one side, for
 * bucket size bucket_bytes (section 6.2: each shard sent once as a contiguous buffer). Host only. */
int emu_bucket_layout(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, int32_t rank,
                      uint64_t* n_buckets, uint64_t* stream_bytes);
/* Buckets [first, first + count) of one side for bucket size bucket_bytes, in pointer-table order (rank
 * 0's first), into out[] (section 6.2: each shard sent once as a contiguous buffer): the sizes a caller
 * allocates and the stream range each bucket carries. EMU_ERR_RANGE if the range passes the side's
 * bucket count (emu_bucket_layout(..., -1, ...)). Host only. */
int emu_bucket_info(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, uint64_t first, uint64_t count,
                    emu_bucket_desc_t* out);

/* Pack one side's tensors into contiguous buckets (section 6.2: each shard is sent once as a contiguous
 * buffer, after the local layout change): bucket k of rank r receives bytes [k*B, (k+1)*B) of r's
 * stream. d_tensor_ptrs lists that side's tensors (as for emu_reshard); d_bucket_ptrs lists all
 * buckets, rank 0 first (emu_bucket_layout(..., -1, ...) of them). Tensor stream offsets (exclusive
 * prefix sums of the ragged tensor sizes, a wave64 scan per rank at upload) come from the workspace;
 * each rank's first bucket index depends on bucket_bytes and is formed per call (on the host for the
 * first 128 ranks, by a wave64 reduction on the device beyond; the persistent fallback kernel scans the
 * tensor sizes on the device). bucket_bytes must be a positive multiple of the element size. */
int emu_pack_buckets(emu_plan_t plan, const void* d_workspace, int32_t side, uint64_t bucket_bytes,
                     const uint64_t* d_tensor_ptrs, const uint64_t* d_bucket_ptrs, void* hip_stream);
/* The inverse of emu_pack_buckets on the receiver side (section 6.2: the receiver restores its shards
 * from the contiguous buffers): buckets -> that side's tensors. */
int emu_unpack_buckets(emu_plan_t plan, const void* d_workspace, int32_t side, uint64_t bucket_bytes,
                       const uint64_t* d_bucket_ptrs, const uint64_t* d_tensor_ptrs, void* hip_stream);

/* Host-side checks of pointer tables before an execute call (debug aid; host only, no GPU calls).
 * The tables are HOST copies of the device pointer tables the execute call will receive.
 *
 * emu_check_tables: src_ptrs[n_src_tensors], dst_ptrs[n_dst_tensors] for emu_reshard (for a plan from
 * emu_plan_to_buckets the destination entries are the buckets). Every entry must be non-zero
 * (EMU_ERR_NULL) and 16-byte aligned (EMU_ERR_ALIGN), and no destination byte range may overlap
 * another destination range or a source range (EMU_ERR_OVERLAP); source ranges may overlap each other.
 * The destination entries of alias tensors a plan leaves out of its map (EMU_PLAN_ALIAS_RESIDENT) are
 * not written and take no part in the overlap test.
 *
 * emu_check_bucket_tables: tensor_ptrs of one side and bucket_ptrs of its buckets of size bucket_bytes
 * (as for emu_pack_buckets / emu_unpack_buckets). The same conditions, with every tensor and bucket
 * range pairwise disjoint, since either kind is written by one of the two calls.
 *
 * emu_last_error() names the offending entries. Sorting sweep, O(n log n) in the table sizes. */
int emu_check_tables(emu_plan_t plan, const uint64_t* src_ptrs, const uint64_t* dst_ptrs);
int emu_check_bucket_tables(emu_plan_t plan, int32_t side, uint64_t bucket_bytes, const uint64_t* tensor_ptrs,
                            const uint64_t* bucket_ptrs);

/* ------------------------------------------------------------------------------------------------
 * Transition-DAG planner (host only). From a current to a target plan of several model-stages: the
 * Split / Destroy / Extend / Merge primitives that carry each model-stage's EMU collection over through
 * the largest common layout T_sub, the resource-dependency edges between model-stages that hand GPUs to
 * each other, and the DAG's critical-path cost L_tran (paper section 6.1, decomposition and DAG
 * construction; L_tran from bytes, link bandwidth and communicator setup, section 6 introduction).
 *
 * Readings implemented (the paper gives no listing):
 *   - T_sub = (gcd(tp, tgt_tp), gcd(pp, tgt_pp)); a (tp, pp) unit splits into (tp/tps)(pp/pps) sub-units,
 *     sub-unit (a, b) holding the unit's ranks (a*tps + t', b*pps + p') at its rank (t', p').
 *   - Sub-units whose GPUs all lie in the target GPU set are kept (first fit, as many as the target
 *     needs); the others are destroyed, each only after any Extend copying from it.
 *   - Missing sub-units are extended onto the target GPUs no kept sub-unit holds (ascending ids), each
 *     copied from a replica on a disjoint GPU set (cyclic first fit).
 *   - Every (tgt_tp / tps)(tgt_pp / pps) sub-units (kept first, then extended) merge into one target unit.
 *   - Model-stages of one stage kind run concurrently and hold disjoint GPUs: an Extend onto a GPU
 *     another such model-stage holds waits for the Destroy that releases it (resource edge), resolved
 *     in generation -> inference -> training order; if that Destroy depends on the Extend, no
 *     deadlock-free order exists and emu_dag_plan returns EMU_ERR_INFEASIBLE.
 *   - Costs: Split = setup + (shard_sub - shard_cur)/bw(unit); Extend = setup + max over rank pairs of
 *     shard_sub/bw(pair); Merge = shard_target/hbm_bw; Destroy = 0; bw is intra-node when every GPU
 *     involved sits in one node (id / gpus_per_node), else inter-node. L_tran is the longest path.
 * ------------------------------------------------------------------------------------------------ */

typedef enum { EMU_STAGE_GENERATION = 0, EMU_STAGE_INFERENCE = 1, EMU_STAGE_TRAINING = 2 } emu_stage_kind;
typedef enum { EMU_PRIM_SPLIT = 0, EMU_PRIM_DESTROY = 1, EMU_PRIM_EXTEND = 2, EMU_PRIM_MERGE = 3 } emu_primitive;

typedef struct {
  int32_t kind;                    /* emu_stage_kind */
  int32_t tp, pp, dp;              /* current layout and number of units */
  int32_t tgt_tp, tgt_pp, tgt_dp;  /* target */
  int32_t reserved;
  const int32_t* gpus;             /* dp*tp*pp current GPU ids, unit-major, rank order r = p*tp + t */
  const int32_t* tgt_gpus;         /* tgt_dp*tgt_tp*tgt_pp distinct ids: the target GPU set */
  double state_bytes;              /* logical state (parameters + optimizer) of one replica */
} emu_stage_transition_t;

typedef struct {
  int32_t gpus_per_node, reserved;
  double intra_bw, inter_bw;       /* bytes/s per GPU pair, inside a node / across nodes */
  double hbm_bw;                   /* bytes/s of a local copy */
  double setup_s;                  /* communicator setup per collective */
} emu_link_model_t;

typedef struct {
  int32_t prim, stage;             /* emu_primitive, model-stage index */
  int32_t unit;                    /* SPLIT: current unit; DESTROY: sub-unit; EXTEND: new sub-unit slot;
                                      MERGE: target unit */
  int32_t src;                     /* EXTEND: sub-unit copied from; otherwise -1 */
  int32_t gpu_first, n_gpus;       /* the primitive's GPUs: emu_dag_gpus entries [gpu_first, +n_gpus) */
  double cost_s, start_s, finish_s;
} emu_dag_node_t;

typedef struct { int32_t from, to, resource, reserved; } emu_dag_edge_t;  /* resource: cross-stage edge */

typedef struct {
  int32_t n_nodes, n_edges, n_resource_edges, n_gpu_entries;
  double l_tran_s;                 /* critical-path cost of the transition */
  double plan_ms;                  /* host time emu_dag_plan spent building the DAG */
} emu_dag_info_t;

typedef struct emu_dag_s* emu_dag_t;

/* Plan the transition of n_stages model-stages. Returns EMU_ERR_ARG for invalid input (including
 * overlapping GPU sets of two model-stages of one kind), EMU_ERR_INFEASIBLE when no deadlock-free DAG
 * exists. Nodes are listed per model-stage in input order (Splits, Destroys, Extends, Merges); edges are
 * ordered by (to, from). */
int emu_dag_plan(const emu_stage_transition_t* stages, int32_t n_stages, const emu_link_model_t* links,
                 emu_dag_t* out);
int emu_dag_free(emu_dag_t dag);
int emu_dag_info(emu_dag_t dag, emu_dag_info_t* out);
int emu_dag_nodes(emu_dag_t dag, int32_t first, int32_t count, emu_dag_node_t* out);
int emu_dag_edges(emu_dag_t dag, int32_t first, int32_t count, emu_dag_edge_t* out);
int emu_dag_gpus(emu_dag_t dag, int32_t first, int32_t count, int32_t* out);
/* GPU ids of target unit `unit` of model-stage `stage`, in rank order (tgt_tp*tgt_pp entries). */
int emu_dag_target_unit(emu_dag_t dag, int32_t stage, int32_t unit, int32_t* gpus_out);

#ifdef __cplusplus
}
#endif

#endif /* EMU_H */
