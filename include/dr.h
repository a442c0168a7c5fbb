/*
 * dr.h - C ABI of libdr.so: bounded state staging for the Training->Rollout
 * role switch of DynaResize (arXiv 2607.22614: GPUs move between the training
 * and rollout roles of a disaggregated LLM post-training job while it runs), on
 * one AMD Instinct MI355X (gfx950).
 *
 * The paper (Sec. 3.3, "Staged State Reloading") migrates a GPU's training
 * state (weights and optimizer states, sharded FSDP-style) through host memory
 * in fine-grained, bounded chunks, loads only the weights at the transition and
 * postpones the optimizer-state reload until the first training step after the
 * resize; the rollout role receives the weights through weight synchronization
 * (Sec. 3.2).
 * This library is the data-parallel part of that path on one GPU:
 *
 *   dr_plan_create      compile (model shape, W shards, T ranks, budgets) into
 *                       a device-resident segment table, once per topology
 *                       (the per-topology metadata cache of Sec. 3.2);
 *   dr_stage_chunk      pack + cast one B-byte chunk of the rollout stream and
 *                       its checksum (bounded chunk of Sec. 3.3);
 *   dr_stage_all        the same for every chunk, one call (the weights moved
 *                       on the role-switch critical path, Sec. 3.3);
 *   dr_offload_moments  stream the Adam moments to host memory through two
 *                       bounded pinned buffers (Sec. 3.3);
 *   dr_restore_moments  the deferred reload of those moments (Sec. 3.3, last
 *                       paragraph).
 *
 * Layouts (the paper names them but does not spell them out; this fixes them):
 *
 *   Training layout.  Tensors in model order: embed[V,H]; per layer l:
 *   ln1[H], q[Hq*D,H], k[Hkv*D,H], v[Hkv*D,H], o[H,Hq*D], ln2[H], gate[F,H],
 *   up[F,H], down[H,F]; then final_norm[H], lm_head[V,H].  Each is row-major
 *   [out,in] fp32, packed densely; the flat buffer is zero-padded at its tail to
 *   Npad = a multiple of W*256 elements and cut into W equal contiguous shards
 *   of S = Npad/W elements.  Shard w is passed as its own device pointer.
 *
 *   Rollout layout of TP rank r (qh=Hq/T, kh=Hkv/T, Fr=F/T, Vr=V/T), bf16,
 *   row-major, packed densely in this order:
 *     embed_r   = embed[r*Vr:(r+1)*Vr, :]                         [Vr, H]
 *     per layer:
 *       ln1     (replicated)                                      [H]
 *       qkv_r   = rows [q heads r*qh.. ; k heads r*kh.. ; v heads r*kh..]
 *                                                                 [(qh+2kh)*D, H]
 *       o_r     = o[:, r*qh*D:(r+1)*qh*D]                         [H, qh*D]
 *       ln2     (replicated)                                      [H]
 *       gate_up_r = rows [gate r*Fr.. ; up r*Fr..]                [2Fr, H]
 *       down_r  = down[:, r*Fr:(r+1)*Fr]                          [H, Fr]
 *     final_norm (replicated)                                     [H]
 *     lm_head_r = lm_head[r*Vr:(r+1)*Vr, :]                       [Vr, H]
 *   The rollout stream is rank 0's tensors, then rank 1's, ... (rank-major).
 *
 *   Cast: IEEE 754 round-to-nearest-even fp32 -> bf16 on the bit pattern; fp32
 *   subnormals round (never flushed), overflow gives +-Inf, +-0/+-Inf kept; a
 *   NaN becomes (bits >> 16) | 0x0040 (sign and top payload kept, quiet).
 *
 *   Chunks: chunk c is stream bytes [c*B, min((c+1)*B, total)).
 *
 *   Checksum of a chunk: with w_j the little-endian u32 at chunk bytes
 *   [4j, 4j+4), s1 = sum_j w_j and s2 = sum_j (j+1)*w_j, both mod 2^64.
 *
 *   Moment stream: m_0 || ... || m_{W-1} || v_0 || ... || v_{W-1} as fp32
 *   bytes, padding included, cut every Bm bytes.
 *
 * Conventions for every call:
 *   - Returns DR_OK (0) or a negative DR_E* code; dr_last_error() then holds a
 *     message (thread-local, valid until the next failing call on the thread).
 *     A failed HIP call is reported this way only: the HIP runtime's per-thread
 *     last error is consumed (hipGetLastError) before DR_EHIP or DR_ENOMEM is
 *     returned, so it does not surface again in the caller's own HIP calls.
 *   - Arguments are validated before any HIP call: a call that returns
 *     DR_EINVAL or DR_ERANGE has launched and copied nothing.  A call that
 *     returns DR_EHIP may have launched part of its kernels, and the plan's
 *     checksum accumulators may then hold partial sums: destroy such a plan
 *     and create it again before trusting its checksums.
 *     (dr_stage_chunk_noalloc clears its static array at its next call.)
 *   - No C++ exception crosses the ABI.
 *   - Device pointers belong to the caller and must stay valid until the work
 *     enqueued on them has completed.  Pointer arrays ("shards") are host
 *     arrays of device pointers, read during the call only.
 *   - A plan is used on the device that was current when it was created.
 *   - Threads.  The introspection calls and the staging calls (dr_stage_chunk,
 *     dr_stage_all, dr_reshard) only read the plan on the host and may run on
 *     several threads at once, within the per-chunk rule of dr_stage_chunk.
 *     The moment calls use the plan's bounce buffers: one transfer at a time
 *     per plan (a second one returns DR_EINVAL), on any thread, overlapping
 *     staging calls on other threads.  dr_stage_through_host and
 *     dr_reshard_through_host use the plan's relay buffers and events: one
 *     call at a time per plan.  dr_plan_destroy
 *     runs when no other call on the plan is running.  dr_last_error() is per
 *     thread.
 */
#ifndef DR_H
#define DR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  DR_OK = 0,
  DR_EINVAL = -1, /* bad shape, layout, pointer or alignment */
  DR_ERANGE = -2, /* chunk index out of range */
  DR_ENOMEM = -3, /* host or device allocation failed */
  DR_EHIP = -4,   /* a HIP runtime call failed; its message is in dr_last_error() */
};

enum { DR_MAX_SHARDS = 64 };

typedef struct dr_plan dr_plan; /* opaque; owns the device tables and pinned bounce buffers */

/* Decoder shape.  n_layers >= 0 (0: embed, final_norm and lm_head only), every
 * other field > 0; hidden % 8 == 0; n_q_heads % n_kv_heads == 0. */
typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
} dr_model;

/* Staging layout.  train_shards = W in [1, 64]; tp = T >= 1 must divide
 * n_q_heads, n_kv_heads, ffn and vocab.  chunk_bytes = B: a multiple of 16,
 * >= 16, at most 2^24 chunks, fewer than 2^32 - 2^24 workgroup tiles
 * (dr_plan_info.num_tiles).  moment_chunk_bytes = Bm: 0 (no moment path) or
 * a multiple of 16, at most 2^24 moment chunks.
 * tile_depth: 16-byte groups per lane in a stage-kernel tile (tiles of
 * 1024 * tile_depth elements), a launch-geometry choice that never changes a
 * result: 2 or 4 explicitly, or 0 = automatic.  Depth 2 is fastest for a pack
 * that follows another pack without a pause; depth 4 keeps more bytes in
 * flight per CU and is faster for a pack that follows idle time or other
 * kernels (the usual role switch), for one-chunk launches and past 128 GiB.
 * An automatic plan whose source + rollout bytes stay within 128 GiB holds
 * both tilings.  dr_stage_chunk (and the host relay, chunk by chunk) takes
 * depth 4; dr_stage_all picks per launch: depth 2 when the call comes while
 * the packs this library launched on the device are still expected to run,
 * or within 2 ms of their expected end (estimated on the host from the times
 * their launches returned and their bytes at 6.5 TB/s), else depth 4.  Past
 * 128 GiB an automatic plan uses depth 4. */
typedef struct {
  int32_t train_shards, tp;
  uint64_t chunk_bytes, moment_chunk_bytes;
  int32_t tile_depth;
  int32_t reserved; /* 0 */
} dr_layout;

#define DR_TILE_DEPTH_AUTO 0

typedef struct {
  uint64_t s1, s2;
} dr_checksum;

typedef struct {
  uint64_t n_elems;        /* N: training elements without padding */
  uint64_t padded_elems;   /* Npad */
  uint64_t shard_elems;    /* S = Npad / W */
  uint64_t norm_elems;     /* (2L+1)*H */
  uint64_t rank_elems;     /* bf16 elements of one rollout rank */
  uint64_t rollout_bytes;  /* 2 * T * rank_elems: the whole stream */
  uint64_t num_chunks;     /* ceil(rollout_bytes / B) */
  uint64_t last_chunk_bytes;
  uint64_t moment_bytes;   /* 2 * W * S * 4 (0 when Bm == 0) */
  uint64_t num_moment_chunks;
  uint64_t num_segments;   /* rows of the segment table */
  uint64_t num_tiles;      /* workgroup tiles over all chunks */
  uint64_t device_table_bytes; /* device memory the plan holds (tables, checksum accumulators) */
  uint64_t pinned_bytes;   /* pinned host memory the plan holds (2 * Bm) */
  int32_t device;          /* HIP device of the plan; -1 for a host-only plan */
  int32_t kind;            /* DR_PLAN_ROLLOUT or DR_PLAN_RESHARD */
  uint64_t dst_shard_elems; /* reshard plans: S' = Npad' / W' (rollout_bytes = 4 * Npad') */
  uint64_t tile_elems;     /* elements per workgroup tile on aligned segments (launch geometry) */
  int32_t train_shards;    /* W: shard pointers every staging call reads */
  int32_t tp;              /* T (rollout plans; 0 for reshard plans) */
  int32_t dst_shards;      /* reshard plans: W' destination shard pointers (0 for rollout plans) */
  int32_t reserved;
  uint64_t chunk_bytes;    /* B */
  uint64_t moment_chunk_bytes; /* Bm (0: no moment path) */
  uint64_t deep_tile_elems; /* automatic plans within 128 GiB: tile size (depth 4) of the packs that
                               follow idle time or other work; 0: one tiling for every launch */
  uint64_t deep_num_tiles;  /* tiles of that second tiling (0 without one) */
  int32_t last_tile_depth;  /* tile depth of the latest dr_stage_all / dr_stage_chunk launch on this
                               plan (0 before the first); read when dr_plan_get_info is called */
  int32_t reserved2;
} dr_plan_info;

enum { DR_PLAN_ROLLOUT = 0, DR_PLAN_RESHARD = 1 };

/* One rollout tensor (introspection). */
typedef struct {
  char name[32];        /* "embed", "layers.<l>.qkv", ..., "lm_head" */
  int32_t rank;
  int32_t ndim;         /* 1 (norms) or 2 */
  uint64_t byte_offset; /* offset of its first element in the rollout stream */
  int64_t rows, cols;   /* ndim 1: rows = numel, cols = 1 */
} dr_tensor_desc;

enum { DR_SEG_VEC4 = 1 }; /* segment moves aligned 4-element groups (16-B loads) */
enum {
  DR_OP_CAST_BF16 = 0, /* fp32 source -> bf16 rollout element */
  DR_OP_COPY_F32 = 1,  /* fp32 source -> fp32 destination (reshard) */
  DR_OP_ZERO_F32 = 2,  /* +0.0 padding of the destination (reshard) */
};

/* One row of the segment table (introspection).  The segment writes rows*cols
 * elements densely at element dst_elem of the output stream (the rollout
 * stream, or for a reshard plan the destination flat buffer, whose shard
 * dst_shard holds it); row i reads cols fp32 elements of source shard `shard`
 * starting at element src_elem + i*src_row_stride (op DR_OP_ZERO_F32 reads
 * nothing).  No segment crosses a shard boundary (either side) or a chunk
 * boundary. */
typedef struct {
  uint64_t dst_elem;
  uint64_t src_elem;
  uint32_t shard, chunk;
  uint32_t rows, cols;
  uint32_t src_row_stride;
  uint32_t flags;
  uint32_t dst_shard;
  uint32_t op;
} dr_segment;

/* Builds the segment table for (model, layout) and uploads it to the current
 * HIP device; allocates 2*Bm bytes of pinned host memory when Bm > 0.
 * Cached per topology by the caller (Sec. 3.2 keeps per-topology metadata).
 * out: receives the plan (owned by the caller, freed by dr_plan_destroy).
 * Errors: DR_EINVAL (shape/layout rules above, null pointers, sizes beyond
 * 2^47 elements), DR_ENOMEM, DR_EHIP. */
int dr_plan_create(const dr_model* model, const dr_layout* layout, dr_plan** out);

/* Same table, host only: no HIP call, no device memory.  Usable with the
 * introspection calls (info, tensor, segment); staging calls on it return
 * DR_EINVAL.  For planning on machines without a GPU (the per-topology
 * metadata of Sec. 3.2, prepared ahead of any switch). */
int dr_plan_create_host(const dr_model* model, const dr_layout* layout, dr_plan** out);

/* Frees the plan's device tables and pinned buffers.  The caller must have
 * synchronized every stream that still uses the plan (the plan's own copy
 * streams and a deferred restore are waited for here).  NULL is a no-op. */
void dr_plan_destroy(dr_plan* plan);

/* Sizes and counts of the plan (dr_plan_info), and the tile depth of its
 * latest stage launch.  Errors: DR_EINVAL (null). */
int dr_plan_get_info(const dr_plan* plan, dr_plan_info* out);

/* Rollout tensor `index` (0 .. 3+6L-1, in packing order) of `rank`: the
 * per-rank weights the rollout role loads (Sec. 3.2), located in the stream.
 * Errors: DR_EINVAL (null), DR_ERANGE (rank or index out of range). */
int dr_plan_tensor(const dr_plan* plan, int32_t rank, int32_t index, dr_tensor_desc* out);

/* Segment-table row `index` (0 .. num_segments-1).  Errors: DR_EINVAL, DR_ERANGE. */
int dr_plan_segment(const dr_plan* plan, uint64_t index, dr_segment* out);

/* Pack + cast chunk `chunk` of the rollout stream into dst_chunk and write its
 * checksum to *d_ck (Sec. 3.3: state streamed in bounded chunks).
 *   shards:    host array of W device pointers (16-B aligned), shard w holds
 *              S fp32 elements; read only.
 *   dst_chunk: device buffer of at least chunk_bytes(chunk) bytes, 16-B
 *              aligned; receives exactly the chunk's bytes, nothing beyond.
 *   d_ck:      device pointer to one dr_checksum (16-B aligned); overwritten.
 *   stream:    hipStream_t (NULL: the null stream).  Asynchronous: results
 *              are valid once the stream has reached this point.
 * Two calls in flight at once on one plan must not cover the same chunk
 * (they share that chunk's checksum accumulators in the plan).
 * Graphs: the call only enqueues kernels (no memset, allocation or host
 * synchronization), so it may be recorded into a HIP graph; the recorded
 * launches keep the pointers given here and the plan's device tables, so
 * those must outlive the graph.  An automatic plan's tile depth is chosen when
 * the call is made (see dr_layout), so a recorded call replays with the depth
 * it was recorded with.
 * Errors: DR_EINVAL (host-only plan, null/misaligned pointer), DR_ERANGE
 * (chunk >= num_chunks), DR_EHIP (launch failure). */
int dr_stage_chunk(dr_plan* plan, uint64_t chunk, const float* const* shards, void* dst_chunk,
                   dr_checksum* d_ck, void* stream);

/* dr_stage_chunk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same kernels, but the chunk's checksum accumulators live in a fixed
 * static device array of the library (32 KiB per GPU, kept until the process
 * ends) instead of the plan's.  The call allocates nothing (no hipMalloc, no
 * allocating library call); it launches the stage and chunk-sum kernels.  The
 * first call on a GPU clears the array with a small kernel first, and every
 * call leaves it at zero (the chunk-sum kernel clears the slots it reads);
 * after a call that failed, the following calls clear it first again, up to
 * and including the first one that is not recorded into a graph.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (two streams, two threads) race and must not be issued; calls in order on
 * one stream are safe.
 * The array's device address on a GPU is looked up when a plan is created
 * there, so every call, the first included, may be recorded into a HIP graph;
 * a replay leaves the accumulators at zero for the calls that follow.
 * Arguments, results and errors as dr_stage_chunk, plus DR_EINVAL if the
 * chunk's accumulators would not fit the array (the largest chunk needs
 * 32 KiB, so this does not happen for plans the library builds). */
int dr_stage_chunk_noalloc(dr_plan* plan, uint64_t chunk, const float* const* shards, void* dst_chunk,
                           dr_checksum* d_ck, void* stream);

/* Every chunk at once: dst (rollout_bytes, 16-B aligned) receives the whole
 * rollout stream and d_cks[c] (num_chunks slots, 16-B aligned) the checksum
 * of chunk c.  This is the weight path that sits on the role-switch critical
 * path (Sec. 3.3).  Asynchronous on `stream` and recordable into a HIP graph,
 * as dr_stage_chunk.
 * Errors: DR_EINVAL, DR_EHIP. */
int dr_stage_all(dr_plan* plan, const float* const* shards, void* dst, dr_checksum* d_cks, void* stream);

/* The paper's weight path (Sec. 3.3: states go from the old rank to the new
 * one through host memory in bounded chunks, store and reload pipelined chunk
 * by chunk).  The stage kernel packs chunk c straight into one of two
 * plan-owned pinned host buffers of B bytes (its stores cross PCIe), and a
 * plan-owned copy stream reloads that buffer into dst + c*B, so the store of
 * one chunk and the reload of the previous one use both link directions at
 * once.  Transient memory: 2*B pinned, no device staging, allocated on the
 * first call and held by the plan.  Results (dst bytes, d_cks) are identical
 * to dr_stage_all.
 *   shards, dst, d_cks: as dr_stage_all.  dst may be any device buffer the
 *   current device can copy into.
 *   stream: hipStream_t running the kernels; it also waits for the last copy,
 *   so results are valid once the stream has reached this point.  Does not
 *   block the calling thread.  Calls on one plan are ordered by the plan's
 *   events; the plan must outlive the enqueued work (dr_plan_destroy
 *   synchronizes the copy streams).
 * Errors: DR_EINVAL (as dr_stage_all), DR_ENOMEM, DR_EHIP. */
int dr_stage_through_host(dr_plan* plan, const float* const* shards, void* dst, dr_checksum* d_cks, void* stream);

/* Training -> training move to a new shard count (Sec. 3.3: weights and
 * optimizer states go from the old training ranks to the new ones).  The same
 * N fp32 elements, bit for bit, are re-cut from W = from_shards shards into
 * W' = to_shards shards of S' = Npad'/W' elements, where the destination is
 * re-padded with +0.0 up to Npad' = a multiple of W'*256.  The output stream
 * is the destination flat buffer (4*Npad' bytes, reported as rollout_bytes),
 * cut into chunks of chunk_bytes with the same checksum as the rollout path.
 * The _host variant builds the table without touching the GPU.
 * Errors: DR_EINVAL (model rules as dr_plan_create, shard counts outside
 * [1, 64], chunk_bytes not a positive multiple of 16), DR_ENOMEM, DR_EHIP. */
int dr_reshard_plan_create(const dr_model* model, int32_t from_shards, int32_t to_shards, uint64_t chunk_bytes,
                           dr_plan** out);
int dr_reshard_plan_create_host(const dr_model* model, int32_t from_shards, int32_t to_shards,
                                uint64_t chunk_bytes, dr_plan** out);

/* Runs a reshard plan (Sec. 3.3: the training state moves from the old
 * training ranks to the new ones): src_shards (host array of W device
 * pointers, S fp32 each, 16-B aligned) -> dst_shards (host array of W' device
 * pointers, S' fp32 each, 16-B aligned), every byte of the destination written (padding
 * zeroed); d_cks (num_chunks slots, 16-B aligned) receives the chunk
 * checksums.  Asynchronous on `stream` and recordable into a HIP graph, as
 * dr_stage_all.
 * Errors: DR_EINVAL (not a reshard plan, null/misaligned pointers), DR_EHIP. */
int dr_reshard(dr_plan* plan, const float* const* src_shards, float* const* dst_shards, dr_checksum* d_cks,
               void* stream);

/* The reshard through host memory, as the paper moves training state from the
 * old ranks to the new ones (Sec. 3.3): the reshard kernel packs destination
 * chunk c straight into one of the plan's two pinned B-byte host buffers, and
 * the plan's copy stream reloads it into the destination shards (cut at shard
 * boundaries), store and reload pipelined chunk by chunk as in
 * dr_stage_through_host.  Transient memory: 2*B pinned, no device staging.
 * Results (every destination byte, d_cks) are identical to dr_reshard.
 *   Arguments, stream semantics, ordering and the one-call-at-a-time rule: as
 *   dr_reshard and dr_stage_through_host.
 * Errors: DR_EINVAL (as dr_reshard), DR_ENOMEM, DR_EHIP. */
int dr_reshard_through_host(dr_plan* plan, const float* const* src_shards, float* const* dst_shards,
                            dr_checksum* d_cks, void* stream);

/* Offload the Adam moments to host memory through the plan's two pinned
 * bounce buffers of Bm bytes (Sec. 3.3: bounded host buffers, store pipelined
 * chunk by chunk): device->pinned copies run on side_stream while host
 * threads drain the other buffer into host_store.
 *   m_shards, v_shards: host arrays of W device pointers (S fp32 each).
 *   host_store: moment_bytes of host memory (any kind); receives the moment
 *               stream.  Owned by the caller.
 *   side_stream: hipStream_t used for the copies, so they start after the work
 *               queued on it; pass a stream other than the one running
 *               dr_stage_all so both overlap.  Work the caller queued on other
 *               streams is not waited for: order the moments' producers before
 *               this call.  The call may run on its own host thread while
 *               another thread stages with the same plan.  The first copies
 *               ever issued on a stream set up its copy path, and a pack
 *               running at that moment was measured 0.8 ms slower (8B): a
 *               job that overlaps the two can warm the side stream once
 *               beforehand (e.g. one chunk through dr_offload_moments_range).
 * Blocks the calling thread until every byte is in host_store.
 * Errors: DR_EINVAL (Bm == 0, host-only plan, null pointers), DR_EHIP. */
int dr_offload_moments(dr_plan* plan, const float* const* m_shards, const float* const* v_shards,
                       void* host_store, void* side_stream);

/* Resumable offload (the bounded chunks of Sec. 3.3, a range at a time):
 * moves only moment chunks [first_chunk, first_chunk + num_chunks) through
 * the same bounded pipeline, into their places in the
 * whole host_store (chunk k at byte k*Bm).  An offload interrupted after chunk
 * k restarts here at k; chunks are independent, so pieces in any order give
 * the same store as one dr_offload_moments.  num_chunks == 0 does nothing.
 * Errors: as dr_offload_moments, and DR_ERANGE when the range passes
 * num_moment_chunks. */
int dr_offload_moments_range(dr_plan* plan, const float* const* m_shards, const float* const* v_shards,
                             void* host_store, uint64_t first_chunk, uint64_t num_chunks, void* side_stream);

/* The deferred reload (Sec. 3.3, last paragraph): host_store -> pinned bounce
 * -> device shards, bit-exact, pipelined chunk by chunk on side_stream.
 * Blocks the calling thread until every byte has landed on the device.
 * Errors: as dr_offload_moments. */
int dr_restore_moments(dr_plan* plan, const void* host_store, float* const* m_shards, float* const* v_shards,
                       void* side_stream);

/* Resumable restore (the deferred reload of Sec. 3.3, a range at a time):
 * moment chunks [first_chunk, first_chunk + num_chunks) only, from their
 * places in host_store back into the shards, as
 * dr_restore_moments.  Errors: as dr_restore_moments, and DR_ERANGE when the
 * range passes num_moment_chunks. */
int dr_restore_moments_range(dr_plan* plan, const void* host_store, float* const* m_shards, float* const* v_shards,
                             uint64_t first_chunk, uint64_t num_chunks, void* side_stream);

/* The deferred reload without blocking the caller (Sec. 3.3: optimizer states
 * are needed only at the end of the first training step after the resize, so their
 * reload can run while that step computes).  _begin checks its arguments as
 * dr_restore_moments does, copies the shard pointer arrays and starts the
 * restore on a plan-owned host thread, then returns: the caller's thread is
 * free to launch the step's work on its own streams.  _end blocks until every
 * byte has landed on the device and returns the restore's status (its
 * message in dr_last_error()).  While a restore is in flight the plan's
 * moment calls return DR_EINVAL; dr_plan_destroy waits for it to finish.
 * The host store must stay valid until _end returns.
 * Errors (_begin): as dr_restore_moments, DR_EINVAL if one is in flight,
 * DR_ENOMEM if the thread cannot start; (_end): DR_EINVAL if none is in
 * flight, else the restore's own code. */
int dr_restore_moments_begin(dr_plan* plan, const void* host_store, float* const* m_shards, float* const* v_shards,
                             void* side_stream);
int dr_restore_moments_end(dr_plan* plan);

/* Checksums of the moment chunks (the bounded chunks of Sec. 3.3 that the
 * offload and the restore move): d_cks[k] receives the checksum of bytes
 * [k*Bm, min((k+1)*Bm, moment_bytes)) of the moment stream
 * m_0 || ... || m_{W-1} || v_0 || ... || v_{W-1}, with the same function as
 * the rollout chunks (little-endian u32 words w_j of the chunk: s1 = sum w_j,
 * s2 = sum (j+1)*w_j, mod 2^64), read from the device shards.  Taken before
 * an offload and again after the restore, equal checksums mean every chunk
 * came back; they can also be compared with a checksum of the host store.
 *   m_shards, v_shards: host arrays of W device pointers (16-B aligned), S
 *   fp32 each (padding included); read only.
 *   d_cks: device array of num_moment_chunks dr_checksum (16-B aligned).
 *   stream: hipStream_t; asynchronous, results valid once the stream has
 *   reached this point.  Reads 4 bytes per moment element from HBM.  Two
 *   calls in flight at once on one plan share its moment accumulators: issue
 *   them in order (one stream).
 * Errors: DR_EINVAL (no moment path, host-only plan, null or misaligned
 * pointer, wrong device), DR_EHIP. */
int dr_moment_checksums(dr_plan* plan, const float* const* m_shards, const float* const* v_shards,
                        dr_checksum* d_cks, void* stream);

/* Hysteresis-guided reconfiguration (Sec. 3.4): the decision of when to move
 * between pre-specified Train:Rollout configurations (indices 0 .. K-1, GPU
 * splits train_gpus[i] : rollout_gpus[i], from the most training GPUs to the
 * most rollout GPUs; one position per resize).
 * Fed one (rollout time, training time) pair per step, it resizes only on
 * sustained directional imbalance:
 *   r = (t_rollout - t_train) / max(t_rollout, t_train)   (0 if both are 0)
 *   signal: off -> +1 when r > enter, -1 when r < -enter; +1 holds while
 *     r > exit (turns to -1 when r < -enter, else off); -1 symmetric
 *   run: consecutive steps with the same nonzero signal
 *   each step first advances the steps spent in the configuration and counts
 *   down a pending cooldown (a resize at step k blocks steps k+1..k+cooldown)
 *   resize in the signal's direction when, checked in this order: signal != 0
 *   (else DR_HYST_BALANCED), run >= consecutive (PERSISTENCE), no cooldown
 *   (COOLDOWN), steps in configuration >= dwell (DWELL), the next
 *   configuration exists (EDGE), and the resize pays off (AMORTIZE; Sec. 3.4
 *   asks that a resize raise throughput, and Exp#3 that it amortize its
 *   cost): over the last `consecutive` steps the stages' work
 *   is mean(t_rollout) * rollout_gpus[cur] and mean(t_train) * train_gpus[cur],
 *   the target's step time is max(work_r / rollout_gpus[tgt], work_t /
 *   train_gpus[tgt]), gain = mean(max(t_rollout, t_train)) - that, and the
 *   resize needs gain > 0 and (switch_cost_s == 0 or gain * horizon_steps >=
 *   switch_cost_s)
 *   after a resize the signal, the run and the dwell count restart.
 * The split arrays are copied at creation.
 * Errors: DR_EINVAL (num_configs < 1, null split arrays, a role with no GPU,
 * splits not ordered, initial out of range, not 0 <= exit <= enter < 1,
 * consecutive outside [1, 2^20], negative dwell/cooldown/cost,
 * horizon_steps < 1 with a positive cost; step: negative or non-finite
 * times), DR_ENOMEM. */
typedef struct dr_hyst dr_hyst;
typedef struct {
  int32_t num_configs, initial;
  const int32_t* train_gpus;   /* [num_configs] */
  const int32_t* rollout_gpus; /* [num_configs] */
  double enter, exit;
  int32_t consecutive, dwell, cooldown;
  int32_t horizon_steps;
  double switch_cost_s;
} dr_hyst_params;
enum {
  DR_HYST_BALANCED = 0,
  DR_HYST_PERSISTENCE = 1,
  DR_HYST_COOLDOWN = 2,
  DR_HYST_DWELL = 3,
  DR_HYST_EDGE = 4,
  DR_HYST_AMORTIZE = 5,
  DR_HYST_RESIZE = 6,
};
typedef struct {
  int32_t config; /* configuration after this step */
  int32_t action; /* -1 toward training, 0 none, +1 toward rollout */
  int32_t reason; /* DR_HYST_* */
  int32_t run;
  double imbalance;
  double predicted_gain_s; /* step time saved per step by the move (0 if not evaluated) */
} dr_hyst_decision;
int dr_hyst_create(const dr_hyst_params* params, dr_hyst** out);
int dr_hyst_step(dr_hyst* h, double t_rollout, double t_train, dr_hyst_decision* out);
void dr_hyst_destroy(dr_hyst* h);
/* Steps after which the per-step saving (step_before - step_after) has covered
 * one resize of blocking cost switch_cost_s (Exp#3's amortization).  Plain
 * IEEE division: +Inf when the resize saves nothing, negative when it costs. */
double dr_break_even_steps(double switch_cost_s, double step_before_s, double step_after_s);

/* Message of the last failing call on this thread ("" if none). */
const char* dr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DR_H */
