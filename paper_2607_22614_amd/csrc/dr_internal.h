// Internal declarations of the host library: plan, planner, launches and scheduler.
#pragma once

#include <atomic>
#include <cstdint>
#include <memory>
#include <thread>
#include <string>
#include <vector>

#include "dev_types.h"
#include "dr.h"

namespace dr {

// Host-side limits; the launch geometry and the device records are in dev_types.h.
constexpr uint64_t kLargeFootprint = 128ull << 30;  // automatic plans beyond it: depth 4 only
// Plans hold fewer than kMaxTiles tiles, so a grid-stride tile index (32-bit)
// never wraps: b < kMaxTiles and b + kMaxGrid < 2^32.
constexpr uint64_t kMaxTiles = (1ull << 32) - (1ull << 24);
static_assert(kMaxTiles + kMaxGrid < (1ull << 32), "grid-stride tile index");

// Automatic tile depth of whole-stream launches (dr_stage_all), chosen per
// launch on the host; one-chunk launches always take depth 4 (staging.cpp).
// Measured on the 8B workload: depth 2 wins only for a pack that follows
// another pack without a pause (7.28 against 7.50 ms); after 0.2 s idle depth 4
// takes 7.49 against 7.99 ms, right behind bf16 GEMMs 7.54 against 7.63 ms,
// and 10 ms after a pack 7.50 against 7.71 ms.  Per device the library keeps
// the time at which the packs it launched should have drained: each starts
// when its launch call returns or at the previous drain time, whichever is
// later, and lasts its algorithmic bytes at kPackBytesPerNs.  A launch no later
// than kHotGapNs after that time is "hot" and takes depth 2; any other launch
// of an automatic plan takes depth 4.
constexpr double kPackBytesPerNs = 6500.0;  // 6.5 TB/s
constexpr int64_t kHotGapNs = 2000000;      // 2 ms
constexpr int kClockDevices = 64;

// Drain time after a launch of `bytes` at host time now, given the previous drain time (0: none).
inline int64_t pack_drain_ns(int64_t now, int64_t prev, uint64_t bytes) {
  return (prev > now ? prev : now) + (int64_t)((double)bytes / kPackBytesPerNs);
}

// Whether a launch at host time now follows the device's packs closely enough for depth 2.
inline bool pack_is_hot(int64_t now, int64_t prev_drain) {
  return prev_drain != 0 && now - prev_drain <= kHotGapNs;
}

// Checksum accumulator slots of a tiling whose largest chunk holds max_chunk_tiles tiles (ChunkSum).
// Adds to one cache line are performed one after another, and all tiles of a small chunk run at
// once, so the slots keep to about kTilesPerSumLine tiles' adds per 128-byte line: one slot per
// chunk up to that many tiles, then a power of two of slots (at most kMaxSumSlots), one line each.
// Chunks of at most kPackedSlotTiles tiles pack their single slots 16 bytes apart, 8 chunks to a
// line (at most 64 tiles' adds per line), which keeps a million tiny chunks' accumulators small.
// Measured on the 8B workload at tile depth 2: 256 KiB chunks (64 tiles) with packed single slots,
// 1024 adds per line in a burst, took the stage kernel from 7.3 to 10.6 ms (7.5 ms with two slots
// a line each); 16 KiB chunks (4-5 tiles) took 8.1 ms with a line per chunk against 7.7 packed.
constexpr uint32_t kTilesPerSumLine = 32;
constexpr uint32_t kPackedSlotTiles = 8;
inline uint32_t sum_slots(uint32_t max_chunk_tiles) {
  uint32_t s = 1;
  while (s < kMaxSumSlots && (uint64_t)s * kTilesPerSumLine < max_chunk_tiles) s *= 2;
  return s;
}
inline uint32_t sum_stride(uint32_t slots, uint32_t max_chunk_tiles) {
  return slots > 1 || max_chunk_tiles > kPackedSlotTiles ? kSlotLineWords : 2;
}

enum PlanKind : int { kRollout = 0, kReshard = 1 };

// One tiling of a plan's segments at tile depth K: the tiles in segment order
// and the chunk -> first-tile index, on the host and on the device.
struct Tiling {
  int depth = 0;                           // K; 0: the plan has no such tiling
  uint32_t max_chunk_tiles = 0;            // the most tiles of any chunk
  uint32_t sum_slots = 1;                  // checksum accumulator slots per chunk (ChunkSum)
  uint32_t sum_stride = 2;                 // 64-bit words between consecutive slots
  uint64_t acc0 = 0;                       // first accumulator word of this tiling in the plan
  std::vector<Tile> tiles;
  std::vector<uint32_t> chunk_tile_begin;  // num_chunks + 1 entries
  Tile* d_tiles = nullptr;
  uint32_t* d_chunk_tile_begin = nullptr;
};

struct TensorDesc {
  std::string name;
  int rank;
  int ndim;
  uint64_t elem_offset;
  int64_t rows, cols;
};

struct HostPool;  // drain/fill threads of the moment path (moments.cpp)

}  // namespace dr

struct dr_plan {
  dr_model model{};
  dr_layout layout{};
  dr_plan_info info{};
  int kind = dr::kRollout;
  int dst_shards = 1;  // reshard plans: W'
  uint64_t dst_shard_elems = 0;

  std::vector<dr::DevSeg> segs;
  // [0]: the plan's tiling (info.tile_elems); [1]: an automatic plan's deep
  // tiling (K = 4, info.deep_tile_elems) for packs after idle time or other work
  dr::Tiling tiling[2];
  // the moment stream m_0..m_{W-1} v_0..v_{W-1} cut at piece and Bm-chunk boundaries (plans with a
  // moment path): segment `shard` is the piece (0..2W-1), `chunk` the moment chunk
  std::vector<dr::DevSeg> moment_segs;
  dr::Tiling moment_tiling;
  dr::DevSeg* d_moment_segs = nullptr;
  std::vector<dr::TensorDesc> tensors;  // T * (3 + 6L), rank-major
  std::atomic<int> last_depth{0};       // K of the latest stage launch (info.last_tile_depth)

  // device side (null for a host-only plan)
  int device = -1;
  dr::DevSeg* d_segs = nullptr;
  // checksum accumulators (ChunkSum) of every tiling, each from its acc0; zero between launches
  uint64_t* d_acc = nullptr;

  // moment path
  void* bounce[2] = {nullptr, nullptr};  // pinned, Bm bytes each
  void* events[2] = {nullptr, nullptr};  // hipEvent_t
  dr::HostPool* pool = nullptr;  // owned; freed by free_moment_resources
  // deferred restore running on a background thread (dr_restore_moments_begin/_end)
  std::thread restore_thread;
  std::atomic<bool> restore_in_flight{false};
  // set while an offload or a restore (blocking or deferred) uses the bounce buffers
  std::atomic<bool> moments_busy{false};
  // set while a dr_stage_through_host or dr_reshard_through_host call enqueues its work
  // (one call at a time per plan)
  std::atomic<bool> relay_busy{false};
  int restore_rc = 0;
  char restore_error[512] = "";
  std::vector<float*> restore_m, restore_v;

  // path through host memory (created on the first dr_stage_through_host or
  // dr_reshard_through_host)
  void* relay_pin[2] = {nullptr, nullptr};  // pinned, mapped, B bytes each
  void* relay_stream = nullptr;             // hipStream_t of the host->device reloads
  void* relay_ev[5] = {};                   // hipEvent_t: packed[2], reloaded[2], call start

  ~dr_plan();
};

namespace dr {

// Error reporting: stores the message for dr_last_error() and returns code.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Every tiling of a plan: the rollout or reshard tilings, then the moment stream's.
template <typename Fn>
void for_each_tiling(dr_plan* p, Fn fn) {
  for (Tiling& tl : p->tiling)
    if (tl.depth) fn(tl);
  if (p->moment_tiling.depth) fn(p->moment_tiling);
}

// Planner (plan.cpp): validates and fills segs/tiles/tensors/info of p.
int build_plan(const dr_model* model, const dr_layout* layout, dr_plan* p);
int build_reshard_plan(const dr_model* model, int32_t from_shards, int32_t to_shards, uint64_t chunk_bytes,
                       dr_plan* p);

// Device tables of the plan (staging.cpp).
int upload_plan(dr_plan* p);
// The current device's address of the allocation-free entry point's static scratch (noalloc.hip).
int scratch_on(int dev, uint64_t** out);
void free_device(dr_plan* p);

// Moment path resources (moments.cpp).
int create_moment_resources(dr_plan* p);
void free_moment_resources(dr_plan* p);

// One chunk through the stage and reduce kernels on stream st (staging.cpp):
// dst_chunk receives the chunk's bytes, *ck its checksum.  Arguments checked by the caller.
int launch_chunk(dr_plan* p, uint64_t chunk, const float* const* shards, void* dst_chunk, dr_checksum* ck,
                 void* st);
// Chunk `chunk` with tiling tl into dst_chunk, its checksum from the accumulators of cs; and the
// tiling one-chunk launches use.  Arguments checked by the caller.
int launch_chunk_into(dr_plan* p, const Tiling& tl, uint64_t chunk, const float* const* shards, void* dst_chunk,
                      const ChunkSum& cs, struct ihipStream_t* st, const char* what);
const Tiling& chunk_launch_tiling(const dr_plan* p);

// The checksum accumulators of tiling tl, with chunk c's checksum going to out[c - out_chunk0].
ChunkSum chunk_sum(const dr_plan* p, const Tiling& tl, dr_checksum* out, uint32_t out_chunk0);
int check_stage_args(const dr_plan* p, const float* const* shards, const void* dst, const void* cks,
                     const char* what);

// Reshard plans (reshard.cpp): the argument checks of every reshard entry point, and chunk
// `chunk` of the destination stream into chunk_dst with its checksum in *ck (arguments checked).
int check_reshard_args(const dr_plan* p, const float* const* src_shards, float* const* dst_shards,
                       const dr_checksum* d_cks, const char* what);
int launch_reshard_chunk(dr_plan* p, uint64_t chunk, const float* const* src, void* chunk_dst, dr_checksum* ck,
                         struct ihipStream_t* st, const char* what);

// Paths through host memory (relay.cpp).
void free_relay_resources(dr_plan* p);

}  // namespace dr
