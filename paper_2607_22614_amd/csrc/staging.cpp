// Host side of the stage path: argument checks, the per-launch tile depth of
// automatic plans, the device tables of a plan, and the dr_stage_chunk /
// dr_stage_all entry points (kernels in stage.hip).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>

#include "dr_internal.h"
#include "kernels.h"

namespace dr {
namespace {

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_shards(const dr_plan* p, const float* const* shards, const char* what) {
  if (!shards) return fail(DR_EINVAL, "%s: null shard array", what);
  for (int w = 0; w < p->layout.train_shards; ++w)
    if (!aligned16(shards[w])) return fail(DR_EINVAL, "%s: shard %d pointer is null or not 16-byte aligned", what, w);
  return DR_OK;
}

int check_device(const dr_plan* p, const char* what) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: hipGetDevice: %s", what, hipGetErrorString(e));
  if (dev != p->device) return fail(DR_EINVAL, "%s: plan lives on device %d, current device is %d", what, p->device, dev);
  return DR_OK;
}

// Per-device state of the automatic tile depth (see pack_drain_ns in the
// internal header): when the packs launched so far should have drained.
std::atomic<int64_t> g_packs_drain_ns[kClockDevices];

int64_t host_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

// Index of the tiling of a one-chunk launch (dr_stage_chunk, the host relay): the deep one when the
// plan has it.  Measured on the 8B workload, 60 one-chunk launches of 256 MiB take 7.86 ms back to
// back and 8.14 ms after idle time at depth 4, against 7.88 / 8.56 ms at depth 2.
int chunk_tiling(const dr_plan* p) { return p->tiling[1].depth ? 1 : 0; }

// Index of the tiling that a whole-stream launch (dr_stage_all) starting now uses.
int pick_tiling(const dr_plan* p) {
  if (!p->tiling[1].depth || p->device < 0 || p->device >= kClockDevices) return 0;
  return pack_is_hot(host_ns(), g_packs_drain_ns[p->device].load(std::memory_order_relaxed)) ? 0 : 1;
}

// Advances the device's drain estimate past a pack of `bytes` algorithmic bytes whose launch has
// just returned (a slow launch, e.g. the first on a new stream, delays the pack's start, so the
// estimate starts no earlier than the return).  The estimate only picks between two bit-identical
// kernels, so a race between threads costs nothing else.
void note_pack(const dr_plan* p, uint64_t bytes) {
  if (p->device < 0 || p->device >= kClockDevices) return;
  std::atomic<int64_t>& drain = g_packs_drain_ns[p->device];
  drain.store(pack_drain_ns(host_ns(), drain.load(std::memory_order_relaxed), bytes), std::memory_order_relaxed);
}

// Tiles [tile0, tile0 + ntiles) of tiling tl, which cover chunks [chunk0, chunk0 + nchunks), then
// their checksums from the accumulators of cs.
int launch(dr_plan* p, const Tiling& tl, uint32_t tile0, uint32_t ntiles, const float* const* shards, void* dst,
           uint64_t dst_bias, uint32_t chunk0, uint32_t nchunks, const ChunkSum& cs, hipStream_t st,
           const char* what) {
  StageLaunch l{};
  l.segs = p->d_segs;
  l.tiles = tl.d_tiles;
  l.sum = cs;
  l.dst = dst;
  l.dst_bias = dst_bias;
  l.chunk_elems = p->layout.chunk_bytes / 2;
  l.tile0 = tile0;
  l.ntiles = ntiles;
  l.depth = tl.depth;
  l.num_shards = p->layout.train_shards;
  l.shards = shards;
  hipError_t e = launch_stage_kernel(l, st);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: stage kernel launch: %s", what, hipGetErrorString(e));
  p->last_depth.store(tl.depth, std::memory_order_relaxed);
  e = launch_chunk_sums(l.sum, chunk0, nchunks, st);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: chunk sum launch: %s", what, hipGetErrorString(e));
  return DR_OK;
}

// Chunk `chunk` with tiling tl into dst_chunk, its checksum into *ck.
int launch_one_chunk(dr_plan* p, const Tiling& tl, uint64_t chunk, const float* const* shards, void* dst_chunk,
                     dr_checksum* ck, hipStream_t st, const char* what) {
  return launch_chunk_into(p, tl, chunk, shards, dst_chunk, chunk_sum(p, tl, ck, (uint32_t)chunk), st, what);
}

uint64_t chunk_out_bytes(const dr_plan* p, uint64_t chunk) {
  return chunk + 1 < p->info.num_chunks ? p->layout.chunk_bytes : p->info.last_chunk_bytes;
}

int alloc(void** dptr, size_t bytes, const char* what) {
  bytes = std::max<size_t>(bytes, 16);
  hipError_t e = hipMalloc(dptr, bytes);
  if (e != hipSuccess) {
    *dptr = nullptr;
    return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "hipMalloc(%s, %zu B): %s", what, bytes,
                hipGetErrorString(e));
  }
  return DR_OK;
}

template <typename T>
int upload(T** dptr, const std::vector<T>& host, const char* what) {
  if (int rc = alloc(reinterpret_cast<void**>(dptr), host.size() * sizeof(T), what)) return rc;
  if (!host.empty()) {
    const hipError_t e = hipMemcpy(*dptr, host.data(), host.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(DR_EHIP, "hipMemcpy(%s): %s", what, hipGetErrorString(e));
  }
  return DR_OK;
}

}  // namespace

ChunkSum chunk_sum(const dr_plan* p, const Tiling& tl, dr_checksum* out, uint32_t out_chunk0) {
  ChunkSum cs{};
  cs.acc = p->d_acc + tl.acc0;
  cs.out = out;
  cs.sub = tl.sum_slots;
  cs.stride_words = tl.sum_stride;
  cs.out_chunk0 = out_chunk0;
  cs.chunk_bias = 0;
  return cs;
}

int check_stage_args(const dr_plan* p, const float* const* shards, const void* dst, const void* cks,
                     const char* what) {
  if (int rc = check_shards(p, shards, what)) return rc;
  if (!aligned16(dst)) return fail(DR_EINVAL, "%s: destination is null or not 16-byte aligned", what);
  if (!aligned16(cks)) return fail(DR_EINVAL, "%s: checksum slots are null or not 16-byte aligned", what);
  if (!p->d_segs) return fail(DR_EINVAL, "%s: host-only plan has no device tables", what);
  return check_device(p, what);
}

int launch_chunk_into(dr_plan* p, const Tiling& tl, uint64_t chunk, const float* const* shards, void* dst_chunk,
                      const ChunkSum& cs, hipStream_t st, const char* what) {
  const uint32_t t0 = tl.chunk_tile_begin[chunk], t1 = tl.chunk_tile_begin[chunk + 1];
  return launch(p, tl, t0, t1 - t0, shards, dst_chunk, chunk * (p->layout.chunk_bytes / 2), (uint32_t)chunk, 1, cs,
                st, what);
}

const Tiling& chunk_launch_tiling(const dr_plan* p) { return p->tiling[chunk_tiling(p)]; }

int launch_chunk(dr_plan* p, uint64_t chunk, const float* const* shards, void* dst_chunk, dr_checksum* ck,
                 void* st) {
  return launch_one_chunk(p, p->tiling[chunk_tiling(p)], chunk, shards, dst_chunk, ck,
                          static_cast<hipStream_t>(st), "chunk launch");
}

int upload_plan(dr_plan* p) {
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) return fail(DR_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  int rc;
  if ((rc = upload(&p->d_segs, p->segs, "segments"))) return rc;
  // per tiling: tiles, chunk index and the checksum accumulators, which start at zero (and every
  // launch leaves them at zero: ChunkSum)
  if (!p->moment_segs.empty() && (rc = upload(&p->d_moment_segs, p->moment_segs, "moment segments"))) return rc;
  uint64_t words = 0;
  for_each_tiling(p, [&](Tiling& tl) {
    if (rc) return;
    if ((rc = upload(&tl.d_tiles, tl.tiles, "tiles"))) return;
    if ((rc = upload(&tl.d_chunk_tile_begin, tl.chunk_tile_begin, "chunk tiles"))) return;
    tl.acc0 = words;
    words += (uint64_t)(tl.chunk_tile_begin.size() - 1) * tl.sum_slots * tl.sum_stride;
  });
  if (rc) return rc;
  if ((rc = alloc(reinterpret_cast<void**>(&p->d_acc), words * 8, "checksum accumulators"))) return rc;
  e = hipMemset(p->d_acc, 0, words * 8);
  if (e != hipSuccess) return fail(DR_EHIP, "hipMemset(checksum accumulators): %s", hipGetErrorString(e));
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return fail(DR_EHIP, "hipDeviceSynchronize: %s", hipGetErrorString(e));
  // the static scratch of dr_stage_chunk_noalloc on this device, looked up here rather than in a call
  uint64_t* scratch = nullptr;
  if ((rc = scratch_on(p->device, &scratch))) return rc;
  p->info.device = p->device;
  return DR_OK;
}

void free_device(dr_plan* p) {
  if (p->d_segs) (void)hipFree(p->d_segs);
  if (p->d_acc) (void)hipFree(p->d_acc);
  if (p->d_moment_segs) (void)hipFree(p->d_moment_segs);
  p->d_segs = nullptr;
  p->d_acc = nullptr;
  p->d_moment_segs = nullptr;
  for_each_tiling(p, [](Tiling& tl) {
    if (tl.d_tiles) (void)hipFree(tl.d_tiles);
    if (tl.d_chunk_tile_begin) (void)hipFree(tl.d_chunk_tile_begin);
    tl.d_tiles = nullptr;
    tl.d_chunk_tile_begin = nullptr;
  });
}

}  // namespace dr

using namespace dr;

extern "C" int dr_stage_chunk(dr_plan* p, uint64_t chunk, const float* const* shards, void* dst_chunk,
                              dr_checksum* d_ck, void* stream) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_stage_chunk: null plan");
  if (p->kind != kRollout) return fail(DR_EINVAL, "dr_stage_chunk: not a rollout plan");
  if (chunk >= p->info.num_chunks)
    return fail(DR_ERANGE, "dr_stage_chunk: chunk %llu >= num_chunks %llu", (unsigned long long)chunk,
                (unsigned long long)p->info.num_chunks);
  if (int rc = check_shards(p, shards, "dr_stage_chunk")) return rc;
  if (!aligned16(dst_chunk)) return fail(DR_EINVAL, "dr_stage_chunk: dst_chunk is null or not 16-byte aligned");
  if (!aligned16(d_ck)) return fail(DR_EINVAL, "dr_stage_chunk: d_ck is null or not 16-byte aligned");
  if (!p->d_segs) return fail(DR_EINVAL, "dr_stage_chunk: host-only plan has no device tables");
  if (int rc = check_device(p, "dr_stage_chunk")) return rc;
  const Tiling& tl = p->tiling[chunk_tiling(p)];
  const int rc =
      launch_one_chunk(p, tl, chunk, shards, dst_chunk, d_ck, static_cast<hipStream_t>(stream), "dr_stage_chunk");
  if (rc == DR_OK) note_pack(p, 3 * chunk_out_bytes(p, chunk));
  return rc;
}

extern "C" int dr_stage_all(dr_plan* p, const float* const* shards, void* dst, dr_checksum* d_cks, void* stream) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_stage_all: null plan");
  if (p->kind != kRollout) return fail(DR_EINVAL, "dr_stage_all: not a rollout plan");
  if (int rc = check_shards(p, shards, "dr_stage_all")) return rc;
  if (!aligned16(dst)) return fail(DR_EINVAL, "dr_stage_all: dst is null or not 16-byte aligned");
  if (!aligned16(d_cks)) return fail(DR_EINVAL, "dr_stage_all: d_cks is null or not 16-byte aligned");
  if (!p->d_segs) return fail(DR_EINVAL, "dr_stage_all: host-only plan has no device tables");
  if (int rc = check_device(p, "dr_stage_all")) return rc;
  const Tiling& tl = p->tiling[pick_tiling(p)];
  const int rc = launch(p, tl, 0, (uint32_t)tl.tiles.size(), shards, dst, 0, 0, (uint32_t)p->info.num_chunks,
                        chunk_sum(p, tl, d_cks, 0), static_cast<hipStream_t>(stream), "dr_stage_all");
  if (rc == DR_OK) note_pack(p, 4 * p->info.n_elems + p->info.rollout_bytes);
  return rc;
}
