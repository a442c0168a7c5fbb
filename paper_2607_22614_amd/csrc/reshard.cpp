// Host side of the training -> training reshard: argument checks, launches and
// the dr_reshard entry point (kernel in reshard.hip).
#include <hip/hip_runtime.h>

#include "dr_internal.h"
#include "kernels.h"

namespace dr {
namespace {

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

int check_reshard_args(const dr_plan* p, const float* const* src_shards, float* const* dst_shards,
                       const dr_checksum* d_cks, const char* what) {
  if (!p) return fail(DR_EINVAL, "%s: null plan", what);
  if (p->kind != kReshard) return fail(DR_EINVAL, "%s: not a reshard plan", what);
  if (!src_shards || !dst_shards) return fail(DR_EINVAL, "%s: null shard array", what);
  for (int w = 0; w < p->layout.train_shards; ++w)
    if (!aligned16(src_shards[w])) return fail(DR_EINVAL, "%s: source shard %d is null or not 16-byte aligned", what, w);
  for (int w = 0; w < p->dst_shards; ++w)
    if (!aligned16(dst_shards[w]))
      return fail(DR_EINVAL, "%s: destination shard %d is null or not 16-byte aligned", what, w);
  if (!aligned16(d_cks)) return fail(DR_EINVAL, "%s: d_cks is null or not 16-byte aligned", what);
  if (!p->d_segs) return fail(DR_EINVAL, "%s: host-only plan has no device tables", what);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: hipGetDevice: %s", what, hipGetErrorString(e));
  if (dev != p->device) return fail(DR_EINVAL, "%s: plan lives on device %d, current device is %d", what, p->device, dev);
  return DR_OK;
}

namespace {

// Tiles [tile0, tile0 + ntiles) of a reshard plan; flat (if not null) receives the destination
// elements from flat_bias on instead of the destination shards.  The tiles cover chunks
// [chunk0, chunk0 + nchunks); the checksum of chunk c goes to cks[c - chunk0].
int launch_reshard(dr_plan* p, uint32_t tile0, uint32_t ntiles, const float* const* src, float* const* dst,
                   float* flat, uint64_t flat_bias, uint32_t chunk0, uint32_t nchunks, dr_checksum* cks,
                   hipStream_t st, const char* what) {
  ReshardLaunch l{};
  l.segs = p->d_segs;
  l.tiles = p->tiling[0].d_tiles;
  l.sum = chunk_sum(p, p->tiling[0], cks, chunk0);
  l.chunk_elems = p->layout.chunk_bytes / 4;
  l.dst_shard_elems = p->dst_shard_elems;
  l.tile0 = tile0;
  l.ntiles = ntiles;
  l.flat = flat;
  l.flat_bias = flat_bias;
  l.num_src = p->layout.train_shards;
  l.src = src;
  l.num_dst = p->dst_shards;
  l.dst = dst;
  hipError_t e = launch_reshard_kernel(l, st);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: kernel launch: %s", what, hipGetErrorString(e));
  e = launch_chunk_sums(l.sum, chunk0, nchunks, st);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: chunk sum launch: %s", what, hipGetErrorString(e));
  return DR_OK;
}

}  // namespace

// Chunk `chunk` of the destination stream into chunk_dst (bytes [c*B, ...) of the flat
// destination, read from the source shards) and its checksum into *ck.  Arguments checked.
int launch_reshard_chunk(dr_plan* p, uint64_t chunk, const float* const* src, void* chunk_dst, dr_checksum* ck,
                         hipStream_t st, const char* what) {
  const Tiling& tl = p->tiling[0];
  const uint32_t t0 = tl.chunk_tile_begin[chunk], t1 = tl.chunk_tile_begin[chunk + 1];
  const uint64_t ce = p->layout.chunk_bytes / 4;
  return launch_reshard(p, t0, t1 - t0, src, nullptr, static_cast<float*>(chunk_dst), chunk * ce, (uint32_t)chunk, 1,
                        ck, st, what);
}

}  // namespace dr

using namespace dr;

extern "C" int dr_reshard(dr_plan* p, const float* const* src_shards, float* const* dst_shards, dr_checksum* d_cks,
                          void* stream) {
  clear_error();
  if (int rc = check_reshard_args(p, src_shards, dst_shards, d_cks, "dr_reshard")) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return launch_reshard(p, 0, (uint32_t)p->info.num_tiles, src_shards, dst_shards, nullptr, 0, 0,
                        (uint32_t)p->info.num_chunks, d_cks, st, "dr_reshard");
}
