// Reshard kernel: the training -> training move to a new shard count
// (weights and optimizer states from the old training ranks to the new ones).
// The N elements keep their order and bits; they are re-cut into W' shards and
// the destination padding is zeroed.  Same tiling, XCD order and checksum
// scheme as the stage kernel, with one fp32 word per element: a lane moves a
// 16-byte group (one nontemporal load, one nontemporal store).  HBM-bound: 4 B
// read and 4 B written per element (padding: written only).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "device_common.h"
#include "dr_internal.h"

namespace dr {
namespace {

struct ReshardArgs {
  const DevSeg* segs;
  const Tile* tiles;
  uint64_t* partials;
  uint64_t chunk_elems;      // B / 4
  uint64_t dst_shard_elems;  // S'
  uint32_t tile0, ntiles;
  float* flat;               // non-null: write destination element e to flat[e - flat_bias] (one chunk)
  uint64_t flat_bias;
  const float* src[DR_MAX_SHARDS];
  float* dst[DR_MAX_SHARDS];
};

__global__ __launch_bounds__(kThreads) void reshard_kernel(ReshardArgs args) {
  (void)args;  // read through the kernarg segment (same bytes)
  const ReshardArgs& a = *(const ReshardArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ uint64_t red[2][kThreads / 64];
  for (uint32_t b = blockIdx.x; b < a.ntiles; b += gridDim.x) {
    const uint32_t t = xcd_tile(b, a.ntiles);
    const Tile tile = load_tile(a.tiles, a.tile0 + t);
    const DevSeg s = load_seg(a.segs, tile.seg);
    float* __restrict__ out = a.flat ? a.flat + (s.dst - a.flat_bias)
                                     : a.dst[s.dst_shard] + (s.dst - (uint64_t)s.dst_shard * a.dst_shard_elems);
    const uint64_t pos0 = s.dst - (uint64_t)s.chunk * a.chunk_elems;  // word position in the chunk
    const uint32_t last = s.units - 1;
    uint64_t acc_w = 0, acc_rw = 0;
    if (s.op == DR_OP_ZERO_F32) {
#pragma unroll
      for (int k = 0; k < kReshardIters; ++k) {
        const uint32_t u = tile.unit0 + k * kThreads + threadIdx.x;
        if (u <= last) store_stream((f32x4){0.f, 0.f, 0.f, 0.f}, reinterpret_cast<f32x4*>(out + 4 * u));
      }
    } else {
      const float* __restrict__ src = a.src[s.shard] + s.src;
      u32x4 v[kReshardIters];
#pragma unroll
      for (int k = 0; k < kReshardIters; ++k) {
        const uint32_t u = min(tile.unit0 + k * kThreads + threadIdx.x, last);
        v[k] = load_stream(reinterpret_cast<const u32x4*>(src + 4 * u));
      }
#pragma unroll
      for (int k = 0; k < kReshardIters; ++k) {
        const uint32_t u = tile.unit0 + k * kThreads + threadIdx.x;
        if (u <= last) {
          store_stream(v[k], reinterpret_cast<u32x4*>(out + 4 * u));
          const uint32_t e = 4 * u;  // word index relative to the segment
          acc_w += (uint64_t)v[k].x + v[k].y + (uint64_t)v[k].z + v[k].w;
          acc_rw += (uint64_t)e * v[k].x + (uint64_t)(e + 1) * v[k].y + (uint64_t)(e + 2) * v[k].z +
                    (uint64_t)(e + 3) * v[k].w;
        }
      }
    }
    block_sum2(acc_w, acc_rw, red);
    if (threadIdx.x == 0) {
      *reinterpret_cast<u64x2*>(a.partials + 2ull * (a.tile0 + t)) = (u64x2){acc_w, (pos0 + 1) * acc_w + acc_rw};
    }
  }
}

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
// elements from flat_bias on instead of the destination shards.
int launch_reshard(dr_plan* p, uint32_t tile0, uint32_t ntiles, const float* const* src, float* const* dst,
                   float* flat, uint64_t flat_bias, hipStream_t st, const char* what) {
  ReshardArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = p->d_segs;
  args.tiles = p->tiling[0].d_tiles;
  args.partials = p->d_partials + 2 * p->tiling[0].partial0;
  args.chunk_elems = p->layout.chunk_bytes / 4;
  args.dst_shard_elems = p->dst_shard_elems;
  args.tile0 = tile0;
  args.ntiles = ntiles;
  args.flat = flat;
  args.flat_bias = flat_bias;
  for (int w = 0; w < p->layout.train_shards; ++w) args.src[w] = src[w];
  if (dst)
    for (int w = 0; w < p->dst_shards; ++w) args.dst[w] = dst[w];
  if (ntiles) {
    hipLaunchKernelGGL(reshard_kernel, dim3(std::min(ntiles, kMaxGrid)), dim3(kThreads), 0, st, args);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(DR_EHIP, "%s: kernel launch: %s", what, hipGetErrorString(e));
  }
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
  if (int rc = launch_reshard(p, t0, t1 - t0, src, nullptr, static_cast<float*>(chunk_dst), chunk * ce, st, what))
    return rc;
  return launch_reduce(p, tl, (uint32_t)chunk, 1, ck, st, what);
}

}  // namespace dr

using namespace dr;

extern "C" int dr_reshard(dr_plan* p, const float* const* src_shards, float* const* dst_shards, dr_checksum* d_cks,
                          void* stream) {
  clear_error();
  if (int rc = check_reshard_args(p, src_shards, dst_shards, d_cks, "dr_reshard")) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (int rc = launch_reshard(p, 0, (uint32_t)p->info.num_tiles, src_shards, dst_shards, nullptr, 0, st, "dr_reshard"))
    return rc;
  return launch_reduce(p, p->tiling[0], 0, (uint32_t)p->info.num_chunks, d_cks, st, "dr_reshard");
}
