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
#include "kernels.h"

namespace dr {
namespace {

struct ReshardArgs {
  const DevSeg* segs;
  const Tile* tiles;
  ChunkSum sum;              // the chunks' checksum accumulators and output slots
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
    if (threadIdx.x == 0) add_tile_sums(a.sum, a.tile0 + t, s.chunk, acc_w, (pos0 + 1) * acc_w + acc_rw);
  }
}

}  // namespace

hipError_t launch_reshard_kernel(const ReshardLaunch& l, hipStream_t st) {
  if (!l.ntiles) return hipSuccess;
  ReshardArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = l.segs;
  args.tiles = l.tiles;
  args.sum = l.sum;
  args.chunk_elems = l.chunk_elems;
  args.dst_shard_elems = l.dst_shard_elems;
  args.tile0 = l.tile0;
  args.ntiles = l.ntiles;
  args.flat = l.flat;
  args.flat_bias = l.flat_bias;
  for (int w = 0; w < l.num_src; ++w) args.src[w] = l.src[w];
  if (l.dst)
    for (int w = 0; w < l.num_dst; ++w) args.dst[w] = l.dst[w];
  hipLaunchKernelGGL(reshard_kernel, dim3(std::min(l.ntiles, kMaxGrid)), dim3(kThreads), 0, st, args);
  return hipGetLastError();
}

}  // namespace dr
