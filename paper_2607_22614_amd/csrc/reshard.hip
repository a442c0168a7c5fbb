// Reshard kernel: the training -> training move to a new shard count
// (weights and optimizer states from the old training ranks to the new ones).
// The N elements keep their order and bits; they are re-cut into W' shards and
// the destination padding is zeroed.  Same tiling, XCD order and checksum
// scheme as the stage kernel, with one fp32 word per element: a lane moves a
// 16-byte group (one nontemporal load, one nontemporal store).  HBM-bound: 4 B
// read and 4 B written per element (padding: written only).
#include <hip/hip_runtime.h>

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
    float* __restrict__ out = a.dst[s.dst_shard] + (s.dst - (uint64_t)s.dst_shard * a.dst_shard_elems);
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
}  // namespace dr

using namespace dr;

extern "C" int dr_reshard(dr_plan* p, const float* const* src_shards, float* const* dst_shards, dr_checksum* d_cks,
                          void* stream) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_reshard: null plan");
  if (p->kind != kReshard) return fail(DR_EINVAL, "dr_reshard: not a reshard plan");
  if (!src_shards || !dst_shards) return fail(DR_EINVAL, "dr_reshard: null shard array");
  for (int w = 0; w < p->layout.train_shards; ++w)
    if (!aligned16(src_shards[w])) return fail(DR_EINVAL, "dr_reshard: source shard %d is null or not 16-byte aligned", w);
  for (int w = 0; w < p->dst_shards; ++w)
    if (!aligned16(dst_shards[w]))
      return fail(DR_EINVAL, "dr_reshard: destination shard %d is null or not 16-byte aligned", w);
  if (!aligned16(d_cks)) return fail(DR_EINVAL, "dr_reshard: d_cks is null or not 16-byte aligned");
  if (!p->d_segs) return fail(DR_EINVAL, "dr_reshard: host-only plan has no device tables");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DR_EHIP, "dr_reshard: hipGetDevice: %s", hipGetErrorString(e));
  if (dev != p->device) return fail(DR_EINVAL, "dr_reshard: plan lives on device %d, current device is %d", p->device, dev);
  ReshardArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = p->d_segs;
  args.tiles = p->d_tiles;
  args.partials = p->d_partials;
  args.chunk_elems = p->layout.chunk_bytes / 4;
  args.dst_shard_elems = p->dst_shard_elems;
  args.tile0 = 0;
  args.ntiles = (uint32_t)p->info.num_tiles;
  for (int w = 0; w < p->layout.train_shards; ++w) args.src[w] = src_shards[w];
  for (int w = 0; w < p->dst_shards; ++w) args.dst[w] = dst_shards[w];
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (args.ntiles) {
    hipLaunchKernelGGL(reshard_kernel, dim3(args.ntiles), dim3(kThreads), 0, st, args);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(DR_EHIP, "dr_reshard: kernel launch: %s", hipGetErrorString(e));
  }
  return launch_reduce(p, 0, (uint32_t)p->info.num_chunks, d_cks, st, "dr_reshard");
}
