// Checksums of the moment chunks: the same (s1, s2) as the rollout chunks,
// taken over the fp32 words of the moment stream m_0..m_{W-1} v_0..v_{W-1}
// cut every Bm bytes (the bounded chunks the offload and the restore move).
// A caller takes them on the device before an offload and again after the
// restore, or compares them with the host store's, to check the round trip.
//
// The kernel only reads: a lane loads K = 4 groups of four fp32 words (one
// 16-byte nontemporal load each), adds them into the tile's sums, and the tile
// adds its sums into its chunk's accumulator slots like the stage kernel; the
// chunk-sum kernel behind it writes the checksums.  HBM-bound: 4 bytes read
// per element, nothing written.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "device_common.h"
#include "dr_internal.h"
#include "kernels.h"

namespace dr {
namespace {

constexpr int kPieces = 2 * DR_MAX_SHARDS;  // m_0..m_{W-1}, v_0..v_{W-1}

struct MomentArgs {
  const DevSeg* segs;
  const Tile* tiles;
  ChunkSum sum;
  uint64_t chunk_elems;  // Bm / 4
  uint32_t tile0, ntiles;
  const float* pieces[kPieces];
};

__global__ __launch_bounds__(kThreads) void moment_sum_kernel(MomentArgs args) {
  (void)args;  // read through the kernarg segment (same bytes)
  const MomentArgs& a = *(const MomentArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ uint64_t red[2][kThreads / 64];
  for (uint32_t b = blockIdx.x; b < a.ntiles; b += gridDim.x) {
    const uint32_t t = xcd_tile(b, a.ntiles);
    const Tile tile = load_tile(a.tiles, a.tile0 + t);
    const DevSeg s = load_seg(a.segs, tile.seg);
    const float* __restrict__ src = a.pieces[s.shard] + s.src;
    const uint64_t pos0 = s.dst - (uint64_t)s.chunk * a.chunk_elems;  // word position in the chunk
    const uint32_t last = s.units - 1;
    u32x4 v[kReshardIters];
#pragma unroll
    for (int k = 0; k < kReshardIters; ++k) {
      const uint32_t u = min(tile.unit0 + k * kThreads + threadIdx.x, last);
      v[k] = load_stream(reinterpret_cast<const u32x4*>(src + 4 * u));
    }
    uint64_t acc_w = 0, acc_rw = 0;
#pragma unroll
    for (int k = 0; k < kReshardIters; ++k) {
      const uint32_t u = tile.unit0 + k * kThreads + threadIdx.x;
      if (u <= last) {
        const uint32_t e = 4 * u;  // word index relative to the segment
        acc_w += (uint64_t)v[k].x + v[k].y + (uint64_t)v[k].z + v[k].w;
        acc_rw += (uint64_t)e * v[k].x + (uint64_t)(e + 1) * v[k].y + (uint64_t)(e + 2) * v[k].z +
                  (uint64_t)(e + 3) * v[k].w;
      }
    }
    block_sum2(acc_w, acc_rw, red);
    if (threadIdx.x == 0) add_tile_sums(a.sum, a.tile0 + t, s.chunk, acc_w, (pos0 + 1) * acc_w + acc_rw);
  }
}

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace
}  // namespace dr

using namespace dr;

extern "C" int dr_moment_checksums(dr_plan* p, const float* const* m_shards, const float* const* v_shards,
                                   dr_checksum* d_cks, void* stream) {
  clear_error();
  const char* what = "dr_moment_checksums";
  if (!p) return fail(DR_EINVAL, "%s: null plan", what);
  if (p->kind != kRollout || !p->layout.moment_chunk_bytes)
    return fail(DR_EINVAL, "%s: the plan has no moment path (moment_chunk_bytes is 0)", what);
  if (!m_shards || !v_shards) return fail(DR_EINVAL, "%s: null shard array", what);
  const int W = p->layout.train_shards;
  for (int w = 0; w < W; ++w)
    if (!aligned16(m_shards[w]) || !aligned16(v_shards[w]))
      return fail(DR_EINVAL, "%s: moment shard %d pointer is null or not 16-byte aligned", what, w);
  if (!aligned16(d_cks)) return fail(DR_EINVAL, "%s: d_cks is null or not 16-byte aligned", what);
  if (!p->d_moment_segs) return fail(DR_EINVAL, "%s: host-only plan has no device tables", what);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: hipGetDevice: %s", what, hipGetErrorString(e));
  if (dev != p->device) return fail(DR_EINVAL, "%s: plan lives on device %d, current device is %d", what, p->device, dev);

  const Tiling& tl = p->moment_tiling;
  MomentArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = p->d_moment_segs;
  args.tiles = tl.d_tiles;
  args.sum = chunk_sum(p, tl, d_cks, 0);
  args.chunk_elems = p->layout.moment_chunk_bytes / 4;
  args.tile0 = 0;
  args.ntiles = (uint32_t)tl.tiles.size();
  for (int w = 0; w < W; ++w) {
    args.pieces[w] = m_shards[w];
    args.pieces[W + w] = v_shards[w];
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(moment_sum_kernel, dim3(std::min(args.ntiles, kMaxGrid)), dim3(kThreads), 0, st, args);
  e = hipGetLastError();
  if (e != hipSuccess) return fail(DR_EHIP, "%s: kernel launch: %s", what, hipGetErrorString(e));
  e = launch_chunk_sums(args.sum, 0, (uint32_t)p->info.num_moment_chunks, st);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: chunk sum launch: %s", what, hipGetErrorString(e));
  return DR_OK;
}
