// Stage kernel: pack + cast + per-chunk checksum of the rollout stream on
// gfx950 (CDNA4), and the chunk-sum kernel.  The launches behind
// dr_stage_chunk / dr_stage_all are driven from staging.cpp.
//
// The work is a gather of contiguous runs with a narrowing cast: every output
// element is read once as fp32 and written once as bf16, so the kernel is
// bound by HBM bandwidth (6 bytes of traffic per element) and never touches
// MFMA.  Design points:
//   * the planner cuts the stream into segments that never cross a shard or
//     chunk boundary, and each workgroup tile lies inside one segment, so a
//     tile finds its work with two uniform (scalar) loads, its tile record and
//     then its segment record, and every lane of a tile takes the same branch;
//   * on aligned segments a lane moves groups of 4 elements: one 16-byte
//     nontemporal load, two packed round-to-nearest-even converts (two bf16
//     per instruction), one 8-byte nontemporal store.  Lane l of a wave takes
//     group l, so one wave instruction covers 1 KiB of source and 512 B of
//     destination, contiguous within a row;
//   * every load of a lane is issued before the first convert (K = 2 or 4
//     independent 16-byte loads in flight per lane: the plan's tile depth);
//   * XCD-aware tile order: the hardware hands workgroup b to XCD b % 8, and
//     the kernel maps it to a tile so that each XCD streams through one
//     contiguous eighth of the stream instead of every eighth tile (measured
//     faster on the 8B shape: 6.3 vs 6.0 TB/s);
//   * the chunk checksum is accumulated from the packed words while they are
//     in registers, reduced across the wavefront (DPP moves, no LDS) and the
//     workgroup (LDS), and added with two 64-bit atomic adds (nothing waits
//     for them) into one of the chunk's accumulator slots; a small kernel
//     behind the launch adds a chunk's slots.  The sums are integer, so the
//     bits do not depend on the order of the adds, and there is no extra
//     pass over the data.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "device_common.h"
#include "kernels.h"

namespace dr {
namespace {

// Everything a stage launch needs, passed as the kernel's only argument.  The
// kernel reads it through the kernarg segment pointer, so the shard table is
// indexed with one scalar load instead of being copied into registers.
struct StageArgs {
  const DevSeg* segs;
  const Tile* tiles;
  uint16_t* dst;          // points at stream element dst_bias
  ChunkSum sum;           // the chunks' checksum accumulators and output slots
  uint64_t dst_bias;
  uint64_t chunk_elems;   // B / 2
  uint32_t tile0, ntiles; // tiles [tile0, tile0 + ntiles)
  const float* shards[DR_MAX_SHARDS];
};

// The convert below is exact only in the default FP mode: fast-math may
// assume no NaN or infinity, and a flush-to-zero denormal mode would flush
// fp32 subnormals before rounding.  Fast-math is refused here; the denormal
// mode of every kernel is checked in the built assembly by the test suite.
#if defined(__FAST_MATH__) || __FINITE_MATH_ONLY__
#error "stage.hip needs the default FP mode: build without -ffast-math / -ffinite-math-only"
#endif

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 -> one word of two bf16 (x in the low half), rounded to nearest
// with ties to even by gfx950's packed convert (v_cvt_pk_bf16_f32).  In the
// default FP mode it keeps fp32 subnormals (no flush), rounds overflow to
// infinity and returns a NaN as its upper half with the quiet bit set: equal
// to the integer definition on all 2^32 inputs, checked on the device.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float x, float y) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){x, y}, bf16x2));
}

// q = e / cols, r = e % cols for e < 2^32, from magic = floor(2^32 / cols):
// the estimate is at most one below the quotient, so one correction suffices.
__device__ __forceinline__ uint32_t div_cols(uint32_t e, uint32_t cols, uint32_t magic, uint32_t* rem) {
  uint32_t q = __umulhi(e, magic);
  uint32_t r = e - q * cols;
  if (r >= cols) {
    q += 1;
    r -= cols;
  }
  *rem = r;
  return q;
}

// One workgroup per tile (grid-stride when the grid is capped); K groups of 4
// elements per lane on aligned segments.
template <int K>
__global__ __launch_bounds__(kThreads) void stage_kernel(StageArgs args) {
  (void)args;  // read below through the kernarg segment (same bytes)
  const StageArgs& a = *(const StageArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ uint64_t red[2][kThreads / 64];
  for (uint32_t b = blockIdx.x; b < a.ntiles; b += gridDim.x) {
    const uint32_t t = xcd_tile(b, a.ntiles);
    const Tile tile = load_tile(a.tiles, a.tile0 + t);
    const DevSeg s = load_seg(a.segs, tile.seg);
    const float* __restrict__ src = a.shards[s.shard] + s.src;
    uint16_t* __restrict__ out = a.dst + (s.dst - a.dst_bias);
    // Checksum of the tile: word j of the chunk counts (j+1)*w_j.  With jb the
    // chunk word index of the segment's first element, j = jb + rel where
    // rel < 2^31 is the word index relative to the segment, so lanes sum
    // A = sum w and R = sum rel*w with 32x32->64 multiply-adds and the tile's
    // s2 = (jb+1)*A + R is formed once at the end.
    const uint64_t pos0 = s.dst - (uint64_t)s.chunk * a.chunk_elems;  // element position in the chunk
    const uint32_t odd0 = (uint32_t)(pos0 & 1);
    uint64_t acc_w = 0, acc_rw = 0;
    const uint32_t last = s.units - 1;

    if (s.flags & DR_SEG_VEC4) {
      const bool contiguous = s.rows == 1;
      f32x4 v[K];
      // Loads first, all unconditional: lanes past the end of a ragged tile
      // re-read the segment's last group and store nothing.
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const uint32_t u = min(tile.unit0 + k * kThreads + threadIdx.x, last);
        const uint32_t e = u * 4;
        uint32_t so = e;
        if (!contiguous) {
          uint32_t col;
          const uint32_t row = div_cols(e, s.cols, s.magic, &col);
          so = row * s.stride + col;
        }
        v[k] = load_stream(reinterpret_cast<const f32x4*>(src + so));
      }
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const uint32_t u = tile.unit0 + k * kThreads + threadIdx.x;
        const uint32_t w0 = cvt_pk_bf16(v[k].x, v[k].y);
        const uint32_t w1 = cvt_pk_bf16(v[k].z, v[k].w);
        if (u <= last) {
          const uint32_t e = u * 4;
          store_stream((u32x2){w0, w1}, reinterpret_cast<u32x2*>(out + e));
          const uint32_t rel = e >> 1;  // pos0 is even on aligned segments
          acc_w += (uint64_t)w0 + w1;
          acc_rw += (uint64_t)rel * w0 + (uint64_t)(rel + 1) * w1;
        }
      }
    } else {
      // Unaligned segment (runs that are not whole 4-element groups): one
      // element per lane per step; each element adds its half of a word.
      float h[kScalarIters];
#pragma unroll
      for (int k = 0; k < kScalarIters; ++k) {
        const uint32_t e = min(tile.unit0 + k * kThreads + threadIdx.x, last);
        uint32_t col = e, row = 0;
        if (s.rows > 1) row = div_cols(e, s.cols, s.magic, &col);
        h[k] = load_stream(src + row * s.stride + col);
      }
#pragma unroll
      for (int k = 0; k < kScalarIters; ++k) {
        const uint32_t e = tile.unit0 + k * kThreads + threadIdx.x;
        const uint32_t bf = cvt_pk_bf16(h[k], 0.f) & 0xFFFFu;
        if (e <= last) {
          out[e] = (uint16_t)bf;
          const uint32_t q = odd0 + e;  // element position relative to the word holding the first element
          const uint32_t val = bf << ((q & 1) * 16);
          acc_w += val;
          acc_rw += (uint64_t)(q >> 1) * val;
        }
      }
    }
    block_sum2(acc_w, acc_rw, red);
    if (threadIdx.x == 0) add_tile_sums(a.sum, a.tile0 + t, s.chunk, acc_w, ((pos0 >> 1) + 1) * acc_w + acc_rw);
  }
}

// Chunk sums: for each chunk c in [chunk0, chunk0 + nchunks), out[c - out_chunk0]
// = the sum of the chunk's accumulator slots, which are then set to zero.  Runs
// after the tile kernel on the same stream, so every add has landed.  The sums
// are integer, so the order of the adds does not change the bits.  A lane per
// slot, so every load is in flight at once: one lane per chunk when a chunk has
// one slot (small budgets: up to 10^6 chunks), one wave per chunk up to 64
// slots, one workgroup per chunk beyond; the grid is capped and strides over
// the chunks.
constexpr uint32_t kMaxSumGrid = 1u << 14;
static_assert(kMaxSumSlots <= kThreads, "one lane per accumulator slot");

__global__ __launch_bounds__(kThreads) void chunk_sum_kernel(ChunkSum cs, uint32_t chunk0, uint32_t nchunks) {
  const u64x2 zero = {0, 0};
  if (cs.sub == 1) {
    for (uint32_t i = blockIdx.x * kThreads + threadIdx.x; i < nchunks; i += gridDim.x * kThreads) {
      const uint32_t c = chunk0 + i;
      u64x2* p = reinterpret_cast<u64x2*>(cs.acc + (uint64_t)(c - cs.chunk_bias) * cs.stride_words);
      const u64x2 v = *p;
      *p = zero;
      *reinterpret_cast<u64x2*>(&cs.out[c - cs.out_chunk0]) = v;
    }
    return;
  }
  if (cs.sub <= 64) {
    const uint32_t lane = threadIdx.x & 63, waves = kThreads / 64;
    // i is the same on every lane of a wave, so the whole wave runs each iteration (DPP sums)
    for (uint32_t i = blockIdx.x * waves + threadIdx.x / 64; i < nchunks; i += gridDim.x * waves) {
      const uint32_t c = chunk0 + i;
      uint64_t a1 = 0, a2 = 0;
      if (lane < cs.sub) {
        const uint64_t slot = (uint64_t)(c - cs.chunk_bias) * cs.sub + lane;
        u64x2* p = reinterpret_cast<u64x2*>(cs.acc + slot * cs.stride_words);
        const u64x2 v = *p;
        *p = zero;
        a1 = v.x;
        a2 = v.y;
      }
      a1 = wave_sum_to_lane63(a1);
      a2 = wave_sum_to_lane63(a2);
      if (lane == 63) *reinterpret_cast<u64x2*>(&cs.out[c - cs.out_chunk0]) = (u64x2){a1, a2};
    }
    return;
  }
  __shared__ uint64_t red[2][kThreads / 64];
  for (uint32_t i = blockIdx.x; i < nchunks; i += gridDim.x) {
    const uint32_t c = chunk0 + i;
    uint64_t a1 = 0, a2 = 0;
    if (threadIdx.x < cs.sub) {
      u64x2* p = reinterpret_cast<u64x2*>(cs.acc + ((uint64_t)(c - cs.chunk_bias) * cs.sub + threadIdx.x) *
                                                       cs.stride_words);
      const u64x2 v = *p;
      *p = zero;
      a1 = v.x;
      a2 = v.y;
    }
    block_sum2(a1, a2, red);
    if (threadIdx.x == 0) *reinterpret_cast<u64x2*>(&cs.out[c - cs.out_chunk0]) = (u64x2){a1, a2};
  }
}

}  // namespace

hipError_t launch_chunk_sums(const ChunkSum& cs, uint32_t chunk0, uint32_t nchunks, hipStream_t st) {
  if (!nchunks) return hipSuccess;
  const uint32_t per = cs.sub == 1 ? kThreads : cs.sub <= 64 ? kThreads / 64 : 1;
  const uint32_t grid = std::min((nchunks + per - 1) / per, kMaxSumGrid);
  hipLaunchKernelGGL(chunk_sum_kernel, dim3(grid), dim3(kThreads), 0, st, cs, chunk0, nchunks);
  return hipGetLastError();
}

hipError_t launch_stage_kernel(const StageLaunch& l, hipStream_t st) {
  if (!l.ntiles) return hipSuccess;
  StageArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = l.segs;
  args.tiles = l.tiles;
  args.dst = static_cast<uint16_t*>(l.dst);
  args.sum = l.sum;
  args.dst_bias = l.dst_bias;
  args.chunk_elems = l.chunk_elems;
  args.tile0 = l.tile0;
  args.ntiles = l.ntiles;
  for (int w = 0; w < l.num_shards; ++w) args.shards[w] = l.shards[w];
  const uint32_t cap = DR_GRID_CAP > 0 ? (uint32_t)DR_GRID_CAP : kMaxGrid;
  const uint32_t grid = l.ntiles < cap ? l.ntiles : cap;
  if (l.depth == kVecItersLarge)
    hipLaunchKernelGGL(stage_kernel<kVecItersLarge>, dim3(grid), dim3(kThreads), 0, st, args);
  else
    hipLaunchKernelGGL(stage_kernel<kVecItersSmall>, dim3(grid), dim3(kThreads), 0, st, args);
  return hipGetLastError();
}

}  // namespace dr
