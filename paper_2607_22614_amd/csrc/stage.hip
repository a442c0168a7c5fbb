// Stage kernel: pack + cast + per-chunk checksum of the rollout stream on
// gfx950 (CDNA4), and the chunk launches behind dr_stage_chunk / dr_stage_all.
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
//     workgroup (LDS), and written as one (s1, s2) partial per tile; a second
//     small kernel sums a chunk's partials.  No atomics, no extra pass over
//     the data, and the result is independent of scheduling.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstring>

#include "device_common.h"
#include "dr_internal.h"

namespace dr {
namespace {

// Everything a stage launch needs, passed as the kernel's only argument.  The
// kernel reads it through the kernarg segment pointer, so the shard table is
// indexed with one scalar load instead of being copied into registers.
struct StageArgs {
  const DevSeg* segs;
  const Tile* tiles;
  uint16_t* dst;          // points at stream element dst_bias
  uint64_t* partials;     // (s1, s2) per tile
  uint64_t dst_bias;
  uint64_t chunk_elems;   // B / 2
  uint32_t tile0, ntiles; // tiles [tile0, tile0 + ntiles)
  const float* shards[DR_MAX_SHARDS];
};

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
    if (threadIdx.x == 0) {
      const uint64_t jb1 = (pos0 >> 1) + 1;
      *reinterpret_cast<u64x2*>(a.partials + 2ull * (a.tile0 + t)) = (u64x2){acc_w, jb1 * acc_w + acc_rw};
    }
  }
}

// out[i] = sum of the partials of chunk chunk0+i, i < nchunks, one workgroup
// per chunk (a grid capped at kMaxReduceGrid workgroups strides over the
// chunks).  A chunk can hold 10^5 tiles (1 GiB chunks), so each lane keeps
// kReduceUnroll independent 16-byte loads in flight; the sum is integer, so any
// order gives the same bits.
constexpr int kReduceThreads = 1024;
constexpr int kReduceUnroll = 8;
constexpr uint32_t kMaxReduceGrid = 1u << 20;

__global__ __launch_bounds__(kReduceThreads) void chunk_reduce_kernel(const uint64_t* __restrict__ partials,
                                                                      const uint32_t* __restrict__ chunk_tile_begin,
                                                                      uint32_t chunk0, uint32_t nchunks,
                                                                      dr_checksum* __restrict__ out) {
  __shared__ uint64_t red[2][kReduceThreads / 64];
  for (uint32_t i = blockIdx.x; i < nchunks; i += gridDim.x) {
    const uint32_t c = chunk0 + i;
    const uint32_t first = chunk_tile_begin[c], last = chunk_tile_begin[c + 1];
    const u64x2* p = reinterpret_cast<const u64x2*>(partials);
    uint64_t a1 = 0, a2 = 0;
    uint64_t t = first + threadIdx.x;
    for (; t + (kReduceUnroll - 1) * kReduceThreads < last; t += kReduceUnroll * kReduceThreads) {
      u64x2 v[kReduceUnroll];
#pragma unroll
      for (int k = 0; k < kReduceUnroll; ++k) v[k] = p[t + k * kReduceThreads];
#pragma unroll
      for (int k = 0; k < kReduceUnroll; ++k) {
        a1 += v[k].x;
        a2 += v[k].y;
      }
    }
    for (; t < last; t += kReduceThreads) {
      a1 += p[t].x;
      a2 += p[t].y;
    }
    a1 = wave_sum_to_lane63(a1);
    a2 = wave_sum_to_lane63(a2);
    const int wave = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 63) {
      red[0][wave] = a1;
      red[1][wave] = a2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t s1 = 0, s2 = 0;
#pragma unroll
      for (int w = 0; w < kReduceThreads / 64; ++w) {
        s1 += red[0][w];
        s2 += red[1][w];
      }
      *reinterpret_cast<u64x2*>(&out[i]) = (u64x2){s1, s2};
    }
    __syncthreads();  // red is rewritten by the next chunk of this workgroup
  }
}

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


}  // namespace
int launch_reduce(dr_plan* p, const Tiling& tl, uint32_t chunk0, uint32_t nchunks, dr_checksum* cks, hipStream_t st,
                  const char* what);
namespace {

// Per-device state of the automatic tile depth (see pack_drain_ns in the
// internal header): when the packs launched so far should have drained.
std::atomic<int64_t> g_packs_drain_ns[kClockDevices];

int64_t host_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

// Index of the tiling that the launch starting now uses.
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

int launch(dr_plan* p, const Tiling& tl, uint32_t tile0, uint32_t ntiles, const float* const* shards, void* dst,
           uint64_t dst_bias, uint32_t chunk0, uint32_t nchunks, dr_checksum* cks, hipStream_t st,
           const char* what) {
  StageArgs args;
  std::memset(&args, 0, sizeof(args));
  args.segs = p->d_segs;
  args.tiles = tl.d_tiles;
  args.dst = static_cast<uint16_t*>(dst);
  args.partials = p->d_partials + 2 * tl.partial0;
  args.dst_bias = dst_bias;
  args.chunk_elems = p->layout.chunk_bytes / 2;
  args.tile0 = tile0;
  args.ntiles = ntiles;
  for (int w = 0; w < p->layout.train_shards; ++w) args.shards[w] = shards[w];
  if (ntiles) {
    const uint32_t cap = DR_GRID_CAP > 0 ? (uint32_t)DR_GRID_CAP : kMaxGrid;
    const uint32_t grid = ntiles < cap ? ntiles : cap;
    if (tl.depth == kVecItersLarge)
      hipLaunchKernelGGL(stage_kernel<kVecItersLarge>, dim3(grid), dim3(kThreads), 0, st, args);
    else
      hipLaunchKernelGGL(stage_kernel<kVecItersSmall>, dim3(grid), dim3(kThreads), 0, st, args);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(DR_EHIP, "%s: stage kernel launch: %s", what, hipGetErrorString(e));
  }
  p->last_depth.store(tl.depth, std::memory_order_relaxed);
  return launch_reduce(p, tl, chunk0, nchunks, cks, st, what);
}

// Chunk `chunk` with tiling tl into dst_chunk.
int launch_one_chunk(dr_plan* p, const Tiling& tl, uint64_t chunk, const float* const* shards, void* dst_chunk,
                     dr_checksum* ck, hipStream_t st, const char* what) {
  const uint32_t t0 = tl.chunk_tile_begin[chunk], t1 = tl.chunk_tile_begin[chunk + 1];
  return launch(p, tl, t0, t1 - t0, shards, dst_chunk, chunk * (p->layout.chunk_bytes / 2), (uint32_t)chunk, 1, ck,
                st, what);
}

uint64_t chunk_out_bytes(const dr_plan* p, uint64_t chunk) {
  return chunk + 1 < p->info.num_chunks ? p->layout.chunk_bytes : p->info.last_chunk_bytes;
}

template <typename T>
int upload(T** dptr, const std::vector<T>& host, const char* what) {
  const size_t bytes = std::max<size_t>(host.size() * sizeof(T), 16);
  hipError_t e = hipMalloc(reinterpret_cast<void**>(dptr), bytes);
  if (e != hipSuccess) {
    *dptr = nullptr;
    return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "hipMalloc(%s, %zu B): %s", what, bytes,
                hipGetErrorString(e));
  }
  if (!host.empty()) {
    e = hipMemcpy(*dptr, host.data(), host.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(DR_EHIP, "hipMemcpy(%s): %s", what, hipGetErrorString(e));
  }
  return DR_OK;
}

}  // namespace

int launch_reduce(dr_plan* p, const Tiling& tl, uint32_t chunk0, uint32_t nchunks, dr_checksum* cks, hipStream_t st,
                  const char* what) {
  if (!nchunks) return DR_OK;
  hipLaunchKernelGGL(chunk_reduce_kernel, dim3(std::min(nchunks, kMaxReduceGrid)), dim3(kReduceThreads), 0, st,
                     p->d_partials + 2 * tl.partial0, tl.d_chunk_tile_begin, chunk0, nchunks, cks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DR_EHIP, "%s: reduce kernel launch: %s", what, hipGetErrorString(e));
  return DR_OK;
}

int check_stage_args(const dr_plan* p, const float* const* shards, const void* dst, const void* cks,
                     const char* what) {
  if (int rc = check_shards(p, shards, what)) return rc;
  if (!aligned16(dst)) return fail(DR_EINVAL, "%s: destination is null or not 16-byte aligned", what);
  if (!aligned16(cks)) return fail(DR_EINVAL, "%s: checksum slots are null or not 16-byte aligned", what);
  if (!p->d_segs) return fail(DR_EINVAL, "%s: host-only plan has no device tables", what);
  return check_device(p, what);
}

int launch_chunk(dr_plan* p, uint64_t chunk, const float* const* shards, void* dst_chunk, dr_checksum* ck,
                 void* st) {
  return launch_one_chunk(p, p->tiling[0], chunk, shards, dst_chunk, ck, static_cast<hipStream_t>(st),
                          "chunk launch");
}

int upload_plan(dr_plan* p) {
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) return fail(DR_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  int rc;
  if ((rc = upload(&p->d_segs, p->segs, "segments"))) return rc;
  size_t slots = 0;
  for (Tiling& tl : p->tiling) {
    if (!tl.depth) continue;
    if ((rc = upload(&tl.d_tiles, tl.tiles, "tiles"))) return rc;
    if ((rc = upload(&tl.d_chunk_tile_begin, tl.chunk_tile_begin, "chunk tiles"))) return rc;
    slots = std::max<size_t>(slots, tl.partial0 + tl.tiles.size());
  }
  const size_t pbytes = std::max<size_t>(slots * 16, 16);
  e = hipMalloc(reinterpret_cast<void**>(&p->d_partials), pbytes);
  if (e != hipSuccess) {
    p->d_partials = nullptr;
    return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "hipMalloc(partials, %zu B): %s", pbytes,
                hipGetErrorString(e));
  }
  p->info.device = p->device;
  return DR_OK;
}

void free_device(dr_plan* p) {
  if (p->d_segs) (void)hipFree(p->d_segs);
  if (p->d_partials) (void)hipFree(p->d_partials);
  p->d_segs = nullptr;
  p->d_partials = nullptr;
  for (Tiling& tl : p->tiling) {
    if (tl.d_tiles) (void)hipFree(tl.d_tiles);
    if (tl.d_chunk_tile_begin) (void)hipFree(tl.d_chunk_tile_begin);
    tl.d_tiles = nullptr;
    tl.d_chunk_tile_begin = nullptr;
  }
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
  const Tiling& tl = p->tiling[pick_tiling(p)];
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
  const int rc = launch(p, tl, 0, (uint32_t)tl.tiles.size(), shards, dst, 0, 0, (uint32_t)p->info.num_chunks, d_cks,
                        static_cast<hipStream_t>(stream), "dr_stage_all");
  if (rc == DR_OK) note_pack(p, 4 * p->info.n_elems + p->info.rollout_bytes);
  return rc;
}
