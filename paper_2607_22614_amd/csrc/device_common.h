// Device helpers shared by the staging kernels (stage.hip, reshard.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "dev_types.h"

namespace dr {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

// The segment and tile tables do not change while a kernel runs: reading them
// through the constant address space (4) lets the uniform reads become scalar
// loads (s_load) instead of vector loads.
typedef const u32x4 __attribute__((address_space(4))) ConstU32x4;
typedef const u32x2 __attribute__((address_space(4))) ConstU32x2;
struct SegWords {
  u32x4 w[4];
};
static_assert(sizeof(SegWords) == sizeof(DevSeg), "segment record size");

__device__ __forceinline__ DevSeg load_seg(const DevSeg* table, uint32_t i) {
  ConstU32x4* q = (ConstU32x4*)(table + i);
  return __builtin_bit_cast(DevSeg, SegWords{{q[0], q[1], q[2], q[3]}});
}

__device__ __forceinline__ Tile load_tile(const Tile* table, uint32_t i) {
  const u32x2 v = *(ConstU32x2*)(table + i);
  return Tile{v.x, v.y};
}

template <typename T>
__device__ __forceinline__ T load_stream(const T* p) {
#if DR_NT_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void store_stream(T v, T* p) {
#if DR_NT_STORES
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// v + (v moved across lanes by the DPP control `ctrl`, applied to the rows in
// row_mask); lanes without a source add 0.
template <int ctrl, int row_mask>
__device__ __forceinline__ uint64_t dpp_add(uint64_t v) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const uint32_t mlo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, ctrl, row_mask, 0xf, false);
  const uint32_t mhi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, ctrl, row_mask, 0xf, false);
  return v + (((uint64_t)mhi << 32) | mlo);
}

// Sum over the 64 lanes of a wave with DPP moves only (VALU, no LDS round
// trips); the total lands in lane 63.  Quads first, then rows of 16, then the
// row totals are broadcast upward (row_bcast exists on gfx9-family parts).
__device__ __forceinline__ uint64_t wave_sum_to_lane63(uint64_t v) {
  v = dpp_add<0xb1, 0xf>(v);   // quad_perm [1,0,3,2]
  v = dpp_add<0x4e, 0xf>(v);   // quad_perm [2,3,0,1]: every lane holds its quad's sum
  v = dpp_add<0x114, 0xf>(v);  // row_shr:4
  v = dpp_add<0x118, 0xf>(v);  // row_shr:8: lane 15 of each row holds the row's sum
  v = dpp_add<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  v = dpp_add<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3: lane 63 holds the total
  return v;
}

// Sums (a1, a2) over the workgroup; lane 0 of wave 0 gets the totals.
__device__ __forceinline__ void block_sum2(uint64_t& a1, uint64_t& a2, uint64_t (*red)[kThreads / 64]) {
  a1 = wave_sum_to_lane63(a1);
  a2 = wave_sum_to_lane63(a2);
  const int wave = threadIdx.x / 64;
  if ((threadIdx.x & 63) == 63) {
    red[0][wave] = a1;
    red[1][wave] = a2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    a1 = 0;
    a2 = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
      a1 += red[0][w];
      a2 += red[1][w];
    }
  }
  __syncthreads();
}

// Adds tile g's (s1, s2) into its slot of chunk c (see ChunkSum); one lane calls it.
__device__ __forceinline__ void add_tile_sums(const ChunkSum& cs, uint32_t g, uint32_t c, uint64_t s1, uint64_t s2) {
  const uint64_t slot = (uint64_t)(c - cs.chunk_bias) * cs.sub + (g & (cs.sub - 1));
  unsigned long long* p = reinterpret_cast<unsigned long long*>(cs.acc + slot * cs.stride_words);
  atomicAdd(p, (unsigned long long)s1);
  atomicAdd(p + 1, (unsigned long long)s2);
}

// Tile run by the b-th workgroup: XCD x = b % 8 takes tiles
// [x*per + min(x, rem), ...) in order, where per/rem split n tiles over 8
// XCDs.  A bijection on [0, n) for every n.
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t n) {
  const uint32_t per = n / kXcds, rem = n % kXcds, x = b % kXcds;
  return x * per + min(x, rem) + b / kXcds;
}

}  // namespace dr
