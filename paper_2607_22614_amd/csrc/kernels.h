// Launches of the HIP kernels (stage.hip, reshard.hip), with plain arguments:
// the host library fills these records from a plan and calls the wrappers.
// Each wrapper enqueues its kernel on `st` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>

#include "dev_types.h"

namespace dr {

// Stage kernel over tiles [tile0, tile0 + ntiles) of one tiling of depth `depth`
// (kVecItersSmall or kVecItersLarge).  dst points at stream element dst_bias;
// each tile adds its checksum sums into sum's accumulators (ChunkSum).
struct StageLaunch {
  const DevSeg* segs;
  const Tile* tiles;
  ChunkSum sum;
  void* dst;
  uint64_t dst_bias;
  uint64_t chunk_elems;  // B / 2
  uint32_t tile0, ntiles;
  int depth;
  int num_shards;
  const float* const* shards;  // host array of num_shards device pointers
};
hipError_t launch_stage_kernel(const StageLaunch& l, hipStream_t st);

// The checksums of chunks [chunk0, chunk0 + nchunks) from their accumulator
// slots (written by the tile kernels), which are then set back to zero.
hipError_t launch_chunk_sums(const ChunkSum& cs, uint32_t chunk0, uint32_t nchunks, hipStream_t st);

// Reshard kernel over tiles [tile0, tile0 + ntiles).  Destination element e goes to
// flat[e - flat_bias] when flat is set, else to dst[e / dst_shard_elems]; each
// tile adds its checksum sums into sum's accumulators (ChunkSum).
struct ReshardLaunch {
  const DevSeg* segs;
  const Tile* tiles;
  ChunkSum sum;
  uint64_t chunk_elems;      // B / 4
  uint64_t dst_shard_elems;  // S'
  uint32_t tile0, ntiles;
  float* flat;
  uint64_t flat_bias;
  int num_src;
  const float* const* src;
  int num_dst;
  float* const* dst;
};
hipError_t launch_reshard_kernel(const ReshardLaunch& l, hipStream_t st);

}  // namespace dr
