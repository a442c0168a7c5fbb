// Types and launch-geometry constants that the kernels and the host code driving
// them share.  Everything a kernel's code depends on lives here, in
// device_common.h, kernels.h and the kernel's own .hip file.
#pragma once

#include <cstdint>

#include "dr.h"

namespace dr {

// Launch geometry of the kernels.  A workgroup of kThreads lanes handles one
// tile: K groups of 4 elements per lane on aligned segments, or kScalarIters
// single elements per lane on unaligned ones.  The stage kernel runs at tile
// depth K = kVecItersSmall or kVecItersLarge (the host picks per plan and per
// launch); the reshard kernel at K = kReshardIters.
// Stage grid: 0 launches one workgroup per tile (at most kMaxGrid, which then
// stride over the tiles); N > 0 caps the grid at N workgroups.
#ifndef DR_GRID_CAP
#define DR_GRID_CAP 0
#endif
// Nontemporal (streaming) hints on the source loads / destination stores.
#ifndef DR_NT_LOADS
#define DR_NT_LOADS 1
#endif
#ifndef DR_NT_STORES
#define DR_NT_STORES 1
#endif
#ifndef DR_THREADS
#define DR_THREADS 256
#endif
constexpr int kThreads = DR_THREADS;
constexpr int kVecItersSmall = 2;
constexpr int kVecItersLarge = 4;
constexpr int kReshardIters = 4;
constexpr int kScalarIters = 8;
constexpr uint32_t kXcds = 8;  // MI355X: workgroup b is dispatched to XCD b % 8
constexpr uint32_t kScalarUnitsPerTile = kThreads * kScalarIters;  // single elements
// Largest tile-kernel grid: a launch holds at most 2^32 - 1 lanes in x.  Grids
// this large stride over the tiles; a multiple of kXcds keeps every tile a
// workgroup visits on that workgroup's XCD.
constexpr uint32_t kMaxGrid = (0xFFFFFFFFu / kThreads) / kXcds * kXcds;

// Segment-table row as the kernels read it (64 bytes, one scalar load).
// Offsets within a segment fit in 32 bits: the planner keeps rows*cols at most
// 2^30 and the source span (rows-1)*stride+cols at most 2^31.
struct DevSeg {
  uint64_t dst;        // first element in the output stream
  uint64_t src;        // first element within the source shard
  uint32_t shard;      // source shard
  uint32_t chunk;
  uint32_t rows;
  uint32_t cols;       // elements per row (run length)
  uint32_t stride;     // source elements between row starts
  uint32_t magic;      // floor(2^32 / cols), clamped to 2^32-1 (division by cols)
  uint32_t units;      // vec: rows*cols/4; scalar: rows*cols
  uint32_t flags;      // DR_SEG_VEC4
  uint32_t dst_shard;  // destination shard (reshard plans; 0 for the rollout stream)
  uint32_t op;         // DR_OP_*
  uint64_t reserved;
};
static_assert(sizeof(DevSeg) == 64, "DevSeg layout");

struct Tile {
  uint32_t seg;    // segment index
  uint32_t unit0;  // first unit of the tile within the segment
};

// Per-chunk checksums.  Each tile adds its (s1, s2) with two atomic adds
// (nothing waits for them) into one of `sub` accumulator slots of its chunk,
// slot g % sub for tile g; a small kernel that runs after the tile kernel adds
// a chunk's slots, writes the checksum and sets the slots back to zero, so
// they are zero between launches.  Slots of chunk c start at slot
// (c - chunk_bias) * sub and lie stride_words 64-bit words apart.  How many
// slots, and how far apart, is the host's choice (a plan's tiling): adds to
// one cache line are performed one after another, so the slots spread the
// adds of a chunk's concurrent tiles over lines.
constexpr uint32_t kMaxSumSlots = 256;
constexpr uint32_t kSlotLineWords = 16;  // 128-byte line

struct ChunkSum {
  uint64_t* acc;         // (s1, s2) accumulators
  dr_checksum* out;      // checksum of chunk c at out[c - out_chunk0]
  uint32_t sub;          // slots per chunk (1 .. kMaxSumSlots, a power of two)
  uint32_t stride_words; // 64-bit words between consecutive slots (2 or kSlotLineWords)
  uint32_t out_chunk0;
  uint32_t chunk_bias;
};

}  // namespace dr
