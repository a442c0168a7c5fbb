// Host-only check of the planner under AddressSanitizer/UBSan: builds rollout
// and reshard plans for many random models and layouts and verifies, for every
// segment and tile, the invariants the kernels rely on to stay in bounds:
//   - segments are dense and ordered in the output stream and sum to its size;
//   - every source access lies inside its shard, every destination access
//     inside its chunk (and destination shard for reshard plans);
//   - in-segment offsets fit the kernels' 32-bit arithmetic (rows*cols <= 2^30,
//     source span <= 2^31);
//   - tiles cover every unit of every segment exactly once, in order, and the
//     chunk -> first-tile index brackets each chunk's tiles.
// Exit status 0 when all plans pass.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <random>

#include "dr_internal.h"

// Plans built here hold host tables only (no device memory, streams or threads).
dr_plan::~dr_plan() {}

namespace dr {
int fail(int code, const char* fmt, ...) {
  (void)fmt;
  return code;
}
void clear_error() {}
}  // namespace dr

using namespace dr;

static int errors = 0;
#define CHECK(c, ...)                                   \
  do {                                                  \
    if (!(c)) {                                         \
      if (errors < 20) {                                \
        std::fprintf(stderr, "FAIL %s: ", #c);          \
        std::fprintf(stderr, __VA_ARGS__);              \
        std::fprintf(stderr, "\n");                     \
      }                                                 \
      ++errors;                                         \
    }                                                   \
  } while (0)

static void check_plan(const dr_plan& p, bool reshard) {
  const uint64_t S = p.info.shard_elems, total_elems = p.info.rollout_bytes / (reshard ? 4 : 2);
  const uint64_t ce = p.layout.chunk_bytes / (reshard ? 4 : 2);
  uint64_t pos = 0;
  for (size_t i = 0; i < p.segs.size(); ++i) {
    const DevSeg& s = p.segs[i];
    const uint64_t n = (uint64_t)s.rows * s.cols;
    CHECK(s.dst == pos, "segment %zu not dense", i);
    pos += n;
    CHECK(n > 0 && n <= (1ull << 30), "segment %zu size %llu", i, (unsigned long long)n);
    CHECK(s.chunk == s.dst / ce && (s.dst + n - 1) / ce == s.chunk, "segment %zu crosses a chunk", i);
    if (s.op != DR_OP_ZERO_F32) {
      CHECK(s.shard < (uint32_t)p.layout.train_shards, "segment %zu shard", i);
      const uint64_t span = (uint64_t)(s.rows - 1) * s.stride + s.cols;
      CHECK(span <= (1ull << 31), "segment %zu source span", i);
      CHECK(s.src + span <= S, "segment %zu leaves its shard", i);
      CHECK(s.rows == 1 || s.stride >= s.cols, "segment %zu stride", i);
    }
    if (reshard) {
      const uint64_t S2 = p.dst_shard_elems;
      CHECK(s.dst_shard == s.dst / S2 && (s.dst + n - 1) / S2 == s.dst_shard, "segment %zu crosses a dst shard", i);
    }
    const bool vec = s.flags & DR_SEG_VEC4;
    CHECK(s.units == (vec ? n / 4 : n), "segment %zu units", i);
    if (vec) CHECK(s.src % 4 == 0 && s.dst % 4 == 0 && s.cols % 4 == 0 && (s.rows == 1 || s.stride % 4 == 0),
                   "segment %zu vec alignment", i);
    if (s.rows > 1) {
      const uint32_t magic = s.cols == 1 ? 0xFFFFFFFFu : (uint32_t)((1ull << 32) / s.cols);
      CHECK(s.magic == magic, "segment %zu magic", i);
    }
  }
  CHECK(pos == total_elems, "stream size %llu vs %llu", (unsigned long long)pos, (unsigned long long)total_elems);
  // tiles of every tiling: every unit once, in order; chunk index brackets
  CHECK(p.tiling[0].depth == (reshard ? kReshardIters : (int)(p.info.tile_elems / (4 * kThreads))), "depth");
  CHECK(p.tiling[0].tiles.size() == p.info.num_tiles, "num_tiles");
  CHECK(p.tiling[1].tiles.size() == p.info.deep_num_tiles, "deep_num_tiles");
  CHECK(p.info.deep_tile_elems == (p.tiling[1].depth ? 4ull * kThreads * p.tiling[1].depth : 0), "deep_tile_elems");
  if (p.tiling[1].depth) CHECK(!reshard && p.tiling[0].depth == kVecItersSmall && p.tiling[1].depth == kVecItersLarge,
                               "second tiling");
  for (const Tiling& tl : p.tiling) {
    if (!tl.depth) {
      CHECK(tl.tiles.empty() && tl.chunk_tile_begin.empty(), "empty tiling");
      continue;
    }
    size_t t = 0;
    for (uint32_t i = 0; i < (uint32_t)p.segs.size(); ++i) {
      const DevSeg& s = p.segs[i];
      const uint32_t per = (s.flags & DR_SEG_VEC4) ? (uint32_t)(kThreads * tl.depth) : kScalarUnitsPerTile;
      for (uint64_t u = 0; u < s.units; u += per, ++t) {
        CHECK(t < tl.tiles.size() && tl.tiles[t].seg == i && tl.tiles[t].unit0 == u, "tile %zu", t);
        CHECK(tl.chunk_tile_begin[s.chunk] <= t && t < tl.chunk_tile_begin[s.chunk + 1], "tile %zu chunk index", t);
      }
    }
    CHECK(t == tl.tiles.size(), "tile count");
    uint32_t most = 0;
    for (uint64_t c = 0; c < p.info.num_chunks; ++c)
      most = std::max(most, tl.chunk_tile_begin[c + 1] - tl.chunk_tile_begin[c]);
    CHECK(tl.max_chunk_tiles == most, "max_chunk_tiles %u vs %u", tl.max_chunk_tiles, most);
    // accumulator slots per chunk: a power of two, at most kMaxSumSlots, about kTilesPerSumLine
    // tiles per slot; a line each unless the chunks are small enough to share one
    const uint32_t s = tl.sum_slots;
    CHECK(s >= 1 && s <= kMaxSumSlots && (s & (s - 1)) == 0, "sum slots %u", s);
    CHECK(s == kMaxSumSlots || (uint64_t)s * kTilesPerSumLine >= most, "sum slots %u for %u tiles", s, most);
    CHECK(s == 1 || (uint64_t)s * kTilesPerSumLine < 2ull * most, "sum slots %u for only %u tiles", s, most);
    CHECK(tl.sum_stride == (s > 1 || most > kPackedSlotTiles ? kSlotLineWords : 2u), "sum stride %u",
          tl.sum_stride);
    CHECK(tl.sum_stride == 2 || (uint64_t)most <= (uint64_t)s * kTilesPerSumLine || s == kMaxSumSlots,
          "tiles per line");
    CHECK(tl.chunk_tile_begin.size() == p.info.num_chunks + 1 && tl.chunk_tile_begin.back() == tl.tiles.size(),
          "chunk index size");
  }
}

// The moment table: the moment stream (2W pieces of S elements) covered once, in order, by
// segments inside one piece and one Bm-byte chunk; its tiling covers every unit once.
void check_moments(const dr_plan& p) {
  const uint64_t Bm = p.layout.moment_chunk_bytes;
  if (!Bm) {
    CHECK(p.moment_segs.empty() && !p.moment_tiling.depth, "moment table without a moment path");
    return;
  }
  const uint64_t S = p.info.shard_elems, W = p.layout.train_shards, ce = Bm / 4;
  CHECK(p.info.moment_bytes == 8 * W * S, "moment bytes");
  uint64_t pos = 0;
  for (size_t i = 0; i < p.moment_segs.size(); ++i) {
    const DevSeg& s = p.moment_segs[i];
    CHECK(s.dst == pos && s.rows == 1 && s.cols > 0 && s.cols <= (1u << 30), "moment segment %zu", i);
    CHECK(s.shard == s.dst / S && s.src == s.dst - (uint64_t)s.shard * S && s.src + s.cols <= S,
          "moment segment %zu piece", i);
    CHECK(s.chunk == s.dst / ce && (s.dst + s.cols - 1) / ce == s.chunk, "moment segment %zu chunk", i);
    CHECK((s.flags & DR_SEG_VEC4) && s.units == s.cols / 4 && s.cols % 4 == 0 && s.src % 4 == 0,
          "moment segment %zu alignment", i);
    pos += s.cols;
  }
  CHECK(pos == 2 * W * S, "moment stream %llu vs %llu", (unsigned long long)pos, (unsigned long long)(2 * W * S));
  const Tiling& tl = p.moment_tiling;
  CHECK(tl.depth == kReshardIters && tl.chunk_tile_begin.size() == p.info.num_moment_chunks + 1, "moment tiling");
  size_t t = 0;
  for (uint32_t i = 0; i < (uint32_t)p.moment_segs.size(); ++i) {
    const DevSeg& s = p.moment_segs[i];
    for (uint64_t u = 0; u < s.units; u += kThreads * tl.depth, ++t) {
      CHECK(t < tl.tiles.size() && tl.tiles[t].seg == i && tl.tiles[t].unit0 == u, "moment tile %zu", t);
      CHECK(tl.chunk_tile_begin[s.chunk] <= t && t < tl.chunk_tile_begin[s.chunk + 1], "moment tile %zu chunk", t);
    }
  }
  CHECK(t == tl.tiles.size() && tl.chunk_tile_begin.back() == t, "moment tile count");
  CHECK(tl.sum_slots >= 1 && tl.sum_slots <= kMaxSumSlots, "moment sum slots");
}

int main(int argc, char** argv) {
  const int n = argc > 1 ? std::atoi(argv[1]) : 300;
  std::mt19937_64 rng(12345);
  auto pick = [&](std::initializer_list<int> xs) { return xs.begin()[rng() % xs.size()]; };
  int plans = 0;
  for (int it = 0; it < n; ++it) {
    dr_model m{pick({0, 1, 2, 3}), 8 * pick({1, 2, 3, 5, 8}), pick({1, 2, 4, 6, 8}), 1, pick({1, 2, 3, 4, 8, 64}),
               pick({4, 6, 8, 12, 24, 40}), pick({4, 8, 16, 24, 96})};
    const int kv[] = {1, 2, 4};
    m.n_kv_heads = kv[rng() % 3];
    if (m.n_q_heads % m.n_kv_heads) m.n_kv_heads = 1;
    const int W = pick({1, 2, 3, 4, 7, 8, 64});
    const int T = pick({1, 2, 3, 4, 8});
    const uint64_t B = 16ull * pick({1, 2, 3, 7, 64, 1000, 65536});
    dr_plan p;
    const uint64_t Bm = 16ull * pick({0, 1, 3, 7, 64, 1000, 65536});
    dr_layout l{W, T, B, Bm, pick({0, 2, 4}), 0};
    if (build_plan(&m, &l, &p) == DR_OK) {
      check_plan(p, false);
      check_moments(p);
      ++plans;
    }
    dr_plan q;
    if (build_reshard_plan(&m, W, pick({1, 2, 5, 8, 64}), B, &q) == DR_OK) {
      check_plan(q, true);
      ++plans;
    }
  }
  // the five workloads' shapes at their real sizes (tables only, no data)
  const dr_model shapes[] = {{2, 256, 4, 4, 64, 688, 2048}, {24, 896, 14, 2, 64, 4864, 151936},
                             {32, 4096, 32, 8, 128, 14336, 128256}, {64, 5120, 40, 8, 128, 27648, 152064}};
  const dr_layout lays[] = {{4, 2, 256 << 10, 0}, {8, 1, 64 << 20, 0}, {8, 4, 256 << 20, 0}, {1, 8, 1ull << 30, 0},
                            {8, 4, 256 << 20, 512 << 20}};
  for (int i = 0; i < 5; ++i) {
    dr_plan p;
    CHECK(build_plan(&shapes[i < 4 ? i : 2], &lays[i], &p) == DR_OK, "workload %d", i);
    check_plan(p, false);
    check_moments(p);
    ++plans;
  }
  // a decoder large enough that the planner's run caps split runs: embed and lm_head hold
  // 2^32 elements (> 2^30 per segment) and down's column slice spans 2^31 source elements
  {
    const dr_model big{1, 16384, 128, 8, 128, 131072, 262144};
    for (int depth : {0, 4}) {
      dr_plan p;
      const dr_layout l{1, 2, 1ull << 34, 0, depth, 0};
      CHECK(build_plan(&big, &l, &p) == DR_OK, "capped model, depth %d", depth);
      check_plan(p, false);
      size_t embed_segs = 0;
      for (const DevSeg& s : p.segs) embed_segs += s.dst < (uint64_t)131072 * 16384;
      CHECK(embed_segs > 1, "rank 0 embed was not split by the segment cap (%zu segments)", embed_segs);
      ++plans;
    }
    dr_plan q;
    CHECK(build_reshard_plan(&big, 1, 3, 1ull << 34, &q) == DR_OK, "capped model, reshard");
    check_plan(q, true);
    ++plans;
  }
  // the automatic depth's drain clock, in nanoseconds: the 8B pack (48.18 GB) lasts 7.41 ms at 6.5 TB/s
  {
    const int64_t t0 = 1000000000000;
    const int64_t d = pack_drain_ns(t0, 0, 48183164928ull) - t0;
    CHECK(d > 7400000 && d < 7420000, "8B pack estimate %lld ns", (long long)d);
    CHECK(pack_drain_ns(t0, t0 + 5, 0) == t0 + 5, "queued behind a later drain time");
    CHECK(!pack_is_hot(t0, 0), "no earlier pack");
    CHECK(pack_is_hot(t0, t0 + 1000000), "previous pack still draining");
    CHECK(pack_is_hot(t0 + kHotGapNs, t0), "at the gap");
    CHECK(!pack_is_hot(t0 + kHotGapNs + 1, t0), "past the gap");
  }
  std::printf("%d plans checked, %d errors\n", plans, errors);
  return errors ? 1 : 0;
}
