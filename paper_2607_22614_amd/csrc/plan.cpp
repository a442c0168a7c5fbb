// Layout planner: compiles (model shape, W shards, T ranks, chunk budget B)
// into the segment table the stage kernel walks, plus its workgroup tiles.
//
// The rollout stream is described as a list of "runs": rows x cols elements
// written densely at a stream offset, row i read from the training flat buffer
// at src + i*stride.  Row-sliced tensors (embed, q/k/v rows of a rank's heads,
// gate/up rows, lm_head, norms) are single contiguous runs; column-sliced
// tensors (o, down) are strided runs.  Runs are then cut at every shard
// boundary (so each reads one shard) and at every chunk boundary (so each
// writes one chunk), and capped so that in-segment offsets fit in 32 bits.
// This compiled table is the per-topology metadata the paper caches so that a
// switch only binds and activates (Sec. 3.2).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "dr_internal.h"

namespace dr {
namespace {

struct Run {
  uint64_t dst, src, stride, rows, cols;
};

constexpr uint64_t kMaxElemsPerSeg = 1ull << 30;
constexpr uint64_t kMaxSrcSpan = 1ull << 31;
constexpr uint64_t kMaxTotalElems = 1ull << 47;
constexpr uint64_t kMaxChunks = 1ull << 24;

bool mul(uint64_t a, uint64_t b, uint64_t* out) {
  if (a != 0 && b > UINT64_MAX / a) return false;
  *out = a * b;
  return true;
}

Run take_rows(const Run& r, uint64_t k) { return Run{r.dst, r.src, r.stride, k, r.cols}; }

void advance(Run& r, uint64_t k) {
  r.dst += k * r.cols;
  r.src += k * r.stride;
  r.rows -= k;
}

// Cuts `in` at every multiple of `period` of its source positions (on_src) or
// of its destination positions.  Output runs keep stream order.
void split_runs(const Run& in, uint64_t period, bool on_src, std::vector<Run>& out) {
  Run cur = in;
  while (cur.rows > 0) {
    const uint64_t base = on_src ? cur.src : cur.dst;
    const uint64_t step = on_src ? cur.stride : cur.cols;
    const uint64_t boundary = (base / period + 1) * period;
    if (base + cur.cols <= boundary) {
      // rows i with base + i*step + cols <= boundary end before it
      uint64_t k = 1;
      if (cur.rows > 1) k = std::min<uint64_t>(cur.rows, (boundary - base - cur.cols) / step + 1);
      out.push_back(take_rows(cur, k));
      advance(cur, k);
      continue;
    }
    // the first row crosses one or more boundaries: cut it at each
    uint64_t pos = 0;
    while (pos < cur.cols) {
      const uint64_t here = base + pos;
      const uint64_t next = (here / period + 1) * period;
      const uint64_t len = std::min<uint64_t>(cur.cols - pos, next - here);
      out.push_back(Run{cur.dst + pos, cur.src + pos, len, 1, len});
      pos += len;
    }
    advance(cur, 1);
  }
}

// Caps a run so that rows*cols <= 2^30 and its source span (rows-1)*stride + cols
// <= 2^31: every in-segment element offset (< 2^30) and source offset (< 2^31)
// then fits the kernels' 32-bit arithmetic.
void cap_run(const Run& in, std::vector<Run>& out) {
  if (in.rows == 1 || in.cols > kMaxElemsPerSeg / 2) {
    for (uint64_t i = 0; i < in.rows; ++i) {
      for (uint64_t pos = 0; pos < in.cols; pos += kMaxElemsPerSeg) {
        const uint64_t len = std::min<uint64_t>(kMaxElemsPerSeg, in.cols - pos);
        out.push_back(Run{in.dst + i * in.cols + pos, in.src + i * in.stride + pos, len, 1, len});
      }
    }
    return;
  }
  const uint64_t by_elems = kMaxElemsPerSeg / in.cols;
  const uint64_t by_span = (kMaxSrcSpan - in.cols) / in.stride + 1;
  const uint64_t g = std::max<uint64_t>(1, std::min(by_elems, by_span));
  Run cur = in;
  while (cur.rows > 0) {
    const uint64_t k = std::min(g, cur.rows);
    out.push_back(take_rows(cur, k));
    advance(cur, k);
  }
}

int validate(const dr_model* m, const dr_layout* l) {
  if (!m || !l) return fail(DR_EINVAL, "null model or layout");
  const int32_t f[7] = {m->n_layers, m->hidden, m->n_q_heads, m->n_kv_heads, m->head_dim, m->ffn, m->vocab};
  static const char* names[7] = {"n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "vocab"};
  for (int i = 0; i < 7; ++i)
    if (f[i] < (i == 0 ? 0 : 1))  // no layers is allowed: embed, final_norm and lm_head alone
      return fail(DR_EINVAL, "model.%s must be %s (got %d)", names[i], i == 0 ? ">= 0" : "> 0", f[i]);
  if (m->hidden % 8) return fail(DR_EINVAL, "hidden (%d) must be a multiple of 8", m->hidden);
  if (m->n_q_heads % m->n_kv_heads)
    return fail(DR_EINVAL, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", m->n_q_heads, m->n_kv_heads);
  if (l->train_shards < 1 || l->train_shards > DR_MAX_SHARDS)
    return fail(DR_EINVAL, "train_shards must be in [1, %d] (got %d)", DR_MAX_SHARDS, l->train_shards);
  if (l->tp < 1) return fail(DR_EINVAL, "tp must be >= 1 (got %d)", l->tp);
  const int32_t t = l->tp;
  if (m->n_q_heads % t) return fail(DR_EINVAL, "tp (%d) must divide n_q_heads (%d)", t, m->n_q_heads);
  if (m->n_kv_heads % t) return fail(DR_EINVAL, "tp (%d) must divide n_kv_heads (%d)", t, m->n_kv_heads);
  if (m->ffn % t) return fail(DR_EINVAL, "tp (%d) must divide ffn (%d)", t, m->ffn);
  if (m->vocab % t) return fail(DR_EINVAL, "tp (%d) must divide vocab (%d)", t, m->vocab);
  if (l->chunk_bytes < 16 || l->chunk_bytes % 16)
    return fail(DR_EINVAL, "chunk_bytes must be a positive multiple of 16 (got %llu)",
                (unsigned long long)l->chunk_bytes);
  if (l->moment_chunk_bytes % 16)
    return fail(DR_EINVAL, "moment_chunk_bytes must be 0 or a multiple of 16 (got %llu)",
                (unsigned long long)l->moment_chunk_bytes);
  if (l->tile_depth != DR_TILE_DEPTH_AUTO && l->tile_depth != kVecItersSmall && l->tile_depth != kVecItersLarge)
    return fail(DR_EINVAL, "tile_depth must be 0 (automatic), %d or %d (got %d)", kVecItersSmall, kVecItersLarge,
                l->tile_depth);
  if (l->reserved) return fail(DR_EINVAL, "dr_layout.reserved must be 0");
  if ((uint64_t)m->n_q_heads * (uint64_t)m->head_dim >= kMaxSrcSpan)
    return fail(DR_EINVAL, "n_q_heads * head_dim must be below 2^31");
  return DR_OK;
}

// Element counts of the model's tensors, with overflow checks: V*H, Hq*D*H,
// Hkv*D*H, F*H and N, the unpadded training element count.
int model_sizes(const dr_model* m, uint64_t* VH, uint64_t* qdH, uint64_t* kdH, uint64_t* FH, uint64_t* N) {
  const uint64_t L = m->n_layers, H = m->hidden, Hq = m->n_q_heads, Hkv = m->n_kv_heads, D = m->head_dim,
                 F = m->ffn, V = m->vocab;
  if (!mul(V, H, VH) || !mul(Hq * D, H, qdH) || !mul(Hkv * D, H, kdH) || !mul(F, H, FH))
    return fail(DR_EINVAL, "model too large");
  uint64_t per_layer = 2 * H;
  for (uint64_t x : {*qdH, *kdH, *kdH, *qdH, *FH, *FH, *FH}) {
    if (per_layer > kMaxTotalElems || x > kMaxTotalElems) return fail(DR_EINVAL, "model too large");
    per_layer += x;
  }
  uint64_t layers_total;
  if (!mul(per_layer, L, &layers_total) || layers_total > kMaxTotalElems || *VH > kMaxTotalElems)
    return fail(DR_EINVAL, "model too large");
  *N = 2 * *VH + layers_total + H;
  if (*N > kMaxTotalElems) return fail(DR_EINVAL, "model too large (%llu elements)", (unsigned long long)*N);
  return DR_OK;
}

void add_tensor(dr_plan* p, const std::string& name, int rank, int ndim, uint64_t off, uint64_t rows, uint64_t cols) {
  p->tensors.push_back(TensorDesc{name, rank, ndim, off, (int64_t)rows, (int64_t)cols});
}

// The tiles of every segment in order at tile depth K (vector segments: kThreads*K
// groups of 4 elements per tile; scalar ones: kScalarUnitsPerTile elements) and the
// chunk -> first-tile index.  Refuses, before allocating, kMaxTiles tiles or more.
int build_tiling(const std::vector<DevSeg>& segs, int K, uint64_t num_chunks, Tiling* out) {
  const uint32_t vec_per = (uint32_t)(kThreads * K);
  uint64_t ntiles = 0;
  for (const DevSeg& s : segs) {
    const uint32_t per = (s.flags & DR_SEG_VEC4) ? vec_per : kScalarUnitsPerTile;
    ntiles += (s.units + per - 1) / per;
  }
  if (ntiles >= kMaxTiles)
    return fail(DR_EINVAL, "too many tiles (%llu; the limit is 2^32 - 2^24)", (unsigned long long)ntiles);
  out->depth = K;
  out->tiles.clear();
  out->tiles.reserve(ntiles);
  out->chunk_tile_begin.assign(num_chunks + 1, 0);
  uint64_t next_chunk = 0;
  for (uint32_t i = 0; i < (uint32_t)segs.size(); ++i) {
    const DevSeg& s = segs[i];
    while (next_chunk <= s.chunk) out->chunk_tile_begin[next_chunk++] = (uint32_t)out->tiles.size();
    const uint32_t per = (s.flags & DR_SEG_VEC4) ? vec_per : kScalarUnitsPerTile;
    for (uint64_t u = 0; u < s.units; u += per) out->tiles.push_back(Tile{i, (uint32_t)u});
  }
  while (next_chunk <= num_chunks) out->chunk_tile_begin[next_chunk++] = (uint32_t)out->tiles.size();
  out->max_chunk_tiles = 0;
  for (uint64_t c = 0; c < num_chunks; ++c)
    out->max_chunk_tiles = std::max(out->max_chunk_tiles, out->chunk_tile_begin[c + 1] - out->chunk_tile_begin[c]);
  out->sum_slots = sum_slots(out->max_chunk_tiles);
  out->sum_stride = sum_stride(out->sum_slots, out->max_chunk_tiles);
  return DR_OK;
}

// Device bytes of the plan's tables: segments, and for every tiling its tiles, chunk index and
// checksum accumulators.  Each tiling has its own accumulators, so launches with different
// tilings never share one.
uint64_t table_bytes(dr_plan* p) {
  uint64_t b = (p->segs.size() + p->moment_segs.size()) * sizeof(DevSeg);
  for_each_tiling(p, [&](const Tiling& t) {
    b += t.tiles.size() * sizeof(Tile) + t.chunk_tile_begin.size() * sizeof(uint32_t) +
         (t.chunk_tile_begin.size() - 1) * t.sum_slots * t.sum_stride * 8;
  });
  return b;
}

// The moment stream (2W pieces of S fp32 elements: m_0..m_{W-1}, v_0..v_{W-1}) cut at every piece
// boundary and every Bm-byte chunk boundary, for the checksums of the moment chunks.  S is a
// multiple of 256 and Bm of 16 bytes, so every run is whole groups of 4 elements.
int build_moment_table(dr_plan* p, uint64_t W, uint64_t S, uint64_t Bm, uint64_t num_chunks) {
  const uint64_t total = 2 * W * S, chunk_elems = Bm / 4;
  std::vector<Run> pieces, chunks, capped;
  split_runs(Run{0, 0, total, 1, total}, S, true, pieces);
  for (const Run& r : pieces) split_runs(r, chunk_elems, false, chunks);
  for (const Run& r : chunks) cap_run(r, capped);
  p->moment_segs.clear();
  p->moment_segs.reserve(capped.size());
  for (const Run& r : capped) {
    DevSeg s{};
    s.dst = r.dst;
    s.shard = (uint32_t)(r.src / S);
    s.src = r.src - (uint64_t)s.shard * S;
    s.chunk = (uint32_t)(r.dst / chunk_elems);
    s.rows = 1;
    s.cols = (uint32_t)r.cols;
    s.stride = s.cols;
    if (s.src % 4 || s.dst % 4 || s.cols % 4) return fail(DR_EINVAL, "internal: unaligned moment segment");
    s.flags = DR_SEG_VEC4;
    s.units = s.cols / 4;
    s.op = DR_OP_COPY_F32;
    p->moment_segs.push_back(s);
  }
  return build_tiling(p->moment_segs, kReshardIters, num_chunks, &p->moment_tiling);
}

}  // namespace

int build_plan(const dr_model* m, const dr_layout* l, dr_plan* p) {
  int rc = validate(m, l);
  if (rc) return rc;
  p->model = *m;
  p->layout = *l;

  const uint64_t L = m->n_layers, H = m->hidden, Hq = m->n_q_heads, Hkv = m->n_kv_heads, D = m->head_dim,
                 F = m->ffn, V = m->vocab, W = l->train_shards, T = l->tp;

  // ---- training layout: offsets of every tensor in the flat buffer (model order)
  uint64_t VH, qdH, kdH, FH, N;
  if (int rc2 = model_sizes(m, &VH, &qdH, &kdH, &FH, &N)) return rc2;
  const uint64_t unit = W * 256;
  const uint64_t Npad = (N + unit - 1) / unit * unit;
  const uint64_t S = Npad / W;

  struct LayerOff {
    uint64_t ln1, q, k, v, o, ln2, gate, up, down;
  };
  std::vector<LayerOff> lay(L);
  uint64_t off = 0;
  const uint64_t embed = off;
  off += VH;
  for (uint64_t i = 0; i < L; ++i) {
    LayerOff& x = lay[i];
    x.ln1 = off; off += H;
    x.q = off; off += qdH;
    x.k = off; off += kdH;
    x.v = off; off += kdH;
    x.o = off; off += qdH;
    x.ln2 = off; off += H;
    x.gate = off; off += FH;
    x.up = off; off += FH;
    x.down = off; off += FH;
  }
  const uint64_t final_norm = off;
  off += H;
  const uint64_t lm_head = off;
  off += VH;
  if (off != N) return fail(DR_EINVAL, "internal: training size mismatch");

  // ---- rollout layout: runs in stream order, rank-major
  const uint64_t qh = Hq / T, kh = Hkv / T, Fr = F / T, Vr = V / T;
  std::vector<Run> runs;
  uint64_t dst = 0;
  auto contiguous = [&](uint64_t src, uint64_t n) {
    runs.push_back(Run{dst, src, n, 1, n});
    dst += n;
  };
  auto strided = [&](uint64_t src, uint64_t stride, uint64_t rows, uint64_t cols) {
    if (stride == cols) {
      runs.push_back(Run{dst, src, rows * cols, 1, rows * cols});
    } else {
      runs.push_back(Run{dst, src, stride, rows, cols});
    }
    dst += rows * cols;
  };
  p->tensors.clear();
  for (uint64_t r = 0; r < T; ++r) {
    add_tensor(p, "embed", (int)r, 2, dst, Vr, H);
    contiguous(embed + r * Vr * H, Vr * H);
    for (uint64_t i = 0; i < L; ++i) {
      const LayerOff& x = lay[i];
      const std::string pre = "layers." + std::to_string(i) + ".";
      add_tensor(p, pre + "ln1", (int)r, 1, dst, H, 1);
      contiguous(x.ln1, H);
      add_tensor(p, pre + "qkv", (int)r, 2, dst, (qh + 2 * kh) * D, H);
      contiguous(x.q + r * qh * D * H, qh * D * H);
      contiguous(x.k + r * kh * D * H, kh * D * H);
      contiguous(x.v + r * kh * D * H, kh * D * H);
      add_tensor(p, pre + "o", (int)r, 2, dst, H, qh * D);
      strided(x.o + r * qh * D, Hq * D, H, qh * D);
      add_tensor(p, pre + "ln2", (int)r, 1, dst, H, 1);
      contiguous(x.ln2, H);
      add_tensor(p, pre + "gate_up", (int)r, 2, dst, 2 * Fr, H);
      contiguous(x.gate + r * Fr * H, Fr * H);
      contiguous(x.up + r * Fr * H, Fr * H);
      add_tensor(p, pre + "down", (int)r, 2, dst, H, Fr);
      strided(x.down + r * Fr, F, H, Fr);
    }
    add_tensor(p, "final_norm", (int)r, 1, dst, H, 1);
    contiguous(final_norm, H);
    add_tensor(p, "lm_head", (int)r, 2, dst, Vr, H);
    contiguous(lm_head + r * Vr * H, Vr * H);
  }
  const uint64_t total_elems = dst;
  const uint64_t rank_elems = total_elems / T;
  const uint64_t rollout_bytes = 2 * total_elems;
  const uint64_t B = l->chunk_bytes;
  const uint64_t num_chunks = (rollout_bytes + B - 1) / B;
  if (num_chunks > kMaxChunks)
    return fail(DR_EINVAL, "chunk_bytes %llu gives %llu chunks (limit %llu)", (unsigned long long)B,
                (unsigned long long)num_chunks, (unsigned long long)kMaxChunks);
  if (l->moment_chunk_bytes) {
    const uint64_t moment_chunks = (8 * Npad + l->moment_chunk_bytes - 1) / l->moment_chunk_bytes;  // m and v
    if (moment_chunks > kMaxChunks)
      return fail(DR_EINVAL, "moment_chunk_bytes %llu gives %llu moment chunks (limit %llu)",
                  (unsigned long long)l->moment_chunk_bytes, (unsigned long long)moment_chunks,
                  (unsigned long long)kMaxChunks);
  }
  const uint64_t chunk_elems = B / 2;

  // ---- cut at shard boundaries (source side), then chunk boundaries (stream side)
  std::vector<Run> by_shard, by_chunk, capped;
  by_shard.reserve(runs.size() * 2);
  for (const Run& r : runs) split_runs(r, S, true, by_shard);
  by_chunk.reserve(by_shard.size() + num_chunks * 2);
  for (const Run& r : by_shard) split_runs(r, chunk_elems, false, by_chunk);
  capped.reserve(by_chunk.size());
  for (const Run& r : by_chunk) cap_run(r, capped);

  // ---- segment table and tiles
  const uint64_t footprint = 4 * N + rollout_bytes;
  int depth = l->tile_depth, deep = 0;
  if (depth == DR_TILE_DEPTH_AUTO) {
    depth = footprint > kLargeFootprint ? kVecItersLarge : kVecItersSmall;
    if (depth == kVecItersSmall) deep = kVecItersLarge;
  }
  p->segs.clear();
  p->segs.reserve(capped.size());
  for (const Run& r : capped) {
    DevSeg s{};
    s.dst = r.dst;
    s.shard = (uint32_t)(r.src / S);
    s.src = r.src - (uint64_t)s.shard * S;
    s.chunk = (uint32_t)(r.dst / chunk_elems);
    s.rows = (uint32_t)r.rows;
    s.cols = (uint32_t)r.cols;
    s.stride = (uint32_t)(r.rows > 1 ? r.stride : r.cols);
    s.magic = s.cols == 1 ? 0xFFFFFFFFu : (uint32_t)((1ull << 32) / s.cols);
    const bool vec = s.src % 4 == 0 && s.dst % 4 == 0 && s.cols % 4 == 0 && (s.rows == 1 || s.stride % 4 == 0);
    s.flags = vec ? DR_SEG_VEC4 : 0;
    s.op = DR_OP_CAST_BF16;
    const uint64_t elems = r.rows * r.cols;
    s.units = (uint32_t)(vec ? elems / 4 : elems);
    p->segs.push_back(s);
  }
  p->tiling[1] = Tiling{};
  if (int rc = build_tiling(p->segs, depth, num_chunks, &p->tiling[0])) return rc;
  if (deep)
    if (int rc = build_tiling(p->segs, deep, num_chunks, &p->tiling[1])) return rc;
  p->moment_segs.clear();
  p->moment_tiling = Tiling{};
  if (l->moment_chunk_bytes) {
    const uint64_t Bm = l->moment_chunk_bytes;
    if (int rc = build_moment_table(p, W, S, Bm, (8 * Npad + Bm - 1) / Bm)) return rc;
  }

  // ---- info
  dr_plan_info& in = p->info;
  std::memset(&in, 0, sizeof(in));
  in.n_elems = N;
  in.padded_elems = Npad;
  in.shard_elems = S;
  in.norm_elems = (2 * L + 1) * H;
  in.rank_elems = rank_elems;
  in.rollout_bytes = rollout_bytes;
  in.num_chunks = num_chunks;
  in.last_chunk_bytes = rollout_bytes - (num_chunks - 1) * B;
  if (l->moment_chunk_bytes) {
    in.moment_bytes = 2 * W * S * 4;
    in.num_moment_chunks = (in.moment_bytes + l->moment_chunk_bytes - 1) / l->moment_chunk_bytes;
  }
  in.num_segments = p->segs.size();
  in.num_tiles = p->tiling[0].tiles.size();
  in.device_table_bytes = table_bytes(p);
  in.pinned_bytes = 2 * l->moment_chunk_bytes;
  in.device = -1;
  in.kind = DR_PLAN_ROLLOUT;
  in.tile_elems = 4ull * kThreads * depth;
  in.deep_tile_elems = deep ? 4ull * kThreads * deep : 0;
  in.deep_num_tiles = p->tiling[1].tiles.size();
  in.train_shards = l->train_shards;
  in.tp = l->tp;
  in.chunk_bytes = B;
  in.moment_chunk_bytes = l->moment_chunk_bytes;
  return DR_OK;
}


// Training -> training reshard: the N elements keep their flat order; the
// copy run is cut at source shard, destination shard and chunk boundaries, and
// the destination padding [N, Npad') becomes zero-fill segments.  Every
// boundary is a multiple of 4 elements (N % 8 == 0, shards are multiples of
// 256, chunks of B/4 with B % 16 == 0), so every segment moves whole 16-byte
// groups.
int build_reshard_plan(const dr_model* m, int32_t from_shards, int32_t to_shards, uint64_t chunk_bytes,
                       dr_plan* p) {
  dr_layout l{from_shards, 1, chunk_bytes, 0, DR_TILE_DEPTH_AUTO, 0};
  int rc = validate(m, &l);
  if (rc) return rc;
  if (to_shards < 1 || to_shards > DR_MAX_SHARDS)
    return fail(DR_EINVAL, "to_shards must be in [1, %d] (got %d)", DR_MAX_SHARDS, to_shards);
  uint64_t VH, qdH, kdH, FH, N;
  if ((rc = model_sizes(m, &VH, &qdH, &kdH, &FH, &N))) return rc;
  const uint64_t unit = (uint64_t)from_shards * 256;
  const uint64_t Npad = (N + unit - 1) / unit * unit, S = Npad / from_shards;
  p->model = *m;
  p->layout = l;
  const uint64_t unit2 = (uint64_t)to_shards * 256;
  const uint64_t Npad2 = (N + unit2 - 1) / unit2 * unit2, S2 = Npad2 / to_shards;
  const uint64_t out_bytes = 4 * Npad2;
  const uint64_t num_chunks = (out_bytes + chunk_bytes - 1) / chunk_bytes;
  if (num_chunks > kMaxChunks)
    return fail(DR_EINVAL, "chunk_bytes %llu gives %llu chunks (limit %llu)", (unsigned long long)chunk_bytes,
                (unsigned long long)num_chunks, (unsigned long long)kMaxChunks);
  const uint64_t chunk_elems = chunk_bytes / 4;

  std::vector<Run> a, b, c, d;
  split_runs(Run{0, 0, N, 1, N}, S, true, a);                 // source shards
  for (const Run& r : a) split_runs(r, S2, false, b);         // destination shards
  if (Npad2 > N) split_runs(Run{N, 0, Npad2 - N, 1, Npad2 - N}, S2, false, b);
  for (const Run& r : b) split_runs(r, chunk_elems, false, c);  // chunks
  for (const Run& r : c) cap_run(r, d);

  p->kind = kReshard;
  p->dst_shards = to_shards;
  p->dst_shard_elems = S2;
  p->tensors.clear();
  p->segs.clear();
  p->segs.reserve(d.size());
  for (const Run& r : d) {
    DevSeg s{};
    const bool zero = r.dst >= N;
    s.dst = r.dst;
    s.shard = zero ? 0 : (uint32_t)(r.src / S);
    s.src = zero ? 0 : r.src - (uint64_t)s.shard * S;
    s.chunk = (uint32_t)(r.dst / chunk_elems);
    s.dst_shard = (uint32_t)(r.dst / S2);
    s.rows = 1;
    s.cols = (uint32_t)r.cols;
    s.stride = s.cols;
    s.magic = 0;
    s.op = zero ? DR_OP_ZERO_F32 : DR_OP_COPY_F32;
    if (s.dst % 4 || s.src % 4 || s.cols % 4) return fail(DR_EINVAL, "internal: unaligned reshard segment");
    s.flags = DR_SEG_VEC4;
    s.units = s.cols / 4;
    p->segs.push_back(s);
  }
  p->tiling[1] = Tiling{};
  if (int rc = build_tiling(p->segs, kReshardIters, num_chunks, &p->tiling[0])) return rc;

  dr_plan_info& in = p->info;
  std::memset(&in, 0, sizeof(in));
  in.n_elems = N;
  in.padded_elems = Npad;
  in.shard_elems = S;
  in.norm_elems = (2 * (uint64_t)m->n_layers + 1) * m->hidden;
  in.rollout_bytes = out_bytes;
  in.num_chunks = num_chunks;
  in.last_chunk_bytes = out_bytes - (num_chunks - 1) * chunk_bytes;
  in.num_segments = p->segs.size();
  in.num_tiles = p->tiling[0].tiles.size();
  in.device_table_bytes = table_bytes(p);
  in.device = -1;
  in.kind = DR_PLAN_RESHARD;
  in.tile_elems = 4ull * kThreads * kReshardIters;
  in.dst_shard_elems = S2;
  in.train_shards = from_shards;
  in.dst_shards = to_shards;
  in.chunk_bytes = chunk_bytes;
  return DR_OK;
}

}  // namespace dr
