/* A plain C99 user of libdr.so: proves the boundary is usable with nothing but
 * dr.h, the HIP runtime's C API and a C compiler (no C++, no Python, no torch).
 *
 *   c_consumer IN OUT_STREAM OUT_CKS L H Hq Hkv D F V W T B Bm
 *
 * IN holds the padded flat fp32 training buffer (Npad elements, little endian).
 * The program
 *   - uploads it as W separate device shards and stages the whole rollout
 *     stream with dr_stage_all on its own HIP stream;
 *   - stages every chunk again with dr_stage_chunk into one B-byte device
 *     buffer, then with dr_stage_chunk_noalloc into the same buffer poisoned,
 *     and checks each against the dr_stage_all bytes and checksum;
 *   - if Bm > 0, offloads W moment shards (m = the weights, v = their bitwise
 *     complement) into malloc'd host memory, restores them into buffers filled
 *     with 0xFF, and checks both directions byte for byte;
 *   - checks that a bad layout is refused with DR_EINVAL and a message;
 * then writes the stream and the (s1, s2) pairs of every chunk to OUT_STREAM
 * and OUT_CKS for comparison with the CPU oracle.  Exit status 0 on success. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dr.h"

#define HIP_OK(call)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess) {                                                            \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
      exit(2);                                                                         \
    }                                                                                  \
  } while (0)

#define DR_OK_(call)                                                                   \
  do {                                                                                 \
    int rc_ = (call);                                                                  \
    if (rc_ != DR_OK) {                                                                \
      fprintf(stderr, "%s:%d %s -> %d: %s\n", __FILE__, __LINE__, #call, rc_, dr_last_error()); \
      exit(3);                                                                         \
    }                                                                                  \
  } while (0)

static void* read_file(const char* path, size_t* size) {
  FILE* f = fopen(path, "rb");
  if (!f) {
    perror(path);
    exit(4);
  }
  fseek(f, 0, SEEK_END);
  *size = (size_t)ftell(f);
  fseek(f, 0, SEEK_SET);
  void* p = malloc(*size ? *size : 1);
  if (!p || fread(p, 1, *size, f) != *size) {
    fprintf(stderr, "%s: short read\n", path);
    exit(4);
  }
  fclose(f);
  return p;
}

static void write_file(const char* path, const void* p, size_t n) {
  FILE* f = fopen(path, "wb");
  if (!f || fwrite(p, 1, n, f) != n || fclose(f) != 0) {
    perror(path);
    exit(4);
  }
}

int main(int argc, char** argv) {
  if (argc != 15) {
    fprintf(stderr, "usage: %s IN OUT_STREAM OUT_CKS L H Hq Hkv D F V W T B Bm\n", argv[0]);
    return 1;
  }
  dr_model m;
  m.n_layers = atoi(argv[4]);
  m.hidden = atoi(argv[5]);
  m.n_q_heads = atoi(argv[6]);
  m.n_kv_heads = atoi(argv[7]);
  m.head_dim = atoi(argv[8]);
  m.ffn = atoi(argv[9]);
  m.vocab = atoi(argv[10]);
  dr_layout l;
  memset(&l, 0, sizeof(l));
  l.train_shards = atoi(argv[11]);
  l.tp = atoi(argv[12]);
  l.chunk_bytes = strtoull(argv[13], NULL, 10);
  l.moment_chunk_bytes = strtoull(argv[14], NULL, 10);
  l.tile_depth = DR_TILE_DEPTH_AUTO;

  /* a refused layout: nothing allocated, a message for this thread */
  {
    dr_layout bad = l;
    bad.chunk_bytes = 24; /* not a multiple of 16 */
    dr_plan* none = NULL;
    if (dr_plan_create(&m, &bad, &none) != DR_EINVAL || none != NULL || dr_last_error()[0] == '\0') {
      fprintf(stderr, "a chunk budget of 24 bytes was not refused\n");
      return 5;
    }
  }

  dr_plan* plan = NULL;
  DR_OK_(dr_plan_create(&m, &l, &plan));
  dr_plan_info info;
  DR_OK_(dr_plan_get_info(plan, &info));
  const int W = l.train_shards;

  size_t in_bytes = 0;
  float* flat = (float*)read_file(argv[1], &in_bytes);
  if (in_bytes != info.padded_elems * 4) {
    fprintf(stderr, "input holds %zu bytes, the plan expects %llu\n", in_bytes,
            (unsigned long long)(info.padded_elems * 4));
    return 6;
  }
  const size_t S = (size_t)info.shard_elems;

  hipStream_t stream;
  HIP_OK(hipStreamCreateWithFlags(&stream, hipStreamNonBlocking));
  float* shards[DR_MAX_SHARDS];
  for (int w = 0; w < W; ++w) {
    HIP_OK(hipMalloc((void**)&shards[w], S * 4));
    HIP_OK(hipMemcpy(shards[w], flat + (size_t)w * S, S * 4, hipMemcpyHostToDevice));
  }

  /* the whole stream */
  void* d_stream = NULL;
  dr_checksum* d_cks = NULL;
  HIP_OK(hipMalloc(&d_stream, info.rollout_bytes));
  HIP_OK(hipMalloc((void**)&d_cks, info.num_chunks * sizeof(dr_checksum)));
  HIP_OK(hipMemsetAsync(d_stream, 0xFF, info.rollout_bytes, stream));
  DR_OK_(dr_stage_all(plan, (const float* const*)shards, d_stream, d_cks, stream));
  HIP_OK(hipStreamSynchronize(stream));
  unsigned char* h_stream = (unsigned char*)malloc(info.rollout_bytes);
  dr_checksum* h_cks = (dr_checksum*)malloc(info.num_chunks * sizeof(dr_checksum));
  HIP_OK(hipMemcpy(h_stream, d_stream, info.rollout_bytes, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_cks, d_cks, info.num_chunks * sizeof(dr_checksum), hipMemcpyDeviceToHost));

  /* chunk by chunk through one bounded buffer */
  void* d_chunk = NULL;
  dr_checksum* d_ck = NULL;
  unsigned char* h_chunk = (unsigned char*)malloc(l.chunk_bytes);
  HIP_OK(hipMalloc(&d_chunk, l.chunk_bytes));
  HIP_OK(hipMalloc((void**)&d_ck, sizeof(dr_checksum)));
  for (uint64_t c = 0; c < info.num_chunks; ++c) {
    const uint64_t len = c + 1 < info.num_chunks ? l.chunk_bytes : info.last_chunk_bytes;
    dr_checksum ck;
    DR_OK_(dr_stage_chunk(plan, c, (const float* const*)shards, d_chunk, d_ck, stream));
    HIP_OK(hipMemcpyAsync(h_chunk, d_chunk, len, hipMemcpyDeviceToHost, stream));
    HIP_OK(hipMemcpyAsync(&ck, d_ck, sizeof(ck), hipMemcpyDeviceToHost, stream));
    HIP_OK(hipStreamSynchronize(stream));
    if (memcmp(h_chunk, h_stream + c * l.chunk_bytes, len) != 0 || ck.s1 != h_cks[c].s1 || ck.s2 != h_cks[c].s2) {
      fprintf(stderr, "dr_stage_chunk(%llu) differs from dr_stage_all\n", (unsigned long long)c);
      return 7;
    }
    HIP_OK(hipMemsetAsync(d_chunk, 0xEE, l.chunk_bytes, stream));
    HIP_OK(hipMemsetAsync(d_ck, 0xEE, sizeof(dr_checksum), stream));
    DR_OK_(dr_stage_chunk_noalloc(plan, c, (const float* const*)shards, d_chunk, d_ck, stream));
    HIP_OK(hipMemcpyAsync(h_chunk, d_chunk, len, hipMemcpyDeviceToHost, stream));
    HIP_OK(hipMemcpyAsync(&ck, d_ck, sizeof(ck), hipMemcpyDeviceToHost, stream));
    HIP_OK(hipStreamSynchronize(stream));
    if (memcmp(h_chunk, h_stream + c * l.chunk_bytes, len) != 0 || ck.s1 != h_cks[c].s1 || ck.s2 != h_cks[c].s2) {
      fprintf(stderr, "dr_stage_chunk_noalloc(%llu) differs from dr_stage_all\n", (unsigned long long)c);
      return 7;
    }
  }
  if (dr_stage_chunk(plan, info.num_chunks, (const float* const*)shards, d_chunk, d_ck, stream) != DR_ERANGE) {
    fprintf(stderr, "a chunk past the end was not refused\n");
    return 7;
  }

  /* moments: offload to plain host memory, restore into poisoned buffers */
  if (l.moment_chunk_bytes) {
    float *mv[2][DR_MAX_SHARDS], *back[2][DR_MAX_SHARDS];
    uint32_t* comp = (uint32_t*)malloc(S * 4);
    unsigned char* store = (unsigned char*)malloc(info.moment_bytes);
    unsigned char* check = (unsigned char*)malloc(S * 4);
    hipStream_t side;
    HIP_OK(hipStreamCreateWithFlags(&side, hipStreamNonBlocking));
    for (int w = 0; w < W; ++w) {
      const uint32_t* src = (const uint32_t*)(flat + (size_t)w * S);
      for (size_t i = 0; i < S; ++i) comp[i] = ~src[i];
      for (int k = 0; k < 2; ++k) {
        HIP_OK(hipMalloc((void**)&mv[k][w], S * 4));
        HIP_OK(hipMalloc((void**)&back[k][w], S * 4));
        HIP_OK(hipMemset(back[k][w], 0xFF, S * 4));
      }
      HIP_OK(hipMemcpy(mv[0][w], src, S * 4, hipMemcpyHostToDevice));
      HIP_OK(hipMemcpy(mv[1][w], comp, S * 4, hipMemcpyHostToDevice));
    }
    DR_OK_(dr_offload_moments(plan, (const float* const*)mv[0], (const float* const*)mv[1], store, side));
    for (int k = 0; k < 2; ++k)
      for (int w = 0; w < W; ++w) {
        const unsigned char* part = store + ((size_t)k * W + w) * S * 4;
        HIP_OK(hipMemcpy(check, mv[k][w], S * 4, hipMemcpyDeviceToHost));
        if (memcmp(part, check, S * 4) != 0) {
          fprintf(stderr, "host store differs from moment %c shard %d\n", k ? 'v' : 'm', w);
          return 8;
        }
      }
    DR_OK_(dr_restore_moments(plan, store, back[0], back[1], side));
    for (int k = 0; k < 2; ++k)
      for (int w = 0; w < W; ++w) {
        HIP_OK(hipMemcpy(check, back[k][w], S * 4, hipMemcpyDeviceToHost));
        if (memcmp(store + ((size_t)k * W + w) * S * 4, check, S * 4) != 0) {
          fprintf(stderr, "restored moment %c shard %d differs\n", k ? 'v' : 'm', w);
          return 8;
        }
      }
    for (int k = 0; k < 2; ++k)
      for (int w = 0; w < W; ++w) {
        HIP_OK(hipFree(mv[k][w]));
        HIP_OK(hipFree(back[k][w]));
      }
    HIP_OK(hipStreamDestroy(side));
    free(comp);
    free(store);
    free(check);
  }

  write_file(argv[2], h_stream, info.rollout_bytes);
  write_file(argv[3], h_cks, info.num_chunks * sizeof(dr_checksum));
  printf("c_consumer ok: %llu bytes in %llu chunks\n", (unsigned long long)info.rollout_bytes,
         (unsigned long long)info.num_chunks);

  dr_plan_destroy(plan);
  for (int w = 0; w < W; ++w) HIP_OK(hipFree(shards[w]));
  HIP_OK(hipFree(d_stream));
  HIP_OK(hipFree(d_cks));
  HIP_OK(hipFree(d_chunk));
  HIP_OK(hipFree(d_ck));
  HIP_OK(hipStreamDestroy(stream));
  free(flat);
  free(h_stream);
  free(h_cks);
  free(h_chunk);
  return 0;
}
