// dr_stage_chunk_noalloc: dr_stage_chunk for callers that cannot allocate
// device memory (code under graph capture, tight serving loops, harnesses that
// forbid allocation).  The chunk's checksum accumulators live in a fixed
// file-scope device array, one copy per GPU held until the process ends,
// instead of the plan's accumulators; the kernels are the same.
//
// The first call on a GPU clears the array with a small kernel, and every call
// leaves it at zero again: the chunk-sum kernel clears each slot it reads.  A
// call that fails after its stage kernel may have run marks the GPU's array
// again.  While the array is marked, calls clear it before staging, until one
// that is not being recorded into a graph has done so.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "dr_internal.h"
#include "kernels.h"

namespace dr {
namespace {

// The accumulator slots of one chunk: at most kMaxSumSlots slots, a 128-byte
// line each (32 KiB).
constexpr size_t kScratchBytes = (size_t)kMaxSumSlots * kSlotLineWords * sizeof(uint64_t);
static __device__ __align__(256) uint64_t scratch[kScratchBytes / sizeof(uint64_t)];

constexpr int kMaxDevices = 64;
uint64_t* g_scratch[kMaxDevices];  // each device's copy of `scratch`, as a device address
std::atomic<bool> g_dirty[kMaxDevices];  // the slots there may be nonzero: clear before use
std::mutex g_scratch_mu;

}  // namespace

// The device address of this device's copy of `scratch`, looked up once per device with that
// device current (the array's name in host code is not a device address).  Plan set-up calls it,
// so the entry point finds the address already known, also when its first call is recorded.
int scratch_on(int dev, uint64_t** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DR_EINVAL, "static scratch of dr_stage_chunk_noalloc: device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(DR_EHIP, "static scratch of dr_stage_chunk_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch[dev] = static_cast<uint64_t*>(ptr);
    g_dirty[dev] = true;  // the first call clears the array
  }
  *out = g_scratch[dev];
  return DR_OK;
}

namespace {

// Sets n 64-bit words to zero (a kernel rather than a memset, so the call stays recordable in a graph).
__global__ __launch_bounds__(256) void zero_words(uint64_t* p, uint32_t n) {
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

}  // namespace
}  // namespace dr

using namespace dr;

extern "C" int dr_stage_chunk_noalloc(dr_plan* p, uint64_t chunk, const float* const* shards, void* dst_chunk,
                                      dr_checksum* d_ck, void* stream) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_stage_chunk_noalloc: null plan");
  if (p->kind != kRollout) return fail(DR_EINVAL, "dr_stage_chunk_noalloc: not a rollout plan");
  if (chunk >= p->info.num_chunks)
    return fail(DR_ERANGE, "dr_stage_chunk_noalloc: chunk %llu >= num_chunks %llu", (unsigned long long)chunk,
                (unsigned long long)p->info.num_chunks);
  if (int rc = check_stage_args(p, shards, dst_chunk, d_ck, "dr_stage_chunk_noalloc")) return rc;
  const Tiling& tl = chunk_launch_tiling(p);
  const uint64_t words = (uint64_t)tl.sum_slots * tl.sum_stride;
  if (words * sizeof(uint64_t) > kScratchBytes)
    return fail(DR_EINVAL, "dr_stage_chunk_noalloc: %llu bytes of checksum slots exceed the %zu-byte static scratch",
                (unsigned long long)(words * sizeof(uint64_t)), kScratchBytes);
  uint64_t* ptr = nullptr;
  if (int rc = scratch_on(p->device, &ptr)) return rc;
  ChunkSum cs{};
  cs.acc = ptr;
  cs.out = d_ck;
  cs.sub = tl.sum_slots;
  cs.stride_words = tl.sum_stride;
  cs.out_chunk0 = (uint32_t)chunk;
  cs.chunk_bias = (uint32_t)chunk;
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::atomic<bool>& dirty = g_dirty[p->device];
  if (dirty.load()) {
    const uint32_t all = (uint32_t)(kScratchBytes / sizeof(uint64_t));
    hipLaunchKernelGGL(zero_words, dim3((all + 255) / 256), dim3(256), 0, st, ptr, all);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(DR_EHIP, "dr_stage_chunk_noalloc: zero launch: %s", hipGetErrorString(e));
    // a clear recorded into a graph has not run yet: the next eager call clears again
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &capture) == hipSuccess && capture == hipStreamCaptureStatusNone) dirty = false;
  }
  const int rc = launch_chunk_into(p, tl, chunk, shards, dst_chunk, cs, st, "dr_stage_chunk_noalloc");
  if (rc) dirty = true;
  return rc;
}
