// The paper's weight path (Sec. 3.3): the training rank's state goes to the
// new rank through host memory, cut into bounded chunks, with store and reload
// pipelined chunk by chunk.  Here the stage kernel packs chunk c straight into
// one of two pinned host buffers of B bytes (its stores cross PCIe: the store
// half of the path), and a copy stream reloads that buffer into the chunk's
// place in the rollout buffer (SDMA, host->device), so storing chunk c+1 and
// reloading chunk c use both directions of the link at once.  The transient
// memory is 2*B pinned and no device staging, whatever the model size.
//
// Everything is enqueued with events; the call never blocks the host.  The
// caller's stream finally waits on the last reload, so the result is valid
// once that stream reaches this point, as for dr_stage_all.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "dr_internal.h"

namespace dr {

void free_relay_resources(dr_plan* p) {
  if (p->relay_stream) (void)hipStreamSynchronize(static_cast<hipStream_t>(p->relay_stream));
  if (p->relay_pin[0]) (void)hipDeviceSynchronize();  // kernels writing the pinned buffers
  for (int i = 0; i < 5; ++i) {
    if (p->relay_ev[i]) (void)hipEventDestroy(static_cast<hipEvent_t>(p->relay_ev[i]));
    p->relay_ev[i] = nullptr;
  }
  if (p->relay_stream) (void)hipStreamDestroy(static_cast<hipStream_t>(p->relay_stream));
  p->relay_stream = nullptr;
  for (int i = 0; i < 2; ++i) {
    if (p->relay_pin[i]) (void)hipHostFree(p->relay_pin[i]);
    p->relay_pin[i] = nullptr;
  }
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "dr_stage_through_host: %s: %s", what,
              hipGetErrorString(e));
}

int create_relay(dr_plan* p) {
  const size_t b = p->layout.chunk_bytes;
  for (int i = 0; i < 2; ++i) {
    hipError_t e = hipHostMalloc(&p->relay_pin[i], b, hipHostMallocDefault);  // mapped: kernels write it
    if (e != hipSuccess) return p->relay_pin[i] = nullptr, hip_fail(e, "hipHostMalloc(relay)");
  }
  hipStream_t s;
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);  // default priority
  if (e != hipSuccess) return hip_fail(e, "hipStreamCreate");
  p->relay_stream = s;
  for (int i = 0; i < 5; ++i) {
    hipEvent_t ev;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    p->relay_ev[i] = ev;
    // a recorded event: the first waits of the first call find it complete
    e = hipEventRecord(ev, s);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  return DR_OK;
}

}  // namespace
}  // namespace dr

using namespace dr;

extern "C" int dr_stage_through_host(dr_plan* p, const float* const* shards, void* dst, dr_checksum* d_cks,
                                     void* stream) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_stage_through_host: null plan");
  if (p->kind != kRollout) return fail(DR_EINVAL, "dr_stage_through_host: not a rollout plan");
  if (int rc = check_stage_args(p, shards, dst, d_cks, "dr_stage_through_host")) return rc;
  bool idle = false;
  if (!p->relay_busy.compare_exchange_strong(idle, true))
    return fail(DR_EINVAL, "dr_stage_through_host: another call on this plan is running on another thread");
  struct Release {
    dr_plan* p;
    ~Release() { p->relay_busy = false; }
  } release{p};
  if (!p->relay_pin[0]) {
    if (int rc = create_relay(p)) {
      free_relay_resources(p);
      return rc;
    }
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipStream_t in = static_cast<hipStream_t>(p->relay_stream);  // host -> device
  hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(p->relay_ev);
  hipEvent_t* packed = ev;         // chunk packed into relay_pin[b]
  hipEvent_t* copied_in = ev + 2;  // relay_pin[b] -> dst done: relay_pin[b] free
  hipEvent_t start = ev[4];        // the caller's earlier work on `stream` (e.g. readers of dst)
  const uint64_t B = p->layout.chunk_bytes, n = p->info.num_chunks;
  char* d = static_cast<char*>(dst);
  hipError_t e;
#define DR_RELAY(call, what)             \
  if ((e = (call)) != hipSuccess) {      \
    (void)hipStreamSynchronize(in);      \
    return hip_fail(e, what);            \
  }
  DR_RELAY(hipEventRecord(start, st), "record start");
  DR_RELAY(hipStreamWaitEvent(in, start, 0), "wait start");
  for (uint64_t c = 0; c < n; ++c) {
    const int b = (int)(c & 1);
    const uint64_t len = c + 1 < n ? B : p->info.last_chunk_bytes;
    // relay_pin[b] still holds chunk c-2 until its reload has finished (events of earlier
    // calls on this plan order the first two chunks after the previous call's reloads)
    DR_RELAY(hipStreamWaitEvent(st, copied_in[b], 0), "wait pinned buffer");
    if (int rc = launch_chunk(p, c, shards, p->relay_pin[b], d_cks + c, st)) return rc;
    DR_RELAY(hipEventRecord(packed[b], st), "record packed");
    DR_RELAY(hipStreamWaitEvent(in, packed[b], 0), "wait packed");
    DR_RELAY(hipMemcpyAsync(d + c * B, p->relay_pin[b], len, hipMemcpyHostToDevice, in), "H2D");
    DR_RELAY(hipEventRecord(copied_in[b], in), "record copied in");
  }
  DR_RELAY(hipStreamWaitEvent(st, copied_in[0], 0), "final wait");
  DR_RELAY(hipStreamWaitEvent(st, copied_in[1], 0), "final wait");
#undef DR_RELAY
  return DR_OK;
}
