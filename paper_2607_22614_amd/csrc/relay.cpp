// The paper's state path (Sec. 3.3): the training rank's state goes to the
// new rank through host memory, cut into bounded chunks, with store and reload
// pipelined chunk by chunk.  Here a kernel packs chunk c straight into one of
// two pinned host buffers of B bytes (its stores cross PCIe: the store half of
// the path), and a copy stream reloads that buffer into the chunk's place at
// the destination (SDMA, host->device), so storing chunk c+1 and reloading
// chunk c use both directions of the link at once.  The transient memory is
// 2*B pinned and no device staging, whatever the model size.  Two forms share
// the pipeline: the weights to the rollout layout (stage kernel) and the
// training state to W' training shards (reshard kernel).
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
  return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "host relay buffers: %s: %s", what,
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

// The relay pipeline shared by the rollout and reshard plans.  pack(c, buf) enqueues on st the
// kernels that write chunk c into pinned buffer buf; reload(c, buf, in) enqueues on the plan's
// copy stream the host->device copies that move it to its destination.
template <typename Pack, typename Reload>
int relay_run(dr_plan* p, hipStream_t st, const char* what, Pack pack, Reload reload) {
  bool idle = false;
  if (!p->relay_busy.compare_exchange_strong(idle, true))
    return fail(DR_EINVAL, "%s: another call on this plan is running on another thread", what);
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
  hipStream_t in = static_cast<hipStream_t>(p->relay_stream);  // host -> device
  hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(p->relay_ev);
  hipEvent_t* packed = ev;         // chunk packed into relay_pin[b]
  hipEvent_t* copied_in = ev + 2;  // relay_pin[b] reloaded: relay_pin[b] free
  hipEvent_t start = ev[4];        // the caller's earlier work on `st` (e.g. readers of the destination)
  hipError_t e;
#define DR_RELAY(call, step)                                                        \
  if ((e = (call)) != hipSuccess) {                                                 \
    (void)hipStreamSynchronize(in);                                                 \
    return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "%s: %s: %s", what, \
                step, hipGetErrorString(e));                                        \
  }
  DR_RELAY(hipEventRecord(start, st), "record start");
  DR_RELAY(hipStreamWaitEvent(in, start, 0), "wait start");
  for (uint64_t c = 0; c < p->info.num_chunks; ++c) {
    const int b = (int)(c & 1);
    // relay_pin[b] still holds chunk c-2 until its reload has finished (events of earlier
    // calls on this plan order the first two chunks after the previous call's reloads)
    DR_RELAY(hipStreamWaitEvent(st, copied_in[b], 0), "wait pinned buffer");
    if (int rc = pack(c, p->relay_pin[b])) return rc;
    DR_RELAY(hipEventRecord(packed[b], st), "record packed");
    DR_RELAY(hipStreamWaitEvent(in, packed[b], 0), "wait packed");
    DR_RELAY(reload(c, static_cast<const char*>(p->relay_pin[b]), in), "host-to-device reload");
    DR_RELAY(hipEventRecord(copied_in[b], in), "record copied in");
  }
  DR_RELAY(hipStreamWaitEvent(st, copied_in[0], 0), "final wait");
  DR_RELAY(hipStreamWaitEvent(st, copied_in[1], 0), "final wait");
#undef DR_RELAY
  return DR_OK;
}

}  // namespace
}  // namespace dr

using namespace dr;

extern "C" int dr_stage_through_host(dr_plan* p, const float* const* shards, void* dst, dr_checksum* d_cks,
                                     void* stream) {
  clear_error();
  const char* what = "dr_stage_through_host";
  if (!p) return fail(DR_EINVAL, "%s: null plan", what);
  if (p->kind != kRollout) return fail(DR_EINVAL, "%s: not a rollout plan", what);
  if (int rc = check_stage_args(p, shards, dst, d_cks, what)) return rc;
  const uint64_t B = p->layout.chunk_bytes, n = p->info.num_chunks;
  char* d = static_cast<char*>(dst);
  hipStream_t st = static_cast<hipStream_t>(stream);
  return relay_run(
      p, st, what, [&](uint64_t c, void* buf) { return launch_chunk(p, c, shards, buf, d_cks + c, st); },
      [&](uint64_t c, const char* buf, hipStream_t in) {
        const uint64_t len = c + 1 < n ? B : p->info.last_chunk_bytes;
        return hipMemcpyAsync(d + c * B, buf, len, hipMemcpyHostToDevice, in);
      });
}

extern "C" int dr_reshard_through_host(dr_plan* p, const float* const* src_shards, float* const* dst_shards,
                                       dr_checksum* d_cks, void* stream) {
  clear_error();
  const char* what = "dr_reshard_through_host";
  if (int rc = check_reshard_args(p, src_shards, dst_shards, d_cks, what)) return rc;
  const uint64_t ce = p->layout.chunk_bytes / 4, S2 = p->dst_shard_elems, total = p->info.rollout_bytes / 4;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return relay_run(
      p, st, what,
      [&](uint64_t c, void* buf) { return launch_reshard_chunk(p, c, src_shards, buf, d_cks + c, st, what); },
      [&](uint64_t c, const char* buf, hipStream_t in) {
        // the chunk's destination elements [e0, e1), cut at the destination shard boundaries
        const uint64_t e0 = c * ce, e1 = std::min(total, e0 + ce);
        for (uint64_t e = e0; e < e1;) {
          const uint64_t w = e / S2, n = std::min(e1, (w + 1) * S2) - e;
          hipError_t err = hipMemcpyAsync(dst_shards[w] + (e - w * S2), buf + (e - e0) * 4, n * 4,
                                          hipMemcpyHostToDevice, in);
          if (err != hipSuccess) return err;
          e += n;
        }
        return hipSuccess;
      });
}
