// The paper's state path (Sec. 3.3): the training rank's state goes to the
// new rank through host memory, cut into bounded chunks, with store and reload
// pipelined chunk by chunk.  Here the stage (or reshard) kernel packs chunk c
// into one of two device staging buffers of B bytes on the caller's stream;
// one SDMA engine stores that buffer into one of two pinned host buffers
// (device -> host) and a second SDMA engine reloads the pinned buffer into the
// chunk's place at the destination (host -> device), so the store of chunk c
// and the reload of chunk c-1 use both link directions at once.  Transient
// memory: 2*B device and 2*B pinned, whatever the model size.
//
// The two directions run on two SDMA engines chosen explicitly through the
// HSA runtime (hsa_amd_memory_async_copy_on_engine).  HIP's own copies let the
// runtime pick the engines; when it puts both directions on one engine the
// two share its ~57 GB/s.  Measured on MI355X, 4 GiB each way at once: engines
// 0 and 1 gave 48.4 GB/s each way in every run, the runtime's choice 43-49.
//
// The host orders the pipeline: it waits for a chunk's pack (HIP event) before
// issuing its store, the reload depends on the store through an HSA signal,
// a staging buffer is packed again only after its store has finished, and a
// pinned buffer is stored into again only after its reload has finished.  The
// call returns when every chunk is at the destination.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <algorithm>
#include <chrono>
#include <cstring>
#include <new>

#include "dr_internal.h"

namespace dr {

struct RelayState {
  bool hsa_up = false;
  void* stage[2] = {nullptr, nullptr};  // device, B bytes each
  void* pin[2] = {nullptr, nullptr};    // pinned host, B bytes each
  hipEvent_t packed[2] = {nullptr, nullptr};
  hsa_signal_t stored[2] = {};    // device -> host copy of buffer b: 1 in flight, 0 done
  hsa_signal_t reloaded[2] = {};  // host -> device copies out of pin[b]: pieces in flight
  int signals = 0;                // signals created (stored[0..1], then reloaded[0..1])
  hsa_agent_t gpu{}, cpu{};
  uint32_t engine_out = 0, engine_in = 0;  // hsa_amd_sdma_engine_id_t bits; 0: the runtime's choice
};

namespace {

constexpr double kCopyWaitLimitS = 120.0;  // a copy that has not finished by then is reported

hsa_status_t find_cpu(hsa_agent_t a, void* out) {
  hsa_device_type_t t;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) == HSA_STATUS_SUCCESS && t == HSA_DEVICE_TYPE_CPU) {
    *static_cast<hsa_agent_t*>(out) = a;
    return HSA_STATUS_INFO_BREAK;
  }
  return HSA_STATUS_SUCCESS;
}

// Waits until signal s reaches 0 (bounded); false if it has not after kCopyWaitLimitS.
bool wait_zero(hsa_signal_t s) {
  const auto t0 = std::chrono::steady_clock::now();
  while (hsa_signal_wait_scacquire(s, HSA_SIGNAL_CONDITION_EQ, 0, 1000000, HSA_WAIT_STATE_BLOCKED) != 0)
    if (std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count() > kCopyWaitLimitS) return false;
  return true;
}

int hip_fail(hipError_t e, const char* what, const char* step) {
  return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "%s: host relay: %s: %s", what, step,
              hipGetErrorString(e));
}

int hsa_fail(hsa_status_t s, const char* what, const char* step) {
  const char* msg = nullptr;
  if (hsa_status_string(s, &msg) != HSA_STATUS_SUCCESS || !msg) msg = "unknown HSA status";
  return fail(s == HSA_STATUS_ERROR_OUT_OF_RESOURCES ? DR_ENOMEM : DR_EHIP, "%s: host relay: %s: %s", what, step,
              msg);
}

// Lowest engine bit in mask other than `taken`; 0 if none.
uint32_t pick_engine(uint32_t mask, uint32_t taken) {
  for (uint32_t bit = 1; bit && bit <= mask; bit <<= 1)
    if ((mask & bit) && bit != taken) return bit;
  return 0;
}

int create_relay(dr_plan* p, const char* what) {
  RelayState* r = new (std::nothrow) RelayState();
  if (!r) return fail(DR_ENOMEM, "%s: host relay: host allocation failed", what);
  p->relay = r;
  const size_t b = p->layout.chunk_bytes;
  for (int i = 0; i < 2; ++i) {
    hipError_t e = hipMalloc(&r->stage[i], b);
    if (e != hipSuccess) return r->stage[i] = nullptr, hip_fail(e, what, "hipMalloc(staging)");
    e = hipHostMalloc(&r->pin[i], b, hipHostMallocDefault);
    if (e != hipSuccess) return r->pin[i] = nullptr, hip_fail(e, what, "hipHostMalloc(pinned)");
    e = hipEventCreateWithFlags(&r->packed[i], hipEventDisableTiming);
    if (e != hipSuccess) return r->packed[i] = nullptr, hip_fail(e, what, "hipEventCreate");
  }
  hsa_status_t s = hsa_init();  // reference counted; the HIP runtime has initialized HSA already
  if (s != HSA_STATUS_SUCCESS) return hsa_fail(s, what, "hsa_init");
  r->hsa_up = true;
  hsa_amd_pointer_info_t info;
  std::memset(&info, 0, sizeof(info));
  info.size = sizeof(info);
  s = hsa_amd_pointer_info(r->stage[0], &info, nullptr, nullptr, nullptr);
  if (s != HSA_STATUS_SUCCESS) return hsa_fail(s, what, "hsa_amd_pointer_info");
  r->gpu = info.agentOwner;
  if (hsa_iterate_agents(find_cpu, &r->cpu) != HSA_STATUS_INFO_BREAK)
    return fail(DR_EHIP, "%s: host relay: no CPU agent", what);
  for (hsa_signal_t* sig : {&r->stored[0], &r->stored[1], &r->reloaded[0], &r->reloaded[1]}) {
    s = hsa_signal_create(0, 0, nullptr, sig);
    if (s != HSA_STATUS_SUCCESS) return hsa_fail(s, what, "hsa_signal_create");
    ++r->signals;
  }
  uint32_t out_mask = 0, in_mask = 0;
  if (hsa_amd_memory_copy_engine_status(r->cpu, r->gpu, &out_mask) == HSA_STATUS_SUCCESS &&
      hsa_amd_memory_copy_engine_status(r->gpu, r->cpu, &in_mask) == HSA_STATUS_SUCCESS) {
    r->engine_out = pick_engine(out_mask, 0);
    r->engine_in = pick_engine(in_mask, r->engine_out);
    if (!r->engine_out || !r->engine_in) r->engine_out = r->engine_in = 0;
  }
  return DR_OK;
}

hsa_status_t copy(void* dst, hsa_agent_t dst_agent, const void* src, hsa_agent_t src_agent, size_t n,
                  const hsa_signal_t* dep, hsa_signal_t done, uint32_t engine) {
  if (engine)
    return hsa_amd_memory_async_copy_on_engine(dst, dst_agent, src, src_agent, n, dep ? 1 : 0, dep, done,
                                               static_cast<hsa_amd_sdma_engine_id_t>(engine), true);
  return hsa_amd_memory_async_copy(dst, dst_agent, src, src_agent, n, dep ? 1 : 0, dep, done);
}

}  // namespace

void free_relay_resources(dr_plan* p) {
  RelayState* r = p->relay;
  if (!r) return;
  // calls return only once their copies have finished; wait anyway before freeing the buffers
  for (int i = 0; i < r->signals; ++i) {
    hsa_signal_t s = i < 2 ? r->stored[i] : r->reloaded[i - 2];
    (void)wait_zero(s);
    (void)hsa_signal_destroy(s);
  }
  if (r->stage[0] || r->packed[0]) (void)hipDeviceSynchronize();  // kernels writing the staging buffers
  for (int i = 0; i < 2; ++i) {
    if (r->packed[i]) (void)hipEventDestroy(r->packed[i]);
    if (r->stage[i]) (void)hipFree(r->stage[i]);
    if (r->pin[i]) (void)hipHostFree(r->pin[i]);
  }
  if (r->hsa_up) (void)hsa_shut_down();
  delete r;
  p->relay = nullptr;
}

// Defined with the reshard host code (reshard.cpp).
int check_reshard_args(const dr_plan* p, const float* const* src_shards, float* const* dst_shards,
                       const dr_checksum* d_cks, const char* what);
int launch_reshard_chunk(dr_plan* p, uint64_t chunk, const float* const* src, void* chunk_dst, dr_checksum* ck,
                         hipStream_t st, const char* what);

namespace {

// The relay pipeline shared by the rollout and reshard plans.  pack(c, buf) enqueues on st the
// kernels that write chunk c into device buffer buf; pieces(c, fn) calls fn(dst, offset, bytes)
// for every destination piece of chunk c (its bytes [offset, offset + bytes) go to dst).
template <typename Pack, typename Pieces>
int relay_run(dr_plan* p, hipStream_t st, const char* what, Pack pack, Pieces pieces) {
  bool idle = false;
  if (!p->relay_busy.compare_exchange_strong(idle, true))
    return fail(DR_EINVAL, "%s: another call on this plan is running on another thread", what);
  struct Release {
    dr_plan* p;
    ~Release() { p->relay_busy = false; }
  } release{p};
  if (!p->relay) {
    if (int rc = create_relay(p, what)) {
      free_relay_resources(p);
      return rc;
    }
  }
  RelayState* r = p->relay;
  const uint64_t n = p->info.num_chunks, B = p->layout.chunk_bytes;
  auto len = [&](uint64_t c) { return c + 1 < n ? B : p->info.last_chunk_bytes; };
  int rc = DR_OK;

  // Store and reload chunk c, whose pack was recorded on packed[c % 2].
  auto issue = [&](uint64_t c) -> int {
    const int b = (int)(c & 1);
    hipError_t e = hipEventSynchronize(r->packed[b]);
    if (e != hipSuccess) return hip_fail(e, what, "wait for the pack");
    if (!wait_zero(r->reloaded[b])) return fail(DR_EHIP, "%s: host relay: a reload did not finish", what);
    int64_t count = 0;
    pieces(c, [&](void*, uint64_t, uint64_t) { ++count; });
    hsa_signal_store_screlease(r->stored[b], 1);
    hsa_signal_store_screlease(r->reloaded[b], count);
    hsa_status_t s = copy(r->pin[b], r->cpu, r->stage[b], r->gpu, len(c), nullptr, r->stored[b], r->engine_out);
    if (s != HSA_STATUS_SUCCESS) {
      hsa_signal_store_screlease(r->stored[b], 0);
      hsa_signal_store_screlease(r->reloaded[b], 0);
      return hsa_fail(s, what, "device-to-host store");
    }
    int64_t issued = 0;
    pieces(c, [&](void* dst, uint64_t off, uint64_t bytes) {
      if (s != HSA_STATUS_SUCCESS) return;
      s = copy(dst, r->gpu, static_cast<char*>(r->pin[b]) + off, r->cpu, bytes, &r->stored[b], r->reloaded[b],
               r->engine_in);
      if (s == HSA_STATUS_SUCCESS) ++issued;
    });
    if (s != HSA_STATUS_SUCCESS) {
      hsa_signal_subtract_screlease(r->reloaded[b], count - issued);  // the pieces never issued
      return hsa_fail(s, what, "host-to-device reload");
    }
    return DR_OK;
  };

  for (uint64_t c = 0; c < n && rc == DR_OK; ++c) {
    const int b = (int)(c & 1);
    // staging[b] still holds chunk c-2 until its store has finished
    if (!wait_zero(r->stored[b])) {
      rc = fail(DR_EHIP, "%s: host relay: a store did not finish", what);
      break;
    }
    if ((rc = pack(c, r->stage[b]))) break;
    hipError_t e = hipEventRecord(r->packed[b], st);
    if (e != hipSuccess) {
      rc = hip_fail(e, what, "record the pack");
      break;
    }
    if (c >= 1) rc = issue(c - 1);
  }
  if (rc == DR_OK && n) rc = issue(n - 1);
  // every copy of this call has finished before it returns, whatever happened
  for (int b = 0; b < 2; ++b) {
    const bool ok = wait_zero(r->stored[b]) && wait_zero(r->reloaded[b]);
    if (!ok && rc == DR_OK) rc = fail(DR_EHIP, "%s: host relay: a copy did not finish", what);
  }
  if (rc != DR_OK) (void)hipStreamSynchronize(st);  // no pack left writing the staging buffers
  return rc;
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
      [&](uint64_t c, auto&& fn) { fn(d + c * B, 0, c + 1 < n ? B : p->info.last_chunk_bytes); });
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
      [&](uint64_t c, auto&& fn) {
        // the chunk's destination elements [e0, e1), cut at the destination shard boundaries
        const uint64_t e0 = c * ce, e1 = std::min(total, e0 + ce);
        for (uint64_t e = e0; e < e1;) {
          const uint64_t w = e / S2, m = std::min(e1, (w + 1) * S2) - e;
          fn(static_cast<void*>(dst_shards[w] + (e - w * S2)), (e - e0) * 4, m * 4);
          e += m;
        }
      });
}
