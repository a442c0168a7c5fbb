// Bounded moment offload / deferred restore (Sec. 3.3): the Adam moments
// stream between the device and a caller-owned host store through two pinned
// bounce buffers of Bm bytes, so pinned host memory stays at 2*Bm however large
// the state is.  Copies run on a side stream (SDMA engines), host threads move
// bytes between the bounce buffers and the store, and the two overlap:
//
//   offload, chunk k:  D2H(k) -> bounce[k%2]   while   drain(k-1) bounce -> store
//   restore, chunk k:  fill(k) store -> bounce[k%2]   while   H2D(k-1) bounce -> device
//
// The moment stream is m_0 .. m_{W-1} v_0 .. v_{W-1} (S fp32 each, padding
// included); chunk k is its bytes [k*Bm, (k+1)*Bm).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <thread>

#include "dr_internal.h"

namespace dr {

// A fixed set of host threads that run one parallel byte copy at a time.
struct HostPool {
  explicit HostPool(int n) {
    for (int i = 0; i < n; ++i) workers_.emplace_back([this, i] { loop(i); });
  }
  ~HostPool() {
    {
      std::lock_guard<std::mutex> g(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : workers_) t.join();
  }
  int size() const { return (int)workers_.size(); }

  // Starts copying `bytes` from src to dst split over the workers; returns at once.
  void copy_async(void* dst, const void* src, size_t bytes) {
    wait();
    std::lock_guard<std::mutex> g(mu_);
    dst_ = static_cast<char*>(dst);
    src_ = static_cast<const char*>(src);
    bytes_ = bytes;
    pending_ = (int)workers_.size();
    ++generation_;
    cv_.notify_all();
  }

  // Blocks until the last copy has finished.
  void wait() {
    std::unique_lock<std::mutex> lk(mu_);
    done_.wait(lk, [this] { return pending_ == 0; });
  }

 private:
  void loop(int id) {
    uint64_t seen = 0;
    for (;;) {
      char* d;
      const char* s;
      size_t n;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || generation_ != seen; });
        if (stop_) return;
        seen = generation_;
        d = dst_;
        s = src_;
        n = bytes_;
      }
      // slice i of the copy, on 4 KiB boundaries
      const size_t parts = workers_.size();
      const size_t per = ((n + parts - 1) / parts + 4095) & ~size_t(4095);
      const size_t a = std::min(n, per * (size_t)id), b = std::min(n, a + per);
      if (b > a) std::memcpy(d + a, s + a, b - a);
      {
        std::lock_guard<std::mutex> g(mu_);
        if (--pending_ == 0) done_.notify_all();
      }
    }
  }

  std::vector<std::thread> workers_;
  std::mutex mu_;
  std::condition_variable cv_, done_;
  char* dst_ = nullptr;
  const char* src_ = nullptr;
  size_t bytes_ = 0;
  int pending_ = 0;
  uint64_t generation_ = 0;
  bool stop_ = false;
};

int create_moment_resources(dr_plan* p) {
  const size_t bm = p->layout.moment_chunk_bytes;
  for (int i = 0; i < 2; ++i) {
    hipError_t e = hipHostMalloc(&p->bounce[i], bm, hipHostMallocDefault);
    if (e != hipSuccess) {
      p->bounce[i] = nullptr;
      return fail(e == hipErrorOutOfMemory ? DR_ENOMEM : DR_EHIP, "hipHostMalloc(%zu B): %s", bm,
                  hipGetErrorString(e));
    }
    hipEvent_t ev;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return fail(DR_EHIP, "hipEventCreate: %s", hipGetErrorString(e));
    p->events[i] = ev;
  }
  const unsigned hw = std::thread::hardware_concurrency();
  p->pool = new HostPool((int)std::max(1u, std::min(16u, hw ? hw : 1u)));
  return DR_OK;
}

void free_moment_resources(dr_plan* p) {
  if (p->restore_thread.joinable()) p->restore_thread.join();
  p->restore_in_flight = false;
  p->moments_busy = false;
  delete p->pool;
  p->pool = nullptr;
  for (int i = 0; i < 2; ++i) {
    if (p->events[i]) (void)hipEventDestroy(static_cast<hipEvent_t>(p->events[i]));
    if (p->bounce[i]) (void)hipHostFree(p->bounce[i]);
    p->events[i] = nullptr;
    p->bounce[i] = nullptr;
  }
}

namespace {

// Calls fn(device_ptr, offset_in_chunk, bytes) for every shard piece of moment chunk k.
template <typename Fn>
int for_each_piece(const dr_plan* p, uint64_t k, const void* const* m, const void* const* v, Fn fn) {
  const uint64_t W = p->layout.train_shards;
  const uint64_t shard_bytes = p->info.shard_elems * 4;
  const uint64_t begin = k * p->layout.moment_chunk_bytes;
  const uint64_t end = std::min(p->info.moment_bytes, begin + p->layout.moment_chunk_bytes);
  for (uint64_t pos = begin; pos < end;) {
    const uint64_t q = pos / shard_bytes;  // 0..2W-1: m shards then v shards
    const uint64_t within = pos - q * shard_bytes;
    const uint64_t n = std::min(end - pos, shard_bytes - within);
    const char* base = static_cast<const char*>(q < W ? m[q] : v[q - W]);
    if (int rc = fn(base + within, pos - begin, n)) return rc;
    pos += n;
  }
  return DR_OK;
}

int check_moment_args(const dr_plan* p, const void* const* m, const void* const* v, const void* host,
                      const char* what) {
  if (!p) return fail(DR_EINVAL, "%s: null plan", what);
  if (!p->layout.moment_chunk_bytes) return fail(DR_EINVAL, "%s: plan was created with moment_chunk_bytes = 0", what);
  if (!m || !v) return fail(DR_EINVAL, "%s: null shard array", what);
  for (int w = 0; w < p->layout.train_shards; ++w)
    if (!m[w] || !v[w]) return fail(DR_EINVAL, "%s: null moment shard %d", what, w);
  if (!host) return fail(DR_EINVAL, "%s: null host store", what);
  if (!p->d_segs || !p->bounce[0]) return fail(DR_EINVAL, "%s: host-only plan has no moment buffers", what);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DR_EHIP, "%s: hipGetDevice: %s", what, hipGetErrorString(e));
  if (dev != p->device) return fail(DR_EINVAL, "%s: plan lives on device %d, current device is %d", what, p->device, dev);
  return DR_OK;
}

uint64_t chunk_len(const dr_plan* p, uint64_t k) {
  const uint64_t begin = k * p->layout.moment_chunk_bytes;
  return std::min(p->info.moment_bytes, begin + p->layout.moment_chunk_bytes) - begin;
}

// Takes the plan's bounce buffers for one moment transfer; DR_EINVAL while
// another transfer (from any thread, or a deferred restore) holds them.
int acquire_bounce(dr_plan* p, const char* what) {
  bool idle = false;
  if (!p->moments_busy.compare_exchange_strong(idle, true))
    return fail(DR_EINVAL, "%s: another moment transfer on this plan is in flight (offload, restore or deferred restore)",
                what);
  return DR_OK;
}

// Releases the bounce buffers when a blocking transfer returns.
struct BounceHeld {
  dr_plan* p;
  ~BounceHeld() { p->moments_busy = false; }
};

}  // namespace
}  // namespace dr

using namespace dr;

namespace dr {
namespace {

// The offload pipeline over moment chunks [k0, k1); arguments already checked
// and the bounce buffers held.  Blocks until the last chunk is in the store.
int offload_loop(dr_plan* p, const void* const* m, const void* const* v, char* store, uint64_t k0, uint64_t k1,
                 hipStream_t st, const char* what) {
  hipEvent_t ev[2] = {static_cast<hipEvent_t>(p->events[0]), static_cast<hipEvent_t>(p->events[1])};
  const uint64_t Bm = p->layout.moment_chunk_bytes;
  HostPool& pool = *p->pool;
  int rc = DR_OK;
  for (uint64_t k = k0; k < k1 && rc == DR_OK; ++k) {
    const int b = (int)((k - k0) & 1);
    pool.wait();  // bounce[b] held chunk k-2, drained by now
    rc = for_each_piece(p, k, m, v, [&](const void* dev, uint64_t off, uint64_t n) {
      hipError_t e = hipMemcpyAsync(static_cast<char*>(p->bounce[b]) + off, dev, n, hipMemcpyDeviceToHost, st);
      return e == hipSuccess ? DR_OK : fail(DR_EHIP, "%s: D2H: %s", what, hipGetErrorString(e));
    });
    if (rc) break;
    hipError_t e = hipEventRecord(ev[b], st);
    if (e != hipSuccess) {
      rc = fail(DR_EHIP, "%s: event record: %s", what, hipGetErrorString(e));
      break;
    }
    if (k > k0) {
      e = hipEventSynchronize(ev[b ^ 1]);
      if (e != hipSuccess) {
        rc = fail(DR_EHIP, "%s: event sync: %s", what, hipGetErrorString(e));
        break;
      }
      pool.copy_async(store + (k - 1) * Bm, p->bounce[b ^ 1], chunk_len(p, k - 1));
    }
  }
  pool.wait();
  if (rc == DR_OK && k1 > k0) {
    const int b = (int)((k1 - 1 - k0) & 1);
    hipError_t e = hipEventSynchronize(ev[b]);
    if (e != hipSuccess) {
      rc = fail(DR_EHIP, "%s: event sync: %s", what, hipGetErrorString(e));
    } else {
      pool.copy_async(store + (k1 - 1) * Bm, p->bounce[b], chunk_len(p, k1 - 1));
      pool.wait();
    }
  }
  if (rc != DR_OK) (void)hipStreamSynchronize(st);  // leave no copy in flight into the bounce buffers
  return rc;
}

int check_range(const dr_plan* p, uint64_t first, uint64_t count, const char* what) {
  const uint64_t K = p->info.num_moment_chunks;
  if (first > K || count > K - first)
    return fail(DR_ERANGE, "%s: chunks [%llu, %llu + %llu) exceed the %llu moment chunks", what,
                (unsigned long long)first, (unsigned long long)first, (unsigned long long)count,
                (unsigned long long)K);
  return DR_OK;
}

int offload(dr_plan* p, const float* const* m_shards, const float* const* v_shards, void* host_store, bool whole,
            uint64_t first, uint64_t count, void* side_stream, const char* what) {
  clear_error();
  const void* const* m = reinterpret_cast<const void* const*>(m_shards);
  const void* const* v = reinterpret_cast<const void* const*>(v_shards);
  if (int rc = check_moment_args(p, m, v, host_store, what)) return rc;
  if (whole) {
    first = 0;
    count = p->info.num_moment_chunks;
  }
  if (int rc = check_range(p, first, count, what)) return rc;
  if (int rc = acquire_bounce(p, what)) return rc;
  BounceHeld held{p};
  return offload_loop(p, m, v, static_cast<char*>(host_store), first, first + count,
                      static_cast<hipStream_t>(side_stream), what);
}

}  // namespace
}  // namespace dr

extern "C" int dr_offload_moments(dr_plan* p, const float* const* m_shards, const float* const* v_shards,
                                  void* host_store, void* side_stream) {
  return offload(p, m_shards, v_shards, host_store, true, 0, 0, side_stream, "dr_offload_moments");
}

extern "C" int dr_offload_moments_range(dr_plan* p, const float* const* m_shards, const float* const* v_shards,
                                        void* host_store, uint64_t first_chunk, uint64_t num_chunks,
                                        void* side_stream) {
  return offload(p, m_shards, v_shards, host_store, false, first_chunk, num_chunks, side_stream,
                 "dr_offload_moments_range");
}

namespace dr {
namespace {

// The restore pipeline itself; arguments already checked.  Blocks until every
// byte has landed on the device.
int restore_loop(dr_plan* p, const void* host_store, const void* const* m, const void* const* v, uint64_t k0,
                 uint64_t k1, void* side_stream, const char* what) {
  hipStream_t st = static_cast<hipStream_t>(side_stream);
  hipEvent_t ev[2] = {static_cast<hipEvent_t>(p->events[0]), static_cast<hipEvent_t>(p->events[1])};
  const char* store = static_cast<const char*>(host_store);
  const uint64_t Bm = p->layout.moment_chunk_bytes;
  HostPool& pool = *p->pool;
  int rc = DR_OK;
  for (uint64_t k = k0; k < k1 && rc == DR_OK; ++k) {
    const int b = (int)((k - k0) & 1);
    if (k - k0 >= 2) {
      hipError_t e = hipEventSynchronize(ev[b]);  // H2D(k-2) out of bounce[b] has finished
      if (e != hipSuccess) {
        rc = fail(DR_EHIP, "%s: event sync: %s", what, hipGetErrorString(e));
        break;
      }
    }
    pool.copy_async(p->bounce[b], store + k * Bm, chunk_len(p, k));
    pool.wait();
    rc = for_each_piece(p, k, m, v, [&](const void* dev, uint64_t off, uint64_t n) {
      hipError_t e = hipMemcpyAsync(const_cast<void*>(dev), static_cast<const char*>(p->bounce[b]) + off, n,
                                    hipMemcpyHostToDevice, st);
      return e == hipSuccess ? DR_OK : fail(DR_EHIP, "%s: H2D: %s", what, hipGetErrorString(e));
    });
    if (rc) break;
    hipError_t e = hipEventRecord(ev[b], st);
    if (e != hipSuccess) rc = fail(DR_EHIP, "%s: event record: %s", what, hipGetErrorString(e));
  }
  for (int b = 0; b < 2 && k1 - k0 > (uint64_t)b; ++b) {
    hipError_t e = hipEventSynchronize(ev[b]);
    if (e != hipSuccess && rc == DR_OK) rc = fail(DR_EHIP, "%s: event sync: %s", what, hipGetErrorString(e));
  }
  if (rc != DR_OK) (void)hipStreamSynchronize(st);
  return rc;
}

}  // namespace
}  // namespace dr

extern "C" int dr_restore_moments(dr_plan* p, const void* host_store, float* const* m_shards, float* const* v_shards,
                                  void* side_stream) {
  clear_error();
  const void* const* m = reinterpret_cast<const void* const*>(m_shards);
  const void* const* v = reinterpret_cast<const void* const*>(v_shards);
  if (int rc = check_moment_args(p, m, v, host_store, "dr_restore_moments")) return rc;
  if (int rc = acquire_bounce(p, "dr_restore_moments")) return rc;
  BounceHeld held{p};
  return restore_loop(p, host_store, m, v, 0, p->info.num_moment_chunks, side_stream, "dr_restore_moments");
}

extern "C" int dr_restore_moments_range(dr_plan* p, const void* host_store, float* const* m_shards,
                                        float* const* v_shards, uint64_t first_chunk, uint64_t num_chunks,
                                        void* side_stream) {
  clear_error();
  const void* const* m = reinterpret_cast<const void* const*>(m_shards);
  const void* const* v = reinterpret_cast<const void* const*>(v_shards);
  if (int rc = check_moment_args(p, m, v, host_store, "dr_restore_moments_range")) return rc;
  if (int rc = check_range(p, first_chunk, num_chunks, "dr_restore_moments_range")) return rc;
  if (int rc = acquire_bounce(p, "dr_restore_moments_range")) return rc;
  BounceHeld held{p};
  return restore_loop(p, host_store, m, v, first_chunk, first_chunk + num_chunks, side_stream,
                      "dr_restore_moments_range");
}

extern "C" int dr_restore_moments_begin(dr_plan* p, const void* host_store, float* const* m_shards,
                                        float* const* v_shards, void* side_stream) {
  clear_error();
  const void* const* m = reinterpret_cast<const void* const*>(m_shards);
  const void* const* v = reinterpret_cast<const void* const*>(v_shards);
  if (int rc = check_moment_args(p, m, v, host_store, "dr_restore_moments_begin")) return rc;
  // held until dr_restore_moments_end (or dr_plan_destroy)
  if (int rc = acquire_bounce(p, "dr_restore_moments_begin")) return rc;
  if (p->restore_thread.joinable()) p->restore_thread.join();  // a finished run not yet ended
  const int W = p->layout.train_shards;
  p->restore_rc = DR_OK;
  p->restore_error[0] = '\0';
  p->restore_in_flight = true;
  try {
    p->restore_m.assign(m_shards, m_shards + W);
    p->restore_v.assign(v_shards, v_shards + W);
    p->restore_thread = std::thread([p, host_store, side_stream] {
      int rc;
      hipError_t e = hipSetDevice(p->device);  // the current device is per thread
      if (e != hipSuccess) {
        rc = fail(DR_EHIP, "dr_restore_moments_begin: hipSetDevice: %s", hipGetErrorString(e));
      } else {
        rc = restore_loop(p, host_store, reinterpret_cast<const void* const*>(p->restore_m.data()),
                          reinterpret_cast<const void* const*>(p->restore_v.data()), 0, p->info.num_moment_chunks,
                          side_stream, "dr_restore_moments_begin");
      }
      if (rc != DR_OK) std::snprintf(p->restore_error, sizeof(p->restore_error), "%s", dr_last_error());
      p->restore_rc = rc;
    });
  } catch (...) {
    p->restore_in_flight = false;
    p->moments_busy = false;
    return fail(DR_ENOMEM, "dr_restore_moments_begin: cannot start the restore thread");
  }
  return DR_OK;
}

extern "C" int dr_restore_moments_end(dr_plan* p) {
  clear_error();
  if (!p) return fail(DR_EINVAL, "dr_restore_moments_end: null plan");
  if (!p->restore_in_flight) return fail(DR_EINVAL, "dr_restore_moments_end: no deferred restore in flight");
  p->restore_thread.join();
  p->restore_in_flight = false;
  p->moments_busy = false;
  if (p->restore_rc != DR_OK) return fail(p->restore_rc, "%s", p->restore_error);
  return DR_OK;
}
