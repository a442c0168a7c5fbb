// Plan lifetime, introspection and error reporting of the C ABI (dr.h).
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "dr_internal.h"

namespace dr {
namespace {
thread_local char g_error[512] = "";
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_error, sizeof(g_error), fmt, ap);
  va_end(ap);
  // The returned code and the message report a failed HIP call to the caller; the runtime's
  // per-thread last error is consumed here, so that it does not surface again in the caller's
  // own later HIP calls (a framework that checks hipGetLastError after its launches would
  // otherwise raise on an error the library has already reported).
  if (code == DR_EHIP || code == DR_ENOMEM) (void)hipGetLastError();
  return code;
}

void clear_error() { g_error[0] = '\0'; }

}  // namespace dr

using namespace dr;

dr_plan::~dr_plan() {
  free_relay_resources(this);
  free_moment_resources(this);
  free_device(this);
}

namespace {

template <typename Build>
int create(dr_plan** out, bool device, Build build) {
  clear_error();
  if (!out) return fail(DR_EINVAL, "dr_plan_create: null output pointer");
  *out = nullptr;
  dr_plan* p = nullptr;
  try {
    p = new dr_plan();
    int rc = build(p);
    if (rc == DR_OK && device) {
      rc = upload_plan(p);
      if (rc == DR_OK && p->layout.moment_chunk_bytes) rc = create_moment_resources(p);
    }
    if (rc != DR_OK) {
      delete p;
      return rc;
    }
  } catch (const std::bad_alloc&) {
    delete p;
    return fail(DR_ENOMEM, "dr_plan_create: host allocation failed");
  } catch (...) {
    delete p;
    return fail(DR_EINVAL, "dr_plan_create: unexpected internal error");
  }
  *out = p;
  return DR_OK;
}

}  // namespace

extern "C" int dr_plan_create(const dr_model* model, const dr_layout* layout, dr_plan** out) {
  return create(out, true, [&](dr_plan* p) { return build_plan(model, layout, p); });
}

extern "C" int dr_plan_create_host(const dr_model* model, const dr_layout* layout, dr_plan** out) {
  return create(out, false, [&](dr_plan* p) { return build_plan(model, layout, p); });
}

extern "C" int dr_reshard_plan_create(const dr_model* model, int32_t from_shards, int32_t to_shards,
                                      uint64_t chunk_bytes, dr_plan** out) {
  return create(out, true, [&](dr_plan* p) { return build_reshard_plan(model, from_shards, to_shards, chunk_bytes, p); });
}

extern "C" int dr_reshard_plan_create_host(const dr_model* model, int32_t from_shards, int32_t to_shards,
                                           uint64_t chunk_bytes, dr_plan** out) {
  return create(out, false,
                [&](dr_plan* p) { return build_reshard_plan(model, from_shards, to_shards, chunk_bytes, p); });
}

extern "C" void dr_plan_destroy(dr_plan* plan) { delete plan; }

extern "C" int dr_plan_get_info(const dr_plan* plan, dr_plan_info* out) {
  clear_error();
  if (!plan || !out) return fail(DR_EINVAL, "dr_plan_get_info: null argument");
  *out = plan->info;
  out->last_tile_depth = plan->last_depth.load(std::memory_order_relaxed);
  return DR_OK;
}

extern "C" int dr_plan_tensor(const dr_plan* plan, int32_t rank, int32_t index, dr_tensor_desc* out) {
  clear_error();
  if (!plan || !out) return fail(DR_EINVAL, "dr_plan_tensor: null argument");
  const int32_t per_rank = 3 + 6 * plan->model.n_layers;
  if (plan->kind != kRollout) return fail(DR_EINVAL, "dr_plan_tensor: not a rollout plan");
  if (rank < 0 || rank >= plan->layout.tp || index < 0 || index >= per_rank)
    return fail(DR_ERANGE, "dr_plan_tensor: rank %d / index %d out of range (tp %d, %d tensors per rank)", rank,
                index, plan->layout.tp, per_rank);
  const TensorDesc& t = plan->tensors[(size_t)rank * per_rank + index];
  std::memset(out, 0, sizeof(*out));
  std::snprintf(out->name, sizeof(out->name), "%s", t.name.c_str());
  out->rank = t.rank;
  out->ndim = t.ndim;
  out->byte_offset = 2 * t.elem_offset;
  out->rows = t.rows;
  out->cols = t.cols;
  return DR_OK;
}

extern "C" int dr_plan_segment(const dr_plan* plan, uint64_t index, dr_segment* out) {
  clear_error();
  if (!plan || !out) return fail(DR_EINVAL, "dr_plan_segment: null argument");
  if (index >= plan->segs.size())
    return fail(DR_ERANGE, "dr_plan_segment: index %llu >= %zu", (unsigned long long)index, plan->segs.size());
  const DevSeg& s = plan->segs[index];
  out->dst_elem = s.dst;
  out->src_elem = s.src;
  out->shard = s.shard;
  out->chunk = s.chunk;
  out->rows = s.rows;
  out->cols = s.cols;
  out->src_row_stride = s.stride;
  out->flags = s.flags;
  out->dst_shard = s.dst_shard;
  out->op = s.op;
  return DR_OK;
}

extern "C" const char* dr_last_error(void) { return dr::g_error; }
