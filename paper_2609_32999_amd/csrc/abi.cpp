// Exported C entry points of libtsr.  Every function validates on the host
// before enqueueing anything, converts failures into a status plus a
// thread-local message, and lets no exception cross the ABI.
#include <cmath>
#include <cstring>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "tsr_internal.h"

namespace tsr {

namespace {
thread_local std::string g_error;

tsr_status check_exec(const tsr_plan* p) {
  if (!p) {
    set_error("plan is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  if (!p->ws) {
    set_error("plan was created without a device workspace (host-only plan)");
    return TSR_ERR_INVALID_ARG;
  }
  return check_static_plan(p);
}

bool is_e4m3(const tsr_plan* p) { return p->model.kv_dtype == TSR_E4M3; }

// e4m3 plans need every scale array the call touches; other plans take none.
tsr_status check_scales(const tsr_plan* p, const float* a, const float* b,
                        bool need_a, bool need_b) {
  if (!is_e4m3(p)) {
    if (a || b) {
      set_error("scale arrays apply to e4m3 pools only; pass NULL");
      return TSR_ERR_INVALID_ARG;
    }
    return TSR_OK;
  }
  if ((need_a && !a) || (need_b && !b)) {
    set_error("e4m3 pools need their page-scale arrays");
    return TSR_ERR_INVALID_ARG;
  }
  return TSR_OK;
}

tsr_status attn_common(const tsr_plan* p, int32_t part, const void* q, const void* req_k,
                       const void* req_v, const void* pool_k, const void* pool_v,
                       const float* req_scale, void* out, float* lse, void* stream,
                       bool aliased_entry) {
  tsr_status st = check_exec(p);
  if (st != TSR_OK) return st;
  if (part < TSR_ATTN_ALL || part > TSR_ATTN_AFTER_COMPOSE) {
    set_error("attn: part must be TSR_ATTN_ALL, _BEFORE_COMPOSE or _AFTER_COMPOSE");
    return TSR_ERR_INVALID_ARG;
  }
  if ((st = check_scales(p, nullptr, req_scale, false, true)) != TSR_OK) return st;
  const bool aliased = p->alias_v || p->alias_k;
  if (aliased != aliased_entry) {
    set_error(aliased ? "the plan reads K or V from the pool: use tsr_attn_aliased"
                      : "tsr_attn_aliased needs a plan created with alias_v or alias_k");
    return TSR_ERR_INVALID_ARG;
  }
  if (p->alias_v != (pool_v != nullptr) || p->alias_k != (pool_k != nullptr)) {
    set_error("tsr_attn_aliased: pass pool_v exactly for alias_v plans and pool_k exactly "
              "for alias_k plans");
    return TSR_ERR_INVALID_ARG;
  }
  if (p->T == 0) return TSR_OK;
  if (!q || !req_k || !req_v || !out) {
    set_error("attn: a required pointer is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  const AttnItem* items = part == TSR_ATTN_ALL ? p->dev.items : p->dev.items_part[part - 1];
  const int32_t n = part == TSR_ATTN_ALL ? p->n_items : p->n_items_part[part - 1];
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = is_e4m3(p)
                     ? launch_attn_e4m3(p, items, n, q, req_k, req_v, req_scale, out, lse, s)
                     : launch_attn(p, part, items, n, pool_k, pool_v, q, req_k, req_v, out,
                                   lse, s);
  if (e != hipSuccess) return device_fail("attention launch", e);
  return TSR_OK;
}


// Options as build_plan takes them; a static plan's automatic split is off
// (its image must fit the static plan area).
tsr_status resolve_options(const tsr_plan_options* options, bool static_plan, bool* alias_v,
                           bool* alias_k, int32_t* split, int32_t* attn_kernel) {
  *alias_v = *alias_k = false;
  *split = static_plan ? -1 : 0;
  *attn_kernel = 0;
  if (!options) return TSR_OK;
  for (int32_t r : options->reserved)
    if (r != 0) {
      set_error("tsr_plan_options.reserved must be zero");
      return TSR_ERR_INVALID_ARG;
    }
  if (options->alias_v != 0 && options->alias_v != 1) {
    set_error("tsr_plan_options.alias_v must be 0 or 1");
    return TSR_ERR_INVALID_ARG;
  }
  if (options->alias_k != 0 && options->alias_k != 1) {
    set_error("tsr_plan_options.alias_k must be 0 or 1");
    return TSR_ERR_INVALID_ARG;
  }
  if (options->split_tiles < -1) {
    set_error("tsr_plan_options.split_tiles must be -1, 0 or positive");
    return TSR_ERR_INVALID_ARG;
  }
  if (options->attn_kernel < 0 || options->attn_kernel > 4) {
    set_error("tsr_plan_options.attn_kernel must be 0 .. 4");
    return TSR_ERR_INVALID_ARG;
  }
  *alias_v = options->alias_v == 1;
  *alias_k = options->alias_k == 1;
  if (options->split_tiles != 0) *split = options->split_tiles;
  *attn_kernel = options->attn_kernel;
  return TSR_OK;
}

}  // namespace

size_t plan_workspace_size(const tsr_model* model, const tsr_request* reqs, int32_t n_req,
                           int32_t n_pool_pages, int32_t n_req_pages,
                           const tsr_plan_options* options, bool static_plan) {
  size_t bytes = 0;
  guarded([&]() -> tsr_status {
    bool alias_v, alias_k;
    int32_t split, attn_kernel;
    tsr_status st =
        resolve_options(options, static_plan, &alias_v, &alias_k, &split, &attn_kernel);
    if (st != TSR_OK) return st;
    tsr_plan tmp{};
    st = build_plan(model, reqs, n_req, n_pool_pages, n_req_pages, alias_v, alias_k, split,
                    attn_kernel, &tmp);
    if (st == TSR_OK) bytes = tmp.ws_bytes;
    return st;
  });
  return bytes;
}

tsr_status create_plan(const tsr_model* model, const tsr_request* reqs, int32_t n_req,
                       int32_t n_pool_pages, int32_t n_req_pages,
                       const tsr_plan_options* options, bool static_plan,
                       const void* dev_rope_table, void* dev_workspace,
                       size_t workspace_bytes, void* stream, tsr_plan** out_plan) {
  return guarded([&]() -> tsr_status {
    if (!out_plan) {
      set_error("out_plan is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    *out_plan = nullptr;
    bool alias_v, alias_k;
    int32_t split, attn_kernel;
    tsr_status st =
        resolve_options(options, static_plan, &alias_v, &alias_k, &split, &attn_kernel);
    if (st != TSR_OK) return st;
    tsr_plan* p = new tsr_plan();
    st = build_plan(model, reqs, n_req, n_pool_pages, n_req_pages, alias_v, alias_k, split,
                    attn_kernel, p);
    if (st != TSR_OK) {
      delete p;
      return st;
    }
    if (dev_workspace) {
      if (workspace_bytes < p->ws_bytes) {
        set_error("workspace smaller than tsr_plan_workspace_size_ex() = " +
                  std::to_string(p->ws_bytes));
        delete p;
        return TSR_ERR_INVALID_ARG;
      }
      if (!dev_rope_table) {
        set_error("dev_rope_table is NULL");
        delete p;
        return TSR_ERR_INVALID_ARG;
      }
      hipError_t e = hipMemcpyAsync(dev_workspace, p->image.data(), p->image_bytes,
                                    hipMemcpyHostToDevice,
                                    static_cast<hipStream_t>(stream));
      if (e != hipSuccess) {
        delete p;
        return device_fail("hipMemcpyAsync(plan)", e);
      }
      char* base = static_cast<char*>(dev_workspace);
      const size_t half = (size_t)p->model.max_position * (p->model.head_dim / 2);
      const float* table = static_cast<const float*>(dev_rope_table);
      p->dev.gather = reinterpret_cast<const GatherDesc*>(base + p->off_gather);
      p->dev.rows = reinterpret_cast<const RowDesc*>(base + p->off_rows);
      p->dev.attn_rows = reinterpret_cast<const AttnRow*>(base + p->off_attn_rows);
      p->dev.retain = reinterpret_cast<const RetainDesc*>(base + p->off_retain);
      p->dev.items = reinterpret_cast<const AttnItem*>(base + p->off_items);
      for (int q = 0; q < 2; ++q)
        p->dev.items_part[q] = reinterpret_cast<const AttnItem*>(base + p->off_items_part[q]);
      p->dev.block_tables = reinterpret_cast<const int32_t*>(base + p->off_bt);
      p->dev.v_block_tables = reinterpret_cast<const int32_t*>(base + p->off_vbt);
      p->dev.k_block_tables = reinterpret_cast<const int32_t*>(base + p->off_kbt);
      p->dev.gpages = reinterpret_cast<const PageDesc*>(base + p->off_gpages);
      p->dev.apages = reinterpret_cast<const PageDesc*>(base + p->off_apages);
      p->dev.rpages = reinterpret_cast<const PageDesc*>(base + p->off_rpages);
      p->dev.combine = reinterpret_cast<const CombineDesc*>(base + p->off_combine);
      p->dev.split_o = reinterpret_cast<float*>(base + p->off_split_o);
      p->dev.split_lse = reinterpret_cast<float*>(base + p->off_split_lse);
      p->dev.rope_cos = table;
      p->dev.rope_sin = table + half;
    }
    p->rope_table = dev_rope_table;
    p->ws = dev_workspace;
    *out_plan = p;
    return TSR_OK;
  });
}

void set_error(const std::string& msg) { g_error = msg; }

}  // namespace tsr

using namespace tsr;

extern "C" {

int32_t tsr_abi_version(void) { return TSR_ABI_VERSION; }

const char* tsr_last_error(void) { return g_error.c_str(); }

size_t tsr_rope_table_bytes(const tsr_model* model) {
  if (check_model(model) != TSR_OK) return 0;
  return 2 * (size_t)model->max_position * (size_t)(model->head_dim / 2) * sizeof(float);
}

tsr_status tsr_rope_table_init(const tsr_model* model, void* dev_table,
                               size_t table_bytes, void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_model(model);
    if (st != TSR_OK) return st;
    const size_t need = tsr_rope_table_bytes(model);
    if (!dev_table || table_bytes < need) {
      set_error("RoPE table buffer is NULL or smaller than tsr_rope_table_bytes()");
      return TSR_ERR_INVALID_ARG;
    }
    const int half = model->head_dim / 2;
    const size_t n = (size_t)model->max_position * half;
    std::vector<double> inv(half);
    for (int i = 0; i < half; ++i)
      inv[i] = std::pow(model->rope_theta, -2.0 * i / model->head_dim);
    std::vector<float> host(2 * n);
    for (int p = 0; p < model->max_position; ++p)
      for (int i = 0; i < half; ++i) {
        const double a = (double)p * inv[i];
        host[(size_t)p * half + i] = (float)std::cos(a);
        host[n + (size_t)p * half + i] = (float)std::sin(a);
      }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(dev_table, host.data(), 2 * n * sizeof(float),
                                  hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return device_fail("hipMemcpyAsync(rope table)", e);
    e = hipStreamSynchronize(s);  // the host image dies with this call
    if (e != hipSuccess) return device_fail("hipStreamSynchronize(rope table)", e);
    return TSR_OK;
  });
}

size_t tsr_plan_workspace_size(const tsr_model* model, const tsr_request* reqs,
                               int32_t n_req, int32_t n_pool_pages,
                               int32_t n_req_pages) {
  return tsr_plan_workspace_size_ex(model, reqs, n_req, n_pool_pages, n_req_pages, nullptr);
}

size_t tsr_plan_workspace_size_ex(const tsr_model* model, const tsr_request* reqs,
                                  int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                                  const tsr_plan_options* options) {
  return plan_workspace_size(model, reqs, n_req, n_pool_pages, n_req_pages, options, false);
}

tsr_status tsr_plan_create(const tsr_model* model, const tsr_request* reqs,
                           int32_t n_req, int32_t n_pool_pages,
                           int32_t n_req_pages, const void* dev_rope_table,
                           void* dev_workspace, size_t workspace_bytes,
                           void* stream, tsr_plan** out_plan) {
  return tsr_plan_create_ex(model, reqs, n_req, n_pool_pages, n_req_pages, nullptr,
                            dev_rope_table, dev_workspace, workspace_bytes, stream, out_plan);
}

tsr_status tsr_plan_create_ex(const tsr_model* model, const tsr_request* reqs,
                              int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                              const tsr_plan_options* options, const void* dev_rope_table,
                              void* dev_workspace, size_t workspace_bytes, void* stream,
                              tsr_plan** out_plan) {
  return create_plan(model, reqs, n_req, n_pool_pages, n_req_pages, options, false,
                     dev_rope_table, dev_workspace, workspace_bytes, stream, out_plan);
}

int32_t tsr_plan_num_compute_tokens(const tsr_plan* p) { return p ? p->T : -1; }
int32_t tsr_plan_num_gather_tokens(const tsr_plan* p) { return p ? p->n_gather : -1; }
int32_t tsr_plan_num_retain_tokens(const tsr_plan* p) { return p ? p->n_retain : -1; }
int32_t tsr_plan_num_attn_items(const tsr_plan* p) { return p ? p->n_items : -1; }
int32_t tsr_plan_attn_rows_per_item(const tsr_plan* p) {
  return p ? kTileRows * p->row_blocks : -1;
}
int32_t tsr_plan_num_aliased_pages(const tsr_plan* p) { return p ? p->n_aliased : -1; }
int32_t tsr_plan_num_attn_splits(const tsr_plan* p) { return p ? p->n_split_items : -1; }
int32_t tsr_plan_num_aliased_k_pages(const tsr_plan* p) { return p ? p->n_aliased_k : -1; }

int32_t tsr_plan_num_attn_items_part(const tsr_plan* p, int32_t part) {
  if (!p || part < TSR_ATTN_ALL || part > TSR_ATTN_AFTER_COMPOSE) return -1;
  return part == TSR_ATTN_ALL ? p->n_items : p->n_items_part[part - 1];
}

tsr_status tsr_plan_compute_positions(const tsr_plan* p, int32_t* host_positions,
                                      int32_t* host_requests) {
  if (!p || !host_positions) {
    set_error("plan or host_positions is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  if (p->T) std::memcpy(host_positions, p->row_pos.data(), p->T * sizeof(int32_t));
  if (host_requests && p->T)
    std::memcpy(host_requests, p->row_req.data(), p->T * sizeof(int32_t));
  return TSR_OK;
}

tsr_status tsr_plan_row_kv_lo(const tsr_plan* p, int32_t* host_kv_lo) {
  if (!p || !host_kv_lo) {
    set_error("plan or host_kv_lo is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  if (p->T) std::memcpy(host_kv_lo, p->row_lo.data(), p->T * sizeof(int32_t));
  return TSR_OK;
}

void tsr_plan_destroy(tsr_plan* p) { delete p; }

tsr_status tsr_compose_kv(const tsr_plan* p, const void* pool_k,
                          const void* pool_v, const float* pool_scale,
                          void* req_k, void* req_v, float* req_scale,
                          int32_t n_layers, int64_t pool_layer_stride,
                          int64_t req_layer_stride, void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_exec(p);
    if (st != TSR_OK) return st;
    if ((st = check_scales(p, pool_scale, req_scale, true, true)) != TSR_OK) return st;
    if (n_layers < 1 || n_layers > 65535) {
      set_error("n_layers must be in [1, 65535]");
      return TSR_ERR_INVALID_ARG;
    }
    if (n_layers > 1 && (pool_layer_stride <= 0 || req_layer_stride <= 0)) {
      set_error("layer strides must be positive when n_layers > 1");
      return TSR_ERR_INVALID_ARG;
    }
    const int64_t elem = p->model.kv_dtype == TSR_F32 ? 4 : is_e4m3(p) ? 1 : 2;
    if (pool_layer_stride % (16 * elem) || req_layer_stride % (16 * elem)) {
      set_error("layer strides must be multiples of 16 elements");
      return TSR_ERR_INVALID_ARG;
    }
    if (p->n_gather == 0) return TSR_OK;
    if (!pool_k || !pool_v || !req_k || !req_v) {
      set_error("compose: a KV pointer is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e =
        is_e4m3(p)
            ? launch_compose_e4m3(p, pool_k, pool_v, pool_scale, req_k, req_v, req_scale,
                                  n_layers, pool_layer_stride, req_layer_stride,
                                  2 * (int64_t)p->n_pool_pages, 2 * (int64_t)p->n_req_pages, s)
            : launch_compose(p, pool_k, pool_v, req_k, req_v, n_layers, pool_layer_stride,
                             req_layer_stride, s);
    if (e != hipSuccess) return device_fail("compose launch", e);
    return TSR_OK;
  });
}

tsr_status tsr_prefill_attn(const tsr_plan* p, const void* q, const void* k,
                            const void* v, void* req_k, void* req_v,
                            float* req_scale, void* out, float* lse,
                            void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_exec(p);
    if (st != TSR_OK) return st;
    if ((st = check_scales(p, nullptr, req_scale, false, true)) != TSR_OK) return st;
    if (p->T == 0) return TSR_OK;
    if (!q || !k || !v || !req_k || !req_v || !out) {
      set_error("prefill_attn: a required pointer is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    if (p->alias_v || p->alias_k) {
      set_error("the plan reads K or V from the pool: use tsr_append_kv and tsr_attn_aliased");
      return TSR_ERR_INVALID_ARG;
    }
    // Every check is above: from here on only a launch failure reported by
    // the runtime can fail the call (append then stays enqueued if the
    // attention launch is the one that fails).
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = is_e4m3(p) ? launch_append_e4m3(p, k, v, req_k, req_v, req_scale, s)
                              : launch_append(p, k, v, req_k, req_v, s);
    if (e != hipSuccess) return device_fail("append launch", e);
    e = is_e4m3(p) ? launch_attn_e4m3(p, p->dev.items, p->n_items, q, req_k, req_v,
                                      req_scale, out, lse, s)
                   : launch_attn(p, TSR_ATTN_ALL, p->dev.items, p->n_items, nullptr, nullptr, q,
                                 req_k, req_v, out,
                                 lse, s);
    if (e != hipSuccess) return device_fail("attention launch", e);
    return TSR_OK;
  });
}

tsr_status tsr_append_kv(const tsr_plan* p, const void* k, const void* v,
                         void* req_k, void* req_v, float* req_scale,
                         void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_exec(p);
    if (st != TSR_OK) return st;
    if ((st = check_scales(p, nullptr, req_scale, false, true)) != TSR_OK) return st;
    if (p->T == 0) return TSR_OK;
    if (!k || !v || !req_k || !req_v) {
      set_error("append_kv: a required pointer is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = is_e4m3(p) ? launch_append_e4m3(p, k, v, req_k, req_v, req_scale, s)
                              : launch_append(p, k, v, req_k, req_v, s);
    if (e != hipSuccess) return device_fail("append launch", e);
    return TSR_OK;
  });
}


tsr_status tsr_assemble_kv(const tsr_plan* p, const void* pool_k, const void* pool_v,
                           const float* pool_scale, const void* k, const void* v,
                           void* req_k, void* req_v, float* req_scale, void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_exec(p);
    if (st != TSR_OK) return st;
    if ((st = check_scales(p, pool_scale, req_scale, p->n_gather > 0, true)) != TSR_OK)
      return st;
    if (p->n_gather == 0 && p->T == 0) return TSR_OK;
    if (!req_k || !req_v || (p->n_gather > 0 && (!pool_k || !pool_v)) ||
        (p->T > 0 && (!k || !v))) {
      set_error("assemble_kv: a required pointer is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = is_e4m3(p) ? launch_assemble_e4m3(p, pool_k, pool_v, pool_scale, k, v,
                                                     req_k, req_v, req_scale, s)
                              : launch_assemble(p, pool_k, pool_v, k, v, req_k, req_v, s);
    if (e != hipSuccess) return device_fail("assembly launch", e);
    return TSR_OK;
  });
}

tsr_status tsr_attn_part(const tsr_plan* p, int32_t part, const void* q,
                         const void* req_k, const void* req_v, const float* req_scale,
                         void* out, float* lse, void* stream) {
  return guarded([&]() -> tsr_status {
    return attn_common(p, part, q, req_k, req_v, nullptr, nullptr, req_scale, out, lse, stream,
                       false);
  });
}

tsr_status tsr_attn_aliased(const tsr_plan* p, int32_t part, const void* q,
                            const void* req_k, const void* req_v, const void* pool_k,
                            const void* pool_v, void* out, float* lse, void* stream) {
  return guarded([&]() -> tsr_status {
    if (!pool_k && !pool_v) {
      set_error("tsr_attn_aliased: pool_k and pool_v are both NULL");
      return TSR_ERR_INVALID_ARG;
    }
    return attn_common(p, part, q, req_k, req_v, pool_k, pool_v, nullptr, out, lse, stream,
                       true);
  });
}

tsr_status tsr_attn(const tsr_plan* p, const void* q, const void* req_k,
                    const void* req_v, const float* req_scale, void* out,
                    float* lse, void* stream) {
  return tsr_attn_part(p, TSR_ATTN_ALL, q, req_k, req_v, req_scale, out, lse, stream);
}

tsr_status tsr_retain_kv(const tsr_plan* p, const void* k, const void* v,
                         void* pool_k, void* pool_v, float* pool_scale,
                         void* stream) {
  return guarded([&]() -> tsr_status {
    tsr_status st = check_exec(p);
    if (st != TSR_OK) return st;
    if ((st = check_scales(p, nullptr, pool_scale, false, true)) != TSR_OK) return st;
    if (p->n_retain == 0) return TSR_OK;
    if (!k || !v || !pool_k || !pool_v) {
      set_error("retain: a required pointer is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = is_e4m3(p) ? launch_retain_e4m3(p, k, v, pool_k, pool_v, pool_scale, s)
                              : launch_retain(p, k, v, pool_k, pool_v, s);
    if (e != hipSuccess) return device_fail("retain launch", e);
    return TSR_OK;
  });
}

}  // extern "C"
