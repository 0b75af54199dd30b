// A plan whose device image lives in a library-owned device array instead
// of a caller workspace, for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// allocation).  Each GPU the library runs on holds one such array,
// `scratch`, until the process ends; the last plan created this way on a
// device owns it, and plans it replaced are refused from then on.
#include <atomic>
#include <mutex>

#include "tsr_internal.h"

namespace tsr {

// Largest device image a static plan may have (the RAG-8B batch needs about
// 1 MiB, the 32-request agent-memory batch about 6 MiB).
constexpr size_t kStaticPlanBytes = size_t(16) << 20;

static __device__ __align__(256) uint8_t scratch[kStaticPlanBytes];

namespace {

constexpr int kMaxDevices = 64;

std::mutex g_mu;
// device address of `scratch` on each device (set once, with that device
// current) and the generation of the static plan that owns it
void* g_addr[kMaxDevices] = {};
std::atomic<uint64_t> g_gen[kMaxDevices];

}  // namespace

tsr_status check_static_plan(const tsr_plan* p) {
  if (p->static_gen == 0) return TSR_OK;
  if (g_gen[p->static_device].load() != p->static_gen) {
    set_error("static plan superseded: a later tsr_plan_create_static on this device "
              "rewrote the shared plan area");
    return TSR_ERR_STATE;
  }
  return TSR_OK;
}

}  // namespace tsr

using namespace tsr;

extern "C" tsr_status tsr_plan_create_static(const tsr_model* model, const tsr_request* reqs,
                                             int32_t n_req, int32_t n_pool_pages,
                                             int32_t n_req_pages,
                                             const tsr_plan_options* options,
                                             const void* dev_rope_table, void* stream,
                                             tsr_plan** out_plan) {
  return guarded([&]() -> tsr_status {
    if (!out_plan) {
      set_error("out_plan is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    *out_plan = nullptr;
    // size first, on the host, so an oversized batch is refused before any
    // HIP call
    const size_t need =
        plan_workspace_size(model, reqs, n_req, n_pool_pages, n_req_pages, options, true);
    if (need == 0) return TSR_ERR_INVALID_ARG;   // error set by the size query
    if (need > kStaticPlanBytes) {
      set_error("plan image of " + std::to_string(need) + " bytes exceeds the static plan "
                "area of " + std::to_string(kStaticPlanBytes) + " bytes; use tsr_plan_create "
                "with a workspace");
      return TSR_ERR_OUT_OF_RANGE;
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return device_fail("hipGetDevice", e);
    if (dev < 0 || dev >= kMaxDevices) {
      set_error("device ordinal out of range for the static plan area");
      return TSR_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_addr[dev]) {
      void* ptr = nullptr;
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return device_fail("hipGetSymbolAddress(scratch)", e);
      g_addr[dev] = ptr;
    }
    tsr_plan* p = nullptr;
    tsr_status st = create_plan(model, reqs, n_req, n_pool_pages, n_req_pages, options, true,
                                dev_rope_table, g_addr[dev], kStaticPlanBytes, stream, &p);
    if (st != TSR_OK) return st;
    p->static_device = dev;
    p->static_gen = g_gen[dev].fetch_add(1) + 1;
    *out_plan = p;
    return TSR_OK;
  });
}
