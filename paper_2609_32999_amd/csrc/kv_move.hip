// KV movement kernels of the composed-prefill path.  All three are bound by
// HBM bandwidth: every byte is read once and written once.
//
//   compose  cached HIT tokens: pool slot -> request slot; V copied bit for
//            bit, K re-rotated from its pre-RoPE form to the token's new
//            prompt position (Section 5.3, "Preparing cache hits").
//   append   computed rows: k rotated at its own position and v written into
//            the request slots before attention (Section 5.3, "Completing
//            prefill").
//   retain   computed MISS units: pre-RoPE k and v copied into the unit's
//            pool blocks, token j at block j / B, slot j % B (Sections 5.1,
//            5.4).
//
// Layout of pages: [page][H_kv][B][d].  A thread owns 8 elements of the low
// half of a (token, head) row and the 8 matching elements of the high half,
// which are exactly the RoPE pairs (i, i + d/2) it rotates.  A workgroup owns
// 16 tokens and walks all KV heads, so consecutive threads touch consecutive
// slots of a page and each thread loads its cos/sin row once.
#include "kernels_common.h"
#include "tsr_internal.h"

namespace tsr {

namespace {

enum MoveMode { kCompose = 0, kAppend = 1, kRetain = 2 };

constexpr int kTok = 16;     // descriptors per workgroup
constexpr int kThreads = 256;

template <int D, typename T, int MODE>
__global__ __launch_bounds__(kThreads) void kv_move_kernel(
    const void* __restrict__ descs, int n, const float* __restrict__ rope_cos,
    const float* __restrict__ rope_sin, const T* __restrict__ src_k,
    const T* __restrict__ src_v, T* __restrict__ dst_k, T* __restrict__ dst_v,
    int n_kv_heads, int log2_page, int64_t src_layer_stride,
    int64_t dst_layer_stride) {
  constexpr int kCh = D / 16;                       // threads per (token, head)
  constexpr int kHeadStep = kThreads / (kCh * kTok);
  static_assert(kHeadStep >= 1, "head_dim too large for the thread mapping");
  const int tid = threadIdx.x;
  const int c = tid % kCh;
  const int tl = (tid / kCh) % kTok;
  const int h0 = tid / (kCh * kTok);
  const int i = blockIdx.x * kTok + tl;
  if (i >= n) return;  // this kernel has no barriers

  const int64_t layer = blockIdx.y;
  src_k += layer * src_layer_stride;
  src_v += layer * src_layer_stride;
  dst_k += layer * dst_layer_stride;
  dst_v += layer * dst_layer_stride;

  int32_t src, dst, pos = 0;
  if constexpr (MODE == kCompose) {
    const GatherDesc gd = static_cast<const GatherDesc*>(descs)[i];
    src = gd.src; dst = gd.dst; pos = gd.pos;
  } else if constexpr (MODE == kAppend) {
    const RowDesc rd = static_cast<const RowDesc*>(descs)[i];
    src = i; dst = rd.dst; pos = rd.pos;
  } else {
    const RetainDesc rd = static_cast<const RetainDesc*>(descs)[i];
    src = rd.row; dst = rd.dst;
  }
  const int page_mask = (1 << log2_page) - 1;

  float cs[8], sn[8];
  if constexpr (MODE != kRetain) {
    load8(rope_cos + (int64_t)pos * (D / 2) + c * 8, cs);
    load8(rope_sin + (int64_t)pos * (D / 2) + c * 8, sn);
  }
  for (int h = h0; h < n_kv_heads; h += kHeadStep) {
    int64_t sb;
    if constexpr (MODE == kCompose)
      sb = ((((int64_t)(src >> log2_page) * n_kv_heads + h) << log2_page) +
            (src & page_mask)) * D;
    else
      sb = ((int64_t)src * n_kv_heads + h) * D;
    const int64_t db = ((((int64_t)(dst >> log2_page) * n_kv_heads + h) << log2_page) +
                        (dst & page_mask)) * D;
    const int lo = c * 8, hi = D / 2 + c * 8;
    copy8(dst_v + db + lo, src_v + sb + lo);
    copy8(dst_v + db + hi, src_v + sb + hi);
    if constexpr (MODE == kRetain) {
      copy8(dst_k + db + lo, src_k + sb + lo);
      copy8(dst_k + db + hi, src_k + sb + hi);
    } else {
      float a[8], b[8];
      load8(src_k + sb + lo, a);
      load8(src_k + sb + hi, b);
      rope_rotate<8>(a, b, cs, sn);
      store8(dst_k + db + lo, a);
      store8(dst_k + db + hi, b);
    }
  }
}

int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

template <typename T, int MODE>
hipError_t launch_move_t(const tsr_plan* p, const void* descs, int n,
                         const void* sk, const void* sv, void* dk, void* dv,
                         int n_layers, int64_t src_stride_bytes,
                         int64_t dst_stride_bytes, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const tsr_model& m = p->model;
  const dim3 grid((n + kTok - 1) / kTok, n_layers);
  const int64_t ss = src_stride_bytes / (int64_t)sizeof(T);
  const int64_t ds = dst_stride_bytes / (int64_t)sizeof(T);
  const int lp = ilog2(m.page_size);
#define TSR_MOVE(DIM)                                                          \
  hipLaunchKernelGGL((kv_move_kernel<DIM, T, MODE>), grid, dim3(kThreads), 0, s, \
                     descs, n, p->dev.rope_cos, p->dev.rope_sin,                \
                     static_cast<const T*>(sk), static_cast<const T*>(sv),      \
                     static_cast<T*>(dk), static_cast<T*>(dv), m.n_kv_heads,    \
                     lp, ss, ds)
  switch (m.head_dim) {
    case 64: TSR_MOVE(64); break;
    case 128: TSR_MOVE(128); break;
    case 256: TSR_MOVE(256); break;
    default: return hipErrorInvalidValue;
  }
#undef TSR_MOVE
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_move(const tsr_plan* p, const void* descs, int n,
                       const void* sk, const void* sv, void* dk, void* dv,
                       int n_layers, int64_t ss, int64_t ds, hipStream_t s) {
  if (p->model.kv_dtype == TSR_F32)
    return launch_move_t<float, MODE>(p, descs, n, sk, sv, dk, dv, n_layers, ss, ds, s);
  return launch_move_t<uint16_t, MODE>(p, descs, n, sk, sv, dk, dv, n_layers, ss, ds, s);
}

}  // namespace

hipError_t launch_compose(const tsr_plan* p, const void* pool_k,
                          const void* pool_v, void* req_k, void* req_v,
                          int32_t n_layers, int64_t pool_stride,
                          int64_t req_stride, hipStream_t s) {
  return launch_move<kCompose>(p, p->dev.gather, p->n_gather, pool_k, pool_v,
                               req_k, req_v, n_layers, pool_stride, req_stride, s);
}

hipError_t launch_append(const tsr_plan* p, const void* k, const void* v,
                         void* req_k, void* req_v, hipStream_t s) {
  return launch_move<kAppend>(p, p->dev.rows, p->T, k, v, req_k, req_v, 1, 0, 0, s);
}

hipError_t launch_retain(const tsr_plan* p, const void* k, const void* v,
                         void* pool_k, void* pool_v, hipStream_t s) {
  return launch_move<kRetain>(p, p->dev.retain, p->n_retain, k, v, pool_k, pool_v,
                              1, 0, 0, s);
}

}  // namespace tsr
