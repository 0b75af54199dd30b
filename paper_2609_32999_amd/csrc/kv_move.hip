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

// Eight raw storage elements held in registers (16 bytes for bf16, 32 for
// fp32), loaded non-temporally: every source row is read exactly once.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Vec8;
template <> struct Vec8<uint16_t> {
  u32x4 u;
  __device__ void load(const uint16_t* p) {
    u = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  }
  __device__ void store(uint16_t* p) const { *reinterpret_cast<u32x4*>(p) = u; }
  __device__ void to_f32(float* o) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = bf16_to_f32(u[i] & 0xffffu);
      o[2 * i + 1] = bf16_to_f32(u[i] >> 16);
    }
  }
};
template <> struct Vec8<float> {
  f32x4 a, b;
  __device__ void load(const float* p) {
    a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
  }
  __device__ void store(float* p) const {
    *reinterpret_cast<f32x4*>(p) = a;
    *reinterpret_cast<f32x4*>(p + 4) = b;
  }
  __device__ void to_f32(float* o) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[i] = a[i];
      o[4 + i] = b[i];
    }
  }
};

constexpr int kTok = 16;     // descriptors per workgroup
constexpr int kThreads = 256;

// The tokens of one workgroup: descriptor i = blk * kTok + (thread's token)
// of `descs` (n of them), moved as MODE says.  No barriers.
template <int D, typename T, int MODE>
__device__ __forceinline__ void move_tokens(
    int blk, const void* __restrict__ descs, int n, const float* __restrict__ rope_cos,
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
  const int i = blk * kTok + tl;
  if (i >= n) return;

  const int64_t layer = blockIdx.y;
  src_k += layer * src_layer_stride;
  src_v += layer * src_layer_stride;
  dst_k += layer * dst_layer_stride;
  dst_v += layer * dst_layer_stride;

  int32_t src, dst, pos = 0;
  // false: attention reads this token's V (K) from the pool (aliasing)
  bool move_v = true, move_k = true;
  if constexpr (MODE == kCompose) {
    const GatherDesc gd = static_cast<const GatherDesc*>(descs)[i];
    src = gd.src; dst = gd.dst; pos = gd.pos;
    move_v = (gd.skip & kSkipV) == 0;
    move_k = (gd.skip & kSkipK) == 0;
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
  // Issue the loads of up to kBatch heads before any store so that each
  // thread keeps several 16-byte requests in flight.
  constexpr int kBatch = 4;
  const int lo = c * 8, hi = D / 2 + c * 8;
  auto src_off = [&](int h) -> int64_t {
    if constexpr (MODE == kCompose)
      return ((((int64_t)(src >> log2_page) * n_kv_heads + h) << log2_page) +
              (src & page_mask)) * D;
    else
      return ((int64_t)src * n_kv_heads + h) * D;
  };
  auto dst_off = [&](int h) -> int64_t {
    return ((((int64_t)(dst >> log2_page) * n_kv_heads + h) << log2_page) +
            (dst & page_mask)) * D;
  };
  for (int hb = h0; hb < n_kv_heads; hb += kBatch * kHeadStep) {
    Vec8<T> kl[kBatch], kh[kBatch], vl[kBatch], vh[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int h = hb + b * kHeadStep;
      if (h < n_kv_heads) {
        const int64_t sb = src_off(h);
        if (move_k) {
          kl[b].load(src_k + sb + lo);
          kh[b].load(src_k + sb + hi);
        }
        if (move_v) {
          vl[b].load(src_v + sb + lo);
          vh[b].load(src_v + sb + hi);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int h = hb + b * kHeadStep;
      if (h < n_kv_heads) {
        const int64_t db = dst_off(h);
        if (move_v) {
          vl[b].store(dst_v + db + lo);
          vh[b].store(dst_v + db + hi);
        }
        if constexpr (MODE == kRetain) {
          kl[b].store(dst_k + db + lo);
          kh[b].store(dst_k + db + hi);
        } else if (move_k) {
          float a[8], bb[8];
          kl[b].to_f32(a);
          kh[b].to_f32(bb);
          rope_rotate<8>(a, bb, cs, sn);
          store8(dst_k + db + lo, a);
          store8(dst_k + db + hi, bb);
        }
      }
    }
  }
}

template <int D, typename T, int MODE>
__global__ __launch_bounds__(kThreads) void kv_move_kernel(
    const void* __restrict__ descs, int n, const float* __restrict__ rope_cos,
    const float* __restrict__ rope_sin, const T* __restrict__ src_k,
    const T* __restrict__ src_v, T* __restrict__ dst_k, T* __restrict__ dst_v,
    int n_kv_heads, int log2_page, int64_t src_layer_stride,
    int64_t dst_layer_stride) {
  move_tokens<D, T, MODE>(blockIdx.x, descs, n, rope_cos, rope_sin, src_k, src_v, dst_k,
                          dst_v, n_kv_heads, log2_page, src_layer_stride,
                          dst_layer_stride);
}

// Assembly of one layer's request KV in a single launch: the first
// ceil(n_gather / kTok) workgroups compose cached tokens, the rest append
// the computed rows.  Both movers are bound by HBM bandwidth; one launch
// spares the second kernel's launch and ramp.
template <int D, typename T>
__global__ __launch_bounds__(kThreads) void kv_assemble_kernel(
    const GatherDesc* __restrict__ gather, int n_gather, const RowDesc* __restrict__ rows,
    int n_rows, const float* __restrict__ rope_cos, const float* __restrict__ rope_sin,
    const T* __restrict__ pool_k, const T* __restrict__ pool_v, const T* __restrict__ k,
    const T* __restrict__ v, T* __restrict__ req_k, T* __restrict__ req_v,
    int n_kv_heads, int log2_page) {
  const int gblocks = (n_gather + kTok - 1) / kTok;
  if ((int)blockIdx.x < gblocks)
    move_tokens<D, T, kCompose>(blockIdx.x, gather, n_gather, rope_cos, rope_sin, pool_k,
                                pool_v, req_k, req_v, n_kv_heads, log2_page, 0, 0);
  else
    move_tokens<D, T, kAppend>(blockIdx.x - gblocks, rows, n_rows, rope_cos, rope_sin, k,
                               v, req_k, req_v, n_kv_heads, log2_page, 0, 0);
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

template <typename T>
hipError_t launch_assemble_t(const tsr_plan* p, const void* pool_k, const void* pool_v,
                             const void* k, const void* v, void* req_k, void* req_v,
                             hipStream_t s) {
  const int gb = (p->n_gather + kTok - 1) / kTok, ab = (p->T + kTok - 1) / kTok;
  if (gb + ab == 0) return hipSuccess;
  const tsr_model& m = p->model;
  const int lp = ilog2(m.page_size);
#define TSR_ASM(DIM)                                                                  \
  hipLaunchKernelGGL((kv_assemble_kernel<DIM, T>), dim3(gb + ab), dim3(kThreads), 0, s, \
                     p->dev.gather, p->n_gather, p->dev.rows, p->T, p->dev.rope_cos,   \
                     p->dev.rope_sin, static_cast<const T*>(pool_k),                   \
                     static_cast<const T*>(pool_v), static_cast<const T*>(k),          \
                     static_cast<const T*>(v), static_cast<T*>(req_k),                 \
                     static_cast<T*>(req_v), m.n_kv_heads, lp)
  switch (m.head_dim) {
    case 64: TSR_ASM(64); break;
    case 128: TSR_ASM(128); break;
    case 256: TSR_ASM(256); break;
    default: return hipErrorInvalidValue;
  }
#undef TSR_ASM
  return hipGetLastError();
}

}  // namespace

hipError_t launch_assemble(const tsr_plan* p, const void* pool_k, const void* pool_v,
                           const void* k, const void* v, void* req_k, void* req_v,
                           hipStream_t s) {
  if (p->model.kv_dtype == TSR_F32)
    return launch_assemble_t<float>(p, pool_k, pool_v, k, v, req_k, req_v, s);
  return launch_assemble_t<uint16_t>(p, pool_k, pool_v, k, v, req_k, req_v, s);
}

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
