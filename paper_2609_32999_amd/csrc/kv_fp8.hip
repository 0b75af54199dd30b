// KV movement for e4m3 pools: codes plus one power-of-two fp32 scale per
// (page, K|V).  Every request page of an e4m3 plan has a single writer, so a
// workgroup owns one whole page and derives the page scale from the page's
// own values:
//   compose  gathered page: V codes and V scale copied bit for bit; K codes
//            dequantized with the pool scale, rotated in fp32 to the new
//            positions (Section 5.3, "Preparing cache hits") and requantized;
//   append   computed page: k rotated at its positions, k and v quantized;
//   retain   retained pool page: pre-RoPE k and v quantized (Section 5.4).
// Page scale = smallest power of two s with amax / s <= 448 (1 if amax = 0);
// codes are round-to-nearest-even, saturating at +-448 (OCP e4m3fn).
#include <cmath>

#include "kernels_common.h"
#include "tsr_internal.h"

namespace tsr {

namespace {

enum Fp8Mode { kFpCompose = 0, kFpAppend = 1, kFpRetain = 2 };

constexpr int kD8 = 128;           // head dim of the e4m3 path
constexpr int kMaxU = 8;           // most (slot, head, pair-chunk) units per thread

// k such that 2^k is the page scale for this amax.
__device__ __forceinline__ int page_scale_exp(float amax) {
  if (!(amax > 0.0f)) return 0;
  int e;
  const float mfr = frexpf(amax, &e);   // amax = mfr * 2^e, mfr in [0.5, 1)
  // 448 = 0.875 * 2^9: amax <= 448 * 2^k  <=>  mfr * 2^e <= 0.875 * 2^(9 + k)
  return mfr <= 0.875f ? e - 9 : e - 8;
}

// Eight e4m3 codes (one uint2) -> fp32.
__device__ __forceinline__ void decode8(uint2 c, float* o) {
  o[0] = __builtin_amdgcn_cvt_f32_fp8((int)c.x, 0);
  o[1] = __builtin_amdgcn_cvt_f32_fp8((int)c.x, 1);
  o[2] = __builtin_amdgcn_cvt_f32_fp8((int)c.x, 2);
  o[3] = __builtin_amdgcn_cvt_f32_fp8((int)c.x, 3);
  o[4] = __builtin_amdgcn_cvt_f32_fp8((int)c.y, 0);
  o[5] = __builtin_amdgcn_cvt_f32_fp8((int)c.y, 1);
  o[6] = __builtin_amdgcn_cvt_f32_fp8((int)c.y, 2);
  o[7] = __builtin_amdgcn_cvt_f32_fp8((int)c.y, 3);
}

// Eight bf16 values (one uint4 of raw bits) -> fp32.
__device__ __forceinline__ void bf16x8_to_f32(uint4 u, float* o) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = bf16_to_f32(w[i] & 0xffffu);
    o[2 * i + 1] = bf16_to_f32(w[i] >> 16);
  }
}

// Eight fp32 values already divided by the page scale -> e4m3 codes.
__device__ __forceinline__ uint2 encode8(const float* y) {
  uint32_t w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    float a[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = fminf(fmaxf(y[4 * h + i], -448.0f), 448.0f);
    int p = __builtin_amdgcn_cvt_pk_fp8_f32(a[0], a[1], 0, false);
    p = __builtin_amdgcn_cvt_pk_fp8_f32(a[2], a[3], p, true);
    w[h] = (uint32_t)p;
  }
  return make_uint2(w[0], w[1]);
}

// U: (slot, head, pair-chunk) units per thread, at least B * H_kv * 8 / 256
// (instantiated for 2, 4 and 8; each unit holds 16 fp32 values and its raw
// V, so U sets the kernel's registers and with them its occupancy).
template <int MODE, int U>
__device__ __forceinline__ void fp8_page(
    const PageDesc pd, const float* __restrict__ rope_cos,
    const float* __restrict__ rope_sin, const void* __restrict__ src_k,
    const void* __restrict__ src_v, const float* __restrict__ src_scale,
    uint8_t* __restrict__ dst_k, uint8_t* __restrict__ dst_v,
    float* __restrict__ dst_scale, int n_kv_heads, int log2_page,
    int64_t src_layer_stride, int64_t dst_layer_stride,
    int64_t src_scale_stride, int64_t dst_scale_stride) {
  __shared__ float red[2][4];
  const int tid = threadIdx.x;
  const int B = 1 << log2_page;
  const int64_t layer = blockIdx.y;
  const int units = B * n_kv_heads * 8;          // (slot, head, pair-chunk)

  // unit u: pair-chunk c (dims 8c.. and 64+8c..), slot s, head h
  float kv[U][16];
  float amax_k = 0.0f, amax_v = 0.0f;
  // a thread's units share their chunk and, for pages of at most 32 slots,
  // their slot: the cos/sin row is then loaded once
  float cs[8], sn[8];
  const bool one_slot = log2_page <= 5;
  uint4 vraw[U][2];         // V source: e4m3 codes (compose, low 8 bytes) or bf16
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = tid + 256 * k;
    if (u >= units) break;
    const int c = u & 7, s = (u >> 3) & (B - 1), h = u >> (3 + log2_page);
    if (s >= pd.n) continue;
    float* x = kv[k];
    if constexpr (MODE == kFpCompose) {
      const uint8_t* sk = static_cast<const uint8_t*>(src_k) + layer * src_layer_stride;
      const uint8_t* sv = static_cast<const uint8_t*>(src_v) + layer * src_layer_stride;
      const int64_t sb = ((((int64_t)pd.src * n_kv_heads + h) << log2_page) + s) * kD8;
      const float ks = src_scale[layer * src_scale_stride + 2 * pd.src];
      decode8(*reinterpret_cast<const uint2*>(sk + sb + 8 * c), x);
      decode8(*reinterpret_cast<const uint2*>(sk + sb + 64 + 8 * c), x + 8);
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] *= ks;       // exact: power of two
      const uint2 a = *reinterpret_cast<const uint2*>(sv + sb + 8 * c);
      const uint2 b = *reinterpret_cast<const uint2*>(sv + sb + 64 + 8 * c);
      vraw[k][0] = make_uint4(a.x, a.y, 0, 0);
      vraw[k][1] = make_uint4(b.x, b.y, 0, 0);
    } else {
      const uint16_t* sk = static_cast<const uint16_t*>(src_k);
      const uint16_t* sv = static_cast<const uint16_t*>(src_v);
      const int64_t sb = ((int64_t)(pd.src + s) * n_kv_heads + h) * kD8;
      load8(sk + sb + 8 * c, x);
      load8(sk + sb + 64 + 8 * c, x + 8);
      vraw[k][0] = *reinterpret_cast<const uint4*>(sv + sb + 8 * c);
      vraw[k][1] = *reinterpret_cast<const uint4*>(sv + sb + 64 + 8 * c);
      float v[16];
      bf16x8_to_f32(vraw[k][0], v);
      bf16x8_to_f32(vraw[k][1], v + 8);
#pragma unroll
      for (int i = 0; i < 16; ++i) amax_v = fmaxf(amax_v, fabsf(v[i]));
    }
    if constexpr (MODE != kFpRetain) {
      if (k == 0 || !one_slot) {
        load8(rope_cos + (int64_t)(pd.pos + s) * (kD8 / 2) + 8 * c, cs);
        load8(rope_sin + (int64_t)(pd.pos + s) * (kD8 / 2) + 8 * c, sn);
      }
      rope_rotate<8>(x, x + 8, cs, sn);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) amax_k = fmaxf(amax_k, fabsf(x[i]));
  }

  // page-wide amax (K and V together)
  for (int o = 32; o > 0; o >>= 1) {
    amax_k = fmaxf(amax_k, __shfl_xor(amax_k, o));
    amax_v = fmaxf(amax_v, __shfl_xor(amax_v, o));
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = amax_k;
    red[1][tid >> 6] = amax_v;
  }
  __syncthreads();
  amax_k = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  amax_v = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
  const int ek = page_scale_exp(amax_k);
  const int ev = page_scale_exp(amax_v);

  uint8_t* dk = dst_k + layer * dst_layer_stride;
  uint8_t* dv = dst_v + layer * dst_layer_stride;
  float* dsc = dst_scale + layer * dst_scale_stride;
  if (tid == 0) {
    dsc[2 * pd.dst] = ldexpf(1.0f, ek);
    dsc[2 * pd.dst + 1] = MODE == kFpCompose
                              ? src_scale[layer * src_scale_stride + 2 * pd.src + 1]
                              : ldexpf(1.0f, ev);
  }
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = tid + 256 * k;
    if (u >= units) break;
    const int c = u & 7, s = (u >> 3) & (B - 1), h = u >> (3 + log2_page);
    if (s >= pd.n) continue;
    const int64_t db = ((((int64_t)pd.dst * n_kv_heads + h) << log2_page) + s) * kD8;
    float y[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) y[i] = ldexpf(kv[k][i], -ek);
    *reinterpret_cast<uint2*>(dk + db + 8 * c) = encode8(y);
    *reinterpret_cast<uint2*>(dk + db + 64 + 8 * c) = encode8(y + 8);
    if constexpr (MODE == kFpCompose) {
      *reinterpret_cast<uint2*>(dv + db + 8 * c) = make_uint2(vraw[k][0].x, vraw[k][0].y);
      *reinterpret_cast<uint2*>(dv + db + 64 + 8 * c) = make_uint2(vraw[k][1].x, vraw[k][1].y);
    } else {
      float v[16];
      bf16x8_to_f32(vraw[k][0], v);
      bf16x8_to_f32(vraw[k][1], v + 8);
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = ldexpf(v[i], -ev);
      *reinterpret_cast<uint2*>(dv + db + 8 * c) = encode8(v);
      *reinterpret_cast<uint2*>(dv + db + 64 + 8 * c) = encode8(v + 8);
    }
  }
}

template <int MODE, int U>
__global__ __launch_bounds__(256) void page_fp8_kernel(
    const PageDesc* __restrict__ pages, const float* __restrict__ rope_cos,
    const float* __restrict__ rope_sin, const void* __restrict__ src_k,
    const void* __restrict__ src_v, const float* __restrict__ src_scale,
    uint8_t* __restrict__ dst_k, uint8_t* __restrict__ dst_v,
    float* __restrict__ dst_scale, int n_kv_heads, int log2_page,
    int64_t src_layer_stride, int64_t dst_layer_stride,
    int64_t src_scale_stride, int64_t dst_scale_stride) {
  fp8_page<MODE, U>(pages[blockIdx.x], rope_cos, rope_sin, src_k, src_v, src_scale, dst_k,
                    dst_v, dst_scale, n_kv_heads, log2_page, src_layer_stride,
                    dst_layer_stride, src_scale_stride, dst_scale_stride);
}

// Assembly of one layer in a single launch: the first n_gpages workgroups
// compose gathered pages, the rest append computed pages.
template <int U>
__global__ __launch_bounds__(256) void page_fp8_assemble_kernel(
    const PageDesc* __restrict__ gpages, int n_gpages, const PageDesc* __restrict__ apages,
    const float* __restrict__ rope_cos, const float* __restrict__ rope_sin,
    const uint8_t* __restrict__ pool_k, const uint8_t* __restrict__ pool_v,
    const float* __restrict__ pool_scale, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint8_t* __restrict__ req_k,
    uint8_t* __restrict__ req_v, float* __restrict__ req_scale, int n_kv_heads,
    int log2_page) {
  if ((int)blockIdx.x < n_gpages)
    fp8_page<kFpCompose, U>(gpages[blockIdx.x], rope_cos, rope_sin, pool_k, pool_v,
                            pool_scale, req_k, req_v, req_scale, n_kv_heads, log2_page,
                            0, 0, 0, 0);
  else
    fp8_page<kFpAppend, U>(apages[blockIdx.x - n_gpages], rope_cos, rope_sin, k, v,
                           nullptr, req_k, req_v, req_scale, n_kv_heads, log2_page, 0, 0,
                           0, 0);
}

int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

template <int MODE>
hipError_t launch_pages(const tsr_plan* p, const PageDesc* pages, int n,
                        const void* sk, const void* sv, const float* ssc,
                        void* dk, void* dv, float* dsc, int n_layers,
                        int64_t ss, int64_t ds, int64_t sss, int64_t dss,
                        hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const tsr_model& m = p->model;
  const int units = m.page_size * m.n_kv_heads * 8;
  if (units > 256 * kMaxU) return hipErrorInvalidValue;   // the planner rejects these
#define TSR_PAGES(UU)                                                                    \
  hipLaunchKernelGGL((page_fp8_kernel<MODE, UU>), dim3(n, n_layers), dim3(256), 0, s, pages, \
                     p->dev.rope_cos, p->dev.rope_sin, sk, sv, ssc,                        \
                     static_cast<uint8_t*>(dk), static_cast<uint8_t*>(dv), dsc,           \
                     m.n_kv_heads, ilog2(m.page_size), ss, ds, sss, dss)
  if (units <= 512) TSR_PAGES(2);
  else if (units <= 1024) TSR_PAGES(4);
  else TSR_PAGES(8);
#undef TSR_PAGES
  return hipGetLastError();
}

}  // namespace

hipError_t launch_assemble_e4m3(const tsr_plan* p, const void* pool_k, const void* pool_v,
                                const float* pool_scale, const void* k, const void* v,
                                void* req_k, void* req_v, float* req_scale, hipStream_t s) {
  const int n = p->n_gpages + p->n_apages;
  if (n <= 0) return hipSuccess;
  const tsr_model& m = p->model;
  const int units = m.page_size * m.n_kv_heads * 8;
  if (units > 256 * kMaxU) return hipErrorInvalidValue;   // the planner rejects these
#define TSR_APAGES(UU)                                                                  \
  hipLaunchKernelGGL((page_fp8_assemble_kernel<UU>), dim3(n), dim3(256), 0, s,          \
                     p->dev.gpages, p->n_gpages, p->dev.apages, p->dev.rope_cos,         \
                     p->dev.rope_sin, static_cast<const uint8_t*>(pool_k),               \
                     static_cast<const uint8_t*>(pool_v), pool_scale,                    \
                     static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),   \
                     static_cast<uint8_t*>(req_k), static_cast<uint8_t*>(req_v), req_scale, \
                     m.n_kv_heads, ilog2(m.page_size))
  if (units <= 512) TSR_APAGES(2);
  else if (units <= 1024) TSR_APAGES(4);
  else TSR_APAGES(8);
#undef TSR_APAGES
  return hipGetLastError();
}

hipError_t launch_compose_e4m3(const tsr_plan* p, const void* pool_k,
                               const void* pool_v, const float* pool_scale,
                               void* req_k, void* req_v, float* req_scale,
                               int32_t n_layers, int64_t pool_stride,
                               int64_t req_stride, int64_t pool_scale_stride,
                               int64_t req_scale_stride, hipStream_t s) {
  return launch_pages<kFpCompose>(p, p->dev.gpages, p->n_gpages, pool_k, pool_v,
                                  pool_scale, req_k, req_v, req_scale, n_layers,
                                  pool_stride, req_stride, pool_scale_stride,
                                  req_scale_stride, s);
}

hipError_t launch_append_e4m3(const tsr_plan* p, const void* k, const void* v,
                              void* req_k, void* req_v, float* req_scale,
                              hipStream_t s) {
  return launch_pages<kFpAppend>(p, p->dev.apages, p->n_apages, k, v, nullptr, req_k,
                                 req_v, req_scale, 1, 0, 0, 0, 0, s);
}

hipError_t launch_retain_e4m3(const tsr_plan* p, const void* k, const void* v,
                              void* pool_k, void* pool_v, float* pool_scale,
                              hipStream_t s) {
  return launch_pages<kFpRetain>(p, p->dev.rpages, p->n_rpages, k, v, nullptr, pool_k,
                                 pool_v, pool_scale, 1, 0, 0, 0, 0, s);
}

}  // namespace tsr
