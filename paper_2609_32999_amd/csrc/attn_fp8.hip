// Causal GQA prefill attention over an e4m3 request KV (codes + one
// power-of-two scale per (page, K|V)).  Same work decomposition, 32-key tile
// schedule and online softmax as the bf16 kernel (attn.hip); what differs:
//
//   * rotated queries are quantized to e4m3 per (row, head) with the
//     smallest power-of-two scale covering the row (a kernel choice that the
//     CPU oracle mirrors exactly);
//   * S^T = K Q^T runs on the codes with v_mfma_scale_f32_32x32x64_f8f6f4
//     (unit block scales); the row's Q scale and each key's page scale are
//     applied to S afterwards (per lane: one row, four pages per tile);
//   * V codes are dequantized to fp16 (exact for e4m3 values times a
//     power-of-two scale up to 2^7, the most that keeps every code inside
//     fp16's range; a page with a larger V scale becomes NaN, so outputs
//     that depend on it are non-finite rather than silently clipped) while
//     being transposed into LDS,
//     and P V runs in fp16 MFMA as in the bf16 kernel, so P keeps fp16
//     precision (e4m3 P would cost several percent of relative error).
#include <cmath>
#include <type_traits>

#include "kernels_common.h"
#include "tsr_internal.h"

namespace tsr {

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

union Frag8 {
  uint4 u;
  uint32_t w[4];
  f16x8 h;
};

constexpr int kD = 128;
// Keys per tile.  With 64 the kernel spilled about 40 registers inside the
// tile loop; with 32 a wave holds 163 registers, three waves per SIMD.
constexpr int kKT = 32;
constexpr int kKStr = kD + 16;         // bytes per e4m3 K row in LDS
// V^T rows (fp16) are 16-byte aligned and hold each 16-key step permuted as
// keys [0..3, 8..11, 4..7, 12..15], so that the eight keys a lane feeds to
// the PV MFMA are one 16-byte LDS read (as in the bf16 kernel).
constexpr int kVStr = kKT + 8;         // fp16 elements per V^T row in LDS
constexpr int kKBytes = kKT * kKStr;
constexpr int kVElems = kD * kVStr;
constexpr float kLazy = 8.0f;          // lazy-rescale threshold (log2 units)
constexpr float kLazySum = 256.0f;     // 2^kLazy

__device__ __forceinline__ int page_scale_exp(float amax) {
  if (!(amax > 0.0f)) return 0;
  int e;
  const float mfr = frexpf(amax, &e);
  return mfr <= 0.875f ? e - 9 : e - 8;
}

// R: row blocks per workgroup.  Waves 4 b .. 4 b + 3 own the 32 rows of
// row block b; the first four waves stage every K/V tile for all of them
// (three row blocks share each staged tile, which cuts the KV reads per row
// threefold).
template <int G, int R>
__global__ __launch_bounds__(256 * R, 3) void attn_fp8_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ kc,
    const uint8_t* __restrict__ vc, const float* __restrict__ scales,
    const AttnItem* __restrict__ items, const int32_t* __restrict__ bts,
    const AttnRow* __restrict__ arows, const float* __restrict__ rope_cos,
    const float* __restrict__ rope_sin, uint16_t* __restrict__ out,
    float* __restrict__ lse, int n_q_heads, int n_kv_heads, int log2_page,
    float scale_log2e) {
  constexpr int HPW = 1;  // query heads per wave
  __shared__ __attribute__((aligned(16))) uint8_t kmem[2][kKBytes];
  __shared__ __attribute__((aligned(16))) uint16_t vmem[2][kVElems];
  // K page scales of each staged tile's two 16-key blocks
  __shared__ float kscl[2][2];
  // cos (dims 0 .. d/2-1) and sin (d/2 ..) at each row's position, per row
  // block, loaded once and shared by its four head waves (rows padded by 4
  // floats so that the 32 rows of a fragment read fall in different banks)
  __shared__ __attribute__((aligned(16))) float rl[R][32][kD + 4];

  const AttnItem it = items[blockIdx.x];
  if (it.n_rows == 0) return;
  const int tid = threadIdx.x;
  const int wg = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int w = wg & 3;                  // query head slot
  const int rb = wg >> 2;                // row block
  const bool stager = wg < 4;            // waves that stage K and V
  const int lane = tid & 63;
  const int lrow = lane & 31;
  const int lh = lane >> 5;
  const int g = it.kv_head;
  const int page_mask = (1 << log2_page) - 1;
  const int32_t* bt = bts + it.bt_off;
  const int rbase = 32 * rb;
  // item rows are entries of arows: the computed row (q, out, lse) and
  // its position (with three row blocks, each request's rows grouped by
  // first visible key)
  const AttnRow ar = arows[it.row0 + min(rbase + lrow, it.n_rows - 1)];
  const int row = ar.row;
  const int pos = ar.pos;
  {
    const int t = tid & 255, lr = t >> 3, c8 = 8 * (t & 7);
    const int ppos = arows[it.row0 + min(rbase + lr, it.n_rows - 1)].pos;
    float c[8], sn[8];
    load8(rope_cos + (int64_t)ppos * (kD / 2) + c8, c);
    load8(rope_sin + (int64_t)ppos * (kD / 2) + c8, sn);
    store8(&rl[rb][lr][c8], c);
    store8(&rl[rb][lr][kD / 2 + c8], sn);
  }
  // key tiles this wave's rows need: up to their largest position
  int my_ntiles = 1 << 30;
  if constexpr (R > 1) {
    int wmax = rbase + lrow < it.n_rows ? pos : -1;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) wmax = max(wmax, __shfl_xor(wmax, o));
    my_ntiles = __builtin_amdgcn_readfirstlane(wmax + kKT) / kKT;
  }
  __syncthreads();

  // ---- queries: rotate in fp32, quantize per (row, head) to e4m3.  Lane
  // half lh holds dims [32 lh, 32 lh + 32) of both RoPE halves, i.e. the
  // B operands of the two 64-deep k steps.
  i32x8 qf[HPW][2];
  float qs[HPW];
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    // wave w owns query head head0 + w of the group; with G < 4 the spare
    // waves recompute head G-1 and store nothing
    const int hl = G >= 4 ? it.head0 + w + 4 * i : min(w + 4 * i, G - 1);
    const uint16_t* qp = q + ((int64_t)row * n_q_heads + g * G + hl) * kD;
    float lo[32], hi[32];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d0 = 32 * lh + 8 * c;
      float cs[8], sn[8];
      load8(qp + d0, lo + 8 * c);
      load8(qp + d0 + kD / 2, hi + 8 * c);
      load8(&rl[rb][lrow][d0], cs);
      load8(&rl[rb][lrow][kD / 2 + d0], sn);
      rope_rotate<8>(lo + 8 * c, hi + 8 * c, cs, sn);
    }
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < 32; ++e) amax = fmaxf(amax, fmaxf(fabsf(lo[e]), fabsf(hi[e])));
    amax = fmaxf(amax, __shfl_xor(amax, 32));
    const int ek = page_scale_exp(amax);
    qs[i] = ldexpf(1.0f, ek);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const float* x = half ? hi : lo;
#pragma unroll
      for (int wd = 0; wd < 8; ++wd) {
        float a[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          a[e] = fminf(fmaxf(ldexpf(x[4 * wd + e], -ek), -448.0f), 448.0f);
        int p = __builtin_amdgcn_cvt_pk_fp8_f32(a[0], a[1], 0, false);
        p = __builtin_amdgcn_cvt_pk_fp8_f32(a[2], a[3], p, true);
        qf[i][half][wd] = p;
      }
    }
  }

  f32x16 o[HPW][4];
  float m[HPW], l[HPW];
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    m[i] = -INFINITY;
    l[i] = 0.0f;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[i][db][r] = 0.0f;
  }
  bool wave_active[HPW];
#pragma unroll
  for (int i = 0; i < HPW; ++i) wave_active[i] = G >= 4 || (w + 4 * i) < G;

  // ---- global -> register staging.  The two 16-key blocks of a tile each
  // lie in one page.
  // K: one 16-byte chunk per thread: key tid / 8 (block tid / 128), dims
  //    16 (tid % 8) ..
  // V: keys 2 (tid % 16) and 2 (tid % 16) + 1, dims 8 (tid / 16) .. +7
  //    (8 bytes per key); the two keys sit next to each other in the
  //    permuted V^T row.
  uint4 kr;
  uint2 vr[2];
  const int kp2 = tid & 15;               // key pair
  const int vq = kp2 >> 3;                // 16-key block of the pair
  const int vk = 2 * kp2 - 16 * vq;       // first key within its block
  const int vc8 = (tid >> 4) * 8;
  const int vcol = 16 * vq + ((vk >> 2) & 1) * 8 + ((vk >> 3) & 1) * 4 + (vk & 3);   // permuted
  float nks[2], nvs[2];   // page scales of the staged tile (uniform)
  auto load_tile = [&](int j) {
    const int key0 = j * kKT;
    int64_t base[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int kq = key0 + 16 * b;
      const int page = bt[min(kq >> log2_page, it.n_pages - 1)];
      base[b] = ((((int64_t)page * n_kv_heads + g) << log2_page) + (kq & page_mask)) * kD;
      nks[b] = scales[2 * page];
      nvs[b] = scales[2 * page + 1];
    }
    kr = *reinterpret_cast<const uint4*>(kc + ((tid >> 7) ? base[1] : base[0]) +
                                         ((tid >> 3) & 15) * kD + (tid & 7) * 16);
    const int64_t vb = vq ? base[1] : base[0];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
      vr[pb] = *reinterpret_cast<const uint2*>(vc + vb + (vk + pb) * kD + vc8);
    if (key0 + kKT > it.kv_len) {  // last, partial tile
      if (key0 + (tid >> 3) >= it.kv_len) kr = make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        if (key0 + 2 * kp2 + pb >= it.kv_len) vr[pb] = make_uint2(0, 0);
    }
  };
  auto store_tile = [&](int buf) {
    *reinterpret_cast<uint4*>(&kmem[buf][(tid >> 3) * kKStr + (tid & 7) * 16]) = kr;
    if (tid == 0) {
      kscl[buf][0] = nks[0];
      kscl[buf][1] = nks[1];
    }
    // V^T[d][key] in fp16: gather byte e of keys (k0, k1) into one word and
    // convert two codes at a time with the page scale.
    // a page scale above 2^7 can take codes (|c| <= 448) past fp16's
    // 65504: such pages are refused loudly, as NaN values
    const float sp = vq ? nvs[1] : nvs[0];
    const float s = sp <= 128.0f ? sp : __builtin_nanf("");
    uint16_t* vs = vmem[buf];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const uint32_t a0 = half ? vr[0].y : vr[0].x, a1 = half ? vr[1].y : vr[1].x;
#pragma unroll
      for (int e2 = 0; e2 < 2; ++e2) {
        // bytes (k0[e], k1[e], k0[e+1], k1[e+1]) for e = 2*e2 within the word
        const uint32_t sel = e2 ? 0x07030602u : 0x05010400u;
        const uint32_t p01 = __builtin_amdgcn_perm(a1, a0, sel);
        // low word: keys (0,1) at dim e; high word: at dim e + 1
        const f16x2 l01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p01, s, false);
        const f16x2 h01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p01, s, true);
        const int d = vc8 + 4 * half + 2 * e2;
        *reinterpret_cast<uint32_t*>(vs + d * kVStr + vcol) = __builtin_bit_cast(uint32_t, l01);
        *reinterpret_cast<uint32_t*>(vs + (d + 1) * kVStr + vcol) = __builtin_bit_cast(uint32_t, h01);
      }
    }
  };

  // MASK: 0 none, 1 keys past the row's position (tiles reaching past the
  // item's smallest position), 2 also keys below kv_lo (the tile holding it)
  auto tile = [&](int j, auto mask_tag) {
    constexpr int MASK = decltype(mask_tag)::value;
    const uint8_t* ks = kmem[j & 1];
    const uint16_t* vs = vmem[j & 1];
    f32x16 s[HPW][1];
#pragma unroll
    for (int i = 0; i < HPW; ++i)
#pragma unroll
      for (int kb = 0; kb < 1; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[i][kb][r] = 0.0f;
#pragma unroll
    for (int kst = 0; kst < 2; ++kst) {
#pragma unroll
      for (int kb = 0; kb < 1; ++kb) {
        const uint8_t* kp = ks + (32 * kb + lrow) * kKStr + 64 * kst + 32 * lh;
        // both 16-byte halves land in adjacent registers of the operand
        union { uint4 u[2]; i32x8 v; } x;
        x.u[0] = *reinterpret_cast<const uint4*>(kp);
        x.u[1] = *reinterpret_cast<const uint4*>(kp + 16);
        const i32x8 a = x.v;
#pragma unroll
        for (int i = 0; i < HPW; ++i)
          s[i][kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              a, qf[i][kst], s[i][kb], 0, 0, 0, 127, 0, 127);
      }
    }
    // page of S register r: r/8 within the tile; its factor f (Q scale x K
    // page scale x softmax scale x log2 e) is > 0, so P = exp2(f s - m) is
    // one fma and one exp2 per score and each page's row max is f times the
    // max of its raw scores.
    // Lazy rescale on the tile's probability sum (as in attn.hip): P is
    // taken against the running max m; while a lane's sum stays <= 2^kLazy
    // (every P is then exact-range for fp16) no max is taken.  Otherwise
    // (or while m is still -inf) the scores are computed again from the
    // tile in LDS, m moves to the row max, O and l are rescaled and P is
    // recomputed.
    auto scores = [&](int i) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[i][0][r] = 0.0f;
#pragma unroll
      for (int kst = 0; kst < 2; ++kst) {
        const uint8_t* kp = ks + lrow * kKStr + 64 * kst + 32 * lh;
        union { uint4 u[2]; i32x8 v; } x;
        x.u[0] = *reinterpret_cast<const uint4*>(kp);
        x.u[1] = *reinterpret_cast<const uint4*>(kp + 16);
        s[i][0] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            x.v, qf[i][kst], s[i][0], 0, 0, 0, 127, 0, 127);
      }
    };
    auto mask = [&](int i) __attribute__((always_inline)) {
      if constexpr (MASK != 0) {
        // score r holds key j kKT + 8 (r / 4) + 4 lh + r % 4: compare its
        // in-tile offset with the row's bounds moved to the same origin
        const int dhi = pos - 4 * lh - j * kKT;
        const int dlo = it.kv_lo - 4 * lh - j * kKT;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = 8 * (r >> 2) + (r & 3);
          const bool out = MASK == 2 ? (off > dhi || off < dlo) : off > dhi;
          s[i][0][r] = out ? -INFINITY : s[i][0][r];
        }
      }
    };
    f16x8 pf[HPW][2];
#pragma unroll
    for (int i = 0; i < HPW; ++i) {
      float f[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) f[b] = qs[i] * kscl[j & 1][b] * scale_log2e;
      mask(i);
      // row sum in fp32 as four independent chains of plain adds; a row with
      // no visible key yet keeps m at -inf and is exponentiated against 0
      const float mi = m[i] == -INFINITY ? 0.0f : m[i];
      float ls[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[i][0][r], f[r >> 3], -mi));
        s[i][0][r] = p;
        ls[r & 3] += p;
      }
      const float lt = (ls[0] + ls[1]) + (ls[2] + ls[3]);
      if (__builtin_amdgcn_ballot_w64(!(lt <= kLazySum) || m[i] == -INFINITY)) {
        scores(i);
        mask(i);
        float mb[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          float x = s[i][0][8 * b];
#pragma unroll
          for (int r = 1; r < 8; ++r) x = fmaxf(x, s[i][0][8 * b + r]);
          mb[b] = x * f[b];
        }
        const float mt = fmaxf(mb[0], mb[1]);
        const float mn = fmaxf(m[i], fmaxf(mt, __shfl_xor(mt, 32)));
        const float alpha = mn == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f(m[i] - mn);
        m[i] = mn;
        l[i] *= alpha;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[i][db][r] *= alpha;
        const float mi2 = m[i] == -INFINITY ? 0.0f : m[i];
#pragma unroll
        for (int r = 0; r < 4; ++r) ls[r] = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[i][0][r], f[r >> 3], -mi2));
          s[i][0][r] = p;
          ls[r & 3] += p;
        }
      }
      l[i] += (ls[0] + ls[1]) + (ls[2] + ls[3]);
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[i][k2][e] = (_Float16)s[i][0][8 * k2 + e];
      }
    }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        Frag8 a;
        a.u = *reinterpret_cast<const uint4*>(vs + (32 * db + lrow) * kVStr + 16 * k2 + 8 * lh);
#pragma unroll
        for (int i = 0; i < HPW; ++i)
          o[i][db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a.h, pf[i][k2], o[i][db], 0, 0, 0);
      }
    }
  };

  // keys kv_lo .. kv_len-1: tiles j0 .. ntiles-1; a tile needs the mask when
  // it reaches past the smallest row position or starts below kv_lo
  const int ntiles = (it.kv_len + kKT - 1) / kKT;
  const int j0 = it.kv_lo / kKT;
  const int jlo = (it.kv_lo + kKT - 1) / kKT;
  const int nfull = min(ntiles, (it.min_pos + 1) / kKT);
  if (stager) {
    load_tile(j0);
    store_tile(j0 & 1);
  }
  __syncthreads();
  // Three loops (masked head, unmasked body, masked tail) rather than one
  // loop that picks the masked or unmasked tile per iteration: with both
  // variants in one loop body the compiler kept about 90 more registers
  // live.  Tiles past a row block's last row are fully masked for it and
  // skipped (only in the masked tail).
  auto run_tiles = [&](int ja, int jb, auto mask_tag) __attribute__((always_inline)) {
    for (int j = ja; j < jb; ++j) {
      const bool more = j + 1 < ntiles;
      if (more) load_tile(j + 1);
      if (j < my_ntiles) tile(j, mask_tag);
      if (more) store_tile((j + 1) & 1);
      __syncthreads();
    }
  };
  // the waves of the other row blocks stage nothing
  auto run_tiles_ns = [&](int ja, int jb, auto mask_tag) __attribute__((always_inline)) {
    for (int j = ja; j < jb; ++j) {
      if (j < my_ntiles) tile(j, mask_tag);
      __syncthreads();
    }
  };
  const int jl = min(ntiles, max(j0, jlo));
  if (stager) {
    run_tiles(j0, jl, std::integral_constant<int, 2>{});
    run_tiles(jl, max(jl, nfull), std::integral_constant<int, 0>{});
    run_tiles(max(jl, nfull), ntiles, std::integral_constant<int, 1>{});
  } else {
    run_tiles_ns(j0, jl, std::integral_constant<int, 2>{});
    run_tiles_ns(jl, max(jl, nfull), std::integral_constant<int, 0>{});
    run_tiles_ns(max(jl, nfull), ntiles, std::integral_constant<int, 1>{});
  }

  // ---- epilogue
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    if (!wave_active[i]) continue;
    const float lt = l[i] + __shfl_xor(l[i], 32);
    if (rbase + lrow >= it.n_rows) continue;
    const float inv = 1.0f / lt;
    const int hq = g * G + (G >= 4 ? it.head0 : 0) + w + 4 * i;
    uint16_t* op = out + ((int64_t)row * n_q_heads + hq) * kD;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int d0 = 32 * db + 8 * rg + 4 * lh;
        uint2 v;
        v.x = f32_to_bf16(o[i][db][4 * rg] * inv) | (f32_to_bf16(o[i][db][4 * rg + 1] * inv) << 16);
        v.y = f32_to_bf16(o[i][db][4 * rg + 2] * inv) | (f32_to_bf16(o[i][db][4 * rg + 3] * inv) << 16);
        *reinterpret_cast<uint2*>(op + d0) = v;
      }
    // lse (natural log) = (m + log2 l) * ln 2 with m in log2 units
    if (lse && lh == 0)
      lse[(int64_t)row * n_q_heads + hq] = (m[i] + log2f(lt)) * 0.69314718055994531f;
  }
}

int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

}  // namespace

hipError_t launch_attn_e4m3(const tsr_plan* p, const AttnItem* items, int32_t n_items,
                            const void* q, const void* req_k,
                            const void* req_v, const float* req_scale, void* out,
                            float* lse, hipStream_t s) {
  if (n_items == 0 || p->T == 0) return hipSuccess;
  const tsr_model& m = p->model;
  const int lp = ilog2(m.page_size);
  const int G = m.n_q_heads / m.n_kv_heads;
  const float sl2e = (float)((double)p->scale * 1.4426950408889634);
#define TSR_FP8(GG)                                                                   \
  if (p->row_blocks == kMaxRowBlocks)                                                 \
    TSR_FP8_R(GG, kMaxRowBlocks);                                                     \
  else                                                                                \
    TSR_FP8_R(GG, 1)
#define TSR_FP8_R(GG, RB)                                                             \
  hipLaunchKernelGGL((attn_fp8_kernel<GG, RB>), dim3(n_items), dim3(256 * (RB)), 0, s, \
                     static_cast<const uint16_t*>(q), static_cast<const uint8_t*>(req_k), \
                     static_cast<const uint8_t*>(req_v), req_scale, items,            \
                     p->dev.block_tables, p->dev.attn_rows, p->dev.rope_cos,          \
                     p->dev.rope_sin, static_cast<uint16_t*>(out), lse, m.n_q_heads,  \
                     m.n_kv_heads, lp, sl2e)
  switch (G) {
    case 1: TSR_FP8(1); break;
    case 2: TSR_FP8(2); break;
    case 4: TSR_FP8(4); break;
    case 8: TSR_FP8(8); break;
    default: return hipErrorInvalidValue;
  }
#undef TSR_FP8
#undef TSR_FP8_R
  return hipGetLastError();
}

}  // namespace tsr
