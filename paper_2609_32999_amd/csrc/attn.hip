// Causal GQA prefill attention of the computed rows over the assembled KV
// (Section 5.3, "Completing prefill": the recompute ranges and the remaining
// prompt are processed in one extend pass).
//
// Row t at prompt position p_t, query head h, KV head g = h / G:
//   o = softmax(scale * q_rot . K[0..p_t, g]^T) V[0..p_t, g]
// with q_rot = RoPE(q, p_t) rounded to the activation dtype and keys visible
// up to and including p_t.
//
// Three kernels:
//   attn_f32_kernel   fp32 reference mode, scalar, one workgroup per item.
//   attn_mfma_kernel  bf16 mode.  Work item = R row blocks of up to 32
//                     rows of one request x one KV head (R = 1 or 3, chosen
//                     per plan), consecutive in the plan's item row order
//                     (AttnRow: with R = 3 the rows of each request grouped
//                     by first visible key); the query heads of that
//                     KV head are packed into the workgroup (four waves per
//                     row block, one head each; G = 8 takes two items), so
//                     every K/V tile staged in LDS feeds all of them.  Per
//                     32-key tile (K loaded straight into
//                     LDS, V staged through registers as V^T in fp16):
//                       S^T = K Q^T        v_mfma_f32_32x32x16_bf16
//                       online softmax     fp32, exp2 with folded scale;
//                                          the running max moves only when
//                                          a tile's probability sum says so
//                       O^T += V^T P^T     v_mfma_f32_32x32x16_f16
//                     Keeping S and O transposed gives every lane one query
//                     row, so row statistics are lane-local except for one
//                     exchange between the two half-waves.  P and V enter the
//                     second product as fp16 (bf16 P would cost ~2e-3
//                     relative error; fp16 keeps it near 2e-4).  A wave
//                     holds at most 168 registers, so three waves share each
//                     SIMD.  LDS per workgroup: 36 KB of K/V tiles plus
//                     16.5 KB of cos/sin rows per row block, 52.5 KB with
//                     one row block (three 4-wave workgroups per CU) and
//                     85.5 KB with three (one 12-wave workgroup per CU).
//                     An item whose key range the plan split writes its
//                     normalized rows and log-sum-exp in fp32 instead (one
//                     split buffer slot per row block).
//   attn_merge_kernel merges the key ranges of split items into out, lse.
#include <cmath>
#include <type_traits>

#include "attn_common.h"
#include "kernels_common.h"
#include "tsr_internal.h"

namespace tsr {

namespace {

// ------------------------------------------------------------- fp32 mode
// The reference mode of the fp32 configurations: operands are fp32 (q_rot
// and K rounded to fp32 like the storage), the arithmetic is fp64 (scores,
// softmax statistics and the weighted sum of V), and the output is rounded
// to fp32 once.  One workgroup per item, scalar code: its job is accuracy.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc,
    const float* __restrict__ vc, const AttnItem* __restrict__ items,
    const int32_t* __restrict__ bts, const RowDesc* __restrict__ rows,
    const float* __restrict__ rope_cos, const float* __restrict__ rope_sin,
    float* __restrict__ out, float* __restrict__ lse, int n_q_heads,
    int n_kv_heads, int log2_page, float scale) {
  __shared__ float qs[D];
  __shared__ double ps[256];
  __shared__ double red[8];
  const AttnItem it = items[blockIdx.x];
  if (it.n_rows == 0) return;
  const int t = threadIdx.x;
  const int G = n_q_heads / n_kv_heads;
  const int g = it.kv_head;
  const int page_mask = (1 << log2_page) - 1;
  const int32_t* bt = bts + it.bt_off;

  auto block_max = [&](double v) {
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    if ((t & 63) == 0) red[t >> 6] = v;
    __syncthreads();
    v = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
    __syncthreads();
    return v;
  };
  auto block_sum = [&](double v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((t & 63) == 0) red[4 + (t >> 6)] = v;
    __syncthreads();
    v = (red[4] + red[5]) + (red[6] + red[7]);
    __syncthreads();
    return v;
  };
  auto key_row = [&](const float* base, int k) {
    const int page = bt[k >> log2_page];
    return base + ((((int64_t)page * n_kv_heads + g) << log2_page) + (k & page_mask)) * D;
  };
  const double sc = scale;

  for (int rr = 0; rr < it.n_rows; ++rr) {
    const int row = it.row0 + rr;
    const int pos = rows[row].pos;
    for (int hh = 0; hh < G; ++hh) {
      const int hq = g * G + hh;
      const float* qp = q + ((int64_t)row * n_q_heads + hq) * D;
      if (t < D / 2) {
        float lo = qp[t], hi = qp[t + D / 2];
        const float c = rope_cos[(int64_t)pos * (D / 2) + t];
        const float s = rope_sin[(int64_t)pos * (D / 2) + t];
        rope_rotate<1>(&lo, &hi, &c, &s);
        qs[t] = lo;
        qs[t + D / 2] = hi;
      }
      __syncthreads();
      double m = -INFINITY, l = 0.0, o = 0.0;
      for (int k0 = it.kv_lo; k0 <= pos; k0 += 256) {
        const int k = k0 + t;
        double s = -INFINITY;
        if (k <= pos) {
          const float* kp = key_row(kc, k);
          double acc = 0.0;
          for (int e = 0; e < D; ++e) acc = fma((double)qs[e], (double)kp[e], acc);
          s = acc * sc;
        }
        const double mn = fmax(m, block_max(s));
        const double p = (k <= pos) ? exp(s - mn) : 0.0;
        ps[t] = p;
        const double alpha = exp(m - mn);
        l = l * alpha + block_sum(p);
        if (t < D) {
          const int nk = min(256, pos + 1 - k0);
          double acc = 0.0;
          for (int j = 0; j < nk; ++j) acc = fma(ps[j], (double)key_row(vc, k0 + j)[t], acc);
          o = o * alpha + acc;
        }
        m = mn;
        __syncthreads();
      }
      if (t < D) out[((int64_t)row * n_q_heads + hq) * D + t] = (float)(o / l);
      if (t == 0 && lse) lse[(int64_t)row * n_q_heads + hq] = (float)(m + log(l));
      __syncthreads();
    }
  }
}

// ------------------------------------------------------------- bf16 mode
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  // bf16 values convert to fp16 exactly inside fp16's normal range (the
  // largest bf16 below fp16's maximum is 65280); the staging code refuses
  // larger magnitudes, which this conversion (toward zero) would clip.
  // (Round-to-nearest-even conversion, which would turn them infinite by
  // itself, made the attention 10 % slower: it sits on the staging waves'
  // path to every tile's barrier.)
  const auto h = __builtin_amdgcn_cvt_pkrtz(a, b);
  return __builtin_bit_cast(uint32_t, h);
}
// fp16 NaN pair: written over a thread's staged V^T values when one of
// them is beyond fp16's range, so outputs that read them are non-finite
// instead of silently clipped.
constexpr uint32_t kF16NaN2 = 0x7E007E00u;

// Masking of a tile's scores (tile loops are instantiated per kind).
constexpr int kNoMask = 0, kMaskCausal = 1, kMaskBoth = 2;
using NoMask = std::integral_constant<int, kNoMask>;
using MaskCausal = std::integral_constant<int, kMaskCausal>;
using MaskBoth = std::integral_constant<int, kMaskBoth>;

// AV: V aliasing -- the V of a 16-key block comes from the page the V block
// table names, a pool page when kPoolPageFlag is set (else the request page
// the K block table names).
// AK: K rotated on load -- the K of a 16-key block comes from the page the K
// block table names; a pool page (kPoolPageFlag) holds the cached keys before
// RoPE, which the staging waves rotate at the keys' positions (fp32 table,
// no fused multiply-add, bf16 rounding: the arithmetic of compose) and write
// to LDS in fragment order.
// R: row blocks per workgroup.  Waves 4 b .. 4 b + 3 own the 32 rows of row
// block b; the first four waves stage every K/V tile for all of them.
template <int G, bool AV, bool AK, int R>
__global__ __launch_bounds__(256 * R, 3) void attn_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, const uint16_t* __restrict__ pool_k,
    const uint16_t* __restrict__ pool_v,
    const AttnItem* __restrict__ items, const int32_t* __restrict__ bts,
    const int32_t* __restrict__ vbts, const int32_t* __restrict__ kbts,
    const AttnRow* __restrict__ arows,
    const float* __restrict__ rope_cos, const float* __restrict__ rope_sin,
    uint16_t* __restrict__ out, float* __restrict__ lse, float* __restrict__ split_o,
    float* __restrict__ split_lse, int n_q_heads, int n_kv_heads, int log2_page, float scale,
    float scale_log2e) {
  // double-buffered K and V^T tiles
  __shared__ __attribute__((aligned(16))) uint8_t kl[2][kKBytes];
  __shared__ __attribute__((aligned(16))) uint16_t vl[2][kVBytes / 2];
  // cos (dims 0 .. d/2-1) and sin (d/2 ..) at each row's position, per row
  // block: loaded once and shared by the block's four head waves (rows
  // padded by 4 floats so that the 32 rows of a fragment read fall in
  // different banks)
  // With K rotated on load the rotated queries move to LDS after the
  // prologue (8 KB per wave, over the cos/sin rows): the staging waves' K
  // rotation needs the 32 registers they would hold, which otherwise spill.
  constexpr int kRlBytes = R * kTileRows * (kD + 4) * 4;
  constexpr bool kQinLds = AK;
  constexpr int kQBytes = kQinLds ? 4 * R * 8 * 1024 : 0;
  __shared__ __attribute__((aligned(16))) uint8_t pro[kRlBytes > kQBytes ? kRlBytes : kQBytes];
  auto rl = reinterpret_cast<float (*)[kTileRows][kD + 4]>(pro);

  const AttnItem it = items[blockIdx.x];
  if (it.n_rows == 0) return;
  const int tid = threadIdx.x;
  const int wg = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int w = R == 1 ? wg : wg & 3;    // query head slot
  const int rb = R == 1 ? 0 : wg >> 2;   // row block
  const bool stager = R == 1 || wg < 4;  // waves that stage K and V
  const int lane = tid & 63;
  const int lrow = lane & 31;
  const int lh = lane >> 5;
  const int g = it.kv_head;
  const int page_mask = (1 << log2_page) - 1;
  // the K block table (pool pages flagged when K is rotated on load)
  const int32_t* bt = (AK ? kbts : bts) + it.bt_off;

  const int rbase = 32 * rb;
  // item rows are entries of arows: the computed row (q, out, lse) and
  // its position; items of consecutive computed rows at consecutive
  // positions carry their first row (crow0) and skip that read
  const int rr = min(rbase + lrow, it.n_rows - 1);
  int row, pos;
  if (it.crow0 >= 0) {
    row = it.crow0 + rr;
    pos = it.min_pos + rr;
  } else {
    const AttnRow ar = arows[it.row0 + rr];
    row = ar.row;
    pos = ar.pos;
  }
  const int pos_l = pos - 4 * lh;   // position less the lane's key offset in a tile
  // key tiles this wave's rows need: up to their largest position
  int my_ntiles = 0;
  if constexpr (R > 1) {
    int wmax = rbase + lrow < it.n_rows ? pos : -1;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) wmax = max(wmax, __shfl_xor(wmax, o));
    my_ntiles = __builtin_amdgcn_readfirstlane(wmax + kKT) / kKT;
  }
  // wave w owns query head head0 + w of the group; with G < 4 the spare
  // waves recompute head G-1 and store nothing
  const int hl = G >= 4 ? it.head0 + w : min(w, G - 1);
  const bool wave_active = G >= 4 || w < G;

  bf16x8 qf[8];
  const uint8_t* qlds = pro + (tid >> 6) * 8192;
  auto qfrag = [&](int kst) __attribute__((always_inline)) -> bf16x8 {
    if constexpr (kQinLds) {
      Frag f;
      f.u = *reinterpret_cast<const uint4*>(qlds + kst * 1024 + lane * 16);
      return f.b;
    } else {
      return qf[kst];
    }
  };
  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;

  // ---- staging.  A tile's 32 keys form two 16-key blocks; with B >= 16
  // each block lies in one page.
  // K: wave w loads fragment blocks kst = 2w, 2w + 1 with direct loads; lane
  //    l fetches key l % 32, in 16-key block (l / 16) % 2.
  // V: thread t owns 16 bytes (dims 8 (t / 16) ..) of keys 2 (t % 16) and
  //    2 (t % 16) + 1, which sit next to each other in the permuted V^T row;
  //    each of its 8 dims takes one 4-byte write.
  const int klane = (lane & 15) * kD + 8 * lh + 32 * w;
  const bool khi = (lane >> 4) & 1;
  uint4 vr[2];
  const int kp = tid & 15;                 // key pair
  const int vb = kp >> 3;                  // 16-key block of the pair
  const int vc8 = (tid >> 4) * 8;          // first dim
  const int voff = (2 * kp - 16 * vb) * kD + vc8;
  const int vk = 2 * kp - 16 * vb;         // key within its block
  const int vcol = 16 * vb + ((vk >> 2) & 1) * 8 + ((vk >> 3) & 1) * 4 + (vk & 3);
  // Page ids of a tile's two 16-key blocks: uniform, so scalar loads, one
  // tile before the tile's loads need them.
  auto fetch_pages = [&](int j, int& q0, int& q1) __attribute__((always_inline)) {
    q0 = bt[min((j * kKT) >> log2_page, it.n_pages - 1)];
    q1 = bt[min((j * kKT + 16) >> log2_page, it.n_pages - 1)];
  };
  auto block_base = [&](int page, int kq) -> int64_t {
    return ((((int64_t)page * n_kv_heads + g) << log2_page) + (kq & page_mask)) * kD;
  };
  // Issues tile j's loads: K directly into the LDS buffer kt, V into
  // registers (written to LDS as V^T by store_tile).
  // K rotated on load: the staging thread's key (kk) and 8-dim chunk of each
  // RoPE half, its raw K, and whether its block is a pool page
  const int kk = tid & 31, kch = (tid >> 5) & 7;
  uint4 kraw[2];
  bool krot = false, kreg = false;
  auto load_tile = [&](int j, int p0, int p1, uint8_t* kt) __attribute__((always_inline)) {
    const int key0 = j * kKT;
    const int64_t b0 = block_base(p0 & ~kPoolPageFlag, key0);
    const int64_t b1 = block_base(p1 & ~kPoolPageFlag, key0 + 16);
    int64_t vbase = vb ? b1 : b0;
    const uint16_t* vsrc = vc;
    if constexpr (AV || AK) {
      // the V page: from the V block table (flagged pool pages) with V
      // aliasing, else the request page of the unflagged block table
      const int kv = key0 + 16 * vb;
      const int32_t vp = (AV ? vbts : bts)[it.bt_off + min(kv >> log2_page, it.n_pages - 1)];
      vsrc = (AV && (vp & kPoolPageFlag)) ? pool_v : vc;
      vbase = block_base(vp & ~kPoolPageFlag, kv);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
      vr[i] = *reinterpret_cast<const uint4*>(vsrc + vbase + voff + i * kD);
    if (key0 + kKT > it.kv_len) {
      // last, partial tile: keys past kv_len may be unwritten slots.  Their
      // scores are masked (a select), but 0 * NaN in P V would not be, so
      // V is zeroed.
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (key0 + 2 * kp + i >= it.kv_len) vr[i] = make_uint4(0, 0, 0, 0);
    }
    if constexpr (AK) {
      kreg = ((p0 | p1) & kPoolPageFlag) != 0;
      if (kreg) {
        // through registers: rotated (pool block) or copied (request block)
        // by store_tile
        const int kb = kk >> 4;
        const int pg = kb ? p1 : p0;
        krot = (pg & kPoolPageFlag) != 0;
        const uint16_t* src = (krot ? pool_k : kc) +
                              block_base(pg & ~kPoolPageFlag, key0 + kk) + 8 * kch;
        kraw[0] = *reinterpret_cast<const uint4*>(src);
        kraw[1] = *reinterpret_cast<const uint4*>(src + kD / 2);
        return;
      }
    }
    const uint16_t* ksrc = kc + (khi ? b1 : b0) + klane;
    const uint32_t kdst = lds_addr(kt) + 2 * w * kKBlk;
    lds_dma16(ksrc, kdst);
    lds_dma16(ksrc + 16, kdst + kKBlk);
  };
  // K through registers (rotated on load): to LDS in fragment order, block
  // kst holding dims 16 kst .. (lane l: key l % 32, dims + 8 (l / 32))
  auto store_k = [&](int j, uint8_t* kt) __attribute__((always_inline)) {
    float lo[8], hi[8];
    const uint32_t wl[4] = {kraw[0].x, kraw[0].y, kraw[0].z, kraw[0].w};
    const uint32_t wh[4] = {kraw[1].x, kraw[1].y, kraw[1].z, kraw[1].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[2 * e] = bf16_to_f32(wl[e] & 0xffffu);
      lo[2 * e + 1] = bf16_to_f32(wl[e] >> 16);
      hi[2 * e] = bf16_to_f32(wh[e] & 0xffffu);
      hi[2 * e + 1] = bf16_to_f32(wh[e] >> 16);
    }
    uint4 a = kraw[0], b = kraw[1];
    if (krot) {
      const int pk = j * kKT + kk;
      float c[8], sn[8];
      load8(rope_cos + (int64_t)pk * (kD / 2) + 8 * kch, c);
      load8(rope_sin + (int64_t)pk * (kD / 2) + 8 * kch, sn);
      rope_rotate<8>(lo, hi, c, sn);
      a.x = f32_to_bf16(lo[0]) | (f32_to_bf16(lo[1]) << 16);
      a.y = f32_to_bf16(lo[2]) | (f32_to_bf16(lo[3]) << 16);
      a.z = f32_to_bf16(lo[4]) | (f32_to_bf16(lo[5]) << 16);
      a.w = f32_to_bf16(lo[6]) | (f32_to_bf16(lo[7]) << 16);
      b.x = f32_to_bf16(hi[0]) | (f32_to_bf16(hi[1]) << 16);
      b.y = f32_to_bf16(hi[2]) | (f32_to_bf16(hi[3]) << 16);
      b.z = f32_to_bf16(hi[4]) | (f32_to_bf16(hi[5]) << 16);
      b.w = f32_to_bf16(hi[6]) | (f32_to_bf16(hi[7]) << 16);
    }
    const int lofs = (kk + 32 * (kch & 1)) * 16;
    *reinterpret_cast<uint4*>(kt + (kch >> 1) * kKBlk + lofs) = a;
    *reinterpret_cast<uint4*>(kt + (4 + (kch >> 1)) * kKBlk + lofs) = b;
  };
  auto store_tile = [&](uint16_t* vs) __attribute__((always_inline)) {
    const uint32_t* v0 = reinterpret_cast<const uint32_t*>(&vr[0]);
    const uint32_t* v1 = reinterpret_cast<const uint32_t*>(&vr[1]);
    float vmax = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int sh = (e & 1) ? 16 : 0;
      const float f0 = bf16_to_f32((v0[e >> 1] >> sh) & 0xffffu);
      const float f1 = bf16_to_f32((v1[e >> 1] >> sh) & 0xffffu);
      vmax = fmaxf(vmax, fmaxf(fabsf(f0), fabsf(f1)));
      *reinterpret_cast<uint32_t*>(vs + (vc8 + e) * kVStr + vcol) = pack_f16x2(f0, f1);
    }
    if (!(vmax <= 65280.0f)) {   // beyond fp16 (or NaN): refuse loudly
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<uint32_t*>(vs + (vc8 + e) * kVStr + vcol) = kF16NaN2;
    }
  };

  // One 32-key tile: S^T = K Q^T, online softmax, O^T += V^T P^T.
  // MASK: kNoMask, kMaskCausal (keys past the row's position: tiles reaching
  // past the smallest row position of the item) or kMaskBoth (also keys
  // below kv_lo: the tile holding kv_lo).
  auto tile = [&](int j, auto mask_tag, const uint8_t* ks, const uint16_t* vs)
      __attribute__((always_inline)) {
    constexpr int MASK = decltype(mask_tag)::value;
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
    for (int kst = 0; kst < 8; ++kst) {
      Frag a;
      a.u = *reinterpret_cast<const uint4*>(ks + kst * kKBlk + lane * 16);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.b, qfrag(kst), s, 0, 0, 0);
    }
    // keep four LDS fragment reads in flight ahead of the MFMAs
    // (scheduling groups: 0x100 = LDS read, 0x008 = MFMA)
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);

    // the V^T fragments of the first 16 keys are read while the softmax runs
    Frag va[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
      va[db].u = *reinterpret_cast<const uint4*>(vs + (32 * db + lrow) * kVStr + 8 * lh);
    if constexpr (MASK != kNoMask) {
      // score r holds key j kKT + 8 (r / 4) + 4 lh + r % 4: compare its
      // offset in the tile with the row's bounds moved to the same origin
      const int dhi = pos_l - j * kKT;
      const int dlo = it.kv_lo - 4 * lh - j * kKT;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = 8 * (r >> 2) + (r & 3);
        const bool out = MASK == kMaskBoth ? (off > dhi || off < dlo) : off > dhi;
        s[r] = out ? -INFINITY : s[r];
      }
    }
    // Online softmax with a lazily updated running max m, common to the
    // row's two half-waves.  P = exp2(s c - m c) is computed against the
    // current m and its per-lane sum checked: while the sum stays <= 2^kLazy
    // (so every P <= 2^kLazy, an exact range for fp16) no maximum is taken
    // and nothing is rescaled.  Otherwise (or while m is still -inf) the
    // tile's scores are computed again from the K tile in LDS, the maximum
    // moves m, O and l are rescaled, and P is recomputed.
    const float mc = m == -INFINITY ? 0.0f : m * scale_log2e;
    float ls[4];
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2e, -mc));
#pragma unroll
    for (int r = 0; r < 4; ++r) ls[r] = (s[r] + s[r + 4]) + (s[r + 8] + s[r + 12]);
    float lt = (ls[0] + ls[1]) + (ls[2] + ls[3]);
    if (__builtin_amdgcn_ballot_w64(!(lt <= kLazySum) || m == -INFINITY)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
      for (int kst = 0; kst < 8; ++kst) {
        Frag a;
        a.u = *reinterpret_cast<const uint4*>(ks + kst * kKBlk + lane * 16);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.b, qfrag(kst), s, 0, 0, 0);
      }
      if constexpr (MASK != kNoMask) {
        const int dhi = pos_l - j * kKT;
        const int dlo = it.kv_lo - 4 * lh - j * kKT;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = 8 * (r >> 2) + (r & 3);
          const bool out = MASK == kMaskBoth ? (off > dhi || off < dlo) : off > dhi;
          s[r] = out ? -INFINITY : s[r];
        }
      }
      float mt = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[r]);
      const float mn = fmaxf(m, fmaxf(mt, __shfl_xor(mt, 32)));
      const float alpha = mn == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f((m - mn) * scale_log2e);
      m = mn;
      l *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      const float mc2 = m == -INFINITY ? 0.0f : m * scale_log2e;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2e, -mc2));
#pragma unroll
      for (int r = 0; r < 4; ++r) ls[r] = (s[r] + s[r + 4]) + (s[r + 8] + s[r + 12]);
    }
    f16x8 pf[2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[h][e] = (_Float16)s[8 * h + e];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[db].h, pf[0], o[db], 0, 0, 0);
      va[db].u = *reinterpret_cast<const uint4*>(vs + (32 * db + lrow) * kVStr + 16 + 8 * lh);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[db].h, pf[1], o[db], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    l += (ls[0] + ls[1]) + (ls[2] + ls[3]);
  };

  // keys kv_lo .. kv_len-1: tiles j0 .. ntiles-1.  A tile needs the mask
  // when it reaches past the smallest row position or starts below kv_lo.
  const int ntiles = (it.kv_len + kKT - 1) / kKT;
  const int j0 = it.kv_lo / kKT;
  const int jlo = min(ntiles, (it.kv_lo + kKT - 1) / kKT);   // first tile without keys < kv_lo
  const int nfull = min(ntiles, (it.min_pos + 1) / kKT);      // tiles ending at or before min_pos
  // page ids of the next tile to load (staging waves; the first tile's
  // come with the item)
  int pp0 = it.pg[0], pp1 = it.pg[1];
  // One tile j: issue the next tile's loads into the other buffers, compute
  // this one, stage the next V^T, wait for this wave's direct K loads, then
  // the workgroup barrier.
  // SKIP: tiles past a row block's last row occur only in the masked tail.
  auto run_tiles = [&](int ja, int jb, auto mask_tag, auto skip_tag)
      __attribute__((always_inline)) {
    constexpr bool SKIP = R > 1 && decltype(skip_tag)::value;
    for (int j = ja; j < jb; ++j) {
      const bool more = j + 1 < ntiles;
      if (more) {
        load_tile(j + 1, pp0, pp1, kl[(j + 1) & 1]);
        fetch_pages(j + 2, pp0, pp1);
      }
      if (!SKIP || j < my_ntiles) tile(j, mask_tag, kl[j & 1], vl[j & 1]);
      if (more) {
        store_tile(vl[(j + 1) & 1]);
        if (AK && kreg) store_k(j + 1, kl[(j + 1) & 1]);
      }
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      __syncthreads();
    }
  };
  // The waves of the other row blocks stage nothing and skip the tiles past
  // their own rows (fully masked for them; all tiles for a row block past
  // the item's last row).  Kept as a separate loop: with the staging under
  // a wave-dependent condition in one loop the compiler kept the staging
  // registers live in every wave and spilled.
  auto run_tiles_ns = [&](int ja, int jb, auto mask_tag) __attribute__((always_inline)) {
    for (int j = ja; j < jb; ++j) {
      if (j < my_ntiles) tile(j, mask_tag, kl[j & 1], vl[j & 1]);
      __syncthreads();
    }
  };
  if (stager) {
    load_tile(j0, pp0, pp1, kl[j0 & 1]);
    fetch_pages(j0 + 1, pp0, pp1);
  }
  // While the first tile is in flight: each row block's cos/sin rows go to
  // LDS (thread t of the block loads 8 dims of cos and sin of row t / 8)
  // and every wave loads its raw queries; the rotation follows the barrier.
  {
    const int t = tid & 255, lr = t >> 3, c8 = 8 * (t & 7);
    const int pr = min(rbase + lr, it.n_rows - 1);
    const int ppos = it.crow0 >= 0 ? it.min_pos + pr : arows[it.row0 + pr].pos;
    float c[8], sn[8];
    load8(rope_cos + (int64_t)ppos * (kD / 2) + c8, c);
    load8(rope_sin + (int64_t)ppos * (kD / 2) + c8, sn);
    store8(&rl[rb][lr][c8], c);
    store8(&rl[rb][lr][kD / 2 + c8], sn);
  }
  uint4 qraw[8];
  {
    const uint16_t* qp = q + ((int64_t)row * n_q_heads + g * G + hl) * kD;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int d0 = 16 * ks + 8 * lh;
      qraw[ks] = *reinterpret_cast<const uint4*>(qp + d0);
      qraw[ks + 4] = *reinterpret_cast<const uint4*>(qp + d0 + kD / 2);
    }
  }
  if (stager) {
    store_tile(vl[j0 & 1]);
    if (AK && kreg) store_k(j0, kl[j0 & 1]);
  }
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  // ---- rotated queries as bf16 B operands: lane = query row, k = head dim
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int d0 = 16 * ks + 8 * lh;
    float lo[8], hi[8], c[8], sn[8];
    const uint32_t wl[4] = {qraw[ks].x, qraw[ks].y, qraw[ks].z, qraw[ks].w};
    const uint32_t wh[4] = {qraw[ks + 4].x, qraw[ks + 4].y, qraw[ks + 4].z, qraw[ks + 4].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[2 * e] = bf16_to_f32(wl[e] & 0xffffu);
      lo[2 * e + 1] = bf16_to_f32(wl[e] >> 16);
      hi[2 * e] = bf16_to_f32(wh[e] & 0xffffu);
      hi[2 * e + 1] = bf16_to_f32(wh[e] >> 16);
    }
    load8(&rl[rb][lrow][d0], c);
    load8(&rl[rb][lrow][kD / 2 + d0], sn);
    rope_rotate<8>(lo, hi, c, sn);
    Frag a, b;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a.w[e] = pack_bf16x2(lo[2 * e], lo[2 * e + 1]);
      b.w[e] = pack_bf16x2(hi[2 * e], hi[2 * e + 1]);
    }
    qf[ks] = a.b;
    qf[ks + 4] = b.b;
  }
  if constexpr (kQinLds) {
    __syncthreads();   // every wave has read its cos/sin rows
#pragma unroll
    for (int kst = 0; kst < 8; ++kst) {
      Frag f;
      f.b = qf[kst];
      *reinterpret_cast<uint4*>(pro + (tid >> 6) * 8192 + kst * 1024 + lane * 16) = f.u;
    }
  }
  if (stager) {
    run_tiles(j0, jlo, MaskBoth{}, std::false_type{});
    run_tiles(jlo, max(jlo, nfull), NoMask{}, std::false_type{});
    run_tiles(max(jlo, nfull), ntiles, MaskCausal{}, std::true_type{});
  } else {
    run_tiles_ns(j0, jlo, MaskBoth{});
    run_tiles_ns(jlo, max(jlo, nfull), NoMask{});
    run_tiles_ns(max(jlo, nfull), ntiles, MaskCausal{});
  }

  // ---- epilogue: normalise, round to bf16, store rows of this tile
  const float lt = l + __shfl_xor(l, 32);
  if (!wave_active || rbase + lrow >= it.n_rows) return;
  const float inv = 1.0f / lt;
  {
    if (it.part_slot >= 0) {
      // one key range of a split item: normalized rows and log-sum-exp in
      // fp32 to this row block's slot, merged by attn_merge_kernel
      const int64_t slot = it.part_slot + (int64_t)rb * it.n_parts;
      const int64_t sr = (slot * kTileRows + lrow) * kSplitHeads + w;
      float* po = split_o + sr * kD;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg)
          *reinterpret_cast<float4*>(po + 32 * db + 8 * rg + 4 * lh) =
              make_float4(o[db][4 * rg] * inv, o[db][4 * rg + 1] * inv,
                          o[db][4 * rg + 2] * inv, o[db][4 * rg + 3] * inv);
      if (lh == 0) split_lse[sr] = m * scale + logf(lt);
      return;
    }
  }
  const int hq = g * G + (G >= 4 ? it.head0 : 0) + w;
  uint16_t* op = out + ((int64_t)row * n_q_heads + hq) * kD;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d0 = 32 * db + 8 * rg + 4 * lh;
      uint2 v;
      v.x = pack_bf16x2(o[db][4 * rg] * inv, o[db][4 * rg + 1] * inv);
      v.y = pack_bf16x2(o[db][4 * rg + 2] * inv, o[db][4 * rg + 3] * inv);
      *reinterpret_cast<uint2*>(op + d0) = v;
    }
  if (lse && lh == 0) lse[(int64_t)row * n_q_heads + hq] = m * scale + logf(lt);
}

int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

// Merge of a split item's key ranges (Section 5.3's extend pass over the
// whole prompt, run as several ranges): for its row r and query head
// hq0 + hs, from the ranges' normalized outputs o_c and log-sum-exps lse_c,
//   lse = log sum_c exp(lse_c),   o = sum_c exp(lse_c - lse) o_c,
// o rounded to bf16 once.  One workgroup per row block of a split item (its
// rows are AttnRow entries), two threads per (row, head), each over half the
// head dims.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(
    const CombineDesc* __restrict__ cds, const AttnRow* __restrict__ arows,
    const float* __restrict__ split_o, const float* __restrict__ split_lse,
    uint16_t* __restrict__ out, float* __restrict__ lse, int n_q_heads) {
  const CombineDesc cd = cds[blockIdx.x];
  const int t = threadIdx.x;
  const int half = t & 1, pair = t >> 1;
  const int r = pair / kSplitHeads, hs = pair % kSplitHeads;
  if (r >= cd.n_rows || hs >= cd.n_heads) return;
  auto slot_row = [&](int c) -> int64_t {
    return ((int64_t)(cd.slot0 + c) * kTileRows + r) * kSplitHeads + hs;
  };
  float mx = -INFINITY;
  for (int c = 0; c < cd.n_slots; ++c) mx = fmaxf(mx, split_lse[slot_row(c)]);
  float den = 0.0f;
  for (int c = 0; c < cd.n_slots; ++c) den += expf(split_lse[slot_row(c)] - mx);
  const float ltot = mx + logf(den);
  constexpr int DH = D / 2;
  float acc[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) acc[d] = 0.0f;
  for (int c = 0; c < cd.n_slots; ++c) {
    const float wc = expf(split_lse[slot_row(c)] - ltot);
    const float* src = split_o + slot_row(c) * D + half * DH;
#pragma unroll
    for (int d = 0; d < DH; d += 4) {
      const float4 v = *reinterpret_cast<const float4*>(src + d);
      acc[d] = fmaf(wc, v.x, acc[d]);
      acc[d + 1] = fmaf(wc, v.y, acc[d + 1]);
      acc[d + 2] = fmaf(wc, v.z, acc[d + 2]);
      acc[d + 3] = fmaf(wc, v.w, acc[d + 3]);
    }
  }
  const int64_t orow = (int64_t)arows[cd.row0 + r].row * n_q_heads + cd.hq0 + hs;
  uint16_t* dst = out + orow * D + half * DH;
#pragma unroll
  for (int d = 0; d < DH; d += 8) {
    uint4 v;
    v.x = f32_to_bf16(acc[d]) | (f32_to_bf16(acc[d + 1]) << 16);
    v.y = f32_to_bf16(acc[d + 2]) | (f32_to_bf16(acc[d + 3]) << 16);
    v.z = f32_to_bf16(acc[d + 4]) | (f32_to_bf16(acc[d + 5]) << 16);
    v.w = f32_to_bf16(acc[d + 6]) | (f32_to_bf16(acc[d + 7]) << 16);
    *reinterpret_cast<uint4*>(dst + d) = v;
  }
  if (lse && half == 0) lse[orow] = ltot;
}

}  // namespace

hipError_t launch_attn(const tsr_plan* p, int32_t part, const AttnItem* items,
                       int32_t n_items, const void* pool_k, const void* pool_v,
                       const void* q, const void* req_k, const void* req_v, void* out,
                       float* lse, hipStream_t s) {
  if (n_items == 0 || p->T == 0) return hipSuccess;
  const tsr_model& m = p->model;
  const int lp = ilog2(m.page_size);
  const int G = m.n_q_heads / m.n_kv_heads;
  const dim3 grid(n_items);
  if (m.act_dtype == TSR_F32) {
    const dim3 block(256);
#define TSR_F32K(DIM)                                                             \
  hipLaunchKernelGGL(attn_f32_kernel<DIM>, grid, block, 0, s,                     \
                     static_cast<const float*>(q), static_cast<const float*>(req_k), \
                     static_cast<const float*>(req_v), items,                       \
                     p->dev.block_tables, p->dev.rows, p->dev.rope_cos,            \
                     p->dev.rope_sin, static_cast<float*>(out), lse, m.n_q_heads,  \
                     m.n_kv_heads, lp, p->scale)
    switch (m.head_dim) {
      case 64: TSR_F32K(64); break;
      case 128: TSR_F32K(128); break;
      case 256: TSR_F32K(256); break;
      default: return hipErrorInvalidValue;
    }
#undef TSR_F32K
    return hipGetLastError();
  }
  if (p->row_blocks == kPipeRowBlocks)
    return launch_attn_pipe(p, items, n_items, pool_v, q, req_k, req_v, out, lse, s);
  const float sl2e = (float)((double)p->scale * 1.4426950408889634);
#define TSR_MFMA(GG, AV, AK)                                                       \
  if (p->row_blocks == kMaxRowBlocks)                                              \
    TSR_MFMA_R(GG, AV, AK, kMaxRowBlocks);                                         \
  else                                                                             \
    TSR_MFMA_R(GG, AV, AK, 1)
#define TSR_MFMA_R(GG, AV, AK, RB)                                                 \
  hipLaunchKernelGGL((attn_mfma_kernel<GG, AV, AK, RB>), grid, dim3(256 * (RB)), 0, s, \
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(req_k), \
                     static_cast<const uint16_t*>(req_v),                          \
                     static_cast<const uint16_t*>(pool_k),                         \
                     static_cast<const uint16_t*>(pool_v), items,                  \
                     p->dev.block_tables, p->dev.v_block_tables,                    \
                     p->dev.k_block_tables, p->dev.attn_rows, p->dev.rope_cos,      \
                     p->dev.rope_sin, static_cast<uint16_t*>(out), lse,             \
                     p->dev.split_o, p->dev.split_lse, m.n_q_heads, m.n_kv_heads, lp, \
                     p->scale, sl2e)
#define TSR_MFMA_G(GG)                                                             \
  if (p->alias_v && p->alias_k) TSR_MFMA(GG, true, true);                          \
  else if (p->alias_v) TSR_MFMA(GG, true, false);                                  \
  else if (p->alias_k) TSR_MFMA(GG, false, true);                                  \
  else TSR_MFMA(GG, false, false)
  switch (G) {
    case 1: TSR_MFMA_G(1); break;
    case 2: TSR_MFMA_G(2); break;
    case 4: TSR_MFMA_G(4); break;
    case 8: TSR_MFMA_G(8); break;
    default: return hipErrorInvalidValue;
  }
#undef TSR_MFMA_G
#undef TSR_MFMA
#undef TSR_MFMA_R
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p->n_combine == 0) return e;
  // the split items of this part: part 0's merge descriptors come first
  const int32_t c0 = part == TSR_ATTN_AFTER_COMPOSE ? p->n_combine_part[0] : 0;
  const int32_t nc = part == TSR_ATTN_ALL ? p->n_combine : p->n_combine_part[part - 1];
  if (nc == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_merge_kernel<kD>, dim3(nc), dim3(256), 0, s, p->dev.combine + c0,
                     p->dev.attn_rows, p->dev.split_o, p->dev.split_lse, static_cast<uint16_t*>(out), lse,
                     m.n_q_heads);
  return hipGetLastError();
}

}  // namespace tsr
