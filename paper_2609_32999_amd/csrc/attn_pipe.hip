// Pipelined bf16 prefill attention of the computed rows over the assembled
// KV (Section 5.3, "Completing prefill": the recompute ranges and the rest
// of the prompt are processed in one extend pass).
//
// Row t at prompt position p_t, query head h, KV head g = h / G:
//   o = softmax(scale * q_rot . K[0..p_t, g]^T) V[0..p_t, g]
// with q_rot = RoPE(q, p_t) rounded to bf16 and keys visible up to and
// including p_t.
//
// The arithmetic is that of attn_mfma_kernel (attn.hip): S^T = K Q^T on
// bf16 MFMA (v_mfma_f32_32x32x16_bf16), an online softmax in fp32 whose
// running max moves only when a tile's probability sum exceeds 2^8, and
// O^T += V^T P^T on fp16 MFMA.  What differs is the schedule, built so that
// each wave keeps the matrix pipe and the vector unit busy at once:
//   - A workgroup is eight waves: two row blocks of 32 consecutive computed
//     rows x the four query heads of one KV head (two waves per SIMD, so a
//     wave may hold 256 registers).  Both row blocks read the same K/V
//     tiles.
//   - Software pipeline inside each wave: the QK^T MFMAs of key tile j+1
//     are issued between the exponentials of tile j's softmax, and the PV
//     MFMAs of tile j between the staging instructions of later tiles.
//   - Every wave stages.  A tile's K and V are loaded straight into LDS,
//     K five tiles ahead (MFMA fragment order), V four (as it lies in the
//     page, 16-byte chunks XOR-swizzled per key pair), into as many
//     buffers; one tile ahead V is converted to fp16 V^T in a pair of
//     buffers.  Loads have two tile steps to land, and the first K
//     fragments of the tile after next are read before each step's
//     barrier; one barrier per tile.
//   - The page ids of the item's keys (one per 16-key block) are copied to
//     LDS once per item.
//   - V converts bf16 -> fp16 with round-to-nearest-even, which is exact up
//     to 65280 in magnitude and turns 65536 and beyond into infinity: rows
//     reading such a value come out non-finite instead of clipped.
#include <cmath>
#include <type_traits>

#include "attn_common.h"
#include "kernels_common.h"
#include "tsr_internal.h"

namespace tsr {

namespace {

constexpr int kPipeThreads = 512;
// K tiles are loaded kPipeAheadK tiles ahead, raw V tiles kPipeAheadV, into
// as many buffers each.
constexpr int kPipeAheadK = 5;
constexpr int kPipeAheadV = 4;
// s_waitcnt immediate leaving the direct loads of the last two tile steps
// (two per wave and step: K and V) outstanding.
constexpr int kWaitVmTwoSteps = 0x0F70 | 4;

// A row's two half-waves (lanes l and l + 32) combined.
__device__ __forceinline__ float half_pair_max(float x) { return fmaxf(x, __shfl_xor(x, 32)); }
__device__ __forceinline__ float half_pair_sum(float x) { return x + __shfl_xor(x, 32); }

// fp32 pair -> fp16 pair, round to nearest even (v_cvt_pk_f16_f32)
__device__ __forceinline__ uint32_t cvt_f16x2(float a, float b) {
  const f16x2 h = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, h);
}

template <int G, bool AV>
__global__ __launch_bounds__(kPipeThreads, 2) void attn_pipe_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, const uint16_t* __restrict__ pool_v,
    const AttnItem* __restrict__ items, const int32_t* __restrict__ bts,
    const int32_t* __restrict__ vbts, const RowDesc* __restrict__ rows,
    const float* __restrict__ rope_cos, const float* __restrict__ rope_sin,
    uint16_t* __restrict__ out, float* __restrict__ lse, int n_q_heads, int n_kv_heads,
    int log2_page, float scale, float scale_log2e) {
  // K tiles in MFMA fragment order; raw V tiles ([key][128 dims], the
  // 16-byte chunk c of key k holding dims 8 (c ^ 2 ((k / 2) % 8)) ..);
  // fp16 V^T tiles
  __shared__ __attribute__((aligned(16))) uint8_t kl[kPipeAheadK][kKBytes];
  __shared__ __attribute__((aligned(16))) uint8_t vraw[kPipeAheadV][kKT * kD * 2];
  __shared__ __attribute__((aligned(16))) uint16_t vl[2][kVBytes / 2];
  // cos (dims 0 .. d/2-1) and sin (d/2 ..) at each row's position, per row
  // block (rows padded by 4 floats against bank conflicts)
  __shared__ __attribute__((aligned(16))) float rl[2][kTileRows][kD + 4];
  // page id of each 16-key block of the item (V pages second, flagged for
  // pool pages, with V aliasing)
  __shared__ int32_t pt[AV ? 2 : 1][kPipeMaxBlocks];

  const AttnItem it = items[blockIdx.x];
  if (it.n_rows == 0) return;
  const int tid = threadIdx.x;
  const int wg = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int w = wg & 3;     // query head slot
  const int rb = wg >> 2;   // row block
  const int lane = tid & 63;
  const int lrow = lane & 31;
  const int lh = lane >> 5;
  const int g = it.kv_head;
  const int page_mask = (1 << log2_page) - 1;

  const int rbase = 32 * rb;
  const int row = it.row0 + min(rbase + lrow, it.n_rows - 1);
  const int pos = rows[row].pos;
  const int pos_l = pos - 4 * lh;   // position less the lane's key offset in a tile
  // key tiles this wave's rows need: up to their largest position (rows
  // past the item's last are that row again, computed and not stored)
  int wmax = pos;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) wmax = max(wmax, __shfl_xor(wmax, o));
  const int my_nt = __builtin_amdgcn_readfirstlane(wmax + kKT) / kKT;
  // wave w owns query head head0 + w of the group; with G < 4 the spare
  // waves recompute head G-1 and store nothing
  const int hl = G >= 4 ? it.head0 + w : min(w, G - 1);
  const bool wave_active = G >= 4 || w < G;

  // keys kv_lo .. kv_len-1: tiles j0 .. ntiles-1.  A tile needs the mask
  // when it reaches past the smallest row position or starts below kv_lo.
  const int ntiles = (it.kv_len + kKT - 1) / kKT;
  const int j0 = it.kv_lo / kKT;
  const int jlo = min(ntiles, (it.kv_lo + kKT - 1) / kKT);
  const int nfull = min(ntiles, (it.min_pos + 1) / kKT);

  // ---- page ids, cos/sin rows and raw queries
  for (int i = tid; i < 2 * (ntiles - j0); i += kPipeThreads) {
    const int ix = min(((2 * j0 + i) * 16) >> log2_page, it.n_pages - 1);
    pt[0][i] = bts[it.bt_off + ix];
    if constexpr (AV) pt[AV ? 1 : 0][i] = vbts[it.bt_off + ix];
  }
  {
    const int t = tid & 255, lr = t >> 3, c8 = 8 * (t & 7);
    const int ppos = rows[it.row0 + min(rbase + lr, it.n_rows - 1)].pos;
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
  __syncthreads();   // page ids in LDS

  // ---- staging.  Tile t's keys 32 t .. 32 t + 31 form two 16-key blocks,
  // each within one page (pages hold 16 or more keys).  Each wave issues
  // one 1 KB direct load of K and one of V per tile:
  // K: wave wg fills fragment block kst = wg; lane l fetches key l % 32,
  //    dims 16 wg + 8 (l / 32) .. + 8.
  // V: wave wg fills keys 4 wg .. 4 wg + 3; lane l fetches 16 bytes of key
  //    4 wg + l / 16 into chunk l % 16 of its row.
  const int kdim = 16 * wg + 8 * lh;
  const int vkey = 4 * wg + (lane >> 4);
  const int vdim = 8 * ((lane & 15) ^ (2 * ((vkey >> 1) & 7)));
  // element offsets of the lane's K and V rows from their 16-key block's
  // first row
  const int64_t koff = (int64_t)((lrow & 15) * kD + kdim);
  const int64_t voff = (int64_t)((vkey & 15) * kD + vdim);
  // element offset of 16-key block b (page id `page`) of tile t
  auto block_base = [&](int page, int t, int b) -> int64_t {
    return ((((int64_t)page * n_kv_heads + g) << log2_page) + ((t * kKT + 16 * b) & page_mask)) *
           kD;
  };
  // Page ids of tile t's two 16-key blocks (K, and V with aliasing): read
  // from LDS ahead of their use, moved to scalar registers by the loads.
  // Past the item's end the last tile again, so that every tile step issues
  // the same loads.
  struct Pages {
    int2 k, v;
  };
  auto read_pages = [&](int t) __attribute__((always_inline)) -> Pages {
    const int i = 2 * (min(t, ntiles - 1) - j0);
    Pages pg;
    pg.k = *reinterpret_cast<const int2*>(&pt[0][i]);
    if constexpr (AV) pg.v = *reinterpret_cast<const int2*>(&pt[AV ? 1 : 0][i]);
    else pg.v = pg.k;
    return pg;
  };
  // K and raw V buffers of tile t
  auto kbuf = [&](int t) __attribute__((always_inline)) -> uint8_t* {
    return kl[(uint32_t)t % kPipeAheadK];
  };
  auto vbuf = [&](int t) __attribute__((always_inline)) -> uint8_t* {
    return vraw[t & (kPipeAheadV - 1)];
  };
  // direct loads of tile t's K (pages pk) and V (pages pv) into their
  // buffers; none past the item's last tile
  auto issue_k = [&](int t, const Pages& pk) __attribute__((always_inline)) {
    if (t >= ntiles) return;
    const int tt = t;
    const int k0 = __builtin_amdgcn_readfirstlane(pk.k.x);
    const int k1 = __builtin_amdgcn_readfirstlane(pk.k.y);
    const uint16_t* kb0 = kc + block_base(k0, tt, 0);
    const uint16_t* kb1 = kc + block_base(k1, tt, 1);
    lds_dma16((lrow < 16 ? kb0 : kb1) + koff, lds_addr(kbuf(t)) + wg * kKBlk);
  };
  auto issue_v = [&](int t, const Pages& pv) __attribute__((always_inline)) {
    if (t >= ntiles) return;
    const int tt = t;
    const int vp = __builtin_amdgcn_readfirstlane(wg < 4 ? pv.v.x : pv.v.y);
    const uint16_t* vsrc = (AV && (vp & kPoolPageFlag)) ? pool_v : vc;
    lds_dma16(vsrc + block_base(vp & ~kPoolPageFlag, tt, wg >> 2) + voff,
              lds_addr(vbuf(t)) + wg * 1024);
  };
  // V of tile t, raw in LDS, to fp16 V^T: thread owns keys 2 kp, 2 kp + 1
  // (kp = tid % 16) at dims 4 c .. 4 c + 3 (c = tid / 16); each dim becomes
  // one 4-byte pair in its V^T row.  Keys past kv_len (slots of the last
  // page that may hold anything) are zeroed: their masked probabilities of
  // 0 would not cancel a NaN in P V.
  const int kp = tid & 15, vc4 = 4 * (tid >> 4);
  const int vrd = (2 * kp) * (kD * 2) + 8 * ((tid >> 4) ^ (4 * (kp & 7)));
  const int vwr = vc4 * kVStr + vt_col(2 * kp);
  struct RawV {
    uint2 a, b;
  };
  auto read_raw = [&](int t) __attribute__((always_inline)) -> RawV {
    const uint8_t* raw = vbuf(t);
    RawV r;
    r.a = *reinterpret_cast<const uint2*>(raw + vrd);
    r.b = *reinterpret_cast<const uint2*>(raw + vrd + kD * 2);
    return r;
  };
  auto write_vt = [&](int t, RawV r, auto last_tag) __attribute__((always_inline)) {
    if (decltype(last_tag)::value && t == ntiles - 1) {
      const int key = t * kKT + 2 * kp;
      if (key >= it.kv_len) r.a = make_uint2(0u, 0u);
      if (key + 1 >= it.kv_len) r.b = make_uint2(0u, 0u);
    }
    uint16_t* vs = vl[t & 1] + vwr;
    *reinterpret_cast<uint32_t*>(vs) =
        cvt_f16x2(__uint_as_float(r.a.x << 16), __uint_as_float(r.b.x << 16));
    *reinterpret_cast<uint32_t*>(vs + kVStr) =
        cvt_f16x2(__uint_as_float(r.a.x & 0xffff0000u), __uint_as_float(r.b.x & 0xffff0000u));
    *reinterpret_cast<uint32_t*>(vs + 2 * kVStr) =
        cvt_f16x2(__uint_as_float(r.a.y << 16), __uint_as_float(r.b.y << 16));
    *reinterpret_cast<uint32_t*>(vs + 3 * kVStr) =
        cvt_f16x2(__uint_as_float(r.a.y & 0xffff0000u), __uint_as_float(r.b.y & 0xffff0000u));
  };

  // K of tiles j0 .. j0+4 and V of j0 .. j0+3 in flight, in the order the
  // tile steps before j0 would have issued them; once all but the last
  // four loads (those steps' last two) have landed, V of j0 goes to LDS as
  // V^T
#pragma unroll
  for (int i = 0; i < kPipeAheadV; ++i) {
    const Pages pg = read_pages(j0 + i);
    issue_k(j0 + i, pg);
    issue_v(j0 + i, pg);
  }
  issue_k(j0 + kPipeAheadV, read_pages(j0 + kPipeAheadV));
  if (j0 + kPipeAheadK <= ntiles) __builtin_amdgcn_s_waitcnt(kWaitVmTwoSteps);
  else __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  write_vt(j0, read_raw(j0), std::true_type{});

  // ---- rotated queries as bf16 B operands: lane = query row, k = head dim
  bf16x8 qf[8];
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
  __syncthreads();   // V^T of tile j0 in LDS

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;

  // S^T of tile t (32 keys x this wave's 32 rows) from K in LDS
  auto qk = [&](int t, f32x16& s) __attribute__((always_inline)) {
    const uint8_t* ks = kbuf(t);
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
    for (int kst = 0; kst < 8; ++kst) {
      Frag a;
      a.u = *reinterpret_cast<const uint4*>(ks + kst * kKBlk + lane * 16);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.b, qf[kst], s, 0, 0, 0);
    }
  };
  // score r holds key t kKT + 8 (r / 4) + 4 lh + r % 4: compare its offset
  // in the tile with the row's bounds moved to the same origin
  auto mask = [&](int t, f32x16& s, bool lo_too) __attribute__((always_inline)) {
    const int dhi = pos_l - t * kKT;
    const int dlo = lo_too ? it.kv_lo - 4 * lh - t * kKT : -1;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int off = 8 * (r >> 2) + (r & 3);
      s[r] = (off > dhi || off < dlo) ? -INFINITY : s[r];
    }
  };
  // P = exp2(s c - m c) as fp16 pairs (the B operand of the PV MFMAs:
  // p[0..3] keys of the tile's first 16, p[4..7] the second) and the fp32
  // sum of P (the log-sum-exp needs the unrounded probabilities)
  auto probs = [&](const f32x16& s, uint32_t (&p)[8], float& lt) __attribute__((always_inline)) {
    const float mc = m == -INFINITY ? 0.0f : m * scale_log2e;
    float e[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2e, -mc));
    float pr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = cvt_f16x2(e[2 * i], e[2 * i + 1]);
      pr[i] = e[2 * i] + e[2 * i + 1];
    }
    lt = ((pr[0] + pr[1]) + (pr[2] + pr[3])) + ((pr[4] + pr[5]) + (pr[6] + pr[7]));
  };
  // The first phase of a steady tile step: QK^T of tile t into sn (eight
  // MFMAs in sequence) with the probabilities of the current tile (scores
  // sc) and one K fragment read (four ahead) in the shadow of each.  kf
  // holds the first four fragments, read ahead by the caller.
  // V^T fragment of head-dim block db, 16-key half h, of tile t
  auto vfrag = [&](int t, int db, int h) __attribute__((always_inline)) -> Frag {
    Frag f;
    f.u = *reinterpret_cast<const uint4*>(vl[t & 1] + (32 * db + lrow) * kVStr + 16 * h + 8 * lh);
    return f;
  };
  auto kfrags = [&](int t, Frag (&kf)[4]) __attribute__((always_inline)) {
    const uint8_t* ks = kbuf(t);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      kf[i].u = *reinterpret_cast<const uint4*>(ks + i * kKBlk + lane * 16);
  };
  // with `va` (vt >= 0): the eight V^T fragments of tile vt, one read per
  // group
  auto qk_probs = [&](int t, Frag (&kf)[4], const f32x16& sc, f32x16& sn, uint32_t (&p)[8],
                      float& lt, Frag (&va)[8], int vt) __attribute__((always_inline)) {
    const uint8_t* ks = kbuf(t);
    const float mc = m == -INFINITY ? 0.0f : m * scale_log2e;
#pragma unroll
    for (int r = 0; r < 16; ++r) sn[r] = 0.0f;
    float e[16], pr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i & 3].b, qf[i], sn, 0, 0, 0);
      if (i < 4)
        kf[i].u = *reinterpret_cast<const uint4*>(ks + (i + 4) * kKBlk + lane * 16);
      if (vt >= 0) va[i] = vfrag(vt, i & 3, i >> 2);
      e[2 * i] = __builtin_amdgcn_exp2f(fmaf(sc[2 * i], scale_log2e, -mc));
      e[2 * i + 1] = __builtin_amdgcn_exp2f(fmaf(sc[2 * i + 1], scale_log2e, -mc));
      if (i > 0) {
        p[i - 1] = cvt_f16x2(e[2 * i - 2], e[2 * i - 1]);
        pr[i - 1] = e[2 * i - 2] + e[2 * i - 1];
      }
      if (i == 3) pr[0] = (pr[0] + pr[1]);
      if (i == 5) pr[2] = (pr[2] + pr[3]);
      if (i == 7) pr[4] = (pr[4] + pr[5]);
    }
    __builtin_amdgcn_sched_barrier(0);
    p[7] = cvt_f16x2(e[14], e[15]);
    pr[7] = e[14] + e[15];
    lt = (pr[0] + pr[2]) + (pr[4] + (pr[6] + pr[7]));
  };
  // Lazy rescale.  The running max m moves (and O, l are rescaled) only
  // when some score of a tile would give P above 2^kLazy (so every P stays
  // within fp16's exact range), or while m is still -inf.  `over` is the
  // lane's test (its 16 scores of the tile against m), taken when the
  // scores are computed.
  auto over = [&](const f32x16& s) __attribute__((always_inline)) -> bool {
    float mt = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[r]);
    return !(fmaf(mt, scale_log2e, -(m * scale_log2e)) <= kLazy);
  };
  auto rescale = [&](const f32x16& s) __attribute__((always_inline)) {
    float mt = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[r]);
    const float mn = fmaxf(m, half_pair_max(mt));
    const float alpha =
        mn == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f((m - mn) * scale_log2e);
    m = mn;
    l *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
  };
  auto pfrags = [&](const uint32_t (&p)[8], Frag& pa, Frag& pb) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pa.w[i] = p[i];
      pb.w[i] = p[4 + i];
    }
  };
  // end of tile step j: the loads of two steps back have landed (each wave
  // waits for its own, the barrier for everyone's); near the item's end,
  // where fewer loads were issued, everything outstanding
  auto step_end = [&](int j) __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    if (j + kPipeAheadK < ntiles) __builtin_amdgcn_s_waitcnt(kWaitVmTwoSteps);
    else __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
  };

  // Tile step j with S^T of tile j in sc; S^T of tile j+1 goes to sn, and
  // `need` to the rescale test of tile j+1.
  // The steady state: every wave needs tiles j and j+1, tile j is unmasked
  // and its rescale test was taken in the previous step.
  bool need = true;
  // kf holds the first four K fragments of tile j+1 on entry and of tile
  // j+2 on exit (read before the barrier: that tile landed two steps ago).
  auto fast_step = [&](int j, f32x16& sc, f32x16& sn, Frag (&kf)[4])
      __attribute__((always_inline)) {
    // the raw V of tile j+1 and the page ids of tiles j+5 (K) and j+4 (V),
    // read ahead of their use in the second phase
    const RawV rv = read_raw(j + 1);
    const Pages pk = read_pages(j + kPipeAheadK);
    const Pages pv = read_pages(j + kPipeAheadV);
    Frag va[8];
    uint32_t p[8];
    float lt;
    qk_probs(j + 1, kf, sc, sn, p, lt, va, j);
    // keep P where it was computed, under the MFMAs (the compiler would
    // otherwise sink it below the rare branch that recomputes it)
#pragma unroll
    for (int i = 0; i < 8; ++i) asm volatile("" ::"v"(p[i]));
    asm volatile("" ::"v"(lt));
    // rare: the tile moves the running max; P is taken again
    if (__builtin_amdgcn_ballot_w64(need)) {
      rescale(sc);
      probs(sc, p, lt);
    }
    l += lt;
    // the second phase: O^T += V^T P^T for tile j (eight MFMAs: four
    // head-dim blocks x two 16-key halves) with the staging and the next
    // tile's rescale test in their shadow
    Frag pa, pb;
    pfrags(p, pa, pb);
    __builtin_amdgcn_sched_barrier(0);
    o[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[0].h, pa.h, o[0], 0, 0, 0);
    write_vt(j + 1, rv, std::false_type{});
    __builtin_amdgcn_sched_barrier(0);
    o[1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[1].h, pa.h, o[1], 0, 0, 0);
    issue_k(j + kPipeAheadK, pk);
    __builtin_amdgcn_sched_barrier(0);
    o[2] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[2].h, pa.h, o[2], 0, 0, 0);
    issue_v(j + kPipeAheadV, pv);
    __builtin_amdgcn_sched_barrier(0);
    o[3] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[3].h, pa.h, o[3], 0, 0, 0);
    need = over(sn);
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      __builtin_amdgcn_sched_barrier(0);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[4 + db].h, pb.h, o[db], 0, 0, 0);
      if (db == 1) kfrags(j + 2, kf);
    }
    step_end(j);
  };
  // Any tile: masks, and waves whose rows end before tile j or j+1 (the
  // rescale test is taken after masking).
  auto gen_step = [&](int j, f32x16& sc, f32x16& sn, Frag (&kf)[4])
      __attribute__((always_inline)) {
    const bool act = j < my_nt;
    const bool nxt = j + 1 < my_nt;
    uint32_t p[8];
    if (act) {
      if (j < jlo) mask(j, sc, true);
      else if (j >= nfull) mask(j, sc, false);
      if (__builtin_amdgcn_ballot_w64(over(sc) || m == -INFINITY)) rescale(sc);
      float lt;
      if (nxt) {
        Frag va[8];
        qk_probs(j + 1, kf, sc, sn, p, lt, va, -1);
      } else {
        probs(sc, p, lt);
      }
      l += lt;
    }
    __builtin_amdgcn_sched_barrier(0);
    write_vt(j + 1, read_raw(j + 1), std::true_type{});
    issue_k(j + kPipeAheadK, read_pages(j + kPipeAheadK));
    issue_v(j + kPipeAheadV, read_pages(j + kPipeAheadV));
    __builtin_amdgcn_sched_barrier(0);
    if (act) {
      Frag pa, pb;
      pfrags(p, pa, pb);
#pragma unroll
      for (int db = 0; db < 4; ++db)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vfrag(j, db, 0).h, pa.h, o[db], 0, 0, 0);
#pragma unroll
      for (int db = 0; db < 4; ++db)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vfrag(j, db, 1).h, pb.h, o[db], 0, 0, 0);
    }
    if (nxt) need = over(sn);
    kfrags(j + 2, kf);
    step_end(j);
  };

  // Tiles jlo .. nmain-1 are unmasked and needed by every wave together
  // with their successor (the first row block's largest position is the
  // smaller of the two row blocks'), and the tile they convert to V^T is
  // not the last (whose keys past kv_len are zeroed).
  const int nt_lo = rows[it.row0 + min(kTileRows, it.n_rows) - 1].pos / kKT + 1;
  const int nmain = max(jlo, min(min(nfull, nt_lo - 1), ntiles - 2));
  f32x16 s0, s1;
  Frag kf[4];
  if (j0 < my_nt) qk(j0, s0);
  kfrags(j0 + 1, kf);
  int j = j0;
  for (; j < jlo; ++j) {
    gen_step(j, s0, s1, kf);
    s0 = s1;
  }
  for (; j + 1 < nmain; j += 2) {
    fast_step(j, s0, s1, kf);
    fast_step(j + 1, s1, s0, kf);
  }
  if (j < nmain) {
    fast_step(j, s0, s1, kf);
    s0 = s1;
    ++j;
  }
  for (; j < ntiles; ++j) {
    gen_step(j, s0, s1, kf);
    s0 = s1;
  }
  // no direct load may still target this workgroup's LDS when it exits
  __builtin_amdgcn_s_waitcnt(kWaitVm0);

  // ---- epilogue: normalise, round to bf16, store the rows of this wave
  const float lt = half_pair_sum(l);
  if (!wave_active || rbase + lrow >= it.n_rows) return;
  const float inv = 1.0f / lt;
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

}  // namespace

hipError_t launch_attn_pipe(const tsr_plan* p, const AttnItem* items, int32_t n_items,
                            const void* pool_v, const void* q, const void* req_k,
                            const void* req_v, void* out, float* lse, hipStream_t s) {
  const tsr_model& m = p->model;
  int lp = 0;
  while ((1 << lp) < m.page_size) ++lp;
  const int G = m.n_q_heads / m.n_kv_heads;
  const float sl2e = (float)((double)p->scale * 1.4426950408889634);
#define TSR_PIPE(GG, AV)                                                                  \
  hipLaunchKernelGGL((attn_pipe_kernel<GG, AV>), dim3(n_items), dim3(kPipeThreads), 0, s, \
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(req_k), \
                     static_cast<const uint16_t*>(req_v),                                 \
                     static_cast<const uint16_t*>(pool_v), items, p->dev.block_tables,    \
                     p->dev.v_block_tables, p->dev.rows, p->dev.rope_cos,                 \
                     p->dev.rope_sin, static_cast<uint16_t*>(out), lse, m.n_q_heads,      \
                     m.n_kv_heads, lp, p->scale, sl2e)
#define TSR_PIPE_G(GG)             \
  if (p->alias_v) TSR_PIPE(GG, true); \
  else TSR_PIPE(GG, false)
  switch (G) {
    case 1: TSR_PIPE_G(1); break;
    case 2: TSR_PIPE_G(2); break;
    case 4: TSR_PIPE_G(4); break;
    case 8: TSR_PIPE_G(8); break;
    default: return hipErrorInvalidValue;
  }
#undef TSR_PIPE_G
#undef TSR_PIPE
  return hipGetLastError();
}

}  // namespace tsr
