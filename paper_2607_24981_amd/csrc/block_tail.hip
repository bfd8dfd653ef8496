// block_tail.hip -- everything of an encoder block after attention, for one
// slab of 16 tokens per workgroup, in a single launch (dim 192, MLP 768):
//
//   x1 = Res(rq(att Wp^T + bp), x)                      (Sec. 3.2.1; residual)
//   h2 = LN2(x1)                                        (I-LayerNorm)
//   g  = rq(SD-ShiftGELU(rq(h2 W1^T + b1)))             (Alg. 1 + requant)
//   y  = Res(rq(g W2^T + b2), x1)                       -> HBM (block output)
//   h  = LN1'(y);  q, k, v^T = rq(h Wq'^T + bq')        -> HBM, window-major,
//                                                          for the next block
//
// Only att and x are read and only y (and the next block's Q, K, V^T) are
// written: x1, h2, g and h live in registers and LDS.  Every weight byte is
// used by exactly one wave of the workgroup (the slab is one 16-token MFMA
// tile), so weights are loaded from global memory straight into MFMA A
// operand registers, without LDS staging, and the loads of the next stage
// are issued before the current stage's math.  At batch 1 this replaces four
// latency-bound launches (each paying dispatch, argument fetch, a load round
// trip and a store drain) by one.
//
// 12 waves: wave w owns output channels 16w..16w+15 of the projection and
// fc2 (so x1 stays in the registers of the lane that produced it), 64w..64w+63
// of fc1 and 48w..48w+47 of the QKV linear.  MFMA layout as in the GEMM: the
// weight tile is the A operand (rows = channels), the activation tile the B
// operand (columns = tokens); a lane ends up with 4 consecutive channels of
// token lane % 16.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int D = 192, HM = 768, NWV = 12, TS = 16;  // dim, MLP, waves, tokens
constexpr int XS = D + 16, GS = HM + 16;             // padded LDS row strides
constexpr int NPROJ = 0, NFC1 = D, NFC2 = D + HM, NQKV = 2 * D + HM;  // channel offsets
constexpr int NCH = NQKV + 3 * D;                    // staged requant channels

struct ChanC {
  int32_t L, mult, shift, bias;
};

__device__ __forceinline__ ChanC make_chan(int32_t mult, int32_t shift, int32_t bias) {
  ChanC r;
  r.mult = mult;
  r.shift = shift;
  r.bias = bias;
  const float am = fabsf((float)r.mult);
  const float bound = am == 0.f ? 1.f : 130.f * exp2f((float)r.shift) * __builtin_amdgcn_rcpf(am);
  r.L = bound >= 2147483520.f ? 0x7fffffff : (int32_t)bound + 1;
  return r;
}

// Exact requantization with the pre-clamped accumulator (as in the GEMM).
__device__ __forceinline__ int32_t rq_chan(int32_t acc, const ChanC& c) {
  int32_t a = acc + c.bias;
  a = min(max(a, -c.L), c.L);
  const int32_t v =
      (int32_t)(((int64_t)a * c.mult + ((int64_t)1 << (c.shift - 1))) >> c.shift);
  return min(max(v, kQmin), kQmax);
}

__device__ __forceinline__ LnChan make_ln(int32_t beta, int32_t mult, int32_t shift) {
  LnChan p;
  p.beta = beta;
  p.mult = mult;
  p.shift = shift;
  const float am = fabsf((float)p.mult);
  const float bound = am == 0.f ? 1.f : 130.f * exp2f((float)p.shift) * __builtin_amdgcn_rcpf(am);
  p.L = bound >= 2147483520.f ? 0x7fffffff : (int32_t)bound + 1;
  return p;
}

// LayerNorm of the slab: each lane holds one word (4 channels of token
// lane % 16) of the wave's 16 channels.  Partial sums go through LDS; the
// caller has made lnred free for writing.  Returns the normalized word.
__device__ __forceinline__ uint32_t slab_layernorm(uint32_t xw, int w, int lane, int ch,
                                                   int32_t* lnred, const LnChan* prm,
                                                   bool wide, int32_t iters) {
  int32_t S = __builtin_amdgcn_sdot4((int32_t)xw, 0x01010101, 0, false);
  int32_t SS = __builtin_amdgcn_sdot4((int32_t)xw, (int32_t)xw, 0, false);
  S += __shfl_xor(S, 16, 64);
  S += __shfl_xor(S, 32, 64);
  SS += __shfl_xor(SS, 16, 64);
  SS += __shfl_xor(SS, 32, 64);
  if (lane < TS) {
    lnred[(w * TS + lane) * 2 + 0] = S;
    lnred[(w * TS + lane) * 2 + 1] = SS;
  }
  __syncthreads();
  const int t = lane & (TS - 1);
  int32_t s = 0, ss = 0;
#pragma unroll
  for (int v = 0; v < NWV; ++v) {
    s += lnred[(v * TS + t) * 2 + 0];
    ss += lnred[(v * TS + t) * 2 + 1];
  }
  const int32_t mu = mean_half_up(s, D);
  const uint32_t V = (uint32_t)(ss - 2 * mu * s + D * mu * mu);
  const uint32_t sigma = newton_isqrt_f64(V, iters);
  const int32_t F = sigma ? (int32_t)div_2p31m1(sigma) : 0;
  int32_t o[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const LnChan p = prm[ch + r];
    const int32_t d = (int8_t)(xw >> (8 * r)) - mu;
    const int32_t n = (d * F) >> 1;  // |d| <= sigma: |d * F| < 2^31
    if (!wide) {
      const int32_t tt = min(max(n + p.beta, -p.L), p.L);
      const int32_t v =
          (int32_t)(((int64_t)tt * p.mult + ((int64_t)1 << (p.shift - 1))) >> p.shift);
      o[r] = min(max(v, kQmin), kQmax);
    } else {
      o[r] = ln_out((int64_t)n + p.beta, p.mult, p.shift);
    }
  }
  return pack4(o[0], o[1], o[2], o[3]);
}

// Window-major offsets of token m (a valid token) for the next attention:
// its row of Q and K, and its column of V^T.
__device__ __forceinline__ void qkv_dest(const TailArgs& a, int64_t m, int64_t& tq, int64_t& tv) {
  const QkvLayout& Lq = a.qkv;
  const int32_t b = fdiv((int32_t)m, Lq.T, a.inv_T);
  const int32_t t = (int32_t)m - b * Lq.T;
  const int32_t ty = fdiv(t, Lq.grid_w, a.inv_gw), tx = t - ty * Lq.grid_w;
  const int32_t wy = fdiv(ty, Lq.win_h, a.inv_wh), iy = ty - wy * Lq.win_h;
  const int32_t wx = fdiv(tx, Lq.win_w, a.inv_ww), ix = tx - wx * Lq.win_w;
  const int64_t bw = (int64_t)b * Lq.nW + wy * Lq.nwx + wx;
  const int32_t li = iy * Lq.win_w + ix;
  tq = (bw * Lq.H * Lq.Tw + li) * 64;
  tv = bw * Lq.H * 64 * Lq.Twp + li;
}

// QKV of the slab from h in bufX (wave w: channels 48w .. 48w + 47, weights
// in wq), requantized with the staged constants qc[0 .. 3D) and scattered
// window-major: the lane's token goes to (tq, tv).
__device__ __forceinline__ void slab_qkv(const TailArgs& a, const v4i (&wq)[3][D / 64],
                                         const int8_t* bufX, const ChanC* qc, int w, int tl,
                                         int cq, int kq, bool tok_ok, int64_t tq, int64_t tv) {
  const v4i zero = {0, 0, 0, 0};
  v4i acc2[3];
#pragma unroll
  for (int t = 0; t < 3; ++t) acc2[t] = zero;
#pragma unroll
  for (int s = 0; s < D / 64; ++s) {
    const v4i fb = *(const v4i*)(bufX + tl * XS + s * 64 + kq);
#pragma unroll
    for (int t = 0; t < 3; ++t)
      acc2[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wq[t][s], fb, acc2[t], 0, 0, 0);
  }
  if (!tok_ok) return;
  const QkvLayout& Lq = a.qkv;
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const int n = 48 * w + 16 * t + cq;  // channel of q | k | v
    int32_t v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = rq_chan(acc2[t][r], qc[n + r]);
    const int32_t part = n / D, rem_n = n - part * D;
    const int32_t h = rem_n >> 6, c = rem_n & 63;
    if (part < 2) {
      int8_t* base = part == 0 ? Lq.q : Lq.k;
      *(uint32_t*)(base + tq + (int64_t)h * Lq.Tw * 64 + c) = pack4(v[0], v[1], v[2], v[3]);
    } else {
      int8_t* dst = Lq.vt + tv + ((int64_t)h * 64 + c) * Lq.Twp;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[(int64_t)r * Lq.Twp] = (int8_t)v[r];
    }
  }
}

template <bool NEXT>
__global__ __launch_bounds__(64 * NWV) void block_tail_kernel(TailArgs a) {
  __shared__ __attribute__((aligned(16))) int8_t bufX[TS * XS];  // att, then h2, then h
  __shared__ __attribute__((aligned(16))) int8_t bufG[TS * GS];  // GELU output
  __shared__ ChanC chan[NEXT ? NCH : NQKV];
  __shared__ LnChan ln2p[D];
  __shared__ LnChan ln1p[NEXT ? D : 1];
  __shared__ int32_t lnred[NWV * TS * 2];
  __shared__ int8_t glut[256];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t M = a.M;
  const int64_t m0 = (int64_t)blockIdx.x * TS;
  const int tl = lane & (TS - 1);    // token of the lane's outputs and B fragments
  const int cq = (lane >> 4) * 4;    // first of the lane's 4 output channels in a 16-tile
  const int kq = (lane >> 4) * 16;   // the lane's 16 bytes of a 64-wide K step
  const int64_t m = m0 + tl;
  const bool tok_ok = m < M;
  const int64_t mc = tok_ok ? m : M - 1;
  const v4i zero = {0, 0, 0, 0};

  // ---- loads, smallest first: every load below is unconditional (indices
  // are clamped, pointers chosen by wave-uniform selects), so the waits for
  // the constants leave the weight loads in flight.
  // (1) per-channel requantization constants.  The four segments start at
  // multiples of 64 channels, so a wave's 64 channels lie in one segment.
  constexpr int NC = NEXT ? NCH : NQKV, NIT = (NC + 64 * NWV - 1) / (64 * NWV);
  int32_t cm[NIT], cs[NIT], cb[NIT];
  bool hasb[NIT];
#pragma unroll
  for (int i = 0; i < NIT; ++i) {
    const int c = min(tid + i * 64 * NWV, NC - 1);
    const int cu = __builtin_amdgcn_readfirstlane(c) >> 6;
    const int seg = (cu >= NFC1 / 64) + (cu >= NFC2 / 64) + (cu >= NQKV / 64);
    const int32_t* mp = seg == 0 ? a.proj_mult : seg == 1 ? a.fc1_mult : seg == 2 ? a.fc2_mult : a.qkv_mult;
    const int32_t* sp = seg == 0 ? a.proj_shift : seg == 1 ? a.fc1_shift : seg == 2 ? a.fc2_shift : a.qkv_shift;
    const int32_t* bp = seg == 0 ? a.b_proj : seg == 1 ? a.b_fc1 : seg == 2 ? a.b_fc2 : a.b_qkv;
    const int32_t nq = seg == 0 ? a.proj_nq : seg == 1 ? a.fc1_nq : seg == 2 ? a.fc2_nq : a.qkv_nq;
    const int base = seg == 0 ? NPROJ : seg == 1 ? NFC1 : seg == 2 ? NFC2 : NQKV;
    const int cc = c - base;
    const int q = nq == 1 ? 0 : cc;
    hasb[i] = bp != nullptr;
    cm[i] = mp[q];
    cs[i] = sp[q];
    cb[i] = (bp ? bp : mp)[bp ? cc : q];
  }
  // (2) LayerNorm constants: waves 0-2 LN2, waves 3-5 the next block's LN1
  const int lrole = __builtin_amdgcn_readfirstlane(tid) / D;  // 0..3, wave-uniform
  const bool l1 = NEXT && lrole == 1;
  const int lc = tid % D;
  int32_t lb, lm, ls;
  {
    const int32_t* bp = l1 ? a.ln1_beta : a.ln2_beta;
    const int32_t* mp = l1 ? a.ln1_mult : a.ln2_mult;
    const int32_t* sp = l1 ? a.ln1_shift : a.ln2_shift;
    const int32_t nq = l1 ? a.ln1_nq : a.ln2_nq;
    const int q = nq == 1 ? 0 : lc;
    lb = bp[lc];
    lm = mp[q];
    ls = sp[q];
  }
  // (3) the attention slab and the residual input
  const int ar = min(tid / (D / 16), TS - 1), ac = tid % (D / 16);
  const v4i att_chunk = *(const v4i*)(a.att + min(m0 + ar, M - 1) * D + ac * 16);
  const int n1 = 16 * w + cq;  // the lane's projection / fc2 channels
  const uint32_t xres = *(const uint32_t*)(a.x + mc * D + n1);
  // (4) weights of the first two stages, issued after everything above (the
  // compiler barrier keeps them last, so that waiting for the small loads
  // leaves these in flight)
  asm volatile("" ::: "memory");
  v4i wp[D / 64];
  {
    const int8_t* src = a.w_proj + (int64_t)(16 * w + tl) * D + kq;
#pragma unroll
    for (int s = 0; s < D / 64; ++s) wp[s] = *(const v4i*)(src + s * 64);
  }
  v4i w1[4][D / 64];
  {
    const int8_t* src = a.w_fc1 + (int64_t)(64 * w + tl) * D + kq;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int s = 0; s < D / 64; ++s) w1[t][s] = *(const v4i*)(src + (int64_t)16 * t * D + s * 64);
  }

  // ---- constants into LDS
#pragma unroll
  for (int i = 0; i < NIT; ++i) {
    const int c = tid + i * 64 * NWV;
    if (c < NC) chan[c] = make_chan(cm[i], cs[i], hasb[i] ? cb[i] : 0);
  }
  int wide = 0;
  if (lrole == 0 || l1) {
    LnChan p = make_ln(lb, lm, ls);
    wide = (lb > (1 << 30) || lb < -(1 << 30)) ? (l1 ? 2 : 1) : 0;
    if (l1) ln1p[lc] = p;
    else ln2p[lc] = p;
  }
  for (int t = tid; t < 256; t += 64 * NWV)
    glut[t] = (int8_t)rq(sd_gelu(t - 128, a.g_I0, a.g_kinter, a.g_kout), a.g_mult, a.g_shift);
  // window-major destination of the lane's token for the next block's Q, K, V^T
  int64_t tq = 0, tv = 0;
  if (NEXT && tok_ok) qkv_dest(a, m, tq, tv);
  if (tid < TS * D / 16) *(v4i*)(bufX + ar * XS + ac * 16) = att_chunk;
  // (__syncthreads_or only tells whether any thread's value is nonzero, so
  // each flag gets its own reduction)
  const bool wide2 = __syncthreads_or(wide & 1) != 0;
  const bool wide1 = __syncthreads_or(wide & 2) != 0;

  // ---- stage 1: projection + residual
  v4i acc = zero;
#pragma unroll
  for (int s = 0; s < D / 64; ++s) {
    const v4i fb = *(const v4i*)(bufX + tl * XS + s * 64 + kq);
    acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(wp[s], fb, acc, 0, 0, 0);
  }
  // fc2 weights: in flight during the LayerNorm and fc1
  v4i w2[HM / 64];
  {
    const int8_t* src = a.w_fc2 + (int64_t)(16 * w + tl) * HM + kq;
#pragma unroll
    for (int s = 0; s < HM / 64; ++s) w2[s] = *(const v4i*)(src + s * 64);
  }
  uint32_t x1w;
  {
    int32_t o[4];
    auto res1 = [&](auto wide) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t v = rq_chan(acc[r], chan[NPROJ + n1 + r]);
        o[r] = rq2i8<decltype(wide)::value>(v, (int8_t)(xres >> (8 * r)), a.res1_ma, a.res1_mb,
                                            a.res1_shift);
      }
    };
    if (a.res1_shift < 9) res1(Flag<true>{});
    else res1(Flag<false>{});
    x1w = pack4(o[0], o[1], o[2], o[3]);
  }
  // h2 = LN2(x1) -> bufX (every wave is past its stage-1 reads of bufX once
  // the statistics barrier inside slab_layernorm is passed)
  {
    const uint32_t hw = slab_layernorm(x1w, w, lane, n1, lnred, ln2p, wide2, a.ln2_iters);
    *(uint32_t*)(bufX + tl * XS + n1) = hw;
  }
  __syncthreads();

  // ---- stage 2: fc1 + SD-ShiftGELU -> bufG
  v4i acc1[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc1[t] = zero;
#pragma unroll
  for (int s = 0; s < D / 64; ++s) {
    const v4i fb = *(const v4i*)(bufX + tl * XS + s * 64 + kq);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      acc1[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(w1[t][s], fb, acc1[t], 0, 0, 0);
  }
  // next block's QKV weights: in flight during fc2
  v4i wq[3][D / 64];
  if (NEXT) {
    const int8_t* src = a.w_qkv + (int64_t)(48 * w + tl) * D + kq;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int s = 0; s < D / 64; ++s) wq[t][s] = *(const v4i*)(src + (int64_t)16 * t * D + s * 64);
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int n = 64 * w + 16 * t + cq;
    int32_t o[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = glut[rq_chan(acc1[t][r], chan[NFC1 + n + r]) + 128];
    *(uint32_t*)(bufG + tl * GS + n) = pack4(o[0], o[1], o[2], o[3]);
  }
  __syncthreads();

  // ---- stage 3: fc2 + residual -> y
  acc = zero;
#pragma unroll
  for (int s = 0; s < HM / 64; ++s) {
    const v4i fb = *(const v4i*)(bufG + tl * GS + s * 64 + kq);
    acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(w2[s], fb, acc, 0, 0, 0);
  }
  uint32_t yw;
  {
    int32_t o[4];
    auto res2 = [&](auto wide) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t v = rq_chan(acc[r], chan[NFC2 + n1 + r]);
        o[r] = rq2i8<decltype(wide)::value>(v, (int8_t)(x1w >> (8 * r)), a.res2_ma, a.res2_mb,
                                            a.res2_shift);
      }
    };
    if (a.res2_shift < 9) res2(Flag<true>{});
    else res2(Flag<false>{});
    yw = pack4(o[0], o[1], o[2], o[3]);
  }
  if (tok_ok) *(uint32_t*)(a.y + m * D + n1) = yw;
  if (!NEXT) return;

  // ---- next block: h = LN1'(y) -> bufX, then QKV scattered window-major.
  // lnred and bufX were last read before the barrier that ended stage 2.
  {
    const uint32_t hw = slab_layernorm(yw, w, lane, n1, lnred, ln1p, wide1, a.ln1_iters);
    *(uint32_t*)(bufX + tl * XS + n1) = hw;
  }
  __syncthreads();
  slab_qkv(a, wq, bufX, chan + NQKV, w, tl, cq, kq, tok_ok, tq, tv);
}

// The first block's h = LN1(x) and Q, K, V^T = rq(h Wq^T + bq), scattered
// window-major, for one 16-token slab per workgroup: the tail kernel's last
// stage applied to the encoder input, so the first block needs no separate
// LayerNorm and QKV launches.  Same wave layout: wave w normalizes channels
// 16w .. 16w + 15 and computes QKV channels 48w .. 48w + 47.
__global__ __launch_bounds__(64 * NWV) void block_head_kernel(TailArgs a) {
  __shared__ __attribute__((aligned(16))) int8_t bufX[TS * XS];  // h
  __shared__ ChanC chan[3 * D];
  __shared__ LnChan ln1p[D];
  __shared__ int32_t lnred[NWV * TS * 2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t M = a.M;
  const int64_t m0 = (int64_t)blockIdx.x * TS;
  const int tl = lane & (TS - 1);
  const int cq = (lane >> 4) * 4;
  const int kq = (lane >> 4) * 16;
  const int64_t m = m0 + tl;
  const bool tok_ok = m < M;
  const int64_t mc = tok_ok ? m : M - 1;

  // loads, smallest first and all unconditional (clamped indices): the QKV
  // and LayerNorm constants, the lane's input word, then the QKV weights
  static_assert(3 * D <= 64 * NWV, "one QKV channel per thread");
  const int c = min(tid, 3 * D - 1);
  const int32_t cm = a.qkv_mult[a.qkv_nq == 1 ? 0 : c];
  const int32_t cs = a.qkv_shift[a.qkv_nq == 1 ? 0 : c];
  const int32_t cb = a.b_qkv ? a.b_qkv[c] : 0;
  const int lc = tid % D;
  const int32_t lb = a.ln1_beta[lc];
  const int32_t lm = a.ln1_mult[a.ln1_nq == 1 ? 0 : lc];
  const int32_t ls = a.ln1_shift[a.ln1_nq == 1 ? 0 : lc];
  const int n1 = 16 * w + cq;  // the lane's 4 LayerNorm channels
  const uint32_t xw = *(const uint32_t*)(a.x + mc * D + n1);
  asm volatile("" ::: "memory");
  v4i wq[3][D / 64];
  {
    const int8_t* src = a.w_qkv + (int64_t)(48 * w + tl) * D + kq;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int s = 0; s < D / 64; ++s) wq[t][s] = *(const v4i*)(src + (int64_t)16 * t * D + s * 64);
  }

  if (tid < 3 * D) chan[tid] = make_chan(cm, cs, cb);
  int wide = 0;
  if (tid < D) {
    ln1p[tid] = make_ln(lb, lm, ls);
    wide = lb > (1 << 30) || lb < -(1 << 30);
  }
  int64_t tq = 0, tv = 0;
  if (tok_ok) qkv_dest(a, m, tq, tv);
  const bool wide1 = __syncthreads_or(wide) != 0;  // also publishes chan and ln1p

  {
    const uint32_t hw = slab_layernorm(xw, w, lane, n1, lnred, ln1p, wide1, a.ln1_iters);
    *(uint32_t*)(bufX + tl * XS + n1) = hw;
  }
  __syncthreads();
  slab_qkv(a, wq, bufX, chan, w, tl, cq, kq, tok_ok, tq, tv);
}

}  // namespace

hipError_t launch_block_head(const TailArgs& a_in, hipStream_t s) {
  if (a_in.M == 0) return hipSuccess;
  TailArgs a = a_in;
  a.inv_T = 1.0f / (float)a.qkv.T;
  a.inv_gw = 1.0f / (float)a.qkv.grid_w;
  a.inv_wh = 1.0f / (float)a.qkv.win_h;
  a.inv_ww = 1.0f / (float)a.qkv.win_w;
  hipLaunchKernelGGL(block_head_kernel, dim3((unsigned)((a.M + TS - 1) / TS)), dim3(64 * NWV),
                     0, s, a);
  return hipGetLastError();
}

hipError_t launch_block_tail(const TailArgs& a_in, hipStream_t s) {
  if (a_in.M == 0) return hipSuccess;
  TailArgs a = a_in;
  if (a.has_next) {
    a.inv_T = 1.0f / (float)a.qkv.T;
    a.inv_gw = 1.0f / (float)a.qkv.grid_w;
    a.inv_wh = 1.0f / (float)a.qkv.win_h;
    a.inv_ww = 1.0f / (float)a.qkv.win_w;
  }
  dim3 grid((unsigned)((a.M + TS - 1) / TS)), block(64 * NWV);
  if (a.has_next)
    hipLaunchKernelGGL(block_tail_kernel<true>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(block_tail_kernel<false>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace ilw
