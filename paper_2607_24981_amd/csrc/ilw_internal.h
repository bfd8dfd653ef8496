// ilw_internal.h -- device helpers and launcher declarations shared by the
// HIP sources of libilw.so.  Not part of the public ABI (include/ilw.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ilw.h"

namespace ilw {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kQmax = 127;   // symmetric int8 range, no zero point
constexpr int kQmin = -127;

// ---------------------------------------------------------------- rescaling
__device__ __forceinline__ int32_t sat8(int64_t v) {
  return v > kQmax ? kQmax : (v < kQmin ? kQmin : (int32_t)v);
}

// Dyadic requantization of a 32-bit accumulator, round half up.  The 64-bit
// product cannot overflow: |acc * mult| < 2^62 and the rounding term <= 2^61.
__device__ __forceinline__ int32_t rq(int32_t acc, int32_t mult, int32_t shift) {
  int64_t v = (int64_t)acc * (int64_t)mult + ((int64_t)1 << (shift - 1));
  return sat8(v >> shift);  // arithmetic shift: floor division by 2^shift
}

// Same for a 64-bit value, through an exact 128-bit product.
__device__ __forceinline__ int32_t rq_wide(int64_t acc, int32_t mult, int32_t shift) {
  __int128 v = (__int128)acc * mult + ((__int128)1 << (shift - 1));
  v >>= shift;
  return v > kQmax ? kQmax : (v < kQmin ? kQmin : (int32_t)v);
}

// Two-input dyadic add onto one scale (|a*ma| + |b*mb| < 2^39).
__device__ __forceinline__ int32_t rq2(int32_t a, int32_t b, int32_t ma, int32_t mb,
                                       int32_t shift) {
  int64_t v = (int64_t)a * ma + (int64_t)b * mb + ((int64_t)1 << (shift - 1));
  return sat8(v >> shift);
}

// The same for int8 inputs and shift >= 9 (wide = false): |v| < 2^39 + 2^61
// but v >> shift < 2^30 + 1 in magnitude, so the shifted value fits int32 and
// one median clamps it.  wide = true is the general form above; the flag is
// uniform across the launch, so callers branch on it outside their loops.
template <bool WIDE>
__device__ __forceinline__ int32_t rq2i8(int32_t a, int32_t b, int32_t ma, int32_t mb,
                                         int32_t shift) {
  if (WIDE) return rq2(a, b, ma, mb, shift);
  const int64_t v = (int64_t)a * ma + (int64_t)b * mb + ((int64_t)1 << (shift - 1));
  return min(max((int32_t)(v >> shift), kQmin), kQmax);
}

// Bytes 0 of a, b, c, d clamped to cap and packed (a in the low byte), for
// a..d < 2^16: the pairs go into 16-bit halves, are clamped two at a time
// (v_pk_min_u16) and their low bytes gathered: 5 instructions for 4 values.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_min_bytes(uint32_t a, uint32_t b, uint32_t c, uint32_t d,
                                                   u16x2 cap) {
  u16x2 lo = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(b, a, 0x05040100u));
  u16x2 hi = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(d, c, 0x05040100u));
  lo = __builtin_elementwise_min(lo, cap);
  hi = __builtin_elementwise_min(hi, cap);
  return __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, hi), __builtin_bit_cast(uint32_t, lo),
                               0x06040200u);
}

// ---------------------------------------------------------------- ShiftExp
// I-ViT's integer exponential for I <= 0 at scale 1/I0: exp(I / I0) =
// 2^(-z / I0) with z = -I log2(e) ~ a + a/2 - a/16 for a = -I, the two
// fractions rounded up (floor shifts of the negative input); z is capped at
// k_inter I0, split as z = n I0 + f (0 <= f < I0), and 2^(-f/I0) is the chord
// 1 - f / (2 I0).  Result (I0 - ceil(f/2)) 2^(k_inter - n) < 2^30 for
// I0 < 2^14 and k_inter <= 16.
__device__ __forceinline__ int32_t shift_exp(int32_t I, int32_t I0, int32_t k_inter) {
  const uint32_t a = (uint32_t)(-I);
  const uint32_t z = min(a + ((a + 1) >> 1) - ((a + 15) >> 4), (uint32_t)(k_inter * I0));
  const uint32_t n = z / (uint32_t)I0;
  const uint32_t f = z - n * (uint32_t)I0;
  return (I0 - (int32_t)((f + 1) >> 1)) << (k_inter - (int32_t)n);
}

// SD-ShiftGELU of one int8 value (Sec. 3.3.1): x sigmoid(z), z = 1.702 x ~
// x + x/2 + x/8 + x/16 (floor shifts), the sigmoid in its sign-dependent
// form: exp(0) / (exp(0) + exp(-z)) for z >= 0, exp(z) / (exp(z) + exp(0))
// for z < 0.  Both are t = exp(-|z|) and one = exp(0) = I0 2^k_inter over the
// same sum; the ratio is floor((2^31 - 1) / sum) times the numerator, kept to
// k_out - 1 fraction bits.  Returns x times it (|result| <= 127 2^(k_out-1)).
__device__ __forceinline__ int32_t sd_gelu(int32_t x, int32_t I0, int32_t k_inter,
                                           int32_t k_out) {
  const int32_t z = x + (x >> 1) + (x >> 3) + (x >> 4);
  const uint32_t one = (uint32_t)I0 << k_inter;
  const uint32_t t = (uint32_t)shift_exp(z < 0 ? z : -z, I0, k_inter);
  const uint32_t f = 0x7fffffffu / (one + t);
  return x * (int32_t)(((uint64_t)f * (z >= 0 ? one : t)) >> (32 - k_out));
}

// Operand tiles in LDS: rows of CPR 16-byte chunks (64 or 128 bytes), not
// padded; chunk c of row r sits at chunk position c ^ s(r), s(r) = 2 (r & 4)
// / 4 for 4 chunks per row and r & 6 for 8.  MFMA fragment reads (lane L:
// row L % 16, chunk L / 16) then hit every LDS bank once per 16-lane group,
// and so do the staging stores of whole rows.  Measured on MI355X with
// ds_read_b128: fragment reads at a padded row stride of 80 or 144 bytes take
// 8.8 cycles per wave instruction and CU, swizzled 5.4; 16-byte-chunk row
// stores 16.3 (80-byte stride) against 13.6.
template <int CPR>
__device__ __forceinline__ int lds_chunk(int r, int c) {
  static_assert(CPR == 4 || CPR == 8, "64- or 128-byte rows");
  const int sw = CPR == 4 ? (r & 4) >> 1 : (r & 6);
  return r * (CPR * 16) + ((c ^ sw) << 4);
}

// Workgroup barrier for LDS hand-offs only: waits for this wave's LDS
// operations (lgkmcnt(0)), then s_barrier.  Unlike __syncthreads() it does
// not wait for outstanding global loads (vmcnt), so loads issued for later K
// steps stay in flight across it.  The empty asm statements keep the
// compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);  // vmcnt 63, expcnt 7: no wait; lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wave-wide reductions (wave64).
__device__ __forceinline__ int32_t wave_sum_i32(int32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, o, 64);
    uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}
__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}

// Denominator shift of Constrained Shiftmax (Alg. 2, CalibrateShift):
// M_req = ceil(log2(S_sum)) = bit length of S_sum - 1, s_d = max(M_req +
// m_p - 31, 0).
__device__ __forceinline__ int32_t calibrate_shift(uint64_t s_sum, int32_t m_p) {
  int32_t m_req = s_sum <= 1 ? 0 : 64 - __clzll((long long)(s_sum - 1));
  return max(m_req + m_p - 31, 0);
}

// Normalization factor F = floor((2^31 - 1) / clamp(S_sum >> s_d, 1, 2^31-1)).
// S_sum >> s_d is exactly the quotient-remainder sum of Alg. 2.
__device__ __forceinline__ uint32_t shiftmax_factor(uint64_t s_sum, int32_t s_d) {
  uint64_t sr = s_sum >> s_d;
  sr = sr < 1 ? 1 : (sr > 0x7fffffffull ? 0x7fffffffull : sr);
  return 0x7fffffffu / (uint32_t)sr;
}

// ---------------------------------------------------------------- LayerNorm
// floor(V / k) for the Newton step.  Newton started at 2^16 >= sqrt(V) never
// drops below floor(sqrt(V)), so the quotient is below 2^17: an fp32
// reciprocal estimate is within one of it and one integer correction makes
// it exact.
__device__ __forceinline__ uint32_t newton_div(uint32_t V, uint32_t k) {
  const float qf = (float)V * __builtin_amdgcn_rcpf((float)k);
  int64_t q = (int64_t)qf;
  const int64_t r = (int64_t)V - q * (int64_t)k;
  q += r < 0 ? -1 : (r >= (int64_t)k ? 1 : 0);
  return (uint32_t)q;
}

// Integer square root by a fixed number of Newton steps from 2^16.
__device__ __forceinline__ uint32_t newton_isqrt(uint32_t V, int32_t iters) {
  if (V == 0) return 0;
  uint32_t k = 65536;
  for (int32_t t = 0; t < iters; ++t) k = (k + newton_div(V, k)) >> 1;
  return k;
}

// floor((2*sum + C) / (2*C)): the row mean rounded half up.
__device__ __forceinline__ int32_t mean_half_up(int32_t s, int32_t C) {
  const int32_t num = 2 * s + C, den = 2 * C;
  int32_t mu = num / den;
  if (num % den != 0 && num < 0) mu -= 1;
  return mu;
}

// n + beta requantized exactly.  |n| <= 2^30 and |beta| < 2^31 give
// |t| < 2^32, so u = t * mult fits int64, and
//   floor((u + 2^(shift-1)) / 2^shift) = ((u >> (shift-1)) + 1) >> 1
// avoids the rounding add that could overflow.
__device__ __forceinline__ int32_t ln_out(int64_t t, int32_t mult, int32_t shift) {
  const int64_t u = t * (int64_t)mult;
  const int64_t r = ((u >> (shift - 1)) + 1) >> 1;
  return sat8(r);
}

// Newton square root with FP64 steps.  k stays >= floor(sqrt(V)) (Newton
// from above), so floor(V / k) < 2^17 and a refined FP64 reciprocal is
// within 2^-33 of V / k; with the 2^-20 bias the floor is exact because a
// non-integer V / k has a fractional part in [2^-16, 1 - 2^-16].
__device__ __forceinline__ uint32_t newton_isqrt_f64(uint32_t V, int32_t iters) {
  if (V == 0) return 0;
  const double Vd = (double)V;
  double k = 65536.0;
  for (int32_t t = 0; t < iters; ++t) {
    double r = __builtin_amdgcn_rcp(k);
    r = fma(r, fma(-k, r, 1.0), r);
    const double q = floor(fma(Vd, r, 0x1p-20));
    k = floor((k + q) * 0.5);
  }
  return (uint32_t)k;
}

// floor((2^31 - 1) / s), exact for every s in [1, 2^31 - 1] (the Shiftmax
// factor F and LayerNorm's 1 / sigma both use it).
// Error bound: the hardware FP64 reciprocal estimate has a relative error of
// at most 2^29 ulp = 2^-23; one Newton step squares it, so with the fma
// roundings |rc - 1/s| / (1/s) < 2^-45.  The product 2^31 * rc is then within
// 2^-14 of the true quotient (plus one rounding of 2^-22 at most), so its
// truncation q is floor - 1, floor or floor + 1, and the remainder
// 2^31 - 1 - q s, taken exactly in int64, tells which: one correction step
// lands on the floor.  Without the Newton step the error near s = 1 would be
// 2^31 * 2^-23 = 2^8 units.
__device__ __forceinline__ uint32_t div_2p31m1(uint32_t s) {
  const double sd = (double)s;
  double r = __builtin_amdgcn_rcp(sd);
  r = fma(r, fma(-sd, r, 1.0), r);
  int64_t q = (int64_t)(2147483647.0 * r);
  const int64_t rem = 2147483647LL - q * (int64_t)s;
  q += rem < 0 ? -1 : (rem >= (int64_t)s ? 1 : 0);
  return (uint32_t)q;
}

// Per-channel output constants: beta, multiplier, shift and the saturation
// bound L (|t| >= L saturates; any L in [129 * 2^s / |m| + 1, 2^30 * 2^s / |m|]
// is exact, so an fp32 estimate with margin is used).
struct LnChan {
  int32_t beta, mult, shift, L;
};

// ---------------------------------------------------------------- launchers
// ---- GEMM epilogue helpers (shared by the GEMM and block-tail kernels)
__device__ __forceinline__ uint32_t pack4(int32_t a, int32_t b, int32_t c, int32_t d) {
  // byte 0 of each (two byte permutes and a shift-or)
  const uint32_t lo = __builtin_amdgcn_perm((uint32_t)b, (uint32_t)a, 0x0c0c0400u);
  const uint32_t hi = __builtin_amdgcn_perm((uint32_t)d, (uint32_t)c, 0x0c0c0400u);
  return lo | (hi << 16);
}

// Requantization of one channel with its accumulator bound L:
// |acc| >= L saturates (|acc * mult| > 129 * 2^shift) and L * |mult| / 2^shift
// stays far inside int32.  Any L in [129 * 2^s / |m| + 1, 2^30 * 2^s / |m|]
// works, so an fp32 estimate with margin is exact enough.
struct ChanRq {
  int32_t L, mult, shift, bias;
  int64_t rnd;
  __device__ __forceinline__ void init(int32_t m, int32_t s, int32_t b) {
    mult = m;
    shift = s;
    bias = b;
    rnd = (int64_t)1 << (s - 1);
    const float am = fabsf((float)m);
    const float bound = am == 0.f ? 1.f : 130.f * exp2f((float)s) * __builtin_amdgcn_rcpf(am);
    L = bound >= 2147483520.f ? 0x7fffffff : (int32_t)bound + 1;
  }
  __device__ __forceinline__ int32_t apply(int32_t acc) const {
    int32_t a = acc + bias;
    a = min(max(a, -L), L);
    const int32_t v = (int32_t)(((int64_t)a * mult + rnd) >> shift);
    return min(max(v, kQmin), kQmax);
  }
};

// The requantization of the GEMM epilogues in four instructions.  Per
// channel, the bias and the rounding are folded into one 64-bit addend
// c = bias * m + 2^(s-1), and the accumulator is clamped to [lo, hi] =
// [-L - bias, L - bias] (saturated to int32), beyond which the result
// saturates anyway: L >= 129 * 2^s / |m| + 1 from an fp32 estimate with
// margin, no clamp when that exceeds 2^30.  Then
//   (acc * m + c) >> s = floor(((acc + bias) m + 2^(s-1)) / 2^s)
// exactly whenever |acc + bias| < 3 * 2^30 (a linear's int32 accumulator;
// LayerNorm's |n| <= 2^30 plus an int32 beta), for every shift in [1, 62]:
// the clamped sum is at most 2^30, an unclamped one comes with |m| <=
// 130 * 2^(s-30) (and |m| < 2^31 anyway), so |(acc + bias) m| + 2^(s-1) <
// 2^63, |c| < 2^62 + 2^61, and the shifted value stays far inside int32.  A clamp, a 64-bit multiply-add,
// a 64-bit shift and a clamp.
struct RqI64 {
  int64_t c;
  int32_t mult, shift, lo, hi;
  __device__ __forceinline__ void init(int32_t m, int32_t s, int32_t b) {
    mult = m;
    shift = s;
    c = (int64_t)b * m + ((int64_t)1 << (s - 1));
    const float am = fabsf((float)m);
    const float bound = am == 0.f ? 1.f : 130.f * exp2f((float)s) * __builtin_amdgcn_rcpf(am);
    if (bound >= 1073741824.f) {
      lo = INT32_MIN;
      hi = INT32_MAX;
    } else {
      const int64_t L = (int64_t)bound + 1;
      lo = (int32_t)max(-L - (int64_t)b, (int64_t)INT32_MIN);
      hi = (int32_t)min(L - (int64_t)b, (int64_t)INT32_MAX);
    }
  }
  __device__ __forceinline__ int32_t apply(int32_t acc) const {
    // the clamp as one median-of-three (lo < hi always holds; the compiler
    // cannot see it and would emit a max and a min)
    int32_t a;
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(a) : "v"(acc), "v"(lo), "v"(hi));
    const int32_t v = (int32_t)(((int64_t)a * mult + c) >> shift);
    return min(max(v, kQmin), kQmax);
  }
  // init for accumulators with |acc| <= acc_max.  Where the bound
  // |mult| (|bias| + acc_max) + 2^(shift - 1) on |acc * mult + c| is below
  // min(2^63, 2^(shift + 31)), the clamp-free form below is exact: the clamp
  // bounds are then the whole int32 range and the float work is skipped.
  // Returns whether that holds.
  __device__ __forceinline__ bool init_bounded(int32_t m, int32_t s, int32_t b, uint32_t acc_max) {
    const uint64_t am = (uint64_t)(m < 0 ? -(int64_t)m : (int64_t)m);
    const uint64_t ab = (uint64_t)(b < 0 ? -(int64_t)b : (int64_t)b);
    // at most 2^31 (2^31 + 2^32) + 2^61 < 2^64: no wrap
    const uint64_t bound = am * (ab + acc_max) + ((uint64_t)1 << (s - 1));
    const uint64_t lim = s >= 32 ? ((uint64_t)1 << 63) : ((uint64_t)1 << (s + 31));
    if (bound >= lim) {
      init(m, s, b);
      return false;
    }
    mult = m;
    shift = s;
    c = (int64_t)b * m + ((int64_t)1 << (s - 1));
    lo = INT32_MIN;
    hi = INT32_MAX;
    return true;
  }
  // The same without the accumulator clamp, for callers that know
  // |acc * mult + c| < min(2^63, 2^(shift + 31)): the 64-bit sum is then
  // exact, its shift lies in int32, and the clamp, which only ever maps
  // saturating accumulators to saturating ones, changes nothing.
  __device__ __forceinline__ int32_t apply_unclamped(int32_t acc) const {
    const int32_t v = (int32_t)(((int64_t)acc * mult + c) >> shift);
    return min(max(v, kQmin), kQmax);
  }
};

template <bool B>
struct Flag {
  static constexpr bool value = B;
};
template <int V>
struct IntC {
  static constexpr int value = V;
};

// n / d for 0 <= n < 2^24 with an fp32 reciprocal and one correction step.
__device__ __forceinline__ int32_t fdiv(int32_t n, int32_t d, float inv) {
  int32_t q = (int32_t)((float)n * inv);
  const int32_t r = n - q * d;
  q += r < 0 ? -1 : (r >= d ? 1 : 0);
  return q;
}

enum GemmEpilogue {
  EPI_STORE = 0,     // y = rq(acc)
  EPI_GELU = 1,      // y = table[rq(acc)] (SD-ShiftGELU + its requantization)
  EPI_RESID = 2,     // y = Res(rq(acc), resid)
  EPI_QKV = 3,       // scatter rq(acc) into window-major Q, K, V^T
  EPI_RESID_LN = 4,  // EPI_RESID, and y2 = LayerNorm(y) (the tile holds whole rows)
  EPI_PATCH = 5      // patch embedding: x gathered from an image, y = Res(rq(acc), pos)
};

// Window-major Q, K, V^T buffers used by the attention kernel:
//   Q, K [B, nW, H, Tw, 64],  V^T [B, nW, H, 64, Twp]  (Twp = Tw rounded to 64)
// Window-major Q, K [B, nW, H, Tw, 64] and V^T [B, nW, H, 64, Twp]: rows of
// 64 bytes per head whatever the head dimension (2^hs, 32 or 64); the bytes
// past the head dimension are never written and never used.
struct QkvLayout {
  int8_t* q;
  int8_t* k;
  int8_t* vt;
  int32_t T, D, H, grid_w, win_h, win_w, nwx, nW, Tw, Twp, hs;
};

struct GemmArgs {
  const int8_t* x;   // [M, K] activations
  const int8_t* w;   // [N, K] weights
  const int32_t* bias;
  const int32_t* mult;
  const int32_t* shift;
  int32_t nq;        // 1 per-tensor, N per-channel
  int64_t M;
  int32_t N, K;
  int8_t* y;         // [M, N] output (STORE, GELU, RESID)
  const int8_t* resid;  // [M, N] skip input (RESID)
  int32_t res_ma, res_mb, res_shift;
  int32_t g_I0, g_kinter, g_kout, g_mult, g_shift;  // GELU
  QkvLayout qkv;     // QKV
  float inv_T, inv_gw, inv_wh, inv_ww;  // QKV: reciprocals for token -> window
  int8_t* y2;        // RESID_LN: LayerNorm of y
  const int32_t* ln_beta;
  const int32_t* ln_mult;
  const int32_t* ln_shift;
  int32_t ln_nq, ln_iters;
  // PATCH: x is an int8 image [B, pC, pH, pW] cut into 16 x 16 patches
  // (pT per image, pgw per row of patches); resid (the positional table)
  // is indexed by the token's position within its image
  int32_t pC, pH, pW, pgw, pT;
  // RESID_LN with N = 384: the weights packed in MFMA fragment order (see
  // PackList), or null for the row-major weights above
  const int8_t* wp;
};

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s);

// Weights packed in MFMA fragment order: for each 16-channel group n16 and
// 64-byte K chunk k64, 1 KB in which lane L's 16 bytes are
// W[16 n16 + L % 16][64 k64 + 16 (L / 16) .. + 15].  The fragments of the 2
// channel groups a wave of the 384-channel kernel owns are packed together,
// K chunk major: fragment (n16, k64) is the ((n16 / 2) KC 2 + 2 k64 + n16 % 2)-th
// KB (KC = K / 64).  One launch packs up to kMaxPack matrices (N x K
// row-major, K % 64 == 0, N % 32 == 0); start[] are the prefix sums of their
// 16-byte chunk counts.
constexpr int kMaxPack = 32;
struct PackList {
  const int8_t* src[kMaxPack];
  int8_t* dst[kMaxPack];
  int32_t K[kMaxPack];
  int64_t start[kMaxPack + 1];
  int32_t n;
};
size_t packed_frag_bytes(int32_t N, int32_t K);
hipError_t launch_pack_frags(const PackList& L, hipStream_t s);
// True where launch_gemm(EPI_RESID_LN or EPI_RESID) takes the packed-weight
// kernel when GemmArgs::wp is set (N = 384, K a multiple of 128, a grid past
// the latency mode).
bool ln384_packed_kernel_applies(int64_t M, int32_t N, int32_t K);
hipError_t launch_ln384_packed(const GemmArgs& a, bool layernorm, hipStream_t s);
// Everything of a 384-wide block after attention in one kernel: fp is the
// projection + residual + LN2 (x = the attention output, wp = packed
// weights, resid = the block input, LN2's fields), f1 fc1 + SD-ShiftGELU
// (wp, N = mlp, K = 384, the GELU fields), f2 fc2 + residual onto x1 (wp,
// N = 384, K = mlp, y, its residual dyadic, and with layernorm the next
// block's LN1 fields and y2).  x1, h and the fc1 output never leave the
// chip.  Applies for mlp a multiple of 384 up to 1536 past the latency mode.
bool tail384_kernel_applies(int64_t M, int32_t D, int32_t mlp);
hipError_t launch_tail384(const GemmArgs& fp, const GemmArgs& f1, const GemmArgs& f2,
                          bool layernorm, hipStream_t s);
bool gemm_latency_mode(int64_t M, int32_t N);

// The rest of an encoder block after attention, for one 16-token slab per
// workgroup (dim 192, MLP 768): projection + residual, LayerNorm, fc1 +
// SD-ShiftGELU, fc2 + residual, and optionally the next block's LayerNorm and
// QKV linear scattered window-major.
struct TailArgs {
  const int8_t* att;  // [M, D] attention output
  const int8_t* x;    // [M, D] block input (first residual)
  int8_t* y;          // [M, D] block output
  int64_t M;
  const int8_t* w_proj; const int32_t* b_proj; const int32_t* proj_mult;
  const int32_t* proj_shift; int32_t proj_nq;
  int32_t res1_ma, res1_mb, res1_shift;
  const int32_t* ln2_beta; const int32_t* ln2_mult; const int32_t* ln2_shift;
  int32_t ln2_nq, ln2_iters;
  const int8_t* w_fc1; const int32_t* b_fc1; const int32_t* fc1_mult;
  const int32_t* fc1_shift; int32_t fc1_nq;
  int32_t g_I0, g_kinter, g_kout, g_mult, g_shift;
  const int8_t* w_fc2; const int32_t* b_fc2; const int32_t* fc2_mult;
  const int32_t* fc2_shift; int32_t fc2_nq;
  int32_t res2_ma, res2_mb, res2_shift;
  // next block (has_next): LayerNorm 1 and QKV
  int32_t has_next;
  const int32_t* ln1_beta; const int32_t* ln1_mult; const int32_t* ln1_shift;
  int32_t ln1_nq, ln1_iters;
  const int8_t* w_qkv; const int32_t* b_qkv; const int32_t* qkv_mult;
  const int32_t* qkv_shift; int32_t qkv_nq;
  QkvLayout qkv;
  float inv_T, inv_gw, inv_wh, inv_ww;
};
hipError_t launch_block_tail(const TailArgs& a, hipStream_t s);
// h = LN1(x) and the window-major Q, K, V^T of the first block (dim 192), from
// TailArgs' x, M, LN1, QKV and layout fields.
hipError_t launch_block_head(const TailArgs& a, hipStream_t s);

// Scale-preserving split convolution (pointwise), up to kMaxBranches branches.
constexpr int kMaxBranches = 8;
struct SplitArgs {
  int32_t nbr;
  const int8_t* x[kMaxBranches];   // [M, C_b]
  const int8_t* w[kMaxBranches];   // [N, C_b]
  int32_t C[kMaxBranches];
  int32_t kstart[kMaxBranches + 1];  // first 64-channel K step of each branch
  const int32_t* bmult[kMaxBranches];
  const int32_t* bshift[kMaxBranches];
  int32_t bnq[kMaxBranches];
  const int32_t* bias;
  const int32_t* omult;
  const int32_t* oshift;
  int32_t onq;
  int8_t* y;  // [M, N]
  int64_t M;
  int32_t N;
};
hipError_t launch_split_conv(const SplitArgs& a, hipStream_t s);

struct AttnArgs {
  const int8_t* q;
  const int8_t* k;
  const int8_t* vt;
  int8_t* out;       // [B, T, D] token-major
  int32_t B, T, D, H, grid_w, win_h, win_w, nwx, nW, Tw, Twp;
  int32_t score_mult, score_shift, I0, k_inter, k_out, m_p, s_d, pv_mult, pv_shift;
  int32_t hd;        // head dimension: 32 or 64
  int32_t rq_fast;   // set by launch_attention: the score shift cannot overflow int32
};
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);
hipError_t launch_qkv_relayout(const int8_t* qkv, int32_t B, const QkvLayout& L,
                               hipStream_t s);

hipError_t launch_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                            const int32_t* beta, const int32_t* mult,
                            const int32_t* shift, int32_t nq, int32_t iters,
                            hipStream_t s);
hipError_t launch_shiftmax_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                               int32_t I0, int32_t k_inter, int32_t k_out, int32_t M,
                               hipStream_t s);
hipError_t launch_shiftgelu_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                                 int32_t I0, int32_t k_inter, int32_t k_out, int32_t mult,
                                 int32_t shift, hipStream_t s);
hipError_t launch_shiftmax(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                           int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                           int32_t s_d, hipStream_t s);
hipError_t launch_gelu(const int8_t* x, int8_t* y, int64_t n, int32_t I0,
                       int32_t k_inter, int32_t k_out, int32_t mult, int32_t shift,
                       hipStream_t s);
hipError_t launch_residual(const int8_t* a, const int8_t* b, int8_t* y, int64_t n,
                           int32_t ma, int32_t mb, int32_t shift, hipStream_t s);

constexpr int kMaxLevels = 8;
struct DeformArgs {
  const int8_t* value;
  const int32_t* ref;
  const int16_t* offs;
  const int8_t* logits;
  int8_t* out;
  int32_t B, Q, H, Dh, L, P, S;
  int32_t hw[kMaxLevels][2];
  int32_t start[kMaxLevels];
  int32_t I0, k_inter, k_out, m_p, s_d, out_mult, out_shift, mode;
  int32_t ref_dims;  // 2: reference points (x, y); 4: reference boxes (cx, cy, w, h)
  const int8_t* offs8;  // when set, int8 offsets used as offs8 << off_shift instead of offs
  int32_t off_shift;
};
hipError_t launch_deform(const DeformArgs& a, hipStream_t s);

}  // namespace ilw
