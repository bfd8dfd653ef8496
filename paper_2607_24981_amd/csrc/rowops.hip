// rowops.hip -- row-wise and element-wise integer operators:
//   integer LayerNorm (Sec. 3.3), Constrained Shiftmax (Sec. 3.3.2, Alg. 2),
//   SD-ShiftGELU (Sec. 3.3.1, Alg. 1) and the dyadic two-input add.
// Row operators run one wave64 per row with wave-shuffle reductions; the
// element-wise operators stream 16-byte chunks.  Every nonlinearity whose
// input is an int8 value is tabulated once per workgroup in LDS, which is
// exact by construction.
#include "ilw_internal.h"

namespace ilw {
namespace {

// ---------------------------------------------------------------- LayerNorm
// LPR lanes per row, JW words (4 channels each) per lane kept in registers:
// C <= 4 * LPR * JW.  The per-channel beta / multiplier / shift of a lane's
// channels are loaded once and reused for every row the wave processes.
template <int LPR, int JW>
__global__ __launch_bounds__(256) void layernorm_kernel(const int8_t* x, int8_t* y,
                                                        int64_t rows, int32_t C,
                                                        const int32_t* beta,
                                                        const int32_t* mult,
                                                        const int32_t* shift, int32_t nq,
                                                        int32_t iters) {
  constexpr int RG = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, k = lane % LPR;
  const int32_t nw = C >> 2;
  int32_t pb[JW][4], pm[JW][4], ps[JW][4];
#pragma unroll
  for (int j = 0; j < JW; ++j) {
    const int32_t wd = k + j * LPR;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t c = wd < nw ? wd * 4 + b : 0;
      const int32_t q = nq == 1 ? 0 : c;
      pb[j][b] = beta[c];
      pm[j][b] = mult[q];
      ps[j][b] = shift[q];
    }
  }
  const int64_t ngroups = (rows + RG - 1) / RG;
  for (int64_t g = (int64_t)blockIdx.x * 4 + wave; g < ngroups; g += (int64_t)gridDim.x * 4) {
    const int64_t row = g * RG + sub;
    const bool live = row < rows;
    const uint32_t* xr = (const uint32_t*)(x + (live ? row : 0) * C);
    uint32_t xw[JW];
    int32_t s = 0;
#pragma unroll
    for (int j = 0; j < JW; ++j) {
      const int32_t wd = k + j * LPR;
      xw[j] = wd < nw ? xr[wd] : 0u;
#pragma unroll
      for (int b = 0; b < 4; ++b) s += (int8_t)(xw[j] >> (8 * b));
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    const int32_t mu = mean_half_up(s, C);
    uint32_t V = 0;
#pragma unroll
    for (int j = 0; j < JW; ++j) {
      if (k + j * LPR >= nw) continue;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int32_t d = (int8_t)(xw[j] >> (8 * b)) - mu;
        V += (uint32_t)(d * d);
      }
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) V += __shfl_xor(V, o, 64);
    const uint32_t sigma = newton_isqrt(V, iters);
    const uint32_t F = sigma ? 0x7fffffffu / sigma : 0u;
    uint32_t* yr = (uint32_t*)(y + (live ? row : 0) * C);
#pragma unroll
    for (int j = 0; j < JW; ++j) {
      const int32_t wd = k + j * LPR;
      uint32_t o = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int32_t d = (int8_t)(xw[j] >> (8 * b)) - mu;
        // |d| <= sigma, so |d * F| < 2^31
        const int64_t n = ((int64_t)d * (int64_t)F) >> 1;
        o |= (uint32_t)(ln_out(n + pb[j][b], pm[j][b], ps[j][b]) & 0xff) << (8 * b);
      }
      if (live && wd < nw) yr[wd] = o;
    }
  }
}

// LPR lanes per row for C a multiple of 16 with C / 16 <= JC * LPR: the row
// stays in registers (16-byte chunks), sum and sum of squares come from byte
// dot products, and the per-channel constants are staged in LDS once per
// workgroup.  V = sum (x - mu)^2 = sum x^2 - 2 mu sum x + C mu^2 (exact).
// Each wave walks several row groups and loads the next group's rows before
// working on the current one; the first group's loads are issued before the
// constants are staged, so the kernel pays about one memory round trip.
// The output requantization of n = (d F) >> 1 (|n| < 2^30) folds beta into
// the per-channel constant (RqI64 with the bias beta); where every channel's
// bound allows it, the accumulator clamp is skipped (one uniform branch).
template <int LPR, int JC>
__global__ __launch_bounds__(256) void layernorm_rows_kernel(const int8_t* x, int8_t* y,
                                                             int64_t rows, int32_t C,
                                                             const int32_t* beta,
                                                             const int32_t* mult,
                                                             const int32_t* shift, int32_t nq,
                                                             int32_t iters) {
  extern __shared__ RqI64 prm[];
  constexpr int RG = 64 / LPR;  // rows per wave and group
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, k = lane % LPR;
  const int32_t n16 = C >> 4;
  const int64_t ngroups = (rows + RG - 1) / RG;
  const int64_t gstride = (int64_t)gridDim.x * 4;
  auto load = [&](int64_t g, v4i (&xv)[JC]) {
    const int64_t row = min(g * RG + sub, rows - 1);
    const v4i* xr = (const v4i*)(x + row * C);
#pragma unroll
    for (int j = 0; j < JC; ++j) xv[j] = xr[min(k + j * LPR, n16 - 1)];
  };
  int64_t g = (int64_t)blockIdx.x * 4 + wave;
  v4i nxt[JC];
  if (g < ngroups) load(g, nxt);

  int clamp = 0;
  for (int32_t c = threadIdx.x; c < C; c += 256) {
    const int32_t q = nq == 1 ? 0 : c;
    RqI64 p;
    clamp |= !p.init_bounded(mult[q], shift[q], beta[c], 1u << 30);
    // chunk-transposed: channel 16 ch + i sits at i * n16 + ch, so the LPR
    // lanes of a row (consecutive chunks ch) read consecutive entries instead
    // of entries 16 * sizeof(RqI64) bytes apart
    prm[(c & 15) * n16 + (c >> 4)] = p;
  }
  clamp = __syncthreads_or(clamp);

  for (; g < ngroups; g += gstride) {
    v4i xv[JC];
#pragma unroll
    for (int j = 0; j < JC; ++j) xv[j] = nxt[j];
    if (g + gstride < ngroups) load(g + gstride, nxt);
    const int64_t row = g * RG + sub;
    const bool live = row < rows;
    int32_t S = 0, SS = 0;
#pragma unroll
    for (int j = 0; j < JC; ++j) {
      if (k + j * LPR < n16) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          S = __builtin_amdgcn_sdot4(xv[j][w], 0x01010101, S, false);
          SS = __builtin_amdgcn_sdot4(xv[j][w], xv[j][w], SS, false);
        }
      }
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) {
      S += __shfl_xor(S, o, 64);
      SS += __shfl_xor(SS, o, 64);
    }
    const int32_t mu = mean_half_up(S, C);
    const uint32_t V = (uint32_t)(SS - 2 * mu * S + C * mu * mu);
    const uint32_t sigma = newton_isqrt_f64(V, iters);
    const int32_t F = sigma ? (int32_t)div_2p31m1(sigma) : 0;
    v4i* yr = (v4i*)(y + (live ? row : rows - 1) * C);
    auto outputs = [&](auto unclamped) {
#pragma unroll
      for (int j = 0; j < JC; ++j) {
        const int32_t ch = k + j * LPR;
        if (ch >= n16) break;
        v4i o;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          int32_t r[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const RqI64& p = prm[(w * 4 + b) * n16 + ch];
            const int32_t d = (int8_t)(xv[j][w] >> (8 * b)) - mu;
            const int32_t n = (d * F) >> 1;  // |d| <= sigma: |d * F| < 2^31
            r[b] = decltype(unclamped)::value ? p.apply_unclamped(n) : p.apply(n);
          }
          o[w] = (int32_t)pack4(r[0], r[1], r[2], r[3]);
        }
        if (live) yr[ch] = o;
      }
    };
    if (clamp)
      outputs(Flag<false>{});
    else
      outputs(Flag<true>{});
  }
}

// Rows longer than 2048 channels: one wave per row, values re-read from
// memory (L1/L2) for each pass.
__global__ __launch_bounds__(256) void layernorm_long_kernel(const int8_t* x, int8_t* y,
                                                             int64_t rows, int32_t C,
                                                             const int32_t* beta,
                                                             const int32_t* mult,
                                                             const int32_t* shift,
                                                             int32_t nq, int32_t iters) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint32_t* xr = (const uint32_t*)(x + row * C);
  uint32_t* yr = (uint32_t*)(y + row * C);
  const int32_t nw = C >> 2;
  int32_t s = 0;
  for (int32_t w = lane; w < nw; w += 64) {
    const uint32_t v = xr[w];
#pragma unroll
    for (int b = 0; b < 4; ++b) s += (int8_t)(v >> (8 * b));
  }
  s = wave_sum_i32(s);
  const int32_t mu = mean_half_up(s, C);
  uint32_t V = 0;
  for (int32_t w = lane; w < nw; w += 64) {
    const uint32_t v = xr[w];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t d = (int8_t)(v >> (8 * b)) - mu;
      V += (uint32_t)(d * d);
    }
  }
  V = wave_sum_u32(V);
  const uint32_t sigma = newton_isqrt(V, iters);
  const uint32_t F = sigma ? 0x7fffffffu / sigma : 0u;
  for (int32_t w = lane; w < nw; w += 64) {
    const uint32_t v = xr[w];
    uint32_t o = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t c = w * 4 + b;
      const int32_t d = (int8_t)(v >> (8 * b)) - mu;
      const int64_t n = ((int64_t)d * (int64_t)F) >> 1;
      const int32_t q = nq == 1 ? 0 : c;
      o |= (uint32_t)(ln_out(n + beta[c], mult[q], shift[q]) & 0xff) << (8 * b);
    }
    yr[w] = o;
  }
}

// ---------------------------------------------------------------- Shiftmax
// One wave per row; three passes over the row (max, exponential sum, output),
// which stays in L1/L2 between passes.
__global__ __launch_bounds__(256) void shiftmax_kernel(const int8_t* x, int8_t* y,
                                                       int64_t rows, int32_t cols,
                                                       int32_t I0, int32_t k_inter,
                                                       int32_t k_out, int32_t m_p,
                                                       int32_t s_d) {
  __shared__ int32_t elut[256];
  elut[threadIdx.x] = shift_exp(-(int32_t)threadIdx.x, I0, k_inter);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int8_t* xr = x + row * cols;
  int8_t* yr = y + row * cols;

  int32_t m = -128;
  for (int32_t j = lane; j < cols; j += 64) m = max(m, (int32_t)xr[j]);
  m = wave_max_i32(m);
  uint64_t sum = 0;
  for (int32_t j = lane; j < cols; j += 64) sum += (uint32_t)elut[m - xr[j]];
  sum = wave_sum_u64(sum);
  const int32_t sd = s_d >= 0 ? s_d : calibrate_shift(sum, m_p);
  const uint32_t F = shiftmax_factor(sum, sd);
  // e F < 2^30 2^31: a shift of 61 or more leaves 0, as does 63, so the cap
  // keeps the 64-bit shift defined (long rows with large m_p: s_d up to 61)
  const int32_t sh = min(32 - k_out + sd, 63);
  const uint64_t cap = (1u << (k_out - 1)) - 1;
  for (int32_t j = lane; j < cols; j += 64) {
    uint64_t p = ((uint64_t)(uint32_t)elut[m - xr[j]] * F) >> sh;
    yr[j] = (int8_t)(p > cap ? cap : p);
  }
}

// Rows of 16-byte chunks (cols % 16 == 0, aligned rows): LPR lanes per row
// hold the row in JC chunks each, so it is read from memory once and written
// once; each wave loads its next row while working on the current one.
// Bytes are biased (x + 128, one XOR per word): max - x is then a byte-wise
// subtraction without borrows, and ShiftExp of it is one lookup in a
// 256-entry LDS table (S_sum >> s_d is exactly the quotient-remainder
// denominator of Alg. 2), kept in registers from the sum to the
// normalization.  The row maximum uses 16-bit packed maxima of the even and
// odd bytes.
template <int LPR, int JC>
__global__ __launch_bounds__(256) void shiftmax_rows_kernel(const int8_t* x, int8_t* y,
                                                            int64_t rows, int32_t cols,
                                                            int32_t I0, int32_t k_inter,
                                                            int32_t k_out, int32_t m_p,
                                                            int32_t s_d) {
  __shared__ uint32_t elut[256];
  constexpr int RG = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, k = lane % LPR;
  const int32_t n16 = cols >> 4;
  const int64_t ngroups = (rows + RG - 1) / RG;
  const int64_t gstride = (int64_t)gridDim.x * 4;
  // chunks past the row repeat the last one: they cannot raise the max
  auto load = [&](int64_t g, v4i(&v)[JC]) {
    const int64_t row = min(g * RG + sub, rows - 1);
    const v4i* xr = (const v4i*)(x + row * cols);
#pragma unroll
    for (int j = 0; j < JC; ++j) v[j] = xr[min(k + j * LPR, n16 - 1)];
  };
  int64_t g = (int64_t)blockIdx.x * 4 + wave;
  v4i nxt[JC];
  if (g < ngroups) load(g, nxt);
  elut[threadIdx.x] = (uint32_t)shift_exp(-(int32_t)threadIdx.x, I0, k_inter);
  __syncthreads();
  const uint32_t cap = (1u << (k_out - 1)) - 1;
  const u16x2 cap2 = {(unsigned short)cap, (unsigned short)cap};
  for (; g < ngroups; g += gstride) {
    uint32_t w[JC][4];
    u16x2 mx = {0, 0};
#pragma unroll
    for (int j = 0; j < JC; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        w[j][q] = (uint32_t)nxt[j][q] ^ 0x80808080u;
        const u16x2 ev = __builtin_bit_cast(u16x2, w[j][q] & 0x00ff00ffu);
        const u16x2 od = __builtin_bit_cast(u16x2, (w[j][q] >> 8) & 0x00ff00ffu);
        mx = __builtin_elementwise_max(mx, __builtin_elementwise_max(ev, od));
      }
    if (g + gstride < ngroups) load(g + gstride, nxt);
    const int64_t row = g * RG + sub;
    const bool live = row < rows;
    uint32_t m = max((uint32_t)mx[0], (uint32_t)mx[1]);
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o, 64));
    const uint32_t m4 = m * 0x01010101u;
    uint32_t e[JC][4][4];
    uint64_t sum = 0;
#pragma unroll
    for (int j = 0; j < JC; ++j) {
      if (k + j * LPR >= n16) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t d4 = m4 - w[j][q];
        uint32_t ws = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          e[j][q][b] = elut[(d4 >> (8 * b)) & 255];
          ws += e[j][q][b];
        }
        sum += ws;  // 4 values of at most 2^30 each
      }
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) {
      const uint32_t lo = __shfl_xor((uint32_t)sum, o, 64);
      const uint32_t hi = __shfl_xor((uint32_t)(sum >> 32), o, 64);
      sum += ((uint64_t)hi << 32) | lo;
    }
    const int32_t sd = s_d >= 0 ? s_d : calibrate_shift(sum, m_p);
    const uint32_t F = shiftmax_factor(sum, sd);
    // e F < 2^30 2^31: a shift of 61 or more leaves 0, as does 63
    const int32_t sh = min(32 - k_out + sd, 63);
    v4i* yr = (v4i*)(y + (live ? row : rows - 1) * cols);
    // With sh < 32 and F < 2^sh, F 2^(32 - sh) fits 32 bits and
    // floor(e F / 2^sh) is the high word of e F 2^(32 - sh); either way the
    // quotient is below 2^k_out <= 2^8, so the 16-bit clamp-and-pack holds
    // it.  (A uniform branch: every row of the wave must qualify.)
    auto outputs = [&](auto hi_word) {
      const uint32_t Fs = F << ((32 - sh) & 31);
#pragma unroll
      for (int j = 0; j < JC; ++j) {
        const int32_t ch = k + j * LPR;
        if (ch >= n16) break;
        v4i o;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t p[4];
#pragma unroll
          for (int b = 0; b < 4; ++b)
            p[b] = decltype(hi_word)::value
                       ? __umulhi(e[j][q][b], Fs)
                       : (uint32_t)min(((uint64_t)e[j][q][b] * F) >> sh, (uint64_t)cap);
          o[q] = (int32_t)pack_min_bytes(p[0], p[1], p[2], p[3], cap2);
        }
        if (live) yr[ch] = o;
      }
    };
    if (__all(sh < 32 && F < (1u << (sh & 31))))
      outputs(Flag<true>{});
    else
      outputs(Flag<false>{});
  }
}

// I-ViT baselines (the forms the paper's operators replace), for comparison.
//
// Shiftmax with a fixed division precision M (eq. shiftmax_original):
// out = (floor((2^M - 1) / S_sum) * I_exp) >> (M - (k_out - 1)).  The factor is
// an exact floor from a correctly rounded FP64 quotient and one integer
// correction (numerator < 2^32, S_sum < 2^47).
__global__ __launch_bounds__(256) void shiftmax_ivit_kernel(const int8_t* x, int8_t* y,
                                                            int64_t rows, int32_t cols,
                                                            int32_t I0, int32_t k_inter,
                                                            int32_t k_out, int32_t M) {
  __shared__ int32_t elut[256];
  elut[threadIdx.x] = shift_exp(-(int32_t)threadIdx.x, I0, k_inter);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int8_t* xr = x + row * cols;
  int8_t* yr = y + row * cols;
  int32_t m = -128;
  for (int32_t j = lane; j < cols; j += 64) m = max(m, (int32_t)xr[j]);
  m = wave_max_i32(m);
  uint64_t sum = 0;
  for (int32_t j = lane; j < cols; j += 64) sum += (uint32_t)elut[m - xr[j]];
  sum = wave_sum_u64(sum);
  const uint64_t num = (1ull << M) - 1;
  int64_t f = (int64_t)((double)num / (double)sum);
  const int64_t r = (int64_t)num - f * (int64_t)sum;
  f += r < 0 ? -1 : (r >= (int64_t)sum ? 1 : 0);
  const int32_t sh = M - (k_out - 1);
  for (int32_t j = lane; j < cols; j += 64)
    yr[j] = (int8_t)(((uint64_t)f * (uint32_t)elut[m - xr[j]]) >> sh);
}

// ShiftGELU with the sigmoid argument shifted by the row maximum of I_p
// (clamped at 0) instead of element-wise by ReLU(I_p), requantized to int8
// like SD-ShiftGELU.  One wave per row.
__global__ __launch_bounds__(256) void shiftgelu_ivit_kernel(const int8_t* x, int8_t* y,
                                                             int64_t rows, int32_t cols,
                                                             int32_t I0, int32_t k_inter,
                                                             int32_t k_out, int32_t mult,
                                                             int32_t shift) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int8_t* xr = x + row * cols;
  int8_t* yr = y + row * cols;
  int32_t mx = -128;
  for (int32_t j = lane; j < cols; j += 64) mx = max(mx, (int32_t)xr[j]);
  mx = wave_max_i32(mx);
  // I_p is non-decreasing in x, so its row maximum is I_p of the row maximum
  const int32_t max_ip = max(mx + (mx >> 1) + (mx >> 3) + (mx >> 4), 0);
  const uint32_t a2 = (uint32_t)shift_exp(-max_ip, I0, k_inter);
  for (int32_t j = lane; j < cols; j += 64) {
    const int32_t v = xr[j];
    const int32_t ip = v + (v >> 1) + (v >> 3) + (v >> 4);
    const uint32_t a = (uint32_t)shift_exp(ip - max_ip, I0, k_inter);
    const uint32_t f = 0x7fffffffu / (a + a2);
    const int32_t d = (int32_t)(((uint64_t)f * a) >> (32 - k_out));
    yr[j] = (int8_t)rq(v * d, mult, shift);
  }
}

// ---------------------------------------------------------------- GELU
// U 16-byte chunks per thread; the first U chunks' loads are issued before
// the table is built (the chunk index clamped: a re-read, never stored).
template <int U>
__global__ __launch_bounds__(256) void gelu_kernel(const int8_t* x, int8_t* y, int64_t n,
                                                   int32_t I0, int32_t k_inter,
                                                   int32_t k_out, int32_t mult,
                                                   int32_t shift) {
  __shared__ int8_t lut[256];
  const int64_t nchunk = n >> 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t c0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  v4i v[U];
  auto load = [&](int64_t cb) {
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = *(const v4i*)(x + min(cb + u * stride, nchunk - 1) * 16);
  };
  if (c0 < nchunk) load(c0);
  lut[threadIdx.x] =
      (int8_t)rq(sd_gelu((int32_t)threadIdx.x - 128, I0, k_inter, k_out), mult, shift);
  __syncthreads();
  for (; c0 < nchunk; c0 += stride * U) {
    if (c0 != (int64_t)blockIdx.x * 256 + threadIdx.x) load(c0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      v4i o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        int32_t r[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) r[b] = lut[(int8_t)(v[u][w] >> (8 * b)) + 128];
        o[w] = (int32_t)pack4(r[0], r[1], r[2], r[3]);
      }
      const int64_t c = c0 + u * stride;
      if (c < nchunk) *(v4i*)(y + c * 16) = o;
    }
  }
  // tail (n not a multiple of 16)
  const int64_t t = (nchunk << 4) + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0 && t < n) y[t] = lut[(int32_t)x[t] + 128];
}

// ---------------------------------------------------------------- residual
// U 16-byte chunks per thread, all loads issued before any arithmetic (the
// chunk index clamped: a re-read, never stored); WIDE as in rq2i8.
template <bool WIDE, int U>
__global__ __launch_bounds__(256) void residual_kernel(const int8_t* a, const int8_t* b,
                                                       int8_t* y, int64_t n, int32_t ma,
                                                       int32_t mb, int32_t shift) {
  const int64_t nchunk = n >> 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t c0 = (int64_t)blockIdx.x * 256 + threadIdx.x; c0 < nchunk; c0 += stride * U) {
    v4i va[U], vb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t c = min(c0 + u * stride, nchunk - 1);
      va[u] = *(const v4i*)(a + c * 16);
      vb[u] = *(const v4i*)(b + c * 16);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      v4i o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        int32_t r[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          r[k] = rq2i8<WIDE>((int8_t)(va[u][w] >> (8 * k)), (int8_t)(vb[u][w] >> (8 * k)), ma, mb,
                             shift);
        o[w] = (int32_t)pack4(r[0], r[1], r[2], r[3]);
      }
      const int64_t c = c0 + u * stride;
      if (c < nchunk) *(v4i*)(y + c * 16) = o;
    }
  }
  const int64_t t = (nchunk << 4) + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0 && t < n) y[t] = (int8_t)rq2(a[t], b[t], ma, mb, shift);
}


}  // namespace

template <int LPR, int JW>
hipError_t launch_ln(const int8_t* x, int8_t* y, int64_t rows, int32_t C, const int32_t* beta,
                     const int32_t* mult, const int32_t* shift, int32_t nq, int32_t iters,
                     hipStream_t s) {
  const int64_t groups = (rows + (64 / LPR) - 1) / (64 / LPR);
  int64_t wgs = (groups + 3) / 4;
  if (wgs > 4096) wgs = 4096;
  hipLaunchKernelGGL((layernorm_kernel<LPR, JW>), dim3((unsigned)wgs), dim3(256), 0, s, x, y,
                     rows, C, beta, mult, shift, nq, iters);
  return hipGetLastError();
}

hipError_t launch_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                            const int32_t* beta, const int32_t* mult, const int32_t* shift,
                            int32_t nq, int32_t iters, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  // Many rows of the encoder widths: LPR lanes per row holding JC 16-byte
  // chunks each.  The 16-byte row loads need 16-byte aligned rows.
  if (C % 16 == 0 && C <= 2048 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)y & 15) == 0) {
    const int32_t n16 = C / 16;
    const size_t smem = (size_t)C * sizeof(RqI64);
    auto go = [&](auto lpr_c, auto jc_c) {
      constexpr int LPR = decltype(lpr_c)::value, JC = decltype(jc_c)::value;
      const int64_t groups = (rows + (64 / LPR) - 1) / (64 / LPR);
      // a few row groups per wave (the next group's loads overlap the
      // current one), and enough workgroups to cover the chip
      int64_t wgs = (groups + 15) / 16;
      if (wgs < 512) wgs = (groups + 3) / 4;
      if (wgs > 2048) wgs = 2048;
      hipLaunchKernelGGL((layernorm_rows_kernel<LPR, JC>), dim3((unsigned)wgs), dim3(256), smem,
                         s, x, y, rows, C, beta, mult, shift, nq, iters);
      return hipGetLastError();
    };
    if (n16 <= 3 * 4) return go(IntC<4>{}, IntC<3>{});    // up to 192 channels
    if (n16 <= 3 * 8) return go(IntC<8>{}, IntC<3>{});    // up to 384
    if (n16 <= 4 * 16) return go(IntC<16>{}, IntC<4>{});  // up to 1024
    return go(IntC<16>{}, IntC<8>{});                     // up to 2048
  }
  const int32_t nw = C / 4;
  if (nw <= 16 * 4) return launch_ln<16, 4>(x, y, rows, C, beta, mult, shift, nq, iters, s);
  if (nw <= 32 * 4) return launch_ln<32, 4>(x, y, rows, C, beta, mult, shift, nq, iters, s);
  if (nw <= 64 * 8) return launch_ln<64, 8>(x, y, rows, C, beta, mult, shift, nq, iters, s);
  dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  hipLaunchKernelGGL(layernorm_long_kernel, grid, block, 0, s, x, y, rows, C, beta, mult,
                     shift, nq, iters);
  return hipGetLastError();
}

hipError_t launch_shiftmax(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                           int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                           int32_t s_d, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (cols % 16 == 0 && cols <= 64 * 16 * 2 && (((uintptr_t)x | (uintptr_t)y) & 15) == 0) {
    const int32_t n16 = cols / 16;
    auto go = [&](auto lpr_c, auto jc_c) {
      constexpr int LPR = decltype(lpr_c)::value, JC = decltype(jc_c)::value;
      const int64_t groups = (rows + (64 / LPR) - 1) / (64 / LPR);
      int64_t wgs = (groups + 3) / 4;
      if (wgs > 4096) wgs = 4096;
      hipLaunchKernelGGL((shiftmax_rows_kernel<LPR, JC>), dim3((unsigned)wgs), dim3(256), 0, s,
                         x, y, rows, cols, I0, k_inter, k_out, m_p, s_d);
      return hipGetLastError();
    };
    if (n16 <= 2 * 8) return go(IntC<8>{}, IntC<2>{});
    if (n16 <= 2 * 32) return go(IntC<32>{}, IntC<2>{});
    return go(IntC<64>{}, IntC<2>{});
  }
  dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  hipLaunchKernelGGL(shiftmax_kernel, grid, block, 0, s, x, y, rows, cols, I0, k_inter,
                     k_out, m_p, s_d);
  return hipGetLastError();
}

hipError_t launch_shiftmax_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                               int32_t I0, int32_t k_inter, int32_t k_out, int32_t M,
                               hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(shiftmax_ivit_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                     x, y, rows, cols, I0, k_inter, k_out, M);
  return hipGetLastError();
}

hipError_t launch_shiftgelu_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                                 int32_t I0, int32_t k_inter, int32_t k_out, int32_t mult,
                                 int32_t shift, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(shiftgelu_ivit_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                     x, y, rows, cols, I0, k_inter, k_out, mult, shift);
  return hipGetLastError();
}



hipError_t launch_gelu(const int8_t* x, int8_t* y, int64_t n, int32_t I0, int32_t k_inter,
                       int32_t k_out, int32_t mult, int32_t shift, hipStream_t s) {
  if (n == 0) return hipSuccess;
  constexpr int U = 4;
  int64_t g = ((n >> 4) + 256 * U - 1) / (256 * U);
  g = g < 1 ? 1 : (g > 4096 ? 4096 : g);
  hipLaunchKernelGGL((gelu_kernel<U>), dim3((unsigned)g), dim3(256), 0, s, x, y, n, I0, k_inter,
                     k_out, mult, shift);
  return hipGetLastError();
}

hipError_t launch_residual(const int8_t* a, const int8_t* b, int8_t* y, int64_t n,
                           int32_t ma, int32_t mb, int32_t shift, hipStream_t s) {
  if (n == 0) return hipSuccess;
  constexpr int U = 4;
  int64_t g = ((n >> 4) + 256 * U - 1) / (256 * U);
  g = g < 1 ? 1 : (g > 2048 ? 2048 : g);
  if (shift >= 9)
    hipLaunchKernelGGL((residual_kernel<false, U>), dim3((unsigned)g), dim3(256), 0, s, a, b, y,
                       n, ma, mb, shift);
  else
    hipLaunchKernelGGL((residual_kernel<true, U>), dim3((unsigned)g), dim3(256), 0, s, a, b, y,
                       n, ma, mb, shift);
  return hipGetLastError();
}

}  // namespace ilw
