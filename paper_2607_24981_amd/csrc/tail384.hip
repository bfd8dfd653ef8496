// tail384.hip -- everything of a 384-wide encoder block after attention in
// one kernel (Sec. 3.2.1 linear and dyadic rescale, Sec. 3.2.2 residual add,
// Sec. 3.3 I-LayerNorm, Sec. 3.3.1 SD-ShiftGELU), weights pre-packed in MFMA
// fragment order.
//
//   x1 = Res(rq(att Wp^T + bp), x)              (registers only)
//   h  = LN2(x1)                                (LDS only)
//   g  = rq(SD-ShiftGELU(rq(h W1^T + b1)))      (LDS only)
//   y  = Res(rq(g W2^T + b2), x1)               -> y   (the block's output)
//   h' = LN1 of the next block (y)              -> y2  (optional)
//
// A workgroup holds 64 tokens.  Each of its 12 waves owns 32 channels of all
// 64 tokens in every 384-wide result (projection, each 384-channel chunk of
// fc1, fc2) and loads its weight fragments from global memory straight into
// MFMA A-operand registers, two K steps ahead in a ring of three register
// sets: the projection's 3 K steps, fc1's 3 per chunk and fc2's mlp / 128
// form one stream.  The activation operands are LDS tiles of 64 rows with
// swizzled 128-byte blocks: the attention output, then h (written by the
// projection's LayerNorm epilogue), then the fc1 output (written chunk by
// chunk, SD-ShiftGELU by table).  In the accumulator layout a lane holds 4
// channels of one token, the same positions in the projection's and fc2's
// results, so x1 -- fc2's residual input -- stays in the registers of the
// lane that produced it.  Only att and x are read from HBM and only y (and
// h') written.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int T_D = 384, T_TM = 64, T_FJ = 4, T_NW = 12, T_FI = 2;
constexpr int T_KB = 128;                    // K bytes per step
constexpr int T_BLK = T_TM * T_KB;           // one 64 x 128 activation block in LDS
constexpr int T_MAXCH = 4;                   // fc1 chunks of 384 channels at most
constexpr int T_OSTR = T_D / 4 + 4;          // output staging: words per token row
constexpr int NXCD_T = 8;
// accumulator bounds for the requantization constants: a 384-deep int8
// product; a LayerNorm's (d F) >> 1, with |d| <= sigma and F < 2^31 / sigma
constexpr uint32_t kAccD = (uint32_t)T_D << 14, kAccLN = 1u << 30;
static_assert(T_FI * T_NW * 16 == T_D, "whole fragments per wave");

// block kb of an activation tile: rows of 128 bytes with swizzled chunks
// (lds_chunk), blocks of 8 KB
__device__ __forceinline__ int blk_off(int kb, int row, int chunk) {
  return kb * T_BLK + lds_chunk<T_KB / 16>(row, chunk);
}

// LayerNorm of one 384-wide result, 4 channels per word: row sums (byte dot
// products, the 4 lanes of a token, the waves through LDS), then wave 0
// turns them into each token's mean and 1 / sigma factor (one serial Newton
// chain per lane, computed once per workgroup), then every lane requantizes
// its words.  lnred: [T_NW][T_TM][2], lnst: [T_TM][2].  `before` runs once
// the sums are written and must end in a barrier; `during` runs on every
// wave while wave 0 computes the statistics (after them on wave 0).
template <typename Before, typename During>
__device__ __forceinline__ void layernorm_words(const uint32_t (&xw)[T_FI][T_FJ],
                                                uint32_t (&yw)[T_FI][T_FJ], const RqI64* lnq,
                                                int32_t iters, int32_t* lnred, int32_t* lnst,
                                                const int32_t (&cw)[T_FI], int wave, int lane,
                                                Before before, During during) {
#pragma unroll
  for (int j = 0; j < T_FJ; ++j) {
    int32_t S = 0, SS = 0;
#pragma unroll
    for (int i = 0; i < T_FI; ++i) {
      S = __builtin_amdgcn_sdot4((int32_t)xw[i][j], 0x01010101, S, false);
      SS = __builtin_amdgcn_sdot4((int32_t)xw[i][j], (int32_t)xw[i][j], SS, false);
    }
    S += __shfl_xor(S, 16, 64);
    S += __shfl_xor(S, 32, 64);
    SS += __shfl_xor(SS, 16, 64);
    SS += __shfl_xor(SS, 32, 64);
    if (lane < 16) {
      lnred[(wave * T_TM + j * 16 + lane) * 2 + 0] = S;
      lnred[(wave * T_TM + j * 16 + lane) * 2 + 1] = SS;
    }
  }
  before();  // ends with a barrier
  if (wave == 0) {
    int32_t s = 0, ss = 0;
#pragma unroll
    for (int w = 0; w < T_NW; ++w) {
      s += lnred[(w * T_TM + lane) * 2 + 0];
      ss += lnred[(w * T_TM + lane) * 2 + 1];
    }
    const int32_t mu = mean_half_up(s, T_D);
    const uint32_t V = (uint32_t)(ss - 2 * mu * s + T_D * mu * mu);
    const uint32_t sigma = newton_isqrt_f64(V, iters);
    lnst[lane * 2 + 0] = mu;
    lnst[lane * 2 + 1] = sigma ? (int32_t)div_2p31m1(sigma) : 0;
  }
  during();
  lds_sync();
#pragma unroll
  for (int j = 0; j < T_FJ; ++j) {
    const int32_t mu = lnst[(j * 16 + (lane & 15)) * 2 + 0];
    const int32_t F = lnst[(j * 16 + (lane & 15)) * 2 + 1];
#pragma unroll
    for (int i = 0; i < T_FI; ++i) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t d = (int8_t)(xw[i][j] >> (8 * r)) - mu;
        o[r] = lnq[cw[i] + r].apply((d * F) >> 1);  // |d| <= sigma: |d * F| < 2^31
      }
      yw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
}

// fp: projection + residual (x = att, wp, resid = the block input, LN2's
// fields); f1: fc1 + SD-ShiftGELU (wp, N = mlp, the GELU fields); f2: fc2 +
// residual (wp, y, with DO_LN the next LayerNorm's fields and y2).
template <bool WIDE1, bool WIDE2, bool DO_LN>
__global__ __launch_bounds__(64 * T_NW) void tail384_kernel(GemmArgs fp, GemmArgs f1, GemmArgs f2,
                                                            int64_t tiles) {
  // sX: h, the fc1 input (3 blocks); after fc1, the fc2 and LayerNorm output
  // constants.  sH: first the attention output (3 blocks), the projection's
  // and LN2's constants and their row sums; then the fc1 output (mlp / 128
  // blocks); after fc2's K loop the output staging rows and row sums.
  __shared__ __attribute__((aligned(16))) int8_t sX[3 * T_BLK];
  __shared__ __attribute__((aligned(16))) int8_t sH[3 * T_MAXCH * T_BLK];
  __shared__ RqI64 rq1[T_MAXCH * T_D];  // fc1 output requantization per channel
  // SD-ShiftGELU of an int8 value, requantized.  Aligned so that it sits at
  // LDS address 0: a lookup's +128 then folds into the instruction offset.
  __shared__ __attribute__((aligned(1024))) int8_t glut[256];
  __shared__ int32_t fc1_needs_clamp[T_NW];  // per wave: see the fc1 constants below
  static_assert(2 * T_D * sizeof(RqI64) <= sizeof(sX), "fc2 constants fit the h tile");
  constexpr int RED = (T_NW + 1) * T_TM * 2 * 4;  // row sums and statistics
  static_assert(3 * T_BLK + 2 * T_D * sizeof(RqI64) + RED <= sizeof(sH), "projection phase fits");
  static_assert(T_TM * T_OSTR * 4 + RED <= sizeof(sH), "staging rows and row sums fit");
  // projection phase
  RqI64* const rqp = (RqI64*)(sH + 3 * T_BLK);  // projection output requantization
  RqI64* const lnq2 = rqp + T_D;                // LN2 output requantization
  int32_t* const red1 = (int32_t*)(lnq2 + T_D);
  // fc2 phase
  RqI64* const rq2 = (RqI64*)sX;
  RqI64* const lnq = (RqI64*)sX + T_D;
  uint32_t* const so = (uint32_t*)sH;
  int32_t* const red2 = (int32_t*)(sH + T_TM * T_OSTR * 4);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware tile order (workgroup i runs on XCD i % 8)
  const int64_t bid = blockIdx.x;
  const int64_t per = tiles / NXCD_T, rem = tiles % NXCD_T, xcd = bid % NXCD_T;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / NXCD_T;
  const int64_t m0 = tile * T_TM;
  const int64_t M = fp.M;
  const int32_t mlp = f1.N, nch = mlp / T_D;
  const int32_t S0 = 3;             // projection K steps
  const int32_t S1 = S0 + 3 * nch;  // + fc1's (3 per chunk of 384 channels)
  const int32_t S = S1 + mlp / T_KB;  // + fc2's: a multiple of 3

  // The weight stream: steps < S0 are the projection's (this wave's group of
  // the packed projection weights), then fc1 chunk q's 3 steps (group q * 12
  // + wave of the packed fc1 weights), then fc2's (group wave).  One step is
  // 2 K chunks x 2 fragments, 4 KB contiguous.
  // (the step's base is wave-uniform; only lane * 16 is per lane)
  auto wload = [&](v4i(&wf)[2][T_FI], int k) {
    const int8_t* base;
    int64_t off;
    if (k < S0) {
      base = fp.wp;
      off = (int64_t)wave * (6 * 2 * 1024) + k * (2 * T_FI * 1024);
    } else if (k < S1) {
      const int q = (k - S0) / 3;
      base = f1.wp;
      off = (int64_t)(q * T_NW + wave) * (6 * 2 * 1024) + (k - S0 - 3 * q) * (2 * T_FI * 1024);
    } else {
      base = f2.wp;
      off = (int64_t)wave * (mlp / 64) * (2 * 1024) + (int64_t)(k - S1) * (2 * T_FI * 1024);
    }
    const int8_t* p = base + off + lane * 16;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < T_FI; ++i) wf[h][i] = *(const v4i*)(p + (h * T_FI + i) * 1024);
  };
  v4i w[3][2][T_FI];
  wload(w[0], 0);
  wload(w[1], 1);

  // the attention output tile: 64 rows x 24 chunks, two chunks per thread
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = tid + u * 64 * T_NW;
    const int r = c / 24, q = c - r * 24;
    const v4i v = *(const v4i*)(fp.x + min(m0 + r, M - 1) * T_D + q * 16);
    *(v4i*)(sH + blk_off(q >> 3, r, q & 7)) = v;
  }
  // Lane: channels c_i .. c_i + 3 (c_i = 32 wave + 16 i + 4 (lane / 16)) of
  // token t_j = 16 j + lane % 16 of every 384-wide result.  Tokens past M
  // read the last row and are never stored.
  int32_t cw[T_FI];
#pragma unroll
  for (int i = 0; i < T_FI; ++i) cw[i] = wave * (16 * T_FI) + i * 16 + (lane >> 4) * 4;
  // constants, while the loads are in flight
  for (int c = tid; c < T_D; c += 64 * T_NW) {
    RqI64 r;
    r.init_bounded(fp.mult[fp.nq == 1 ? 0 : c], fp.shift[fp.nq == 1 ? 0 : c],
                   fp.bias ? fp.bias[c] : 0, kAccD);
    rqp[c] = r;
    const int qn = fp.ln_nq == 1 ? 0 : c;
    r.init_bounded(fp.ln_mult[qn], fp.ln_shift[qn], fp.ln_beta[c], kAccLN);
    lnq2[c] = r;
  }
  // fc1's requantization skips the accumulator clamp when every channel
  // allows it (RqI64::init_bounded)
  bool needs_clamp = false;
  for (int c = tid; c < mlp; c += 64 * T_NW) {
    RqI64 r;
    needs_clamp |= !r.init_bounded(f1.mult[f1.nq == 1 ? 0 : c], f1.shift[f1.nq == 1 ? 0 : c],
                                   f1.bias ? f1.bias[c] : 0, kAccD);
    rq1[c] = r;
  }
  const bool wave_needs = __any(needs_clamp);
  if (lane == 0) fc1_needs_clamp[wave] = wave_needs;
  if (tid < 256)
    glut[tid] = (int8_t)rq(sd_gelu(tid - 128, f1.g_I0, f1.g_kinter, f1.g_kout), f1.g_mult,
                           f1.g_shift);
  lds_sync();
  int32_t any_needs = 0;
#pragma unroll
  for (int w = 0; w < T_NW; ++w) any_needs |= fc1_needs_clamp[w];
  const bool fc1_unclamped = __builtin_amdgcn_readfirstlane(any_needs) == 0;

  v4i acc[T_FI][T_FJ];
  const v4i zero = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < T_FI; ++i)
#pragma unroll
    for (int j = 0; j < T_FJ; ++j) acc[i][j] = zero;
  // fragment rows start at multiples of 16: the swizzle depends on lane % 16
  const int fo[2] = {lds_chunk<T_KB / 16>(lane & 15, lane >> 4),
                     lds_chunk<T_KB / 16>(lane & 15, 4 + (lane >> 4))};
  auto compute = [&](const int8_t* blk, const v4i(&wf)[2][T_FI]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      v4i fb[T_FJ];
#pragma unroll
      for (int j = 0; j < T_FJ; ++j) fb[j] = *(const v4i*)(blk + j * 16 * T_KB + fo[h]);
#pragma unroll
      for (int i = 0; i < T_FI; ++i)
#pragma unroll
        for (int j = 0; j < T_FJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf[h][i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
  // one ring turn: steps k0 .. k0 + 2 from the 3 blocks at base (stride
  // T_BLK); step k loads step k + 2 (clamped to the last step: a re-read,
  // never used)
  auto turn = [&](int k0, const int8_t* base) {
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      wload(w[(u + 2) % 3], min(k0 + u + 2, S - 1));
      compute(base + u * T_BLK, w[u]);
    }
  };
  // a word of 4 channels of token t into block layout tile (channel n, a
  // multiple of 4)
  auto put_word = [&](int8_t* tilebase, int n, int t, uint32_t word) {
    *(uint32_t*)(tilebase + blk_off(n >> 7, t, (n & 127) >> 4) + (n & 15)) = word;
  };

  // The stream, one ring turn (3 K steps) per iteration: the projection's
  // turn, then fc1's chunks, then fc2's turns.  After the projection:
  // x1 = Res(rq(acc), x) stays in xw1, h = LN2(x1) goes to sX.  After each
  // fc1 chunk: requantize, SD-ShiftGELU by table, into sH.
  uint32_t xw1[T_FI][T_FJ];
  for (int k0 = 0; k0 < S; k0 += 3) {
    turn(k0, k0 < S0 ? sH : (k0 < S1 ? sX : sH + (k0 - S1) * T_BLK));
    if (k0 < S0) {
      uint32_t rs[T_FI][T_FJ];  // the block input x: the projection's residual
#pragma unroll
      for (int j = 0; j < T_FJ; ++j) {
        const int64_t m = min(m0 + j * 16 + (lane & 15), M - 1);
#pragma unroll
        for (int i = 0; i < T_FI; ++i) rs[i][j] = *(const uint32_t*)(fp.resid + m * T_D + cw[i]);
      }
#pragma unroll
      for (int i = 0; i < T_FI; ++i) {
        RqI64 rf[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) rf[r] = rqp[cw[i] + r];
#pragma unroll
        for (int j = 0; j < T_FJ; ++j) {
          int32_t o[4];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            o[r] = rq2i8<WIDE1>(rf[r].apply(acc[i][j][r]), (int8_t)(rs[i][j] >> (8 * r)),
                                fp.res_ma, fp.res_mb, fp.res_shift);
          xw1[i][j] = pack4(o[0], o[1], o[2], o[3]);
          acc[i][j] = zero;
        }
      }
      uint32_t hw[T_FI][T_FJ];
      layernorm_words(xw1, hw, lnq2, fp.ln_iters, red1, red1 + T_NW * T_TM * 2, cw, wave, lane,
                      [] { lds_sync(); }, [] {});
#pragma unroll
      for (int i = 0; i < T_FI; ++i)
#pragma unroll
        for (int j = 0; j < T_FJ; ++j) put_word(sX, cw[i], j * 16 + (lane & 15), hw[i][j]);
      lds_sync();  // h complete; the attention tile and its constants no longer read
    } else if (k0 < S1) {
      const int q = (k0 - S0) / 3;
#pragma unroll
      for (int i = 0; i < T_FI; ++i) {
        const int32_t n = q * T_D + cw[i];
        RqI64 rf[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) rf[r] = rq1[n + r];
        if (fc1_unclamped) {
#pragma unroll
          for (int j = 0; j < T_FJ; ++j) {
            int32_t g[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) g[r] = glut[rf[r].apply_unclamped(acc[i][j][r]) + 128];
            put_word(sH, n, j * 16 + (lane & 15), pack4(g[0], g[1], g[2], g[3]));
            acc[i][j] = zero;
          }
        } else {
#pragma unroll
          for (int j = 0; j < T_FJ; ++j) {
            int32_t g[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) g[r] = glut[rf[r].apply(acc[i][j][r]) + 128];
            put_word(sH, n, j * 16 + (lane & 15), pack4(g[0], g[1], g[2], g[3]));
            acc[i][j] = zero;
          }
        }
      }
      if (k0 + 3 == S1) {
        // fc1 done: its outputs complete, the h tile free for the fc2 and
        // LayerNorm constants (first used after the closing barrier)
        lds_sync();
        for (int c = tid; c < T_D; c += 64 * T_NW) {
          RqI64 r;
          r.init_bounded(f2.mult[f2.nq == 1 ? 0 : c], f2.shift[f2.nq == 1 ? 0 : c],
                         f2.bias ? f2.bias[c] : 0, (uint32_t)mlp << 14);
          rq2[c] = r;
          if (DO_LN) {
            const int qn = f2.ln_nq == 1 ? 0 : c;
            r.init_bounded(f2.ln_mult[qn], f2.ln_shift[qn], f2.ln_beta[c], kAccLN);
            lnq[c] = r;
          }
        }
      }
    }
  }

  // ---- fc2's result: residual onto x1, the next LayerNorm
  lds_sync();  // fc2's reads of sH done; its constants visible
  uint32_t xw[T_FI][T_FJ];
#pragma unroll
  for (int i = 0; i < T_FI; ++i) {
    RqI64 rf[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rf[r] = rq2[cw[i] + r];
#pragma unroll
    for (int j = 0; j < T_FJ; ++j) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        o[r] = rq2i8<WIDE2>(rf[r].apply(acc[i][j][r]), (int8_t)(xw1[i][j] >> (8 * r)), f2.res_ma,
                            f2.res_mb, f2.res_shift);
      xw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
  // Both outputs leave through LDS token rows as 16-byte row chunks; wave 0
  // turns the row sums into the tokens' statistics while the others copy the
  // block output out.
  auto stage = [&](const uint32_t(&wd)[T_FI][T_FJ]) {
#pragma unroll
    for (int i = 0; i < T_FI; ++i)
#pragma unroll
      for (int j = 0; j < T_FJ; ++j) so[(j * 16 + (lane & 15)) * T_OSTR + (cw[i] >> 2)] = wd[i][j];
  };
  auto copy_out = [&](int8_t* dst) {
    const bool a16 = ((uintptr_t)dst & 15) == 0;
    for (int c = tid; c < T_TM * (T_D / 16); c += 64 * T_NW) {
      const int r = c / (T_D / 16), q = c - r * (T_D / 16);
      const int64_t m = m0 + r;
      if (m < M) {
        const v4i v = *(const v4i*)(so + r * T_OSTR + q * 4);
        int8_t* p = dst + m * T_D + q * 16;
        if (a16) {
          *(v4i*)p = v;
        } else {
          uint32_t* d = (uint32_t*)p;
          d[0] = (uint32_t)v[0];
          d[1] = (uint32_t)v[1];
          d[2] = (uint32_t)v[2];
          d[3] = (uint32_t)v[3];
        }
      }
    }
  };
  if (!DO_LN) {
    stage(xw);
    lds_sync();
    copy_out(f2.y);
    return;
  }
  uint32_t yw[T_FI][T_FJ];
  // (the barrier after `during` also ends every read of the staged y)
  layernorm_words(
      xw, yw, lnq, f2.ln_iters, red2, red2 + T_NW * T_TM * 2, cw, wave, lane,
      [&] {
        stage(xw);
        lds_sync();
      },
      [&] { copy_out(f2.y); });
  stage(yw);
  lds_sync();
  copy_out(f2.y2);
}

template <bool W1, bool W2>
void tail384_launch(const GemmArgs& fp, const GemmArgs& f1, const GemmArgs& f2, bool layernorm,
                    int64_t tiles, hipStream_t s) {
  const dim3 grid((unsigned)tiles), block(64 * T_NW);
  if (layernorm)
    hipLaunchKernelGGL((tail384_kernel<W1, W2, true>), grid, block, 0, s, fp, f1, f2, tiles);
  else
    hipLaunchKernelGGL((tail384_kernel<W1, W2, false>), grid, block, 0, s, fp, f1, f2, tiles);
}

}  // namespace

// Any token count: at batch 1 to 4 of the 1600-token 384-wide encoder (25 to
// 100 workgroups) the kernel still beats the latency-mode GEMM tiles.
bool tail384_kernel_applies(int64_t M, int32_t D, int32_t mlp) {
  return M > 0 && D == T_D && mlp > 0 && mlp % T_D == 0 && mlp / T_D <= T_MAXCH;
}

hipError_t launch_tail384(const GemmArgs& fp, const GemmArgs& f1, const GemmArgs& f2,
                          bool layernorm, hipStream_t s) {
  if (fp.M == 0) return hipSuccess;
  if (!tail384_kernel_applies(fp.M, fp.N, f1.N) || fp.K != T_D || f1.K != T_D ||
      f2.K != f1.N || f2.N != T_D || !fp.wp || !f1.wp || !f2.wp)
    return hipErrorInvalidValue;
  const int64_t tiles = (fp.M + T_TM - 1) / T_TM;
  const bool w1 = fp.res_shift < 9, w2 = f2.res_shift < 9;
  if (w1 && w2) tail384_launch<true, true>(fp, f1, f2, layernorm, tiles, s);
  else if (w1) tail384_launch<true, false>(fp, f1, f2, layernorm, tiles, s);
  else if (w2) tail384_launch<false, true>(fp, f1, f2, layernorm, tiles, s);
  else tail384_launch<false, false>(fp, f1, f2, layernorm, tiles, s);
  return hipGetLastError();
}

}  // namespace ilw
