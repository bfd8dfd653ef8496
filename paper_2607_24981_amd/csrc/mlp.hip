// mlp.hip -- the 384-wide block's whole MLP in one kernel (Sec. 3.2.1 linear
// and dyadic rescale, Sec. 3.3.1 SD-ShiftGELU, Sec. 3.2.2 residual add,
// Sec. 3.3 I-LayerNorm of the next block), weights pre-packed in MFMA
// fragment order.
//
//   g = rq(SD-ShiftGELU(rq(h W1^T + b1)))      (kept in LDS, never in HBM)
//   y = Res(rq(g W2^T + b2), skip)             -> y   (the residual stream)
//   h' = LN(y)                                 -> y2  (the next block's LN1)
//
// A workgroup holds 64 tokens: their fc1 input (64 x 384) and their whole
// fc1 output (64 x mlp, mlp <= 1536) stay in LDS, so the fc1 output makes no
// HBM round trip and fc2 reads its activations straight from LDS.  As in the
// LayerNorm-fused 384-channel linear, each of the 12 waves owns 32 output
// channels of all 64 tokens and loads its weight fragments from global memory
// straight into MFMA A-operand registers, two K steps ahead in a ring of
// three register sets.  The fc1 and fc2 K steps form one stream: mlp / 384
// chunks of 384 fc1 channels (three 128-byte K steps each, followed by the
// chunk's requantization and SD-ShiftGELU table lookup into LDS), then the
// mlp / 128 K steps of fc2, then the residual and LayerNorm epilogue of the
// 384-channel kernel.  No barrier is needed inside either phase: the
// activation tiles they read are complete before the phase starts.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int M_D = 384, M_TM = 64, M_FJ = 4, M_NW = 12, M_FI = 2;
constexpr int M_KB = 128;                    // K bytes per step
constexpr int M_BLK = M_TM * M_KB;           // one 64 x 128 activation block in LDS
constexpr int M_MAXCH = 4;                   // fc1 chunks of 384 channels at most
constexpr int M_OSTR = M_D / 4 + 4;          // output staging: words per token row
constexpr int NXCD_M = 8;
static_assert(M_FI * M_NW * 16 == M_D, "whole fragments per wave");

// fc1 input block kb of the tile, fc1 output block kb: rows of 128 bytes with
// swizzled chunks (lds_chunk), blocks of 8 KB
__device__ __forceinline__ int blk_off(int kb, int row, int chunk) {
  return kb * M_BLK + lds_chunk<M_KB / 16>(row, chunk);
}

template <bool WIDE_RES, bool DO_LN>
__global__ __launch_bounds__(64 * M_NW) void mlp384_kernel(GemmArgs f1, GemmArgs f2,
                                                           int64_t tiles) {
  // sX: the fc1 input tile (3 blocks); after fc1, the fc2 and LayerNorm
  // output constants.  sH: the fc1 output (mlp / 128 blocks); after fc2's K
  // loop, the output staging rows and the row sums.
  __shared__ __attribute__((aligned(16))) int8_t sX[3 * M_BLK];
  __shared__ __attribute__((aligned(16))) int8_t sH[3 * M_MAXCH * M_BLK];
  __shared__ RqI64 rq1[M_MAXCH * M_D];  // fc1 output requantization per channel
  __shared__ int8_t glut[256];          // SD-ShiftGELU of an int8 value, requantized
  static_assert(2 * M_D * sizeof(RqI64) <= sizeof(sX), "fc2 constants fit the input tile");
  static_assert(M_TM * M_OSTR * 4 + (M_NW + 1) * M_TM * 2 * 4 <= sizeof(sH),
                "staging rows and row sums fit the fc1 output");
  RqI64* const rq2 = (RqI64*)sX;           // fc2 output requantization per channel
  RqI64* const lnq = (RqI64*)sX + M_D;     // LayerNorm output requantization
  uint32_t* const so = (uint32_t*)sH;      // output staging
  int32_t* const lnred = (int32_t*)(sH + M_TM * M_OSTR * 4);  // [M_NW][M_TM][2]
  int32_t* const lnst = lnred + M_NW * M_TM * 2;               // [M_TM][2]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware tile order (workgroup i runs on XCD i % 8)
  const int64_t bid = blockIdx.x;
  const int64_t per = tiles / NXCD_M, rem = tiles % NXCD_M, xcd = bid % NXCD_M;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / NXCD_M;
  const int64_t m0 = tile * M_TM;
  const int64_t M = f1.M;
  const int32_t mlp = f1.N, nch = mlp / M_D;
  const int32_t S1 = 3 * nch;       // fc1 K steps (3 per chunk of 384 channels)
  const int32_t S = S1 + mlp / M_KB;  // with fc2's (a multiple of 3)

  // The weight stream: step k < S1 is K step k % 3 of fc1 chunk k / 3 (this
  // wave's group q * 12 + wave of the packed fc1 weights), later steps are
  // fc2's (group wave of the packed fc2 weights).  One step is 2 K chunks x 2
  // fragments, 4 KB contiguous.
  const int8_t* const w1b = f1.wp + (int64_t)wave * (6 * 2 * 1024) + lane * 16;
  const int8_t* const w2b = f2.wp + (int64_t)wave * (mlp / 64) * (2 * 1024) + lane * 16;
  auto wload = [&](v4i(&wf)[2][M_FI], int k) {
    const int8_t* p;
    if (k < S1) {
      const int q = k / 3;
      p = w1b + (int64_t)q * M_NW * (6 * 2 * 1024) + (k - 3 * q) * (2 * M_FI * 1024);
    } else {
      p = w2b + (int64_t)(k - S1) * (2 * M_FI * 1024);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < M_FI; ++i) wf[h][i] = *(const v4i*)(p + (h * M_FI + i) * 1024);
  };
  v4i w[3][2][M_FI];
  wload(w[0], 0);
  wload(w[1], 1);

  // the fc1 input tile: 64 rows x 24 chunks, two chunks per thread
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = tid + u * 64 * M_NW;
    const int r = c / 24, q = c - r * 24;
    const v4i v = *(const v4i*)(f1.x + min(m0 + r, M - 1) * M_D + q * 16);
    *(v4i*)(sX + blk_off(q >> 3, r, q & 7)) = v;
  }
  // constants, while the loads are in flight
  for (int c = tid; c < mlp; c += 64 * M_NW) {
    RqI64 r;
    r.init(f1.mult[f1.nq == 1 ? 0 : c], f1.shift[f1.nq == 1 ? 0 : c], f1.bias ? f1.bias[c] : 0);
    rq1[c] = r;
  }
  if (tid < 256)
    glut[tid] = (int8_t)rq(sd_gelu(tid - 128, f1.g_I0, f1.g_kinter, f1.g_kout), f1.g_mult,
                           f1.g_shift);
  lds_sync();

  v4i acc[M_FI][M_FJ];
  const v4i zero = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < M_FI; ++i)
#pragma unroll
    for (int j = 0; j < M_FJ; ++j) acc[i][j] = zero;
  // fragment rows start at multiples of 16: the swizzle depends on lane % 16
  const int fo[2] = {lds_chunk<M_KB / 16>(lane & 15, lane >> 4),
                     lds_chunk<M_KB / 16>(lane & 15, 4 + (lane >> 4))};
  auto compute = [&](const int8_t* blk, const v4i(&wf)[2][M_FI]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      v4i fb[M_FJ];
#pragma unroll
      for (int j = 0; j < M_FJ; ++j) fb[j] = *(const v4i*)(blk + j * 16 * M_KB + fo[h]);
#pragma unroll
      for (int i = 0; i < M_FI; ++i)
#pragma unroll
        for (int j = 0; j < M_FJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf[h][i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
  // Lane: channels c_i .. c_i + 3 (c_i = 32 wave + 16 i + 4 (lane / 16)) of
  // token t_j = 16 j + lane % 16 in each chunk / of the fc2 output.
  int32_t cw[M_FI];
#pragma unroll
  for (int i = 0; i < M_FI; ++i) cw[i] = wave * (16 * M_FI) + i * 16 + (lane >> 4) * 4;
  // fc1 chunk q's outputs: requantize, SD-ShiftGELU by table, into sH
  auto fc1_out = [&](int q) {
#pragma unroll
    for (int i = 0; i < M_FI; ++i) {
      const int32_t n = q * M_D + cw[i];
      RqI64 rf[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) rf[r] = rq1[n + r];
      const int kb = n >> 7, nb = n & 127;
#pragma unroll
      for (int j = 0; j < M_FJ; ++j) {
        int32_t g[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) g[r] = glut[rf[r].apply(acc[i][j][r]) + 128];
        const int t = j * 16 + (lane & 15);
        *(uint32_t*)(sH + blk_off(kb, t, nb >> 4) + (nb & 15)) = pack4(g[0], g[1], g[2], g[3]);
        acc[i][j] = zero;
      }
    }
  };

  // The stream, one ring turn (3 steps) per iteration: step k computes from
  // weight set k % 3 and loads step k + 2 (clamped to the last step: a
  // re-read, never used).  fc1 chunks end at steps 3 q + 2, i.e. at the end
  // of a turn; fc2 starts at a turn boundary.
  for (int k0 = 0; k0 < S; k0 += 3) {
    const bool in_fc1 = k0 < S1;
    if (k0 == S1) {
      // fc1 done: its outputs complete, the input tile free for the fc2 and
      // LayerNorm constants (first used after the K loop's closing barrier)
      lds_sync();
      for (int c = tid; c < M_D; c += 64 * M_NW) {
        RqI64 r;
        r.init(f2.mult[f2.nq == 1 ? 0 : c], f2.shift[f2.nq == 1 ? 0 : c],
               f2.bias ? f2.bias[c] : 0);
        rq2[c] = r;
        if (DO_LN) {
          const int qn = f2.ln_nq == 1 ? 0 : c;
          r.init(f2.ln_mult[qn], f2.ln_shift[qn], f2.ln_beta[c]);
          lnq[c] = r;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      const int k = k0 + u;
      wload(w[(u + 2) % 3], min(k + 2, S - 1));
      compute(in_fc1 ? sX + u * M_BLK : sH + (k - S1) * M_BLK, w[u]);
    }
    if (in_fc1) fc1_out(k0 / 3);
  }
  lds_sync();  // fc2's reads of sH done; its constants visible

  // fc2 epilogue: x = Res(rq(acc), skip), 4 channels per word.  Tokens past
  // M read the last row and are never stored.
  uint32_t rs[M_FI][M_FJ];
#pragma unroll
  for (int j = 0; j < M_FJ; ++j) {
    const int64_t m = min(m0 + j * 16 + (lane & 15), M - 1);
#pragma unroll
    for (int i = 0; i < M_FI; ++i) rs[i][j] = *(const uint32_t*)(f2.resid + m * M_D + cw[i]);
  }
  uint32_t xw[M_FI][M_FJ];
#pragma unroll
  for (int i = 0; i < M_FI; ++i) {
    RqI64 rf[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rf[r] = rq2[cw[i] + r];
#pragma unroll
    for (int j = 0; j < M_FJ; ++j) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        o[r] = rq2i8<WIDE_RES>(rf[r].apply(acc[i][j][r]), (int8_t)(rs[i][j] >> (8 * r)),
                               f2.res_ma, f2.res_mb, f2.res_shift);
      xw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
  // row sums: in the lane (byte dot products), across the 4 lanes of a token
  // (shuffles), across the waves (LDS)
#pragma unroll
  for (int j = 0; j < (DO_LN ? M_FJ : 0); ++j) {
    int32_t Sm = 0, SS = 0;
#pragma unroll
    for (int i = 0; i < M_FI; ++i) {
      Sm = __builtin_amdgcn_sdot4((int32_t)xw[i][j], 0x01010101, Sm, false);
      SS = __builtin_amdgcn_sdot4((int32_t)xw[i][j], (int32_t)xw[i][j], SS, false);
    }
    Sm += __shfl_xor(Sm, 16, 64);
    Sm += __shfl_xor(Sm, 32, 64);
    SS += __shfl_xor(SS, 16, 64);
    SS += __shfl_xor(SS, 32, 64);
    if (lane < 16) {
      lnred[(wave * M_TM + j * 16 + lane) * 2 + 0] = Sm;
      lnred[(wave * M_TM + j * 16 + lane) * 2 + 1] = SS;
    }
  }
  // Both outputs leave through LDS token rows as 16-byte row chunks; wave 0
  // turns the row sums into the tokens' statistics while the others copy the
  // residual stream out.
  auto stage = [&](const uint32_t(&wd)[M_FI][M_FJ]) {
#pragma unroll
    for (int i = 0; i < M_FI; ++i)
#pragma unroll
      for (int j = 0; j < M_FJ; ++j) so[(j * 16 + (lane & 15)) * M_OSTR + (cw[i] >> 2)] = wd[i][j];
  };
  auto copy_out = [&](int8_t* dst) {
    const bool a16 = ((uintptr_t)dst & 15) == 0;
    for (int c = tid; c < M_TM * (M_D / 16); c += 64 * M_NW) {
      const int r = c / (M_D / 16), q = c - r * (M_D / 16);
      const int64_t m = m0 + r;
      if (m < M) {
        const v4i v = *(const v4i*)(so + r * M_OSTR + q * 4);
        int8_t* p = dst + m * M_D + q * 16;
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
  stage(xw);
  lds_sync();
  if (!DO_LN) {
    copy_out(f2.y);
    return;
  }
  if (wave == 0) {
    int32_t s = 0, ss = 0;
#pragma unroll
    for (int w2 = 0; w2 < M_NW; ++w2) {
      s += lnred[(w2 * M_TM + lane) * 2 + 0];
      ss += lnred[(w2 * M_TM + lane) * 2 + 1];
    }
    const int32_t mu = mean_half_up(s, M_D);
    const uint32_t V = (uint32_t)(ss - 2 * mu * s + M_D * mu * mu);
    const uint32_t sigma = newton_isqrt_f64(V, f2.ln_iters);
    lnst[lane * 2 + 0] = mu;
    lnst[lane * 2 + 1] = sigma ? (int32_t)div_2p31m1(sigma) : 0;
  }
  copy_out(f2.y);
  lds_sync();  // statistics written; every read of the staged x done
  uint32_t yw[M_FI][M_FJ];
#pragma unroll
  for (int j = 0; j < M_FJ; ++j) {
    const int32_t mu = lnst[(j * 16 + (lane & 15)) * 2 + 0];
    const int32_t F = lnst[(j * 16 + (lane & 15)) * 2 + 1];
#pragma unroll
    for (int i = 0; i < M_FI; ++i) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t d = (int8_t)(xw[i][j] >> (8 * r)) - mu;
        o[r] = lnq[cw[i] + r].apply((d * F) >> 1);  // |d| <= sigma: |d * F| < 2^31
      }
      yw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
  stage(yw);
  lds_sync();
  copy_out(f2.y2);
}

}  // namespace

bool mlp384_kernel_applies(int64_t M, int32_t D, int32_t mlp) {
  return D == M_D && mlp > 0 && mlp % M_D == 0 && mlp / M_D <= M_MAXCH &&
         !gemm_latency_mode(M, D);
}

hipError_t launch_mlp384(const GemmArgs& f1, const GemmArgs& f2, bool layernorm,
                         hipStream_t s) {
  if (f1.M == 0) return hipSuccess;
  if (!mlp384_kernel_applies(f1.M, f2.N, f1.N) || f1.K != M_D || f2.K != f1.N || !f1.wp ||
      !f2.wp)
    return hipErrorInvalidValue;
  const int64_t tiles = (f1.M + M_TM - 1) / M_TM;
  const dim3 grid((unsigned)tiles), block(64 * M_NW);
  if (f2.res_shift < 9) {
    if (layernorm) hipLaunchKernelGGL((mlp384_kernel<true, true>), grid, block, 0, s, f1, f2, tiles);
    else hipLaunchKernelGGL((mlp384_kernel<true, false>), grid, block, 0, s, f1, f2, tiles);
  } else {
    if (layernorm) hipLaunchKernelGGL((mlp384_kernel<false, true>), grid, block, 0, s, f1, f2, tiles);
    else hipLaunchKernelGGL((mlp384_kernel<false, false>), grid, block, 0, s, f1, f2, tiles);
  }
  return hipGetLastError();
}

}  // namespace ilw
