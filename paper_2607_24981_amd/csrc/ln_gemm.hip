// ln_gemm.hip -- the 384-channel residual linear with its LayerNorm fused
// (Sec. 3.2.1 linear and dyadic rescale, Sec. 3.2.2 residual add, Sec. 3.3
// I-LayerNorm), for weights pre-packed in MFMA fragment order.
//
//   x = Res(rq(a W^T + b), skip)          -> y   (the block's residual stream)
//   h = LN(x)                             -> y2  (the next linear's input)
//
// A workgroup holds 64 tokens x all 384 channels, so the LayerNorm
// statistics of a token stay on chip.  Each weight fragment (16 channels x 64
// K bytes) is used by exactly one wave, so the weights skip LDS: a wave loads
// its fragments straight into MFMA A-operand registers.  Packed, the 16 x 64
// bytes of a fragment are 1 KB contiguous in lane order (lane L holds
// channel L % 16, K bytes 16 (L / 16) .. + 15), so each load instruction of
// the wave reads 1 KB contiguous, and the fragments of one wave are grouped
// K-chunk-major, so that one K step of a wave (2 K chunks x 2 fragments) is
// 4 KB contiguous: one address, four immediate offsets.  Only the 64-token
// activation tile is staged through LDS (shared by all waves).  Measured
// against the LDS-staged weight tile on MI355X: 27% less time in the K loop
// of the 1536-deep fc2, 20% at K = 384.
//
// Weights are loaded two K steps ahead (a ring of three register sets) when
// the step count is a multiple of 3 (K = 384, 768, 1152, 1536), one step
// ahead otherwise: fc2 21.4 -> 19.3 us, projection 13.9 -> 13.4 us at batch
// 8.  Every load of the ring is unconditional (the step index clamped to the
// last step) and the loop body holds whole ring turns: with guarded loads the
// compiler waited for each load and spilled the ring.
//
// 12 waves: wave w owns channels 32 w .. 32 w + 31 (2 fragments) of all 64
// tokens (4 fragments); a lane ends up with 4 consecutive channels of token
// lane % 16 of each fragment, as in the other GEMM kernels.  Three waves per
// SIMD hide the epilogue's latencies better than two (8 waves of 48
// channels): projection 14.5 -> 13.9 us, fc2 22.4 -> 21.3 us at batch 8.
#include <algorithm>

#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int LN_N = 384, LN_TM = 64, LN_FJ = 4;
constexpr int LN_KB = 128, LN_LROW = LN_KB;  // 128-byte rows, chunks swizzled (lds_chunk)
constexpr int LN_OSTR = LN_N / 4 + 4;  // output staging: 100 words per token row (odd x 4)
constexpr int LN_XBUF = 3;  // activation tile buffers (the ring's length at most)
constexpr int LN_SBUF = LN_XBUF * LN_TM * LN_LROW > LN_TM * LN_OSTR * 4
                            ? LN_XBUF * LN_TM * LN_LROW
                            : LN_TM * LN_OSTR * 4;
constexpr int NXCD_LN = 8;
constexpr int LN_WAVES = 12;  // waves per workgroup: 12 x 32 channels
constexpr int kPackGroup = LN_N / 16 / LN_WAVES;  // fragments per wave, packed together

// LN_NW waves of LN_FI 16-channel fragments each (LN_NW * LN_FI = 24); RING
// weight register sets (2: one K step ahead, any step count; 3: two steps
// ahead, step count a multiple of 3); DO_LN false: the residual output only
// (the last block's fc2, which no LayerNorm follows)
template <bool WIDE_RES, int LN_NW, int RING, bool DO_LN>
__global__ __launch_bounds__(64 * LN_NW) void ln384_wp_kernel(GemmArgs a, int64_t tiles) {
  constexpr int LN_FI = LN_N / 16 / LN_NW;
  static_assert(LN_FI * LN_NW * 16 == LN_N, "whole fragments per wave");
  static_assert(LN_FI == kPackGroup, "the packing groups this wave's fragments");
  static_assert(RING == 2 || RING == 3, "ring of two or three weight sets");
  // X double buffer during the K loop; after it, the output staging rows
  __shared__ __attribute__((aligned(16))) int8_t sbuf[LN_SBUF];
  __shared__ RqI64 rqc[LN_N];    // linear output requantization per channel
  __shared__ RqI64 lnq[LN_N];    // LayerNorm output requantization per channel
  __shared__ int32_t lnred[LN_NW][LN_TM][2];  // per-wave row sums
  __shared__ int32_t lnst[LN_TM][2];          // per token: mean, 1 / sigma factor

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware tile order (workgroup i runs on XCD i % 8)
  const int64_t bid = blockIdx.x;
  const int64_t per = tiles / NXCD_LN, rem = tiles % NXCD_LN, xcd = bid % NXCD_LN;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / NXCD_LN;
  const int64_t m0 = tile * LN_TM;
  const int64_t M = a.M;
  const int32_t K = a.K, KC = K / 64, nk = K / LN_KB;

  // operands: this thread's 16-byte chunk of the activation tile (row tid / 8)
  // and this wave's weight fragments
  const int8_t* xsrc = a.x + min(m0 + tid / 8, M - 1) * K + (tid % 8) * 16;
  const int xo = lds_chunk<LN_KB / 16>(tid / 8, tid % 8);
  static_assert(64 * LN_NW >= LN_TM * LN_KB / 16, "one activation chunk per thread at most");
  const bool xown = tid < LN_TM * LN_KB / 16;  // threads that stage an activation chunk
  // this wave's fragments: K chunk k64, fragment i at (k64 LN_FI + i) KB
  const int8_t* wb = a.wp + (int64_t)wave * KC * (LN_FI * 1024) + lane * 16;
  auto wload = [&](v4i(&wf)[2][LN_FI], int kt) {
    const int8_t* p = wb + (int64_t)kt * (2 * LN_FI * 1024);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < LN_FI; ++i) wf[h][i] = *(const v4i*)(p + (h * LN_FI + i) * 1024);
  };
  v4i w[RING][2][LN_FI];
  v4i rx = {0, 0, 0, 0};
  if (xown) rx = *(const v4i*)xsrc;
#pragma unroll
  for (int u = 0; u < RING - 1; ++u) wload(w[u], min(u, nk - 1));

  // constants, while the first loads are in flight
  for (int c = tid; c < LN_N; c += 64 * LN_NW) {
    RqI64 r;
    r.init(a.mult[a.nq == 1 ? 0 : c], a.shift[a.nq == 1 ? 0 : c], a.bias ? a.bias[c] : 0);
    rqc[c] = r;
    if (DO_LN) {
      const int q = a.ln_nq == 1 ? 0 : c;
      r.init(a.ln_mult[q], a.ln_shift[q], a.ln_beta[c]);
      lnq[c] = r;
    }
  }

  v4i acc[LN_FI][LN_FJ];
  const v4i zero = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < LN_FI; ++i)
#pragma unroll
    for (int j = 0; j < LN_FJ; ++j) acc[i][j] = zero;
  // fragment rows start at multiples of 16: the swizzle depends on lane % 16
  const int fo[2] = {lds_chunk<LN_KB / 16>(lane & 15, lane >> 4),
                     lds_chunk<LN_KB / 16>(lane & 15, 4 + (lane >> 4))};
  auto compute = [&](const int8_t* sx, const v4i(&wf)[2][LN_FI]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      v4i fb[LN_FJ];
#pragma unroll
      for (int j = 0; j < LN_FJ; ++j) fb[j] = *(const v4i*)(sx + j * 16 * LN_LROW + fo[h]);
#pragma unroll
      for (int i = 0; i < LN_FI; ++i)
#pragma unroll
        for (int j = 0; j < LN_FJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf[h][i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
  if (xown) *(v4i*)(sbuf + xo) = rx;
  lds_sync();
  if constexpr (RING == 3) {
    // nk is a multiple of 3.  Step k computes from LDS buffer k % 3 and
    // weight set k % 3 and loads the activations of step k + 1 and the
    // weights of step k + 2 (clamped to the last step: re-read, never used).
    // Buffer (k + 1) % 3 was last read in step k - 2, before the previous
    // barrier.
    for (int kt = 0; kt < nk; kt += 3) {
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int k = kt + u;
        if (xown) rx = *(const v4i*)(xsrc + min(k + 1, nk - 1) * LN_KB);
        wload(w[(u + 2) % 3], min(k + 2, nk - 1));
        compute(sbuf + u * LN_TM * LN_LROW, w[u]);
        if (xown) *(v4i*)(sbuf + ((u + 1) % 3) * LN_TM * LN_LROW + xo) = rx;
        lds_sync();
      }
    }
  } else {
    // step kt computes from LDS buffer kt % 2 and weight set kt % 2 while
    // step kt + 1 loads
    int8_t* const sX0 = sbuf;
    int8_t* const sX1 = sbuf + LN_TM * LN_LROW;
    for (int kt = 0; kt < nk; kt += 2) {
      if (kt + 1 < nk) {
        if (xown) rx = *(const v4i*)(xsrc + (kt + 1) * LN_KB);
        wload(w[1], kt + 1);
      }
      compute(sX0, w[0]);
      if (kt + 1 < nk && xown) *(v4i*)(sX1 + xo) = rx;
      lds_sync();
      if (kt + 1 >= nk) break;
      if (kt + 2 < nk) {
        if (xown) rx = *(const v4i*)(xsrc + (kt + 2) * LN_KB);
        wload(w[0], kt + 2);
      }
      compute(sX1, w[1]);
      if (kt + 2 < nk && xown) *(v4i*)(sX0 + xo) = rx;
      lds_sync();
    }
  }

  // Epilogue.  Lane: channels n_i .. n_i + 3 of token t_j = 16 j + lane % 16.
  // Tokens past M read the last row and are never stored.
  int32_t nch[LN_FI];
#pragma unroll
  for (int i = 0; i < LN_FI; ++i) nch[i] = wave * (16 * LN_FI) + i * 16 + (lane >> 4) * 4;
  uint32_t rs[LN_FI][LN_FJ];
#pragma unroll
  for (int j = 0; j < LN_FJ; ++j) {
    const int64_t m = min(m0 + j * 16 + (lane & 15), M - 1);
#pragma unroll
    for (int i = 0; i < LN_FI; ++i) rs[i][j] = *(const uint32_t*)(a.resid + m * LN_N + nch[i]);
  }
  // x = Res(rq(acc), skip), 4 channels per word
  uint32_t xw[LN_FI][LN_FJ];
#pragma unroll
  for (int i = 0; i < LN_FI; ++i) {
    RqI64 rf[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rf[r] = rqc[nch[i] + r];
#pragma unroll
    for (int j = 0; j < LN_FJ; ++j) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        o[r] = rq2i8<WIDE_RES>(rf[r].apply(acc[i][j][r]), (int8_t)(rs[i][j] >> (8 * r)),
                               a.res_ma, a.res_mb, a.res_shift);
      xw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
  // row sums: in the lane (byte dot products), across the 4 lanes of a token
  // (shuffles), across the waves (LDS)
#pragma unroll
  for (int j = 0; j < (DO_LN ? LN_FJ : 0); ++j) {
    int32_t S = 0, SS = 0;
#pragma unroll
    for (int i = 0; i < LN_FI; ++i) {
      S = __builtin_amdgcn_sdot4((int32_t)xw[i][j], 0x01010101, S, false);
      SS = __builtin_amdgcn_sdot4((int32_t)xw[i][j], (int32_t)xw[i][j], SS, false);
    }
    S += __shfl_xor(S, 16, 64);
    S += __shfl_xor(S, 32, 64);
    SS += __shfl_xor(SS, 16, 64);
    SS += __shfl_xor(SS, 32, 64);
    if (lane < 16) {
      lnred[wave][j * 16 + lane][0] = S;
      lnred[wave][j * 16 + lane][1] = SS;
    }
  }
  // Both outputs leave through LDS token rows as 16-byte row chunks.  The
  // residual stream x is staged with the row sums (sbuf is free: the K loop
  // ends in a barrier); while the other waves copy it out, wave 0 turns the
  // sums into the 64 tokens' statistics (one serial Newton chain per lane:
  // computed once, not once per wave) and leaves them in LDS.
  uint32_t* so = (uint32_t*)sbuf;
  auto stage = [&](const uint32_t(&wd)[LN_FI][LN_FJ]) {
#pragma unroll
    for (int i = 0; i < LN_FI; ++i)
#pragma unroll
      for (int j = 0; j < LN_FJ; ++j) so[(j * 16 + (lane & 15)) * LN_OSTR + (nch[i] >> 2)] = wd[i][j];
  };
  auto copy_out = [&](int8_t* dst) {
    const bool a16 = ((uintptr_t)dst & 15) == 0;
    for (int c = tid; c < LN_TM * (LN_N / 16); c += 64 * LN_NW) {
      const int r = c / (LN_N / 16), q = c - r * (LN_N / 16);
      const int64_t m = m0 + r;
      if (m < M) {
        const v4i v = *(const v4i*)(so + r * LN_OSTR + q * 4);
        int8_t* p = dst + m * LN_N + q * 16;
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
    copy_out(a.y);
    return;
  }
  if (wave == 0) {
    int32_t s = 0, ss = 0;
#pragma unroll
    for (int w = 0; w < LN_NW; ++w) {
      s += lnred[w][lane][0];
      ss += lnred[w][lane][1];
    }
    const int32_t mu = mean_half_up(s, LN_N);
    const uint32_t V = (uint32_t)(ss - 2 * mu * s + LN_N * mu * mu);
    const uint32_t sigma = newton_isqrt_f64(V, a.ln_iters);
    lnst[lane][0] = mu;
    lnst[lane][1] = sigma ? (int32_t)div_2p31m1(sigma) : 0;
  }
  copy_out(a.y);
  lds_sync();  // statistics written; every read of the staged x done
  uint32_t yw[LN_FI][LN_FJ];
#pragma unroll
  for (int j = 0; j < LN_FJ; ++j) {
    const int32_t mu = lnst[j * 16 + (lane & 15)][0];
    const int32_t F = lnst[j * 16 + (lane & 15)][1];
#pragma unroll
    for (int i = 0; i < LN_FI; ++i) {
      int32_t o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t d = (int8_t)(xw[i][j] >> (8 * r)) - mu;
        o[r] = lnq[nch[i] + r].apply((d * F) >> 1);  // |d| <= sigma: |d * F| < 2^31
      }
      yw[i][j] = pack4(o[0], o[1], o[2], o[3]);
    }
  }
  stage(yw);
  lds_sync();
  copy_out(a.y2);
}

// Weight packing: blockIdx.y picks the matrix, each thread moves 16-byte
// chunks kPackChunks * 256 apart (32-bit indices: a matrix has fewer than
// 2^31 chunks, checked at launch).
constexpr int kPackChunks = 4;
__global__ __launch_bounds__(256) void pack_frags_kernel(PackList L) {
  const int j = blockIdx.y;
  const int32_t n = (int32_t)(L.start[j + 1] - L.start[j]);
  const int32_t K = L.K[j], KC = K / 64;
  const uint32_t per_group = (uint32_t)KC * kPackGroup;  // fragments per group
  const int8_t* const src0 = L.src[j];
  int8_t* const dst0 = L.dst[j];
#pragma unroll
  for (int u = 0; u < kPackChunks; ++u) {
    const int32_t local = (blockIdx.x * kPackChunks + u) * 256 + (int32_t)threadIdx.x;
    if (local >= n) break;
    const int32_t lane = local & 63;
    // fragment (n16, k64) at blk = (n16 / G) KC G + k64 G + n16 % G, G
    // fragments per group (one wave's channels)
    const uint32_t blk = (uint32_t)local >> 6;
    const uint32_t g = blk / per_group;
    const uint32_t rem = blk - g * per_group;
    const int32_t k64 = (int32_t)(rem / kPackGroup);
    const int32_t n16 = (int32_t)(g * kPackGroup + rem % kPackGroup);
    const int8_t* src = src0 + (int64_t)(n16 * 16 + (lane & 15)) * K + k64 * 64 + (lane >> 4) * 16;
    *(v4i*)(dst0 + (int64_t)local * 16) = *(const v4i*)src;
  }
}

}  // namespace

size_t packed_frag_bytes(int32_t N, int32_t K) { return (size_t)N * K; }

bool ln384_packed_kernel_applies(int64_t M, int32_t N, int32_t K) {
  return N == LN_N && K >= LN_KB && K % LN_KB == 0 && !gemm_latency_mode(M, N);
}

hipError_t launch_pack_frags(const PackList& L, hipStream_t s) {
  int64_t most = 0;
  for (int j = 0; j < L.n; ++j) most = std::max(most, L.start[j + 1] - L.start[j]);
  if (most == 0) return hipSuccess;
  if (most >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const int64_t per_block = 256 * kPackChunks;
  hipLaunchKernelGGL(pack_frags_kernel, dim3((unsigned)((most + per_block - 1) / per_block), L.n),
                     dim3(256), 0, s, L);
  return hipGetLastError();
}

template <int NW, int RING, bool DO_LN>
hipError_t launch_ln384_nw(const GemmArgs& a, int64_t tiles, hipStream_t s) {
  if (a.res_shift < 9)
    hipLaunchKernelGGL((ln384_wp_kernel<true, NW, RING, DO_LN>), dim3((unsigned)tiles),
                       dim3(64 * NW), 0, s, a, tiles);
  else
    hipLaunchKernelGGL((ln384_wp_kernel<false, NW, RING, DO_LN>), dim3((unsigned)tiles),
                       dim3(64 * NW), 0, s, a, tiles);
  return hipGetLastError();
}

hipError_t launch_ln384_packed(const GemmArgs& a, bool layernorm, hipStream_t s) {
  const int64_t tiles = (a.M + LN_TM - 1) / LN_TM;
  const bool ring3 = (a.K / LN_KB) % 3 == 0;
  if (layernorm)
    return ring3 ? launch_ln384_nw<LN_WAVES, 3, true>(a, tiles, s)
                 : launch_ln384_nw<LN_WAVES, 2, true>(a, tiles, s);
  return ring3 ? launch_ln384_nw<LN_WAVES, 3, false>(a, tiles, s)
               : launch_ln384_nw<LN_WAVES, 2, false>(a, tiles, s);
}

}  // namespace ilw
