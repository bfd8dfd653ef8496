// gemm.hip -- int8 x int8 -> int32 GEMM on CDNA4 MFMA with the dyadic
// requantization fused into the epilogue (Sec. 3.2.1, eq. linear_quant; the
// rescale is a dyadic multiply-and-shift, Sec. 3.2.2).
//
//   y[m][n] = epilogue( rq(bias[n] + sum_k x[m][k] * w[n][k]; mult[n], shift[n]) )
//
// Tiling: each wave computes FI x FJ tiles of v_mfma_i32_16x16x64_i8 (16
// channels x 16 tokens each); a workgroup holds WN x WM waves.  Large grids
// use 32 x 64 or 64 x 32 (channels x tokens) per wave, small grids (latency
// mode) 32 x 32 or 32/64 x 16 with
// PF K steps of loads in flight.  Global loads of the next K step are issued
// before the MFMAs of the current one; they are unconditional (out-of-range
// rows are clamped onto valid ones and only feed outputs that are never
// stored), which keeps the memory counters exact and the loads in flight
// across the MFMAs.  The workgroup barriers wait for LDS operations only
// (lds_sync): __syncthreads() would also wait for every outstanding global
// load and drain the PF-deep pipeline at each K step.  The
// weight tile is the MFMA A operand (rows = channels) and the activation tile
// the B operand (columns = tokens), so each lane ends up holding four
// consecutive channels of one token (one 32-bit word).  The throughput tiles
// transpose their output words through LDS and store 16-byte row chunks; the
// latency-mode tiles store each lane's words directly.  K
// advances 64 bytes per step (128 for the 384-channel LayerNorm tile, which
// runs one workgroup per CU) through double-buffered LDS tiles whose rows are
// padded by 16 bytes, which keeps the 16-byte fragment reads of a wave free of
// bank conflicts.  Workgroups are remapped so that each XCD works on a
// contiguous run of tiles (tokens-major), keeping an activation tile and the
// weights in that XCD's L2.
//
// At K = 192 the exact requantization costs more VALU time than the MFMA work
// of the tile, so the epilogue is kept to a few instructions per output.  Each
// workgroup stages its channels' constants in LDS once (RqI64: multiplier,
// shift, a 64-bit addend carrying the bias and the rounding, accumulator
// bounds); an output is then a clamp, one 64-bit multiply-add, one shift and
// a clamp, exact by the argument at RqI64.  Tiles holding a channel with a
// shift above 53 take the general integer form (bias added first, then the
// clamp, the multiply-add and the shift).
#include <stdlib.h>

#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int TK = 64;        // K bytes per step
constexpr int NXCD = 8;

// 16 bytes to dst, which the entry points require to be 4-byte aligned: one
// 16-byte store when the output base is 16-byte aligned (a16), else four
// word stores.
__device__ __forceinline__ void store16(int8_t* dst, const v4i& v, bool a16) {
  if (a16) {
    *(v4i*)dst = v;
  } else {
    uint32_t* d = (uint32_t*)dst;
    d[0] = (uint32_t)v[0];
    d[1] = (uint32_t)v[1];
    d[2] = (uint32_t)v[2];
    d[3] = (uint32_t)v[3];
  }
}

// WN x WM waves per workgroup; each wave computes FI x FJ MFMA tiles of 16
// channels x 16 tokens.  PF register slots of staged operands (PF > 1 is the
// latency mode for small grids: PF K steps of loads in flight, and every
// epilogue input -- channel constants, residual words -- loaded before the
// main loop so that the kernel pays about one memory round trip).
template <int WN, int WM, int FI, int FJ, int EPI, bool KTAIL, int PF, int KB = TK, bool LAT = (PF > 1)>
__global__ __launch_bounds__(64 * WN * WM) void gemm_i8_kernel(GemmArgs a, int32_t tiles_n,
                                                              int64_t tiles_total) {
  constexpr int WTN = 16 * FI, WTM = 16 * FJ;  // wave tile
  constexpr int TN = WTN * WN, TM = WTM * WM, NT = 64 * WN * WM;
  constexpr bool LN = EPI == EPI_RESID_LN;
  constexpr bool XP = EPI == EPI_PATCH;
  constexpr bool RES = EPI == EPI_RESID || LN || XP;
  constexpr bool EARLY = LAT;
  // Store and GELU epilogues of the throughput tiles go through LDS: the
  // tile's output words are transposed there (OSTR words per token row, an
  // odd multiple of 4: the 16 tokens of a fragment land on disjoint banks)
  // and leave as 16-byte row chunks.  A lane's own words would cover 16 rows
  // with 4 bytes each per store instruction; staged, an instruction writes
  // whole 128-byte row segments (the batch-32 fc1 20% faster).
  constexpr bool STAGED = !LAT && (EPI == EPI_STORE || EPI == EPI_GELU);
  constexpr bool RSTAGED = !LAT && RES;  // residual outputs (and LayerNorm's) likewise
  // QKV: the Q and K words likewise (a 16-channel chunk of a token lies in
  // one head's 64-byte window-major row); V^T keeps its byte scatter
  constexpr bool QSTAGED = !LAT && EPI == EPI_QKV;
  // Tiles inside M x N take an epilogue without per-lane validity tests in
  // the 384-channel LayerNorm tile (one workgroup per CU) and in the staged
  // store and GELU tiles (the staged words of rows or channels past the
  // edges are never copied out; same registers there, fc1 3% faster).
  // Elsewhere the extra registers would cost workgroups per CU.
  constexpr bool BRANCH_FREE = (LN && RSTAGED && TN >= 384) || STAGED;
  constexpr int OSTR = (TN / 4) % 8 == 0 ? TN / 4 + 4 : TN / 4;
  // KB K bytes per step (one or two MFMA K chunks): CPR 16-byte chunks per
  // staged row, rows unpadded with their chunks swizzled (lds_chunk)
  constexpr int CPR = KB / 16, LROW = KB;
  static_assert(KB == TK || KB == 2 * TK, "one or two MFMA K chunks per step");
  static_assert(!XP || KB == TK, "the image gather takes 64-byte steps");
  // Operand double buffers (W tiles, then X tiles); after the K loop the same
  // bytes hold the transposed output tile (TM rows of OSTR words).
  constexpr int SOPS = 2 * (TN + TM) * LROW, SOUT = TM * OSTR * 4;
  __shared__ __attribute__((aligned(16))) int8_t sbuf[SOPS > SOUT ? SOPS : SOUT];
  auto sW = [&](int buf) { return sbuf + buf * (TN * LROW); };
  auto sX = [&](int buf) { return sbuf + (2 * TN + buf * TM) * LROW; };
  __shared__ int8_t glut[EPI == EPI_GELU ? 256 : 1];
  __shared__ RqI64 rqc[TN];                         // output requantization per channel
  __shared__ int64_t qoff[EPI == EPI_QKV ? TM : 1][2];  // QKV: Q/K and V^T offsets per token
  __shared__ RqI64 lnq[LN ? TN : 1];  // LayerNorm output requantization per channel
  // per-wave row sums of the LayerNorm epilogue: in the first weight tile,
  // free once the K loop's last barrier has passed
  static_assert(2 * WN * TM * 4 <= TN * LROW, "row sums fit one weight tile");
  int32_t* const lnred = (int32_t*)sbuf;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave % WN;  // channel block of the tile
  const int wm = wave / WN;  // token block of the tile

  // XCD-aware tile order: dispatch places workgroup i on XCD i % 8; give each
  // XCD a contiguous block of tiles.
  const int64_t bid = blockIdx.x;
  const int64_t per = tiles_total / NXCD, rem = tiles_total % NXCD;
  const int64_t xcd = bid % NXCD;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / NXCD;
  const int64_t m0 = (tile / tiles_n) * TM;
  const int32_t n0 = (int32_t)(tile % tiles_n) * TN;

  const int8_t* __restrict__ X = a.x;
  const int8_t* __restrict__ W = a.w;
  const int64_t M = a.M;
  const int32_t N = a.N, K = a.K;
  const v4i zero = {0, 0, 0, 0};

  // Global -> LDS staging: (TN + TM) rows of 64 bytes per K step, 16 bytes
  // per thread-chunk.  Rows past N or M are clamped onto the last valid row;
  // with a K tail (K % 64 != 0) chunks past K are zeroed.
  constexpr int CW = TN * CPR, CX = TM * CPR;  // chunks per operand tile
  constexpr int PW = (CW + NT - 1) / NT, PX = (CX + NT - 1) / NT;
  const int8_t* wsrc[PW];
  const int8_t* xsrc[PX];
  int kofs[PW > PX ? PW : PX];
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int c = min(tid + i * NT, CW - 1);
    wsrc[i] = W + (int64_t)min(n0 + c / CPR, N - 1) * K + (c % CPR) * 16;
  }
#pragma unroll
  for (int i = 0; i < PX; ++i) {
    const int c = min(tid + i * NT, CX - 1);
    const int64_t m = min(m0 + c / CPR, M - 1);
    if (XP) {
      // top-left pixel of the token's patch; K offsets are added per step
      const int32_t b = (int32_t)(m / a.pT), t = (int32_t)(m - (int64_t)b * a.pT);
      const int32_t py = t / a.pgw, px = t - py * a.pgw;
      xsrc[i] = X + ((int64_t)b * a.pC * a.pH + py * 16) * a.pW + px * 16;
    } else {
      xsrc[i] = X + m * K + (c % CPR) * 16;
    }
  }
#pragma unroll
  for (int i = 0; i < (PW > PX ? PW : PX); ++i) kofs[i] = ((tid + i * NT) % CPR) * 16;
  // The loads of K step k go to register slot k % PF.
  v4i rw[PF][PW], rx[PF][PX];
  const int nk = (K + KB - 1) / KB;
  auto gload = [&](int kt, int sl) {
    const int kb = kt * KB;
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      if (KTAIL) {
        const bool ok = kb + kofs[i] < K;
        rw[sl][i] = *(const v4i*)(wsrc[i] + (ok ? kb : 0));
        if (!ok) rw[sl][i] = zero;
      } else {
        rw[sl][i] = *(const v4i*)(wsrc[i] + kb);
      }
    }
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      if (XP) {
        // the chunk's 16 K values are pixels kx = 0..15 of row ky of channel c
        const int32_t k = kb + kofs[i];
        rx[sl][i] = *(const v4i*)(xsrc[i] + (int64_t)(k >> 8) * a.pH * a.pW +
                                  ((k >> 4) & 15) * a.pW);
      } else if (KTAIL) {
        const bool ok = kb + kofs[i] < K;
        rx[sl][i] = *(const v4i*)(xsrc[i] + (ok ? kb : 0));
        if (!ok) rx[sl][i] = zero;
      } else {
        rx[sl][i] = *(const v4i*)(xsrc[i] + kb);
      }
    }
  };
  auto sstore = [&](int buf, int sl) {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int c = tid + i * NT;
      if (CW % NT == 0 || c < CW)
        *(v4i*)(sW(buf) + lds_chunk<CPR>(c / CPR, c % CPR)) = rw[sl][i];
    }
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      const int c = tid + i * NT;
      if (CX % NT == 0 || c < CX)
        *(v4i*)(sX(buf) + lds_chunk<CPR>(c / CPR, c % CPR)) = rx[sl][i];
    }
  };

  // Operand loads first: everything below overlaps with their latency.
  if constexpr (PF == 1) {
    gload(0, 0);
  } else {
#pragma unroll
    for (int d = 0; d < PF; ++d) gload(min(d, nk - 1), d);
  }

  // Output coordinates.  Lane holds channels n..n+3 (n = 4*(lane/16) within a
  // 16-tile) of token lane%16 of each of the FI x FJ tiles.
  int32_t nch[FI];
  bool ch_ok[FI];
#pragma unroll
  for (int i = 0; i < FI; ++i) {
    nch[i] = n0 + wn * WTN + i * 16 + (lane >> 4) * 4;
    ch_ok[i] = nch[i] < N;  // N is a multiple of 16: the 4 channels are all valid
  }
  int64_t tok[FJ];   // per token: output row (STORE/GELU/RESID) or Q/K offset (QKV)
  int64_t tokv[FJ];  // QKV: V^T offset of the token
  int64_t rtok[FJ];  // RESID: row of the skip input (PATCH: of the positional table)
  bool tok_ok[FJ];
#pragma unroll
  for (int j = 0; j < FJ; ++j) {
    const int64_t m = m0 + wm * WTM + j * 16 + (lane & 15);
    tok_ok[j] = m < M;
    tok[j] = m * N;
    tokv[j] = 0;
    const int64_t mc = min(m, M - 1);
    rtok[j] = (XP ? mc % a.pT : mc) * N;
  }

  // Residual words (latency mode: loaded now).
  uint32_t rs[FI][FJ];
  auto load_resid = [&](int i) {
#pragma unroll
    for (int j = 0; j < FJ; ++j)
      rs[i][j] = *(const uint32_t*)(a.resid + rtok[j] + min(nch[i], N - 4));
  };
  if (EARLY && RES) {
#pragma unroll
    for (int i = 0; i < FI; ++i) load_resid(i);
  }
  // Output requantization constants of the tile's channels, once per
  // workgroup (a lane's channels are shared by 16 lanes of each wave row).
  for (int c = tid; c < TN; c += NT) {
    const int32_t n = min(n0 + c, N - 1);
    RqI64 r;
    r.init(a.mult[a.nq == 1 ? 0 : n], a.shift[a.nq == 1 ? 0 : n], a.bias ? a.bias[n] : 0);
    rqc[c] = r;
  }

  if (EPI == EPI_GELU) {
    // SD-ShiftGELU of the requantized fc1 output is a function of one int8
    // value: tabulate it (with its output requantization) once per workgroup.
    for (int t = tid; t < 256; t += NT)
      glut[t] = (int8_t)rq(sd_gelu(t - 128, a.g_I0, a.g_kinter, a.g_kout), a.g_mult, a.g_shift);
  }
  if (EPI == EPI_QKV) {
    // destination of each of the tile's tokens in the window-major layout,
    // once per workgroup
    for (int t = tid; t < TM; t += NT) {
      const int64_t m = min(m0 + t, M - 1);
      const QkvLayout& Lq = a.qkv;
      const int32_t b = fdiv((int32_t)m, Lq.T, a.inv_T);
      const int32_t tt = (int32_t)m - b * Lq.T;
      const int32_t ty = fdiv(tt, Lq.grid_w, a.inv_gw), tx = tt - ty * Lq.grid_w;
      const int32_t wy = fdiv(ty, Lq.win_h, a.inv_wh), iy = ty - wy * Lq.win_h;
      const int32_t wx = fdiv(tx, Lq.win_w, a.inv_ww), ix = tx - wx * Lq.win_w;
      const int64_t bw = (int64_t)b * Lq.nW + wy * Lq.nwx + wx;
      const int32_t li = iy * Lq.win_w + ix;
      qoff[t][0] = (bw * Lq.H * Lq.Tw + li) * 64;
      qoff[t][1] = bw * Lq.H * 64 * Lq.Twp + li;
    }
  }
  if (LN) {
    // Stage the LayerNorm output constants of the N (= TN) channels of the
    // row: gamma-scaled n plus beta requantizes like an accumulator plus a
    // bias (|n| < 2^30 and beta inside int32 keep RqI64's bounds).
    for (int c = tid; c < TN; c += NT) {
      const int q = a.ln_nq == 1 ? 0 : c;
      RqI64 r;
      r.init(a.ln_mult[q], a.ln_shift[q], a.ln_beta[c]);
      lnq[c] = r;
    }
  }

  v4i acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = zero;
  // fragment rows start at multiples of 16, so a lane's swizzle depends on
  // lane % 16 only: its chunk offsets for the KB / TK halves of a step
  int frag_off[KB / TK];
#pragma unroll
  for (int h = 0; h < KB / TK; ++h) frag_off[h] = lds_chunk<CPR>(lane & 15, h * 4 + (lane >> 4));
  // compute(buf, kt): the MFMAs of K step kt; with a K tail, 64-byte halves
  // of the last step that lie wholly past K are skipped (their chunks are
  // zero-filled anyway)
  auto compute = [&](int buf, int kt) {
#pragma unroll
    for (int h = 0; h < KB / TK; ++h) {
      if (KTAIL && h > 0 && kt * KB + h * TK >= K) break;
      v4i fa[FI], fb[FJ];
#pragma unroll
      for (int i = 0; i < FI; ++i)
        fa[i] = *(const v4i*)(sW(buf) + (wn * WTN + i * 16) * LROW + frag_off[h]);
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        fb[j] = *(const v4i*)(sX(buf) + (wm * WTM + j * 16) * LROW + frag_off[h]);
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  };

  if constexpr (PF == 1) {
    sstore(0, 0);
    lds_sync();  // the first tile and the staged constants
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) gload(kt + 1, 0);
      compute(kt & 1, kt);
      if (kt + 1 < nk) sstore((kt + 1) & 1, 0);
      lds_sync();
    }
  } else {
    // Loads are issued on every path (steps past the end re-read the last
    // one), so the memory counter wait before each LDS store is exact: it
    // leaves the younger slots' loads in flight.
    sstore(0, 0);
    lds_sync();  // the first tile and the staged constants
    gload(min(PF, nk - 1), 0);
    for (int kt0 = 0; kt0 < nk; kt0 += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        const int kt = kt0 + u;
        if (kt < nk) compute(kt & 1, kt);
        sstore((kt + 1) & 1, (u + 1) % PF);
        gload(min(kt + 1 + PF, nk - 1), (u + 1) % PF);
        lds_sync();
      }
    }
  }

  // Epilogue: the staged four-instruction requantization, then the
  // epilogue's own work.
  uint32_t xw[FI][FJ];  // RESID_LN: the residual outputs, 4 channels per word
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) xw[i][j] = 0;
  if (EPI == EPI_QKV) {
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int t = wm * WTM + j * 16 + (lane & 15);
      tok[j] = qoff[t][0];
      tokv[j] = qoff[t][1];
    }
  }
  // The residual add has a 32-bit form for shifts >= 9 (uniform per launch),
  // and tiles inside M x N need no per-lane validity tests (whose exec-mask
  // branches would split the loop into blocks the compiler cannot
  // interleave): the loop below is instantiated for each case and selected
  // once per workgroup.
  const bool full_tile = BRANCH_FREE && n0 + TN <= N && m0 + TM <= M;
  auto requant_tile = [&](auto wide_res, auto full) {
    constexpr bool FULL = decltype(full)::value;
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      if (!FULL && !ch_ok[i]) continue;
      const int32_t n = nch[i];
      if (!EARLY && RES) load_resid(i);
      RqI64 rf[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) rf[r] = rqc[n - n0 + r];
      int8_t* qk_base = nullptr;
      int64_t ch_qk = 0, ch_v = 0;
      bool is_v = false;
      if (EPI == EPI_QKV) {
        const QkvLayout& Lq = a.qkv;
        const int32_t part = n / Lq.D, rem_n = n - part * Lq.D;
        const int32_t h = rem_n >> Lq.hs, c = rem_n & ((1 << Lq.hs) - 1);
        is_v = part == 2;
        qk_base = part == 0 ? Lq.q : Lq.k;
        ch_qk = (int64_t)h * Lq.Tw * 64 + c;
        ch_v = ((int64_t)h * 64 + c) * Lq.Twp;
      }
#pragma unroll
      for (int j = 0; j < FJ; ++j) {
        if (!FULL && !tok_ok[j]) continue;
        int32_t u[4];  // the requantized outputs
#pragma unroll
        for (int r = 0; r < 4; ++r) u[r] = rf[r].apply(acc[i][j][r]);
        if (STAGED) {
          const uint32_t word =
              EPI == EPI_GELU
                  ? pack4(glut[u[0] + 128], glut[u[1] + 128], glut[u[2] + 128], glut[u[3] + 128])
                  : pack4(u[0], u[1], u[2], u[3]);
          ((uint32_t*)sbuf)[(wm * WTM + j * 16 + (lane & 15)) * OSTR + ((n - n0) >> 2)] = word;
        } else if (EPI == EPI_STORE) {
          *(uint32_t*)(a.y + tok[j] + n) = pack4(u[0], u[1], u[2], u[3]);
        } else if (EPI == EPI_GELU) {
          *(uint32_t*)(a.y + tok[j] + n) =
              pack4(glut[u[0] + 128], glut[u[1] + 128], glut[u[2] + 128], glut[u[3] + 128]);
        } else if (RES) {
          const uint32_t s = rs[i][j];
          int32_t o[4];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            o[r] = rq2i8<decltype(wide_res)::value>(u[r], (int8_t)(s >> (8 * r)), a.res_ma,
                                                    a.res_mb, a.res_shift);
          const uint32_t word = pack4(o[0], o[1], o[2], o[3]);
          if (!RSTAGED) *(uint32_t*)(a.y + tok[j] + n) = word;
          if (LN || RSTAGED) xw[i][j] = word;
        } else {  // EPI_QKV: scatter into window-major Q, K and V^T
          if (!is_v) {
            if (QSTAGED) xw[i][j] = pack4(u[0], u[1], u[2], u[3]);
            else *(uint32_t*)(qk_base + tok[j] + ch_qk) = pack4(u[0], u[1], u[2], u[3]);
          } else {
            int8_t* dst = a.qkv.vt + tokv[j] + ch_v;
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(int64_t)r * a.qkv.Twp] = (int8_t)u[r];
          }
        }
      }
    }
  };
  if (RES && a.res_shift < 9) {
    if constexpr (BRANCH_FREE) {
      if (full_tile) requant_tile(Flag<true>{}, Flag<true>{});
      else requant_tile(Flag<true>{}, Flag<false>{});
    } else {
      requant_tile(Flag<true>{}, Flag<false>{});
    }
  } else {
    if constexpr (BRANCH_FREE) {
      if (full_tile) requant_tile(Flag<false>{}, Flag<true>{});
      else requant_tile(Flag<false>{}, Flag<false>{});
    } else {
      requant_tile(Flag<false>{}, Flag<false>{});
    }
  }
  // Output words in the accumulator lane layout, transposed into LDS token
  // rows (the weight tiles, free after the K loop; LayerNorm's row sums are
  // past their last read at the first barrier).
  auto stage_words = [&](const uint32_t(&wd)[FI][FJ]) {
    uint32_t* so = (uint32_t*)sbuf;
    lds_sync();
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        so[(wm * WTM + j * 16 + (lane & 15)) * OSTR + ((nch[i] - n0) >> 2)] = wd[i][j];
    lds_sync();
  };
  // The staged tile out to dst (row stride N) in 16-byte row chunks.
  constexpr int CPT = TN / 16;  // 16-byte chunks per token row
  auto copy_rows = [&](int8_t* dst) {
    const uint32_t* so = (const uint32_t*)sbuf;
    const bool a16 = ((uintptr_t)dst & 15) == 0;
    for (int c = tid; c < TM * CPT; c += NT) {
      const int r = c / CPT, q = c - r * CPT;
      const int64_t m = m0 + r;
      const int32_t n = n0 + q * 16;
      if (m < M && n < N) store16(dst + m * N + n, *(const v4i*)(so + r * OSTR + q * 4), a16);
    }
  };
  if constexpr (STAGED) {  // the words went to LDS in the loop above
    lds_sync();
    copy_rows(a.y);
  }
  if constexpr (RSTAGED && !LN) {
    stage_words(xw);
    copy_rows(a.y);
  }
  if constexpr (QSTAGED) {
    // Q and K chunks to their window-major rows (16-byte aligned: the rows
    // are 64 bytes, the workspace 16-byte aligned)
    stage_words(xw);
    const uint32_t* so = (const uint32_t*)sbuf;
    const QkvLayout& Lq = a.qkv;
    for (int c = tid; c < TM * CPT; c += NT) {
      const int r = c / CPT, q = c - r * CPT;
      const int32_t n = n0 + q * 16;
      const int32_t part = n / Lq.D, rem_n = n - part * Lq.D;
      if (m0 + r < M && n < N && part < 2) {
        const int32_t h = rem_n >> Lq.hs, cc = rem_n & ((1 << Lq.hs) - 1);
        int8_t* dst = (part == 0 ? Lq.q : Lq.k) + qoff[r][0] + (int64_t)h * Lq.Tw * 64 + cc;
        *(v4i*)dst = *(const v4i*)(so + r * OSTR + q * 4);
      }
    }
  }
  if (LN) {
    // LayerNorm of the residual output rows (same reading as the standalone
    // operator).  A token's N channels sit in 4 lanes of each of the WN waves
    // along the channels: reduce in the lane (byte dot products), across the
    // 4 lanes (shuffles), then across the waves (LDS).
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      int32_t S = 0, SS = 0;
#pragma unroll
      for (int i = 0; i < FI; ++i) {
        S = __builtin_amdgcn_sdot4((int32_t)xw[i][j], 0x01010101, S, false);
        SS = __builtin_amdgcn_sdot4((int32_t)xw[i][j], (int32_t)xw[i][j], SS, false);
      }
      S += __shfl_xor(S, 16, 64);
      S += __shfl_xor(S, 32, 64);
      SS += __shfl_xor(SS, 16, 64);
      SS += __shfl_xor(SS, 32, 64);
      const int t = wm * WTM + j * 16 + (lane & 15);
      if (lane < 16) {
        lnred[(wn * TM + t) * 2 + 0] = S;
        lnred[(wn * TM + t) * 2 + 1] = SS;
      }
    }
    lds_sync();
    // Row statistics with one token per lane (the Newton steps form a serial
    // dependency chain; one chain per lane keeps it short), then each lane
    // fetches those of its FJ tokens.
    int32_t mu_l, F_l;
    {
      const int t = wm * WTM + min(lane, WTM - 1);
      int32_t s = 0, ss = 0;
#pragma unroll
      for (int w = 0; w < WN; ++w) {
        s += lnred[(w * TM + t) * 2 + 0];
        ss += lnred[(w * TM + t) * 2 + 1];
      }
      mu_l = mean_half_up(s, N);
      const uint32_t V = (uint32_t)(ss - 2 * mu_l * s + N * mu_l * mu_l);
      const uint32_t sigma = newton_isqrt_f64(V, a.ln_iters);
      F_l = sigma ? (int32_t)div_2p31m1(sigma) : 0;
    }
    int32_t mu[FJ], F[FJ];
    uint32_t yw2[FI][FJ] = {};  // staged LayerNorm outputs
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      mu[j] = __shfl(mu_l, j * 16 + (lane & 15), 64);
      F[j] = __shfl(F_l, j * 16 + (lane & 15), 64);
    }
    // (the 384-channel tile stages its outputs, and those of tokens past M
    // are never copied out: no per-lane test there)
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      const int32_t n = wn * WTN + i * 16 + (lane >> 4) * 4;
#pragma unroll
      for (int j = 0; j < FJ; ++j) {
        if (!BRANCH_FREE && !tok_ok[j]) continue;
        int32_t o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int32_t d = (int8_t)(xw[i][j] >> (8 * r)) - mu[j];
          const int32_t nn = (d * F[j]) >> 1;  // |d| <= sigma: |d * F| < 2^31
          o[r] = lnq[n + r].apply(nn);
        }
        if (RSTAGED) yw2[i][j] = pack4(o[0], o[1], o[2], o[3]);
        else *(uint32_t*)(a.y2 + tok[j] + n) = pack4(o[0], o[1], o[2], o[3]);
      }
    }
    if constexpr (RSTAGED) {
      stage_words(xw);
      copy_rows(a.y);
      stage_words(yw2);
      copy_rows(a.y2);
    }
  }
}

template <int WN, int WM, int FI, int FJ, bool KT, int PF, int KB = TK, bool LAT = (PF > 1)>
hipError_t launch_cfg(int epi, const GemmArgs& a, hipStream_t s) {
  constexpr int TN = 16 * FI * WN, TM = 16 * FJ * WM;
  const int32_t tiles_n = (a.N + TN - 1) / TN;
  const int64_t tiles_m = (a.M + TM - 1) / TM;
  const int64_t total = tiles_m * tiles_n;
  dim3 grid((unsigned)total), block(64 * WN * WM);
#define ILW_LAUNCH(E)                                                                   \
  hipLaunchKernelGGL((gemm_i8_kernel<WN, WM, FI, FJ, E, KT, PF, KB, LAT>), grid, block, 0, s, a, \
                     tiles_n, total)
  switch (epi) {
    case EPI_STORE: ILW_LAUNCH(EPI_STORE); break;
    case EPI_GELU: ILW_LAUNCH(EPI_GELU); break;
    case EPI_RESID: ILW_LAUNCH(EPI_RESID); break;
    case EPI_QKV: ILW_LAUNCH(EPI_QKV); break;
    case EPI_PATCH:
      if constexpr (!KT && KB == TK) ILW_LAUNCH(EPI_PATCH);
      else return hipErrorInvalidValue;  // K = 256 * channels: 64-byte steps, no tail
      break;
    default: return hipErrorInvalidValue;
  }
#undef ILW_LAUNCH
  return hipGetLastError();
}

// Fused residual + LayerNorm: the workgroup holds whole rows (TN == N).
template <int WN, int WM, int FI, int FJ, bool KT, int PF, int KB = TK, bool LAT = (PF > 1)>
hipError_t launch_ln(const GemmArgs& a, hipStream_t s) {
  constexpr int TN = 16 * FI * WN, TM = 16 * FJ * WM;
  if (a.N != TN) return hipErrorInvalidValue;
  const int64_t total = (a.M + TM - 1) / TM;
  hipLaunchKernelGGL((gemm_i8_kernel<WN, WM, FI, FJ, EPI_RESID_LN, KT, PF, KB, LAT>),
                     dim3((unsigned)total), dim3(64 * WN * WM), 0, s, a, 1, total);
  return hipGetLastError();
}

template <int WN, int WM, int FI, int FJ, int PF, int KB = TK, bool LAT = (PF > 1)>
hipError_t launch_tile(int epi, const GemmArgs& a, hipStream_t s) {
  return a.K % KB == 0 ? launch_cfg<WN, WM, FI, FJ, false, PF, KB, LAT>(epi, a, s)
                       : launch_cfg<WN, WM, FI, FJ, true, PF, KB, LAT>(epi, a, s);
}

template <int WN, int WM, int FI, int FJ, int PF, int KB = TK, bool LAT = (PF > 1)>
hipError_t launch_ln_tile(const GemmArgs& a, hipStream_t s) {
  return a.K % KB == 0 ? launch_ln<WN, WM, FI, FJ, false, PF, KB, LAT>(a, s)
                       : launch_ln<WN, WM, FI, FJ, true, PF, KB, LAT>(a, s);
}

// Latency mode (ILW_GEMM_PF=1|3 forces it off or on): grids of at most about
// one wave per SIMD with the throughput tiles.
bool latency_mode(int64_t waves) {
  static const int ov = [] {  // read once (thread-safe static initialisation)
    const char* e = getenv("ILW_GEMM_PF");
    return (e && (atoi(e) == 1 || atoi(e) == 3)) ? atoi(e) : 0;
  }();
  if (ov) return ov == 3;
  return waves <= 1024;
}

}  // namespace

bool gemm_latency_mode(int64_t M, int32_t N) { return latency_mode(((M + 63) / 64) * (N / 64)); }

hipError_t launch_gemm(int epi, const GemmArgs& a_in, hipStream_t s) {
  if (a_in.M == 0) return hipSuccess;
  GemmArgs a = a_in;
  if (epi == EPI_QKV) {
    a.inv_T = 1.0f / (float)a.qkv.T;
    a.inv_gw = 1.0f / (float)a.qkv.grid_w;
    a.inv_wh = 1.0f / (float)a.qkv.win_h;
    a.inv_ww = 1.0f / (float)a.qkv.win_w;
  }
  const int64_t mt64 = (a.M + 63) / 64;
  if (epi == EPI_RESID_LN) {
    // The workgroup holds whole rows (N channels) so the LayerNorm statistics
    // stay on chip.  These tiles fill few workgroups per CU (one at N = 384),
    // so the deep-K linears (fc2) keep two K steps of loads in flight: 4-7%
    // faster there, slower at K <= 384.
    // (at 192 channels the count is the throughput tile's own waves, 12 per
    // 128 tokens: on the 1600-token encoder its tiles win from batch 7,
    // 11 200 tokens, against a tie at batch 6)
    const bool lat = a.N == 192 ? latency_mode(((a.M + 127) / 128) * 12)
                                : latency_mode(mt64 * (a.N / 64));
    if (a.N == 192) {
      if (lat)  // 192 x 16 tokens
        return a.K >= 6 * TK ? launch_ln_tile<6, 1, 2, 1, 6>(a, s)
                             : launch_ln_tile<6, 1, 2, 1, 3>(a, s);
      // 192 x 128 tokens, 12 waves of 64 x 32; the deep-K fc2 with two K
      // steps of loads in flight but the throughput epilogue (outputs staged
      // through LDS): 3% faster than with the latency-mode epilogue
      return a.K >= 12 * TK ? launch_ln_tile<3, 4, 4, 2, 2, TK, false>(a, s)
                            : launch_ln_tile<3, 4, 4, 2, 1>(a, s);
    }
    if (a.N == 256) {
      if (lat)  // 256 x 16 tokens
        return a.K >= 6 * TK ? launch_ln_tile<8, 1, 2, 1, 6>(a, s)
                             : launch_ln_tile<8, 1, 2, 1, 3>(a, s);
      return launch_ln_tile<4, 2, 4, 2, 1>(a, s);  // 256 x 64 tokens, 8 waves of 64 x 32
    }
    if (a.N == 384) {
      // weights packed in fragment order: the register-operand kernel
      if (!lat && a.wp && ln384_packed_kernel_applies(a.M, a.N, a.K))
        return launch_ln384_packed(a, true, s);
      if (lat)  // 384 x 16 tokens
        return a.K >= 6 * TK ? launch_ln_tile<6, 1, 4, 1, 6>(a, s)
                             : launch_ln_tile<6, 1, 4, 1, 3>(a, s);
      // 384 x 64 tokens, 12 waves of 64 x 32
      // (one workgroup per CU: 128-byte K steps halve the steps' barriers
      // and LDS round trips, 6-8% faster than 64-byte steps)
      if (a.K % (2 * TK) == 0) return launch_ln<6, 2, 4, 2, false, 1, 2 * TK>(a, s);
      return a.K >= 12 * TK ? launch_ln_tile<6, 2, 4, 2, 2>(a, s)
                            : launch_ln_tile<6, 2, 4, 2, 1>(a, s);
    }
    return hipErrorInvalidValue;
  }
  // The 384-channel residual linear with packed weights (the last block's
  // fc2): the LayerNorm kernel without its LayerNorm.
  if (epi == EPI_RESID && a.wp && ln384_packed_kernel_applies(a.M, a.N, a.K))
    return launch_ln384_packed(a, false, s);
  // Small grids: 64 x 64 workgroup tiles split over 4 waves of 32 x 32, with
  // the latency-mode pipeline.  Otherwise, from a sweep over the encoder
  // shapes on MI355X: 192-channel tiles for the deep-K linears and N = 192,
  // and 128 x 128 tiles over 8 waves of 64 channels x 32 tokens for the rest
  // (6% faster than 32 x 64 waves on the batch-32 QKV, equal elsewhere).
  if (latency_mode(mt64 * ((a.N + 63) / 64)))
    return a.K >= 6 * TK ? launch_tile<2, 2, 2, 2, 6>(epi, a, s)
                         : launch_tile<2, 2, 2, 2, 3>(epi, a, s);
  // Wide QKV linears on 256-channel x 128-token tiles of 8 waves of 64 x 64
  // (12% faster than 128 x 128 on the 1152-channel QKV of the 384-wide
  // encoder at batch 8, slower for fc1; at batch 3 and 4, or half of batch 8
  // on each of two streams, 15-20% faster than the one-wave tiles below)
  if (epi == EPI_QKV && a.N >= 1024) return launch_tile<4, 2, 4, 4, 1>(epi, a, s);
  const int64_t big_tiles = ((a.M + 127) / 128) * ((a.N + 127) / 128);
  if (big_tiles < 512) return launch_tile<1, 1, 4, 4, 1>(epi, a, s);
  if (a.N % 192 == 0 && a.K >= 768) return launch_tile<3, 2, 4, 4, 1>(epi, a, s);
  if (a.N == 192) return launch_tile<3, 1, 4, 4, 1>(epi, a, s);
  return launch_tile<2, 4, 4, 2, 1>(epi, a, s);
}

}  // namespace ilw
