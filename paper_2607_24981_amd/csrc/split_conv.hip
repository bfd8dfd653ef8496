// split_conv.hip -- scale-preserving split convolution of the projector
// (Sec. 3.2.2, Fig. projector_split_conv), pointwise:
//
//   acc_b = x_b W_b^T                       (int8 MFMA, int32, per branch)
//   r_b   = floor((acc_b m_b + 2^(s_b-1)) / 2^s_b)   (rescale to the common scale)
//   y     = sat8(rq(bias + sum_b r_b; out))
//
// Each branch is one encoder feature map with its own activation scale; its
// int32 partial is rescaled to the common scale (the largest branch scale)
// before the integer accumulation.  The K loop runs over the branches in
// turn (64 channels per step): at the last step of a branch the accumulators
// are rescaled into an int64 running sum and cleared.  Tiling as in the GEMM:
// weights are the MFMA A operand (a lane ends with 4 consecutive channels of
// one token), double-buffered LDS tiles with 80-byte rows, unconditional
// loads with clamped rows, and PF (two) K steps of loads in flight.  The
// loads walk the branches with a wave-uniform cursor whose pointers and row
// offsets change only at branch boundaries, and the fold is triggered by a
// step count, so a K step issues no scalar loads.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int TK = 64, LDS_ROW = 64, NXCD = 8;  // 64-byte rows, chunks swizzled (lds_chunk)

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

struct BrChan {
  int32_t mult, shift;
};

template <int WN, int WM, int FI, int FJ, int PF>
__global__ __launch_bounds__(64 * WN * WM) void split_conv_kernel(SplitArgs a, int32_t tiles_n,
                                                                 int64_t tiles_total) {
  constexpr int WTN = 16 * FI, WTM = 16 * FJ;
  constexpr int TN = WTN * WN, TM = WTM * WM, NT = 64 * WN * WM;
  // output staging: OSTR words per token row, an odd multiple of 4
  constexpr int OSTR = (TN / 4) % 8 == 0 ? TN / 4 + 4 : TN / 4;
  // operand double buffers (W tiles, then X tiles); after the K loop the
  // same bytes hold the transposed output tile
  constexpr int SOPS = 2 * (TN + TM) * LDS_ROW, SOUT = TM * OSTR * 4;
  __shared__ __attribute__((aligned(16))) int8_t sbuf[SOPS > SOUT ? SOPS : SOUT];
  auto sW = [&](int buf) { return sbuf + buf * (TN * LDS_ROW); };
  auto sX = [&](int buf) { return sbuf + (2 * TN + buf * TM) * LDS_ROW; };
  __shared__ BrChan brc[kMaxBranches][TN];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave % WN, wm = wave / WN;
  const int64_t bid = blockIdx.x;
  const int64_t per = tiles_total / NXCD, rem = tiles_total % NXCD;
  const int64_t xcd = bid % NXCD;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / NXCD;
  const int64_t m0 = (tile / tiles_n) * TM;
  const int32_t n0 = (int32_t)(tile % tiles_n) * TN;
  const int64_t M = a.M;
  const int32_t N = a.N, nbr = a.nbr, S = a.kstart[a.nbr];
  const v4i zero = {0, 0, 0, 0};

  // staging chunks: (TN + TM) rows of 64 bytes per K step, 16 bytes per chunk
  constexpr int CW = TN * 4, CX = TM * 4;
  constexpr int PW = (CW + NT - 1) / NT, PX = (CX + NT - 1) / NT;
  int wrow[PW];
  int64_t xrow[PX];
  int cofs[PW > PX ? PW : PX];
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int c = min(tid + i * NT, CW - 1);
    wrow[i] = min(n0 + (c >> 2), N - 1);
  }
#pragma unroll
  for (int i = 0; i < PX; ++i) {
    const int c = min(tid + i * NT, CX - 1);
    xrow[i] = min(m0 + (c >> 2), M - 1);
  }
#pragma unroll
  for (int i = 0; i < (PW > PX ? PW : PX); ++i) cofs[i] = ((tid + i * NT) & 3) * 16;

  v4i rw[PF][PW], rx[PF][PX];
  // Loads go step by step through the branches: a wave-uniform cursor (the
  // branch lb and the byte offset lk in its rows) whose branch pointers and
  // per-lane row offsets change only at branch boundaries.  Once every step
  // has been loaded the cursor stays on the last one (re-read, never used).
  int lb = 0, lsteps = 0;
  int32_t lk = 0, LC = a.C[0];
  const int8_t* LW = a.w[0];
  const int8_t* LX = a.x[0];
  int64_t wo[PW], xo[PX];  // row * C + chunk offset, for the cursor's branch
  auto set_rows = [&]() {
#pragma unroll
    for (int i = 0; i < PW; ++i) wo[i] = (int64_t)wrow[i] * LC + cofs[i];
#pragma unroll
    for (int i = 0; i < PX; ++i) xo[i] = xrow[i] * LC + cofs[i];
  };
  set_rows();
  auto gload = [&](int sl) {
#pragma unroll
    for (int i = 0; i < PW; ++i) rw[sl][i] = *(const v4i*)(LW + wo[i] + lk);
#pragma unroll
    for (int i = 0; i < PX; ++i) rx[sl][i] = *(const v4i*)(LX + xo[i] + lk);
    if (++lsteps < S) {
      lk += TK;
      if (lk == LC) {
        ++lb;
        lk = 0;
        LW = a.w[lb];
        LX = a.x[lb];
        LC = a.C[lb];
        set_rows();
      }
    }
  };
  auto sstore = [&](int buf, int sl) {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int c = tid + i * NT;
      if (CW % NT == 0 || c < CW)
        *(v4i*)(sW(buf) + lds_chunk<4>(c >> 2, c & 3)) = rw[sl][i];
    }
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      const int c = tid + i * NT;
      if (CX % NT == 0 || c < CX)
        *(v4i*)(sX(buf) + lds_chunk<4>(c >> 2, c & 3)) = rx[sl][i];
    }
  };

  // Operand loads first; then the branch rescale constants of the tile's
  // channels into LDS.
#pragma unroll
  for (int d = 0; d < PF; ++d) gload(d);
  for (int e = tid; e < nbr * TN; e += NT) {
    const int b = e / TN, c = e % TN;
    const int32_t n = min(n0 + c, N - 1);
    const int32_t q = a.bnq[b] == 1 ? 0 : n;
    brc[b][c] = {a.bmult[b][q], a.bshift[b][q]};
  }

  v4i acc[FI][FJ];
  int64_t tot[FI][FJ][4];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      acc[i][j] = zero;
#pragma unroll
      for (int r = 0; r < 4; ++r) tot[i][j][r] = 0;
    }
  const int frag_off = lds_chunk<4>(lane & 15, lane >> 4);  // rows start at multiples of 16
  auto compute = [&](int buf) {
    v4i fa[FI], fb[FJ];
#pragma unroll
    for (int i = 0; i < FI; ++i)
      fa[i] = *(const v4i*)(sW(buf) + (wn * WTN + i * 16) * LDS_ROW + frag_off);
#pragma unroll
    for (int j = 0; j < FJ; ++j)
      fb[j] = *(const v4i*)(sX(buf) + (wm * WTM + j * 16) * LDS_ROW + frag_off);
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  // rescale the finished branch b's partials into the running sums
  auto fold = [&](int b) {
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      const int c = wn * WTN + i * 16 + (lane >> 4) * 4;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const BrChan p = brc[b][c + r];
        const int64_t rnd = (int64_t)1 << (p.shift - 1);
#pragma unroll
        for (int j = 0; j < FJ; ++j)
          tot[i][j][r] += ((int64_t)acc[i][j][r] * p.mult + rnd) >> p.shift;
      }
#pragma unroll
      for (int j = 0; j < FJ; ++j) acc[i][j] = zero;
    }
  };

  sstore(0, 0);
  __syncthreads();
  gload(0);
  int b = 0, ck = 0, csteps = a.C[0] / TK;  // branch of the current step, its steps
  for (int s0 = 0; s0 < S; s0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int s = s0 + u;
      if (s < S) {
        compute(s & 1);
        if (++ck == csteps) {
          fold(b);
          ++b;
          ck = 0;
          csteps = b < nbr ? a.C[b] / TK : 0;
        }
      }
      sstore((s + 1) & 1, (u + 1) % PF);
      gload((u + 1) % PF);
      __syncthreads();
    }
  }

  // Epilogue: bias, output requantization (accumulator pre-clamped to the
  // channel's saturation bound, then exact in 64 bits), store.
#pragma unroll
  for (int i = 0; i < FI; ++i) {
    const int32_t n = n0 + wn * WTN + i * 16 + (lane >> 4) * 4;
    if (n >= N) continue;  // N is a multiple of 16: the 4 channels are all valid
    ChanRq cr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int q = a.onq == 1 ? 0 : n + r;
      cr[r].init(a.omult[q], a.oshift[q], 0);
    }
    int32_t bias[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[r] = a.bias ? a.bias[n + r] : 0;
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int64_t m = m0 + wm * WTM + j * 16 + (lane & 15);
      if (m >= M) continue;
      int32_t v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        int64_t t = tot[i][j][r] + bias[r];
        t = t < -(int64_t)cr[r].L ? -(int64_t)cr[r].L : (t > cr[r].L ? cr[r].L : t);
        v[r] = cr[r].apply((int32_t)t);
      }
      ((uint32_t*)sbuf)[(wm * WTM + j * 16 + (lane & 15)) * OSTR + ((n - n0) >> 2)] =
          pack4(v[0], v[1], v[2], v[3]);
    }
  }
  // The output tile leaves through LDS (the weight tiles, free after the
  // last step's barrier) as 16-byte row chunks: a lane's own words would put
  // 16 rows of 4 bytes each into every store instruction.
  __syncthreads();
  {
    const uint32_t* so = (const uint32_t*)sbuf;
    const bool a16 = ((uintptr_t)a.y & 15) == 0;
    constexpr int CPT = TN / 16;
    for (int c = tid; c < TM * CPT; c += NT) {
      const int r = c / CPT, q = c - r * CPT;
      const int64_t m = m0 + r;
      const int32_t n = n0 + q * 16;
      if (m < M && n < N) store16(a.y + m * N + n, *(const v4i*)(so + r * OSTR + q * 4), a16);
    }
  }
}

template <int WN, int WM, int FI, int FJ, int PF = 2>
hipError_t launch_split_tile(const SplitArgs& a, hipStream_t s) {
  constexpr int TN = 16 * FI * WN, TM = 16 * FJ * WM;
  const int32_t tiles_n = (a.N + TN - 1) / TN;
  const int64_t total = ((a.M + TM - 1) / TM) * tiles_n;
  hipLaunchKernelGGL((split_conv_kernel<WN, WM, FI, FJ, PF>), dim3((unsigned)total),
                     dim3(64 * WN * WM), 0, s, a, tiles_n, total);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_split_conv(const SplitArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  // 32 x 32 per wave (the int64 running sums take 2 registers per output):
  // 64 x 64 workgroups for small grids, 128 x 64 beyond.
  const int64_t waves = ((a.M + 63) / 64) * ((a.N + 63) / 64) * 4;
  if (waves <= 4096) return launch_split_tile<2, 2, 2, 2>(a, s);
  return launch_split_tile<4, 2, 2, 2>(a, s);
}

}  // namespace ilw
