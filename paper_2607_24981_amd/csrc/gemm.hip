// gemm.hip -- int8 x int8 -> int32 GEMM on CDNA4 MFMA with the dyadic
// requantization fused into the epilogue (Sec. 3.2.1, eq. linear_quant; the
// rescale is a dyadic multiply-and-shift, Sec. 3.2.2).
//
//   y[m][n] = epilogue( rq(bias[n] + sum_k x[m][k] * w[n][k]; mult[n], shift[n]) )
//
// Tiling: a workgroup of 4 waves computes 128 channels x 128 tokens; each wave
// a 64 x 64 quadrant as 4 x 4 tiles of v_mfma_i32_16x16x64_i8.  The weight
// tile is the MFMA A operand (rows = channels) and the activation tile the B
// operand (columns = tokens), so each lane ends up holding four consecutive
// channels of one token and stores them as one 32-bit word.  K advances 64
// bytes per step through double-buffered LDS tiles whose rows are padded to
// 80 bytes, which keeps the 16-byte fragment reads of a wave free of bank
// conflicts.  Workgroups are remapped so that each XCD works on a contiguous
// run of tiles (tokens-major), keeping an activation tile and the weights in
// that XCD's L2.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int TN = 128;       // channels per workgroup tile
constexpr int TM = 128;       // tokens per workgroup tile
constexpr int TK = 64;        // K bytes per step
constexpr int LDS_ROW = 80;   // padded LDS row stride (bytes)
constexpr int NXCD = 8;

__device__ __forceinline__ uint32_t pack4(int32_t a, int32_t b, int32_t c, int32_t d) {
  return (uint32_t)(a & 0xff) | ((uint32_t)(b & 0xff) << 8) |
         ((uint32_t)(c & 0xff) << 16) | ((uint32_t)(d & 0xff) << 24);
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_i8_kernel(GemmArgs a, int32_t tiles_n,
                                                      int64_t tiles_total) {
  __shared__ __attribute__((aligned(16))) int8_t sW[2][TN * LDS_ROW];
  __shared__ __attribute__((aligned(16))) int8_t sX[2][TM * LDS_ROW];
  __shared__ int8_t glut[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave & 1;   // channel half of the tile
  const int wm = wave >> 1;  // token half of the tile

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

  if (EPI == EPI_GELU) {
    // SD-ShiftGELU of the requantized fc1 output is a function of one int8
    // value: tabulate it (with its output requantization) once per workgroup.
    int32_t v = tid - 128;
    glut[tid] = (int8_t)rq(sd_gelu(v, a.g_I0, a.g_kinter, a.g_kout), a.g_mult, a.g_shift);
  }

  const v4i zero = {0, 0, 0, 0};
  v4i acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero;

  // Each thread moves two 16-byte chunks of each operand tile per K step.
  v4i rw[2], rx[2];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256;
      const int row = c >> 2;
      const int k = kt * TK + (c & 3) * 16;
      const int32_t n = n0 + row;
      const int64_t m = m0 + row;
      rw[i] = (n < N && k < K) ? *(const v4i*)(W + (int64_t)n * K + k) : zero;
      rx[i] = (m < M && k < K) ? *(const v4i*)(X + m * K + k) : zero;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256;
      const int off = (c >> 2) * LDS_ROW + (c & 3) * 16;
      *(v4i*)(&sW[buf][off]) = rw[i];
      *(v4i*)(&sX[buf][off]) = rx[i];
    }
  };

  const int nk = (K + TK - 1) / TK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int frag_off = (lane & 15) * LDS_ROW + (lane >> 4) * 16;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    v4i fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      fa[i] = *(const v4i*)(&sW[buf][(wn * 64 + i * 16) * LDS_ROW + frag_off]);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      fb[j] = *(const v4i*)(&sX[buf][(wm * 64 + j * 16) * LDS_ROW + frag_off]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  Lane holds channels n..n+3 (n = 4*(lane/16) within a 16-tile)
  // of token lane%16 of each of the 4 x 4 tiles.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int32_t n = n0 + wn * 64 + i * 16 + (lane >> 4) * 4;
    if (n >= N) continue;  // N is a multiple of 16: the 4 channels are all valid
    int32_t bs[4], ml[4], sh[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      bs[r] = a.bias ? a.bias[n + r] : 0;
      const int qi = a.nq == 1 ? 0 : n + r;
      ml[r] = a.mult[qi];
      sh[r] = a.shift[qi];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t m = m0 + wm * 64 + j * 16 + (lane & 15);
      if (m >= M) continue;
      int32_t v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = rq(acc[i][j][r] + bs[r], ml[r], sh[r]);
      if (EPI == EPI_STORE) {
        *(uint32_t*)(a.y + m * N + n) = pack4(v[0], v[1], v[2], v[3]);
      } else if (EPI == EPI_GELU) {
        *(uint32_t*)(a.y + m * N + n) = pack4(glut[v[0] + 128], glut[v[1] + 128],
                                              glut[v[2] + 128], glut[v[3] + 128]);
      } else if (EPI == EPI_RESID) {
        const uint32_t s = *(const uint32_t*)(a.resid + m * N + n);
        int32_t o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          o[r] = rq2(v[r], (int8_t)(s >> (8 * r)), a.res_ma, a.res_mb, a.res_shift);
        *(uint32_t*)(a.y + m * N + n) = pack4(o[0], o[1], o[2], o[3]);
      } else {  // EPI_QKV: scatter into window-major Q, K and V^T
        const QkvLayout& L = a.qkv;
        const int32_t b = (int32_t)(m / L.T), t = (int32_t)(m % L.T);
        const int32_t ty = t / L.grid_w, tx = t % L.grid_w;
        const int32_t w = (ty / L.win_h) * L.nwx + tx / L.win_w;
        const int32_t li = (ty % L.win_h) * L.win_w + tx % L.win_w;
        const int32_t part = n / L.D, rem_n = n % L.D;
        const int32_t h = rem_n >> 6, c = rem_n & 63;
        const int64_t slice = ((int64_t)b * L.nW + w) * L.H + h;
        if (part < 2) {
          int8_t* dst = (part == 0 ? L.q : L.k) + (slice * L.Tw + li) * 64 + c;
          *(uint32_t*)dst = pack4(v[0], v[1], v[2], v[3]);
        } else {
          int8_t* dst = L.vt + (slice * 64 + c) * L.Twp + li;
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[(int64_t)r * L.Twp] = (int8_t)v[r];
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  const int32_t tiles_n = (a.N + TN - 1) / TN;
  const int64_t tiles_m = (a.M + TM - 1) / TM;
  const int64_t total = tiles_m * tiles_n;
  dim3 grid((unsigned)total), block(256);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL(gemm_i8_kernel<EPI_STORE>, grid, block, 0, s, a, tiles_n, total); break;
    case EPI_GELU: hipLaunchKernelGGL(gemm_i8_kernel<EPI_GELU>, grid, block, 0, s, a, tiles_n, total); break;
    case EPI_RESID: hipLaunchKernelGGL(gemm_i8_kernel<EPI_RESID>, grid, block, 0, s, a, tiles_n, total); break;
    default: hipLaunchKernelGGL(gemm_i8_kernel<EPI_QKV>, grid, block, 0, s, a, tiles_n, total); break;
  }
  return hipGetLastError();
}

}  // namespace ilw
