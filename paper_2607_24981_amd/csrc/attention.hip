// attention.hip -- fused integer attention for one (image, window, head,
// 32-query block) per workgroup:
//
//   S = Q K^T (MFMA int8) -> per-tensor dyadic -> int8 scores held in LDS
//   P = Constrained Shiftmax of every score row (Alg. 2)      (int8 in LDS)
//   O = P V   (MFMA int8) -> per-tensor dyadic -> int8 output (token order)
//
// Constrained Shiftmax needs the exact row maximum before any exponential
// (ShiftExp of x - max cannot be rescaled bit-exactly when the maximum
// changes), so a whole score row block is kept in LDS instead of the online
// rescaling used by float attention: 32 rows x Tw int8 scores (51 KB at
// Tw = 1600).  Because the scores are int8, x - max only takes the values
// 0 .. -255, so ShiftExp is one table of 256 entries per workgroup, and
// S_sum >> s_d is exactly the quotient-remainder denominator of Alg. 2.
#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int AR = 32;  // query rows per workgroup

__global__ __launch_bounds__(256) void attention_kernel(AttnArgs a, int32_t lds_row) {
  extern __shared__ __attribute__((aligned(16))) int8_t sS[];  // [AR][lds_row]
  __shared__ int32_t elut[256];
  __shared__ int32_t pmax[4][AR];
  __shared__ int32_t rmax[AR];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t Tw = a.Tw, Twp = a.Twp;
  const int32_t i0 = blockIdx.x * AR;
  const int32_t h = blockIdx.y;
  const int32_t bw = blockIdx.z;  // image * nW + window
  const int64_t slice = (int64_t)bw * a.H + h;
  const int8_t* __restrict__ Q = a.q + slice * Tw * 64;
  const int8_t* __restrict__ K = a.k + slice * Tw * 64;
  const int8_t* __restrict__ Vt = a.vt + slice * 64 * Twp;

  elut[tid] = shift_exp(-tid, a.I0, a.k_inter);  // ShiftExp(-d), d = 0..255

  // Query fragments (MFMA B operand: columns = query rows).  Rows past the
  // window are clamped to a valid row; their results are never stored.
  v4i qf[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int32_t r = min(i0 + f * 16 + (lane & 15), Tw - 1);
    qf[f] = *(const v4i*)(Q + (int64_t)r * 64 + (lane >> 4) * 16);
  }

  // ---- phase 1: scores.  Waves split the keys in blocks of 16; the key
  // fragment is the A operand, so a lane holds 4 consecutive keys of one row.
  const v4i zero = {0, 0, 0, 0};
  int32_t mx[2] = {-128, -128};
  const int32_t nkb = (Tw + 15) >> 4;
  for (int32_t kb = wave; kb < nkb; kb += 4) {
    const int32_t key = min(kb * 16 + (lane & 15), Tw - 1);
    const v4i kf = *(const v4i*)(K + (int64_t)key * 64 + (lane >> 4) * 16);
    const int32_t kcol = kb * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const v4i s = __builtin_amdgcn_mfma_i32_16x16x64_i8(kf, qf[f], zero, 0, 0, 0);
      uint32_t packed = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int32_t v = rq(s[r], a.score_mult, a.score_shift);
        if (kcol + r < Tw) mx[f] = max(mx[f], v);
        packed |= (uint32_t)(v & 0xff) << (8 * r);
      }
      *(uint32_t*)(sS + (f * 16 + (lane & 15)) * lds_row + kcol) = packed;
    }
  }
  // row maxima: combine the 4 lanes sharing a row, then the 4 waves
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    mx[f] = max(mx[f], __shfl_xor(mx[f], 16, 64));
    mx[f] = max(mx[f], __shfl_xor(mx[f], 32, 64));
    if (lane < 16) pmax[wave][f * 16 + lane] = mx[f];
  }
  __syncthreads();
  if (tid < AR)
    rmax[tid] = max(max(pmax[0][tid], pmax[1][tid]), max(pmax[2][tid], pmax[3][tid]));
  __syncthreads();

  // ---- phase 2: Constrained Shiftmax of each row, in place.  8 rows per wave.
  const int32_t nword = (Tw + 3) >> 2;
  const int32_t pword = Twp >> 2;
  const int32_t pcap = (1 << (a.k_out - 1)) - 1;
  for (int rr = wave * 8; rr < wave * 8 + 8; ++rr) {
    if (i0 + rr >= Tw) break;
    uint32_t* row = (uint32_t*)(sS + rr * lds_row);
    const int32_t m = rmax[rr];
    uint64_t sum = 0;
    for (int32_t wd = lane; wd < nword; wd += 64) {
      const uint32_t word = row[wd];
#pragma unroll
      for (int b = 0; b < 4; ++b)
        if (wd * 4 + b < Tw) sum += (uint32_t)elut[m - (int8_t)(word >> (8 * b))];
    }
    sum = wave_sum_u64(sum);
    const int32_t sd = a.s_d >= 0 ? a.s_d : calibrate_shift(sum, a.m_p);
    const uint32_t F = shiftmax_factor(sum, sd);
    const int32_t sh = 32 - a.k_out + sd;
    for (int32_t wd = lane; wd < pword; wd += 64) {
      const uint32_t word = row[wd];
      uint32_t outw = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (wd * 4 + b < Tw) {
          const uint32_t e = (uint32_t)elut[m - (int8_t)(word >> (8 * b))];
          uint64_t p = ((uint64_t)e * F) >> sh;
          p = p > (uint64_t)pcap ? (uint64_t)pcap : p;
          outw |= (uint32_t)p << (8 * b);
        }
      }
      row[wd] = outw;  // padding columns become 0
    }
  }
  __syncthreads();

  // ---- phase 3: O = P V.  Wave w owns channels 16w..16w+15; V^T is the A
  // operand (rows = channels), P^T the B operand (columns = query rows), so a
  // lane holds 4 consecutive channels of one query row.
  v4i o[2] = {zero, zero};
  const int32_t c0 = wave * 16;
  const int8_t* vrow = Vt + (int64_t)(c0 + (lane & 15)) * Twp + (lane >> 4) * 16;
  const int8_t* prow = sS + (lane & 15) * lds_row + (lane >> 4) * 16;
  for (int32_t j0 = 0; j0 < Twp; j0 += 64) {
    const v4i vf = *(const v4i*)(vrow + j0);
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const v4i pf = *(const v4i*)(prow + f * 16 * lds_row + j0);
      o[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(vf, pf, o[f], 0, 0, 0);
    }
  }
  const int32_t b_img = bw / a.nW, w = bw % a.nW;
  const int32_t wy = w / a.nwx, wx = w % a.nwx;
  const int32_t c = c0 + (lane >> 4) * 4;
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int32_t i = i0 + f * 16 + (lane & 15);
    if (i >= Tw) continue;
    const int32_t t = (wy * a.win_h + i / a.win_w) * a.grid_w + wx * a.win_w + i % a.win_w;
    uint32_t packed = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      packed |= (uint32_t)(rq(o[f][r], a.pv_mult, a.pv_shift) & 0xff) << (8 * r);
    *(uint32_t*)(a.out + ((int64_t)b_img * a.T + t) * a.D + h * 64 + c) = packed;
  }
}

// [B, T, 3D] token-major QKV -> window-major Q, K and V^T.  One thread per
// 16-byte chunk of a token's 3D channels.
__global__ __launch_bounds__(256) void qkv_relayout_kernel(const int8_t* qkv, int32_t B,
                                                           QkvLayout L) {
  const int32_t chunks = 3 * L.D / 16;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (g >= (int64_t)B * L.T * chunks) return;
  const int64_t m = g / chunks;
  const int32_t n = (int32_t)(g % chunks) * 16;
  const int32_t b = (int32_t)(m / L.T), t = (int32_t)(m % L.T);
  const int32_t ty = t / L.grid_w, tx = t % L.grid_w;
  const int32_t w = (ty / L.win_h) * L.nwx + tx / L.win_w;
  const int32_t li = (ty % L.win_h) * L.win_w + tx % L.win_w;
  const int32_t part = n / L.D, rem_n = n % L.D;
  const int32_t h = rem_n >> 6, c = rem_n & 63;
  const int64_t slice = ((int64_t)b * L.nW + w) * L.H + h;
  const v4i v = *(const v4i*)(qkv + m * 3 * L.D + n);
  if (part < 2) {
    *(v4i*)((part == 0 ? L.q : L.k) + (slice * L.Tw + li) * 64 + c) = v;
  } else {
    int8_t* dst = L.vt + (slice * 64 + c) * L.Twp + li;
    const int8_t* bytes = (const int8_t*)&v;
#pragma unroll
    for (int r = 0; r < 16; ++r) dst[(int64_t)r * L.Twp] = bytes[r];
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  const int32_t lds_row = a.Twp + 16;
  const size_t smem = (size_t)AR * lds_row;
  static size_t configured = 0;
  if (smem > 65536 && smem > configured) {
    hipError_t e = hipFuncSetAttribute((const void*)attention_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)smem);
    if (e != hipSuccess) return e;
    configured = smem;
  }
  dim3 grid((a.Tw + AR - 1) / AR, a.H, a.B * a.nW), block(256);
  hipLaunchKernelGGL(attention_kernel, grid, block, smem, s, a, lds_row);
  return hipGetLastError();
}

hipError_t launch_qkv_relayout(const int8_t* qkv, int32_t B, const QkvLayout& L,
                               hipStream_t s) {
  const int64_t n = (int64_t)B * L.T * (3 * L.D / 16);
  if (n == 0) return hipSuccess;
  dim3 grid((unsigned)((n + 255) / 256)), block(256);
  hipLaunchKernelGGL(qkv_relayout_kernel, grid, block, 0, s, qkv, B, L);
  return hipGetLastError();
}

}  // namespace ilw
