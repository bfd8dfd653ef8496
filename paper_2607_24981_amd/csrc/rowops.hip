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
// One wave per row of C (multiple of 4) int8 channels.
__global__ __launch_bounds__(256) void layernorm_kernel(const int8_t* x, int8_t* y,
                                                        int64_t rows, int32_t C,
                                                        const int32_t* beta,
                                                        const int32_t* mult,
                                                        const int32_t* shift, int32_t nq,
                                                        int32_t iters) {
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
  // mean rounded half up: floor((2*sum + C) / (2*C)), numerator may be < 0
  const int32_t num = 2 * s + C, den = 2 * C;
  int32_t mu = num / den;
  if (num % den != 0 && num < 0) mu -= 1;

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
  // Newton's integer square root from 2^16, a fixed number of steps; the
  // iterate never drops below floor(sqrt(V)) >= 1 when V > 0.
  uint32_t sigma = 0;
  if (V != 0) {
    uint32_t k = 65536;
    for (int32_t t = 0; t < iters; ++t) k = (k + V / k) >> 1;
    sigma = k;
  }
  const uint32_t F = sigma ? 0x7fffffffu / sigma : 0u;

  for (int32_t w = lane; w < nw; w += 64) {
    const uint32_t v = xr[w];
    uint32_t o = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t c = w * 4 + b;
      const int32_t d = (int8_t)(v >> (8 * b)) - mu;
      // |d| <= sigma, so |d * F| < 2^31 and n fits 31 bits
      const int64_t n = ((int64_t)d * (int64_t)F) >> 1;
      const int32_t q = nq == 1 ? 0 : c;
      const int32_t r = rq_wide(n + beta[c], mult[q], shift[q]);
      o |= (uint32_t)(r & 0xff) << (8 * b);
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
  const int32_t sh = 32 - k_out + sd;
  const uint64_t cap = (1u << (k_out - 1)) - 1;
  for (int32_t j = lane; j < cols; j += 64) {
    uint64_t p = ((uint64_t)(uint32_t)elut[m - xr[j]] * F) >> sh;
    yr[j] = (int8_t)(p > cap ? cap : p);
  }
}

// ---------------------------------------------------------------- GELU
__global__ __launch_bounds__(256) void gelu_kernel(const int8_t* x, int8_t* y, int64_t n,
                                                   int32_t I0, int32_t k_inter,
                                                   int32_t k_out, int32_t mult,
                                                   int32_t shift) {
  __shared__ int8_t lut[256];
  lut[threadIdx.x] =
      (int8_t)rq(sd_gelu((int32_t)threadIdx.x - 128, I0, k_inter, k_out), mult, shift);
  __syncthreads();
  const int64_t nchunk = n >> 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < nchunk; c += stride) {
    v4i v = *(const v4i*)(x + c * 16);
    int8_t* b = (int8_t*)&v;
#pragma unroll
    for (int i = 0; i < 16; ++i) b[i] = lut[(int32_t)b[i] + 128];
    *(v4i*)(y + c * 16) = v;
  }
  // tail (n not a multiple of 16)
  const int64_t t = (nchunk << 4) + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0 && t < n) y[t] = lut[(int32_t)x[t] + 128];
}

// ---------------------------------------------------------------- residual
__global__ __launch_bounds__(256) void residual_kernel(const int8_t* a, const int8_t* b,
                                                       int8_t* y, int64_t n, int32_t ma,
                                                       int32_t mb, int32_t shift) {
  const int64_t nchunk = n >> 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < nchunk; c += stride) {
    v4i va = *(const v4i*)(a + c * 16);
    const v4i vb = *(const v4i*)(b + c * 16);
    int8_t* pa = (int8_t*)&va;
    const int8_t* pb = (const int8_t*)&vb;
#pragma unroll
    for (int i = 0; i < 16; ++i) pa[i] = (int8_t)rq2(pa[i], pb[i], ma, mb, shift);
    *(v4i*)(y + c * 16) = va;
  }
  const int64_t t = (nchunk << 4) + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0 && t < n) y[t] = (int8_t)rq2(a[t], b[t], ma, mb, shift);
}

unsigned stream_grid(int64_t n) {
  const int64_t chunks = (n >> 4) + 1;
  int64_t g = (chunks + 255) / 256;
  if (g > 4096) g = 4096;
  return (unsigned)g;
}

}  // namespace

hipError_t launch_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                            const int32_t* beta, const int32_t* mult, const int32_t* shift,
                            int32_t nq, int32_t iters, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  hipLaunchKernelGGL(layernorm_kernel, grid, block, 0, s, x, y, rows, C, beta, mult, shift,
                     nq, iters);
  return hipGetLastError();
}

hipError_t launch_shiftmax(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                           int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                           int32_t s_d, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  hipLaunchKernelGGL(shiftmax_kernel, grid, block, 0, s, x, y, rows, cols, I0, k_inter,
                     k_out, m_p, s_d);
  return hipGetLastError();
}

hipError_t launch_gelu(const int8_t* x, int8_t* y, int64_t n, int32_t I0, int32_t k_inter,
                       int32_t k_out, int32_t mult, int32_t shift, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gelu_kernel, dim3(stream_grid(n)), dim3(256), 0, s, x, y, n, I0,
                     k_inter, k_out, mult, shift);
  return hipGetLastError();
}

hipError_t launch_residual(const int8_t* a, const int8_t* b, int8_t* y, int64_t n,
                           int32_t ma, int32_t mb, int32_t shift, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(residual_kernel, dim3(stream_grid(n)), dim3(256), 0, s, a, b, y, n,
                     ma, mb, shift);
  return hipGetLastError();
}

}  // namespace ilw
