// deform.hip -- multi-scale deformable sampling core with integer weights
// (Sec. 3.1.1: the sampled value is the nearest grid point instead of a
// bilinear blend; Sec. 3.3.2: the sampling weights are Constrained Shiftmax
// of the L*P logits of each (image, query, head)).
//
// A group of head_dim/4 lanes serves one (image, query, head); each lane owns
// four channels, so the head slice of one sample (head_dim bytes) is read by
// the group as consecutive 32-bit words.  The L*P weights are recomputed by
// every lane of the group from a per-workgroup ShiftExp table: it costs a few
// table reads and saves a cross-lane exchange.
#include "ilw_internal.h"

namespace ilw {
namespace {

__global__ __launch_bounds__(256) void deform_kernel(DeformArgs a) {
  __shared__ int32_t elut[256];
  elut[threadIdx.x] = shift_exp(-(int32_t)threadIdx.x, a.I0, 16);
  __syncthreads();

  const int32_t G = a.Dh >> 2;  // lanes per (b, q, h)
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t grp = gid / G;
  const int32_t cl = (int32_t)(gid % G);
  if (grp >= (int64_t)a.B * a.Q * a.H) return;
  const int32_t h = (int32_t)(grp % a.H);
  const int64_t bq = grp / a.H;
  const int32_t b = (int32_t)(bq / a.Q);
  const int32_t LP = a.L * a.P;

  // Constrained Shiftmax over the L*P logits of this (b, q, h)
  const int8_t* lg = a.logits + grp * LP;
  int32_t m = -128;
  for (int32_t i = 0; i < LP; ++i) m = max(m, (int32_t)lg[i]);
  uint64_t sum = 0;
  for (int32_t i = 0; i < LP; ++i) sum += (uint32_t)elut[m - lg[i]];
  const int32_t sd = a.s_d >= 0 ? a.s_d : calibrate_shift(sum, 4);
  const uint32_t F = shiftmax_factor(sum, sd);
  const int32_t sh = 24 + sd;  // 32 - k_out with k_out = 8

  const int64_t rx = a.ref[bq * 2 + 0], ry = a.ref[bq * 2 + 1];
  const int16_t* off = a.offs + grp * LP * 2;
  const int64_t head_stride = (int64_t)a.H * a.Dh;
  const int8_t* vbase = a.value + (int64_t)b * a.S * head_stride + (int64_t)h * a.Dh + cl * 4;

  int32_t acc[4] = {0, 0, 0, 0};
  int64_t accw[4] = {0, 0, 0, 0};
  for (int32_t l = 0; l < a.L; ++l) {
    const int32_t Hl = a.hw[l][0], Wl = a.hw[l][1];
    const int64_t X0 = (rx * Wl) >> 8, Y0 = (ry * Hl) >> 8;  // Q8 pixel coordinates
    const int8_t* vl = vbase + (int64_t)a.start[l] * head_stride;
    for (int32_t p = 0; p < a.P; ++p) {
      const int32_t i = l * a.P + p;
      uint64_t pw = ((uint64_t)(uint32_t)elut[m - lg[i]] * F) >> sh;
      const int32_t wgt = (int32_t)(pw > 127 ? 127 : pw);
      const int64_t X = X0 + off[2 * i], Y = Y0 + off[2 * i + 1];
      if (a.mode == 0) {
        const int64_t ix = X >> 8, iy = Y >> 8;  // floor
        if (ix < 0 || ix >= Wl || iy < 0 || iy >= Hl) continue;
        const uint32_t v = *(const uint32_t*)(vl + (iy * Wl + ix) * head_stride);
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] += wgt * (int32_t)(int8_t)(v >> (8 * c));
      } else {
        const int64_t Xc = X - 128, Yc = Y - 128;  // half-pixel grid
        const int64_t x0 = Xc >> 8, y0 = Yc >> 8;
        const int32_t fx = (int32_t)(Xc & 255), fy = (int32_t)(Yc & 255);
#pragma unroll
        for (int dy = 0; dy < 2; ++dy)
#pragma unroll
          for (int dx = 0; dx < 2; ++dx) {
            const int64_t xi = x0 + dx, yi = y0 + dy;
            if (xi < 0 || xi >= Wl || yi < 0 || yi >= Hl) continue;
            const int32_t wc = (dx ? fx : 256 - fx) * (dy ? fy : 256 - fy);
            const uint32_t v = *(const uint32_t*)(vl + (yi * Wl + xi) * head_stride);
            const int64_t pwc = (int64_t)wgt * wc;
#pragma unroll
            for (int c = 0; c < 4; ++c) accw[c] += pwc * (int32_t)(int8_t)(v >> (8 * c));
          }
      }
    }
  }
  uint32_t packed = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int32_t r = a.mode == 0 ? rq(acc[c], a.out_mult, a.out_shift)
                                  : rq_wide(accw[c], a.out_mult, a.out_shift + 16);
    packed |= (uint32_t)(r & 0xff) << (8 * c);
  }
  *(uint32_t*)(a.out + grp * a.Dh + cl * 4) = packed;
}

}  // namespace

hipError_t launch_deform(const DeformArgs& a, hipStream_t s) {
  const int64_t threads = (int64_t)a.B * a.Q * a.H * (a.Dh / 4);
  if (threads == 0) return hipSuccess;
  dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  hipLaunchKernelGGL(deform_kernel, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace ilw
