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
//
// Sampling locations are Q8 pixels of each level.  A reference point (x, y)
// lands at floor(x W / 2^8) and the offset adds Q8 pixels.  A reference box
// (cx, cy, w, h) takes the offset in units of the box, location = c +
// (off / 2^8) / P * size / 2, floored once in Q8 pixels:
// X = floor((cx 2^9 P + off_x w) W / (2^17 P)).
#include "ilw_internal.h"

namespace ilw {
namespace {

// floor(n / d) for d > 0
__device__ __forceinline__ int64_t floor_div_pos(int64_t n, int64_t d) {
  const int64_t q = n / d;
  return (n % d != 0 && n < 0) ? q - 1 : q;
}

__global__ __launch_bounds__(256) void deform_kernel(DeformArgs a) {
  __shared__ int32_t elut[256];
  elut[threadIdx.x] = shift_exp(-(int32_t)threadIdx.x, a.I0, a.k_inter);
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
  const int32_t sd = a.s_d >= 0 ? a.s_d : calibrate_shift(sum, a.m_p);
  const uint32_t F = shiftmax_factor(sum, sd);
  // e F < 2^30 2^31: a shift of 61 or more leaves 0, as does 63, so the cap
  // keeps the 64-bit shift defined (s_d reaches 36 with m_p = 31)
  const int32_t sh = min(32 - a.k_out + sd, 63);
  const uint64_t cap = (1u << (a.k_out - 1)) - 1;

  const bool box = a.ref_dims == 4;
  const int32_t* r = a.ref + bq * a.ref_dims;
  const int64_t rx = r[0], ry = r[1];
  const int64_t bw = box ? r[2] : 0, bh = box ? r[3] : 0;
  // box locations divide by 2^17 P: a shift when P is a power of two
  const int32_t pshift = (a.P & (a.P - 1)) == 0 ? 17 + __builtin_ctz(a.P) : -1;
  const int64_t den = (int64_t)131072 * a.P;
  const int64_t cxs = rx * 512 * a.P, cys = ry * 512 * a.P;
  auto box_loc = [&](int64_t num) {
    return pshift >= 0 ? num >> pshift : floor_div_pos(num, den);
  };
  const int16_t* off = a.offs + grp * LP * 2;
  const int8_t* off8 = a.offs8 + grp * LP * 2;
  auto offset = [&](int32_t k) {  // offset word k of this (b, q, h)
    return a.offs8 ? (int64_t)off8[k] << a.off_shift : (int64_t)off[k];
  };
  const int64_t head_stride = (int64_t)a.H * a.Dh;
  const int8_t* vbase = a.value + (int64_t)b * a.S * head_stride + (int64_t)h * a.Dh + cl * 4;

  // The samples go in chunks whose gathers are all issued before any is
  // used: addresses of samples outside the map are clamped onto the base
  // row (a valid address) and their weights are 0.
  int32_t acc[4] = {0, 0, 0, 0};
  int64_t accw[4] = {0, 0, 0, 0};
  int32_t l = 0, p = 0;  // level and point of sample i0
  constexpr int CH = 8;
  for (int32_t i0 = 0; i0 < LP; i0 += CH) {
    uint32_t v[CH][4];
    int64_t wt[CH][4];
    int32_t ll = l, pp = p;
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int32_t i = i0 + u;
      const bool live = i < LP;
      const int32_t Hl = a.hw[ll][0], Wl = a.hw[ll][1];
      const int8_t* vl = vbase + (int64_t)a.start[ll] * head_stride;
      const int32_t ic = live ? i : LP - 1;
      const uint64_t pw = ((uint64_t)(uint32_t)elut[m - lg[ic]] * F) >> sh;
      const int32_t wgt = live ? (int32_t)(pw > cap ? cap : pw) : 0;
      const int64_t ox = offset(2 * ic), oy = offset(2 * ic + 1);
      const int64_t X = box ? box_loc((cxs + ox * bw) * Wl) : ((rx * Wl) >> 8) + ox;
      const int64_t Y = box ? box_loc((cys + oy * bh) * Hl) : ((ry * Hl) >> 8) + oy;
      if (a.mode == 0) {
        const int64_t ix = X >> 8, iy = Y >> 8;  // floor
        const bool in = ix >= 0 && ix < Wl && iy >= 0 && iy < Hl;
        v[u][0] = *(const uint32_t*)(in ? vl + (iy * Wl + ix) * head_stride : vbase);
        wt[u][0] = in ? wgt : 0;
      } else {
        const int64_t Xc = X - 128, Yc = Y - 128;  // half-pixel grid
        const int64_t x0 = Xc >> 8, y0 = Yc >> 8;
        const int32_t fx = (int32_t)(Xc & 255), fy = (int32_t)(Yc & 255);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int dx = c & 1, dy = c >> 1;
          const int64_t xi = x0 + dx, yi = y0 + dy;
          const bool in = xi >= 0 && xi < Wl && yi >= 0 && yi < Hl;
          const int32_t wc = (dx ? fx : 256 - fx) * (dy ? fy : 256 - fy);
          v[u][c] = *(const uint32_t*)(in ? vl + (yi * Wl + xi) * head_stride : vbase);
          wt[u][c] = in ? (int64_t)wgt * wc : 0;
        }
      }
      if (++pp == a.P) {
        pp = 0;
        ll = min(ll + 1, a.L - 1);
      }
    }
    l = ll;
    p = pp;
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      if (a.mode == 0) {
        const int32_t w0 = (int32_t)wt[u][0];
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] += w0 * (int32_t)(int8_t)(v[u][0] >> (8 * c));
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int c = 0; c < 4; ++c) accw[c] += wt[u][k] * (int32_t)(int8_t)(v[u][k] >> (8 * c));
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

// The same sampler without the per-lane redundancy, for G = head_dim / 4 a
// power of two in [4, 64] (groups then align with waves): lane k of a group
// owns samples k, k + G, ..., computes their Shiftmax weights and value rows
// once, the group combines the row maximum and the exponential sum with XOR
// shuffles, and each sample's (row, weight) reaches the G lanes of its group
// by shuffle.  J = ceil(L*P / G) samples per lane; MODE 0 nearest, 1 bilinear.
template <int MODE, int J>
__global__ __launch_bounds__(256) void deform_group_kernel(DeformArgs a) {
  constexpr int NC = MODE == 0 ? 1 : 4;  // value rows per sample
  __shared__ int32_t elut[256];
  elut[threadIdx.x] = shift_exp(-(int32_t)threadIdx.x, a.I0, a.k_inter);
  __syncthreads();

  const int32_t G = a.Dh >> 2;
  const int lane = threadIdx.x & 63;
  const int32_t cl = lane & (G - 1);
  const int gbase = lane & ~(G - 1);
  const int64_t ngrp = (int64_t)a.B * a.Q * a.H;
  const int64_t grp0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) / G;
  const bool live = grp0 < ngrp;
  const int64_t grp = live ? grp0 : ngrp - 1;  // idle lanes still join the shuffles
  const int32_t h = (int32_t)(grp % a.H);
  const int64_t bq = grp / a.H;
  const int32_t b = (int32_t)(bq / a.Q);
  const int32_t LP = a.L * a.P;

  // Constrained Shiftmax over the group's L*P logits
  const int8_t* lg = a.logits + grp * LP;
  int32_t lgv[J];
  int32_t m = -128;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int32_t i = cl + j * G;
    lgv[j] = i < LP ? (int32_t)lg[i] : -128;
    m = max(m, lgv[j]);
  }
  for (int o = 1; o < G; o <<= 1) m = max(m, __shfl_xor(m, o, 64));
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (cl + j * G < LP) sum += (uint32_t)elut[m - lgv[j]];
  for (int o = 1; o < G; o <<= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)sum, o, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(sum >> 32), o, 64);
    sum += ((uint64_t)hi << 32) | lo;
  }
  const int32_t sd = a.s_d >= 0 ? a.s_d : calibrate_shift(sum, a.m_p);
  const uint32_t F = shiftmax_factor(sum, sd);
  // e F < 2^30 2^31: a shift of 61 or more leaves 0, as does 63, so the cap
  // keeps the 64-bit shift defined (s_d reaches 36 with m_p = 31)
  const int32_t sh = min(32 - a.k_out + sd, 63);
  const uint64_t cap = (1u << (a.k_out - 1)) - 1;

  const bool box = a.ref_dims == 4;
  const int32_t* r = a.ref + bq * a.ref_dims;
  const int64_t rx = r[0], ry = r[1];
  const int64_t bw = box ? r[2] : 0, bh = box ? r[3] : 0;
  const int32_t pshift = (a.P & (a.P - 1)) == 0 ? 17 + __builtin_ctz(a.P) : -1;
  const int64_t den = (int64_t)131072 * a.P;
  const int64_t cxs = rx * 512 * a.P, cys = ry * 512 * a.P;
  auto box_loc = [&](int64_t num) {
    return pshift >= 0 ? num >> pshift : floor_div_pos(num, den);
  };
  const int16_t* off = a.offs + grp * LP * 2;
  const int8_t* off8 = a.offs8 + grp * LP * 2;
  auto offset = [&](int32_t k) {  // offset word k of this (b, q, h)
    return a.offs8 ? (int64_t)off8[k] << a.off_shift : (int64_t)off[k];
  };

  // the lane's own samples: value rows (0 with weight 0 when off the map)
  int32_t row[J][NC], wt[J][NC];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int32_t i = cl + j * G;
    const bool valid = i < LP;
    const int32_t ic = valid ? i : 0;
    const int32_t l = ic / a.P;
    const int32_t Hl = a.hw[l][0], Wl = a.hw[l][1], st = a.start[l];
    const uint64_t pw = ((uint64_t)(uint32_t)elut[m - lgv[j]] * F) >> sh;
    const int32_t wgt = valid ? (int32_t)(pw > cap ? cap : pw) : 0;
    const int64_t ox = offset(2 * ic), oy = offset(2 * ic + 1);
    const int64_t X = box ? box_loc((cxs + ox * bw) * Wl) : ((rx * Wl) >> 8) + ox;
    const int64_t Y = box ? box_loc((cys + oy * bh) * Hl) : ((ry * Hl) >> 8) + oy;
    if (MODE == 0) {
      const int64_t ix = X >> 8, iy = Y >> 8;  // floor
      const bool in = ix >= 0 && ix < Wl && iy >= 0 && iy < Hl;
      row[j][0] = in ? st + (int32_t)(iy * Wl + ix) : 0;
      wt[j][0] = in ? wgt : 0;
    } else {
      const int64_t Xc = X - 128, Yc = Y - 128;  // half-pixel grid
      const int64_t x0 = Xc >> 8, y0 = Yc >> 8;
      const int32_t fx = (int32_t)(Xc & 255), fy = (int32_t)(Yc & 255);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int dx = c & 1, dy = c >> 1;
        const int64_t xi = x0 + dx, yi = y0 + dy;
        const bool in = xi >= 0 && xi < Wl && yi >= 0 && yi < Hl;
        row[j][c] = in ? st + (int32_t)(yi * Wl + xi) : 0;
        wt[j][c] = in ? wgt * (dx ? fx : 256 - fx) * (dy ? fy : 256 - fy) : 0;
      }
    }
  }

  // every sample of the group, its (row, weight) from the owning lane; the
  // loads of four samples are issued before their products
  const int64_t head_stride = (int64_t)a.H * a.Dh;
  const int8_t* vbase = a.value + (int64_t)b * a.S * head_stride + (int64_t)h * a.Dh + cl * 4;
  int32_t acc[4] = {0, 0, 0, 0};
  int64_t accw[4] = {0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < J; ++j) {
    for (int k0 = 0; k0 < G && j * G + k0 < LP; k0 += 4) {
      uint32_t v[4][NC];
      int32_t w[4][NC];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int owner = gbase + min(k0 + u, G - 1);
        const bool use = k0 + u < G && j * G + k0 + u < LP;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int32_t rr = __shfl(row[j][c], owner, 64);
          const int32_t ww = __shfl(wt[j][c], owner, 64);
          w[u][c] = use ? ww : 0;
          v[u][c] = *(const uint32_t*)(vbase + (int64_t)rr * head_stride);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int32_t x = (int32_t)(int8_t)(v[u][c] >> (8 * q));
            if (MODE == 0) acc[q] += w[u][c] * x;
            else accw[q] += (int64_t)w[u][c] * x;
          }
    }
  }
  if (!live) return;
  uint32_t packed = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int32_t rv = MODE == 0 ? rq(acc[c], a.out_mult, a.out_shift)
                                 : rq_wide(accw[c], a.out_mult, a.out_shift + 16);
    packed |= (uint32_t)(rv & 0xff) << (8 * c);
  }
  *(uint32_t*)(a.out + grp * a.Dh + cl * 4) = packed;
}

template <int MODE>
hipError_t launch_group(const DeformArgs& a, int32_t J, dim3 grid, hipStream_t s) {
  switch (J) {
    case 1: hipLaunchKernelGGL((deform_group_kernel<MODE, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((deform_group_kernel<MODE, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((deform_group_kernel<MODE, 3>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((deform_group_kernel<MODE, 4>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_deform(const DeformArgs& a, hipStream_t s) {
  const int64_t threads = (int64_t)a.B * a.Q * a.H * (a.Dh / 4);
  if (threads == 0) return hipSuccess;
  dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  const int32_t G = a.Dh / 4, LP = a.L * a.P, J = (LP + G - 1) / G;
  if (G >= 4 && G <= 64 && (G & (G - 1)) == 0 && J <= 4)
    return a.mode == 0 ? launch_group<0>(a, J, grid, s) : launch_group<1>(a, J, grid, s);
  hipLaunchKernelGGL(deform_kernel, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace ilw
