// attention.hip -- fused integer attention for one (image, window, head,
// block of query rows) per workgroup:
//
//   S = Q K^T (MFMA int8) -> per-tensor dyadic -> int8 scores held in LDS
//   P = Constrained Shiftmax of every score row (Alg. 2)      (int8 in LDS)
//   O = P V   (MFMA int8) -> per-tensor dyadic -> int8 output (token order)
//
// Constrained Shiftmax needs the exact row maximum before any exponential
// (ShiftExp of x - max cannot be rescaled bit-exactly when the maximum
// changes), so a whole block of score rows is kept in LDS instead of the
// online rescaling used by float attention: R rows x Tw int8 scores (51 KB
// for 32 rows at Tw = 1600).  Because the scores are int8, max - score only
// takes the values 0..254: ShiftExp is one 256-entry table per workgroup,
// looked up once per score; the looked-up values stay in registers for the
// normalization, and S_sum >> s_d is exactly the quotient-remainder
// denominator of Alg. 2.
//
// Per score, the exact integer work is a handful of VALU operations while the
// two matmuls are 256 int8 MFMA ops (about two VALU lane-ops at the chip's
// MFMA:VALU ratio), so this kernel is bound by the VALU work of the exact
// Shiftmax, not by the matrix cores.
#include <map>
#include <mutex>
#include <utility>

#include "ilw_internal.h"

namespace ilw {
namespace {

constexpr int kXcds = 8;  // accelerator complex dies, each with its own L2

// Score requantization, stored biased: the result is q + 128 in [1, 255]
// (q in [-127, 127]).  c = 2^(s-1) + 128 * 2^s, so
//   floor((acc * m + c) / 2^s) = floor((acc * m + 2^(s-1)) / 2^s) + 128,
// exact in 64 bits (|acc| <= 64 * 128 * 128 = 2^20 for a 64-channel head,
// |m| < 2^31 and s <= 54).  The host checks that this value always fits in
// int32 (always true for s >= 32); then the low word of the 64-bit shift is
// the value itself and one clamp finishes the job.
__device__ __forceinline__ int32_t rq_fast(int32_t acc, int32_t mult, int64_t c, int32_t shift) {
  const int64_t v = ((int64_t)acc * mult + c) >> shift;
  return min(max((int32_t)v, 128 + kQmin), 128 + kQmax);
}

// Otherwise (any s up to 62) the accumulator is clamped to [-L, L] first:
// that keeps every saturated result saturated and the shifted value inside
// int32; rnd = 2^(s-1) and the bias is added after the shift.
__device__ __forceinline__ int32_t rq_clamped(int32_t acc, int32_t L, int32_t mult,
                                              int64_t rnd, int32_t shift) {
  acc = min(max(acc, -L), L);
  const int64_t v = ((int64_t)acc * mult + rnd) >> shift;
  return min(max((int32_t)v, kQmin), kQmax) + 128;
}

// Bytes 0 of a, b, c, d packed into one word (a in the low byte).
__device__ __forceinline__ uint32_t pack_bytes(int32_t a, int32_t b, int32_t c, int32_t d) {
  const uint32_t lo = __builtin_amdgcn_perm((uint32_t)b, (uint32_t)a, 0x0c0c0400u);
  const uint32_t hi = __builtin_amdgcn_perm((uint32_t)d, (uint32_t)c, 0x0c0c0400u);
  return lo | (hi << 16);
}

// NW waves per workgroup (4, 8 or 16): keys are split over all waves for the
// scores, rows for the Shiftmax (R / NW rows per wave), and (channel group,
// key range) pairs for P V, whose int32 partial sums are added through LDS.
// MASK says which Shiftmax words may hold no key: 0 any word past the keys
// (whole words, T_w % 4 == 0), 1 any byte past the keys (T_w % 4 != 0),
// 2 only the last word step's (T_w = Twp and (JW - 1) LPR <= Twp / 4),
// 3 only the last two steps' (whole words, JW LPR = Twp / 4 and
// (JW - 2) LPR <= T_w / 4: every step stays inside the row).
template <int R, int LPR, bool NARROW, int MASK, int NW, int JW, bool P3K>
__global__ __launch_bounds__(64 * NW) void attention_kernel(AttnArgs a, int32_t lds_row,
                                                            int32_t clampL, int32_t nrb,
                                                            int64_t ntiles) {
  constexpr bool RAGGED = MASK == 1;
  extern __shared__ __attribute__((aligned(16))) int8_t sS[];  // [R][lds_row]
  __shared__ uint32_t elut[256];
  __shared__ int32_t pmax[NW][R];
  constexpr int KP = NW / 4;  // key ranges of the P V phase
  __shared__ v4i ored[KP > 1 ? (KP - 1) * 4 * (R / 16) * 64 : 1];

  constexpr int NF = R / 16;  // query fragments of 16 rows
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int32_t Tw = a.Tw, Twp = a.Twp;
  // Workgroups go to the 8 XCDs round-robin; XCD x takes the contiguous
  // tiles x * per + min(x, rem) + ..., so the row blocks of one (window,
  // head) share one XCD's L2 for their keys and values.
  const int64_t bid = blockIdx.x;
  const int64_t per = ntiles / kXcds, rem = ntiles % kXcds, xcd = bid % kXcds;
  const int64_t tile = xcd * per + (xcd < rem ? xcd : rem) + bid / kXcds;
  const int64_t hs = tile / nrb;  // bw * H + h
  const int32_t i0 = (int32_t)(tile - hs * nrb) * R;
  const int32_t h = (int32_t)(hs % a.H);
  const int32_t bw = (int32_t)(hs / a.H);  // image * nW + window
  const int64_t slice = (int64_t)bw * a.H + h;
  const int8_t* __restrict__ Q = a.q + slice * Tw * 64;
  const int8_t* __restrict__ K = a.k + slice * Tw * 64;
  const int8_t* __restrict__ Vt = a.vt + slice * 64 * Twp;

  // ShiftExp(-d) for d = 0..254 (entry 255 is never a valid max - score)
  if (tid < 256) elut[tid] = tid < 255 ? (uint32_t)shift_exp(-tid, a.I0, a.k_inter) : 0u;

  // Query fragments (MFMA B operand: columns = query rows).  Rows past the
  // window are clamped to a valid row; their results are never stored.
  // Past the head dimension (32-dim heads) the query fragment is zero, so
  // the unused key bytes there contribute nothing.
  const v4i zero4 = {0, 0, 0, 0};
  v4i qf[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int32_t r = min(i0 + f * 16 + (lane & 15), Tw - 1);
    qf[f] = *(const v4i*)(Q + (int64_t)r * 64 + (lane >> 4) * 16);
    if ((lane >> 4) * 16 >= a.hd) qf[f] = zero4;
  }

  // ---- phase 1: scores.  Waves split the keys in blocks of 16; the key
  // fragment is the A operand, so a lane holds 4 consecutive keys of one row.
  // Scores and row maxima are kept biased (q + 128).
  const v4i zero = {0, 0, 0, 0};
  const int32_t sm = a.score_mult, ss = a.score_shift;
  const int64_t srnd = (int64_t)1 << (ss - 1);
  const int64_t sc = srnd + (a.rq_fast ? (int64_t)128 << ss : 0);  // s <= 54 when fast
  int32_t mx[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) mx[f] = 0;
  const int32_t nkb = (Tw + 15) >> 4;
  const int32_t kc = (lane >> 4) * 4;  // first of this lane's 4 keys in a block
  // The nkf whole 16-key blocks go through a ring of loads from a per-lane
  // base (block kb, wave-uniform, clamped to the last whole block); a
  // partial last block (T_w % 16 != 0) is done on its own afterwards, its
  // keys past the window clamped to the last key.
  const int32_t nkf = Tw >> 4;
  const int8_t* const kbase = K + (lane & 15) * 64 + (lane >> 4) * 16;
  auto kload = [&](int32_t kb) { return *(const v4i*)(kbase + (int64_t)min(kb, nkf - 1) * 1024); };
  auto phase1 = [&](auto fast) {
    // requantize block kb's products, fold them into the row maxima and store
    // them biased as bytes
    auto emit = [&](int32_t kb, const v4i(&sc4)[NF]) {
      const int32_t col = kb * 16 + kc;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        int32_t v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          v[r] = decltype(fast)::value ? rq_fast(sc4[f][r], sm, sc, ss)
                                       : rq_clamped(sc4[f][r], clampL, sm, srnd, ss);
        // keys past the window repeat the last key (clamped rows), so they
        // never raise the maximum
        mx[f] = max(max(mx[f], v[0]), v[1]);
        mx[f] = max(max(mx[f], v[2]), v[3]);
        *(uint32_t*)(sS + (f * 16 + (lane & 15)) * lds_row + col) =
            pack_bytes(v[0], v[1], v[2], v[3]);
      }
    };
    auto products = [&](v4i(&sc4)[NF], const v4i& kf) {
#pragma unroll
      for (int f = 0; f < NF; ++f) sc4[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(kf, qf[f], zero, 0, 0, 0);
    };
    if (nkf < nkb && wave == nkf % NW) {  // the partial last block
      const int32_t key = min(nkf * 16 + (lane & 15), Tw - 1);
      v4i sp[NF];
      products(sp, *(const v4i*)(K + (int64_t)key * 64 + (lane >> 4) * 16));
      emit(nkf, sp);
    }
    if (wave >= nkf) return;
    // A ring of four key fragments in flight: slot u holds block kb + u NW
    // and is reloaded with block kb + 4 NW once its products are issued.
    // Loads past the last block re-read the clamped last key and are never
    // used.  The products of the next block are issued before the current
    // block is requantized, so the matrix core and the vector unit overlap;
    // two product sets alternate.
    v4i kr[4] = {kload(wave), kload(wave + NW), kload(wave + 2 * NW), kload(wave + 3 * NW)};
    v4i s0[NF], s1[NF];
    products(s0, kr[0]);
    kr[0] = kload(wave + 4 * NW);
    int32_t kb = wave;
    // one block: kr slot U + 1 feeds the next block's products; true when kb
    // was the last block
    auto step = [&](auto U, v4i(&cur)[NF], v4i(&nxt)[NF]) {
      constexpr int un = (decltype(U)::value + 1) & 3;
      const bool more = kb + NW < nkf;
      if (more) products(nxt, kr[un]);
      emit(kb, cur);
      if (!more) return true;
      kr[un] = kload(kb + 5 * NW);
      kb += NW;
      return false;
    };
    for (;;) {
      if (step(IntC<0>{}, s0, s1)) break;
      if (step(IntC<1>{}, s1, s0)) break;
      if (step(IntC<2>{}, s0, s1)) break;
      if (step(IntC<3>{}, s1, s0)) break;
    }
  };
  if (a.rq_fast)
    phase1(Flag<true>{});
  else
    phase1(Flag<false>{});
  // row maxima: combine the 4 lanes sharing a row, then the waves
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    mx[f] = max(mx[f], __shfl_xor(mx[f], 16, 64));
    mx[f] = max(mx[f], __shfl_xor(mx[f], 32, 64));
    if (lane < 16) pmax[wave][f * 16 + lane] = mx[f];
  }
  __syncthreads();

  // ---- phase 2: Constrained Shiftmax of each row, in place.  LPR lanes
  // share one row; a lane keeps the ShiftExp values of its elements in
  // registers between the sum and the normalization.
  {
    constexpr int RG = 64 / LPR;   // rows processed together by one wave
    // JW words per lane: Twp / 4 <= JW * LPR (the host picks the smallest
    // JW it has for the window)
    const int sub = lane / LPR, k = lane % LPR;
    const int32_t nword = Twp >> 2;
    const int32_t pcap = (1 << (a.k_out - 1)) - 1;
    const u16x2 pcap2 = {(unsigned short)pcap, (unsigned short)pcap};
    static_assert(R / NW >= RG, "a wave must own at least RG rows");
    for (int rr0 = wave * (R / NW); rr0 < (wave + 1) * (R / NW); rr0 += RG) {
      const int rr = rr0 + sub;
      uint32_t* row = (uint32_t*)(sS + rr * lds_row);
      int32_t m = pmax[0][rr];
#pragma unroll
      for (int w = 1; w < NW; ++w) m = max(m, pmax[w][rr]);
      const uint32_t m4 = (uint32_t)m * 0x01010101u;  // biased maximum per byte
      uint32_t e[JW][4];
      uint64_t sum = 0;
      uint32_t sum32 = 0;
#pragma unroll
      for (int j = 0; j < JW; ++j) {
        const int32_t wd = k + j * LPR;
        // a step that may pass the keys
        const bool tail = MASK == 2 ? j == JW - 1 : (MASK == 3 ? j >= JW - 2 : true);
        const uint32_t word = row[tail && MASK != 3 ? min(wd, nword - 1) : wd];  // inside the row
        // max - score per byte (both biased): every valid byte is >= 0, and a
        // borrow from an invalid (higher) byte never reaches a valid one.
        // Words past the window index table entry 255, which is 0.
        uint32_t d4 = m4 - word;
        if (!RAGGED && tail) d4 = wd * 4 < Tw ? d4 : 0xffffffffu;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          uint32_t ev = elut[(d4 >> (8 * b)) & 255];
          if (RAGGED) ev = wd * 4 + b < Tw ? ev : 0u;
          e[j][b] = ev;
          if (NARROW) sum32 += ev; else sum += ev;
        }
      }
      if (NARROW) sum = sum32;
#pragma unroll
      for (int o = LPR / 2; o > 0; o >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)sum, o, 64);
        const uint32_t hi = __shfl_xor((uint32_t)(sum >> 32), o, 64);
        sum += ((uint64_t)hi << 32) | lo;
      }
      const int32_t sd = a.s_d >= 0 ? a.s_d : calibrate_shift(sum, a.m_p);
      uint64_t sr = sum >> sd;
      sr = sr < 1 ? 1 : (sr > 0x7fffffffull ? 0x7fffffffull : sr);
      const uint32_t F = div_2p31m1((uint32_t)sr);
      // e F < 2^30 2^31: a shift of 61 or more leaves 0, as does 63, so
      // the cap keeps the 64-bit shift defined (large m_p gives s_d up to 41)
      const int32_t sh = min(32 - a.k_out + sd, 63);
      // With sh < 32 and F < 2^sh (the usual case: F is small once s_d > 0,
      // and S_sum >= 2^16 bounds it otherwise), Fs = F 2^(32-sh) fits in 32
      // bits and floor(e F / 2^sh) is the high word of e Fs: one multiply.
      // Taken when every row of the wave qualifies (a uniform branch).
      // Either way the quotient is below 2^k_out <= 2^8 (e F < 2^(32 + s_d)
      // when S_sum >> s_d fits S_R; smaller when S_R is clamped), so the
      // 16-bit clamp-and-pack holds it.
      if (__all(sh < 32 && F < (1u << (sh & 31)))) {
        const uint32_t Fs = F << ((32 - sh) & 31);
#pragma unroll
        for (int j = 0; j < JW; ++j) {
          const int32_t wd = k + j * LPR;
          const uint32_t pw = pack_min_bytes(__umulhi(e[j][0], Fs), __umulhi(e[j][1], Fs),
                                             __umulhi(e[j][2], Fs), __umulhi(e[j][3], Fs), pcap2);
          if ((MASK == 2 && j < JW - 1) || MASK == 3 || wd < nword) row[wd] = pw;  // padding -> 0
        }
      } else {
#pragma unroll
        for (int j = 0; j < JW; ++j) {
          const int32_t wd = k + j * LPR;
          uint32_t p[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) p[b] = (uint32_t)(((uint64_t)e[j][b] * F) >> sh);
          if ((MASK == 2 && j < JW - 1) || MASK == 3 || wd < nword)
            row[wd] = pack_min_bytes(p[0], p[1], p[2], p[3], pcap2);  // padding -> 0
        }
      }
    }
  }
  __syncthreads();

  // ---- phase 3: O = P V.  V^T is the A operand (rows = channels), P^T the
  // B operand (columns = query rows), so a lane holds 4 consecutive channels
  // of one query row.  Two ways to split the work over the waves:
  //  * P3K (4 waves, rows of at least 752 keys): wave w takes the 64-key
  //    blocks w, w + 4, ... for all 64 channels, so P is read from LDS once
  //    per workgroup; the four partial sums of each 16-channel group are then
  //    added through LDS (the score rows, free by then) by the wave that
  //    owns the group (channels 16 w .. 16 w + 15);
  //  * otherwise wave w owns channels 16 (w % 4) .. + 15 over key range
  //    w / 4 (64-key blocks kp, kp + KP, ...), reading all of its key range
  //    of P.
  v4i o[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) o[f] = zero;
  const int cg = P3K ? wave : (wave & 3);
  const int32_t c0 = cg * 16;
  if constexpr (P3K) {
    static_assert(NW == 4, "one 16-channel group per wave");
    v4i og[4][NF];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int f = 0; f < NF; ++f) og[g][f] = zero;
    const int8_t* vrow = Vt + (int64_t)(lane & 15) * Twp + (lane >> 4) * 16;
    const int8_t* prow = sS + (lane & 15) * lds_row + (lane >> 4) * 16;
    const int32_t last = Twp - 64;  // loads past the end re-read the last block
    auto vload4 = [&](v4i(&vf)[4], int32_t j0) {
      const int32_t jj = min(j0, last);
#pragma unroll
      for (int g = 0; g < 4; ++g) vf[g] = *(const v4i*)(vrow + (int64_t)g * 16 * Twp + jj);
    };
    auto pv4 = [&](int32_t j0, const v4i(&vf)[4]) {
      v4i pf[NF];
#pragma unroll
      for (int f = 0; f < NF; ++f) pf[f] = *(const v4i*)(prow + f * 16 * lds_row + j0);
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int f = 0; f < NF; ++f)
          og[g][f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(vf[g], pf[f], og[g][f], 0, 0, 0);
    };
    // the next block's V^T fragments are in flight while this one is used
    v4i va[4], vb[4];
    int32_t j0 = wave * 64;
    vload4(va, j0);
    for (;;) {
      if (j0 >= Twp) break;
      vload4(vb, j0 + 4 * 64);
      pv4(j0, va);
      j0 += 4 * 64;
      if (j0 >= Twp) break;
      vload4(va, j0 + 4 * 64);
      pv4(j0, vb);
      j0 += 4 * 64;
    }
    // partial sums of the other waves' groups to LDS: [wave][g][f][lane]
    __syncthreads();  // every wave is past its reads of P
    v4i* part = (v4i*)sS;
    auto publish = [&](auto G) {
      constexpr int g = decltype(G)::value;
      if (g != wave) {
#pragma unroll
        for (int f = 0; f < NF; ++f) part[((wave * 4 + g) * NF + f) * 64 + lane] = og[g][f];
      } else {
#pragma unroll
        for (int f = 0; f < NF; ++f) o[f] = og[g][f];
      }
    };
    publish(IntC<0>{});
    publish(IntC<1>{});
    publish(IntC<2>{});
    publish(IntC<3>{});
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q == wave) continue;
#pragma unroll
      for (int f = 0; f < NF; ++f) o[f] += part[((q * 4 + wave) * NF + f) * 64 + lane];
    }
  } else {
  const int kp = wave >> 2;
  const int8_t* vrow = Vt + (int64_t)(c0 + (lane & 15)) * Twp + (lane >> 4) * 16;
  const int8_t* prow = sS + (lane & 15) * lds_row + (lane >> 4) * 16;
  const int32_t last = Twp - 64;  // loads past the end re-read the last block
  auto vload = [&](int32_t j0) { return *(const v4i*)(vrow + min(j0, last)); };
  auto pv = [&](int32_t j0, const v4i& vf) {
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const v4i pf = *(const v4i*)(prow + f * 16 * lds_row + j0);
      o[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(vf, pf, o[f], 0, 0, 0);
    }
  };
  // four V^T fragments in flight, as for the keys
  constexpr int32_t SJ = 64 * KP;  // key stride of one wave
  const int32_t j00 = kp * 64;
  v4i v0 = vload(j00), v1 = vload(j00 + SJ), v2 = vload(j00 + 2 * SJ), v3 = vload(j00 + 3 * SJ);
  for (int32_t j0 = j00; j0 < Twp; j0 += 4 * SJ) {
    pv(j0, v0);
    v0 = vload(j0 + 4 * SJ);
    if (j0 + SJ >= Twp) break;
    pv(j0 + SJ, v1);
    v1 = vload(j0 + 5 * SJ);
    if (j0 + 2 * SJ >= Twp) break;
    pv(j0 + 2 * SJ, v2);
    v2 = vload(j0 + 6 * SJ);
    if (j0 + 3 * SJ >= Twp) break;
    pv(j0 + 3 * SJ, v3);
    v3 = vload(j0 + 7 * SJ);
  }
  if (KP > 1) {
    // add the partial sums of the other key ranges into the kp = 0 waves
    if (kp > 0) {
#pragma unroll
      for (int f = 0; f < NF; ++f) ored[(((kp - 1) * 4 + cg) * NF + f) * 64 + lane] = o[f];
    }
    __syncthreads();
    if (kp > 0) return;
#pragma unroll
    for (int q = 0; q < KP - 1; ++q)
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const v4i t = ored[((q * 4 + cg) * NF + f) * 64 + lane];
        o[f] += t;
      }
  }
  }
  const int32_t b_img = bw / a.nW, w = bw % a.nW;
  const int32_t wy = w / a.nwx, wx = w % a.nwx;
  const int32_t c = c0 + (lane >> 4) * 4;
  if (c0 >= a.hd) return;  // channel group past the head dimension
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int32_t i = i0 + f * 16 + (lane & 15);
    if (i >= Tw) continue;
    const int32_t t = (wy * a.win_h + i / a.win_w) * a.grid_w + wx * a.win_w + i % a.win_w;
    uint32_t packed = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      packed |= (uint32_t)(rq(o[f][r], a.pv_mult, a.pv_shift) & 0xff) << (8 * r);
    *(uint32_t*)(a.out + ((int64_t)b_img * a.T + t) * a.D + h * a.hd + c) = packed;
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
  const int32_t h = rem_n >> L.hs, c = rem_n & ((1 << L.hs) - 1);
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

// Dynamic LDS above 64 KB must be allowed per kernel; the attribute is set
// once per (device, kernel) and size high-water mark, under a lock so that
// threads launching on several devices at once all see it set.
hipError_t allow_dynamic_lds(const void* kern, size_t smem) {
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, size_t> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  size_t& have = done[{dev, kern}];
  if (smem <= have) return hipSuccess;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e == hipSuccess) have = smem;
  return e;
}

template <int R, int LPR, bool NARROW, int MASK, int NW, int JW, bool P3K>
hipError_t launch_variant(const AttnArgs& a, int32_t clampL, hipStream_t s) {
  const int32_t lds_row = a.Twp + 16;
  const size_t smem = (size_t)R * lds_row;
  // the split-key P V exchange needs 16 KB per 16 query rows of score rows
  if (P3K && lds_row < 1024) return hipErrorInvalidValue;
  auto kern = attention_kernel<R, LPR, NARROW, MASK, NW, JW, P3K>;
  if (smem > 65536) {
    const hipError_t e = allow_dynamic_lds((const void*)kern, smem);
    if (e != hipSuccess) return e;
  }
  const int32_t nrb = (a.Tw + R - 1) / R;
  const int64_t ntiles = (int64_t)nrb * a.H * a.B * a.nW;
  hipLaunchKernelGGL(kern, dim3((unsigned)ntiles), dim3(64 * NW), smem, s, a, lds_row, clampL,
                     nrb, ntiles);
  return hipGetLastError();
}

template <int R, int LPR, int NW, int JW = 8, bool P3K = false>
hipError_t launch_rows(const AttnArgs& a, int32_t clampL, int64_t emax, hipStream_t s) {
  // A lane sums at most 4 JW ShiftExp values, each at most emax = ShiftExp(0)
  // = I0 * 2^k_inter: 32-bit partial sums are exact while 4 JW emax < 2^32.
  const bool narrow = emax * 4 * JW < ((int64_t)1 << 32);
  int mask = (a.Tw & 3) ? 1 : (a.Tw == a.Twp && (JW - 1) * LPR <= (a.Twp >> 2) ? 2 : 0);
  // exact fit: mask only the last two word steps (the 400-token windows, 3%)
  if (mask == 0 && JW * LPR == (a.Twp >> 2) && (JW - 2) * LPR <= (a.Tw >> 2)) mask = 3;
  if (narrow) {
    if (mask == 3) return launch_variant<R, LPR, true, 3, NW, JW, P3K>(a, clampL, s);
    if (mask == 2) return launch_variant<R, LPR, true, 2, NW, JW, P3K>(a, clampL, s);
    return mask ? launch_variant<R, LPR, true, 1, NW, JW, P3K>(a, clampL, s)
                : launch_variant<R, LPR, true, 0, NW, JW, P3K>(a, clampL, s);
  }
  if (mask == 3) return launch_variant<R, LPR, false, 3, NW, JW, P3K>(a, clampL, s);
  if (mask == 2) return launch_variant<R, LPR, false, 2, NW, JW, P3K>(a, clampL, s);
  return mask ? launch_variant<R, LPR, false, 1, NW, JW, P3K>(a, clampL, s)
              : launch_variant<R, LPR, false, 0, NW, JW, P3K>(a, clampL, s);
}

// The 16-word variants with the smallest word count the window needs: 13
// words cover 1600-token rows over 32 lanes, 14 rows of up to 1792 bytes
// over 32 lanes, 10 the 320-byte padded 300-query rows.
template <int R, int LPR, int NW, bool P3K = false>
hipError_t launch_fit16(const AttnArgs& a, int32_t clampL, int64_t emax, hipStream_t s) {
  const int32_t jw = ((a.Twp >> 2) + LPR - 1) / LPR;
  if (jw <= 10) return launch_rows<R, LPR, NW, 10, P3K>(a, clampL, emax, s);
  if (jw <= 13) return launch_rows<R, LPR, NW, 13, P3K>(a, clampL, emax, s);
  if (jw == 14) return launch_rows<R, LPR, NW, 14, P3K>(a, clampL, emax, s);
  return launch_rows<R, LPR, NW, 16, P3K>(a, clampL, emax, s);
}

template <int R>
hipError_t launch_lpr(const AttnArgs& a, int32_t clampL, int64_t emax, int64_t wgs,
                      hipStream_t s) {
  // Rows per wave: a lane holds JW words (4 JW scores) of its row, and the
  // LPR lanes of a row combine their sums in log2(LPR) shuffle steps.  With
  // 32-row blocks each wave normalizes 8 rows; doing them 4 or 8 (windows)
  // or 2 (long rows) at a time overlaps the rows' serial sum-shuffle-divide
  // chains (measured against one row group of 16 or 64 lanes).
  if (a.Twp <= 512) {
    // 7 words over 16 lanes fit the 448-byte padded 400-token rows exactly;
    // in 32-row blocks that variant needs 60 VGPRs against 95 for 8 lanes of
    // 14 words (two row groups per wave instead of one), which fits more
    // workgroups per CU: the medium encoder 3.9% faster
    if constexpr (R == 32) {
      if ((a.Twp >> 2) <= 7 * 16) return launch_rows<32, 16, 4, 7>(a, clampL, emax, s);
      return launch_fit16<32, 8, 4>(a, clampL, emax, s);
    }
    if ((a.Twp >> 2) <= 7 * 16) return launch_rows<R, 16, 4, 7>(a, clampL, emax, s);
    return launch_rows<R, 16, 4>(a, clampL, emax, s);
  }
  if (a.Twp <= 1024) return launch_rows<R, 32, 4>(a, clampL, emax, s);
  // Long rows: small grids spread a 32-row block over 16 waves so that every
  // SIMD holds several, each wave normalizing its 2 rows together (measured
  // best of 16 or 32 rows over 4, 8 or 16 waves for 1600-token rows at
  // batch 1).
  if (wgs * 4 <= 2048) return launch_fit16<32, 32, 16>(a, clampL, emax, s);
  // (P V split by key blocks over the 4 waves: P read from LDS once)
  if constexpr (R == 32) {
    // Padded rows of more than 1408 and at most 1600 bytes with 32-bit lane
    // sums: 16 lanes per row,
    // 25 words each, so a wave normalizes 4 rows at a time and the per-row
    // work (sum shuffles, shift calibration, reciprocal) is shared by twice
    // the scores: 130 VGPRs, global attention of the 384-wide encoder 5%
    // faster than 32 lanes of 13 words.  (With 64-bit lane sums the
    // variant needs over 200 VGPRs.)
    const int32_t words = a.Twp >> 2;
    if (words > 22 * 16 && words <= 25 * 16 && emax * 4 * 25 < ((int64_t)1 << 32))
      return launch_rows<32, 16, 4, 25, true>(a, clampL, emax, s);
    return launch_fit16<32, 32, 4, true>(a, clampL, emax, s);
  }
  return launch_rows<R, 64, 4>(a, clampL, emax, s);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  // Accumulator clamp for the score requantization: beyond |acc| = L the
  // result saturates (|acc * mult| >= 129 * 2^shift) and the product of the
  // clamped value stays far inside 64 bits.
  const int64_t am = a.score_mult < 0 ? -(int64_t)a.score_mult : (int64_t)a.score_mult;
  int64_t L = am == 0 ? 1 : (129 * ((int64_t)1 << a.score_shift)) / am + 1;
  if (L > ((int64_t)1 << 30)) L = (int64_t)1 << 30;
  const int64_t emax = (int64_t)a.I0 << a.k_inter;  // ShiftExp(0), the largest value
  // The unclamped score form: |acc| <= 2^20 keeps the 64-bit value below
  // 2^62 for s <= 54, and the shifted value (below 2^51 / 2^s + 129) inside
  // int32 for s >= 32, or for smaller s when |m| 2^20 / 2^s is small enough.
  AttnArgs b = a;
  b.rq_fast = a.score_shift <= 54 &&
              (a.score_shift >= 32 || ((am << 20) >> a.score_shift) + 257 < ((int64_t)1 << 31));
  // Fill the chip: fall back to 16-row blocks when 32-row blocks would give
  // fewer than two workgroups per CU.
  const int64_t wg32 = (int64_t)((a.Tw + 31) / 32) * a.H * a.B * a.nW;
  const int64_t wg16 = (int64_t)((a.Tw + 15) / 16) * a.H * a.B * a.nW;
  if (wg32 < 512) return launch_lpr<16>(b, (int32_t)L, emax, wg16, s);
  return launch_lpr<32>(b, (int32_t)L, emax, wg32, s);
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
