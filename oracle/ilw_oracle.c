/*
 * ilw_oracle.c -- CPU oracle for the integer-only I-LW-DETR operators.
 *
 * TEST INFRASTRUCTURE ONLY: the plain, slow, obviously correct reference the
 * GPU library is checked against.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load it; the GPU library never does, and the
 * two share no code.
 *
 * Each function follows one statement of the paper, named at its definition:
 *   Sec. 3.2.1 / eq. (linear_quant)  integer linear layer, dyadic rescale
 *   Sec. 3.2.2                       dyadic multiply-and-shift rescale
 *   Sec. 3.3 (opening paragraph)     I-ViT integer LayerNorm, Newton sqrt
 *   Sec. 3.3.1 (ShiftExp of I-ViT)   ShiftExp, SD-ShiftGELU
 *   Sec. 3.3.2                       Constrained Shiftmax, denominator shift
 *   Sec. 3.1.1                       nearest-neighbour deformable sampling
 * Readings of points the paper leaves open are stated where they are used.
 *
 * Intermediates that could leave 64 bits are computed in __int128; all
 * divisions are written as explicit floor divisions, so nothing here relies
 * on implementation-defined shifts of negative numbers.
 */
#include "ilw_oracle.h"

#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* Symmetric int8 activations without zero point (Sec. 4.4, "8/8/16"):
 * reading: the saturation range is the symmetric [-127, 127]. */
#define ORC_QMAX 127
#define ORC_QMIN (-127)

static void orc_require(int cond, const char* what) {
  if (!cond) {
    fprintf(stderr, "ilw oracle: precondition violated: %s\n", what);
    abort();
  }
}

/* floor(a / b) for b != 0, written out from the definition. */
static __int128 floor_div(__int128 a, __int128 b) {
  __int128 q = a / b; /* C truncates toward zero */
  if ((a % b) != 0 && ((a < 0) != (b < 0))) q -= 1;
  return q;
}

static __int128 pow2(int32_t s) { return (__int128)1 << s; }

int64_t orc_floor_div_pow2(int64_t v, int32_t s) {
  orc_require(s >= 0 && s <= 62, "shift in [0, 62]");
  return (int64_t)floor_div(v, pow2(s));
}

static int32_t sat8(__int128 v) {
  if (v > ORC_QMAX) return ORC_QMAX;
  if (v < ORC_QMIN) return ORC_QMIN;
  return (int32_t)v;
}

/* Dyadic requantization (Sec. 3.2.1, eq. linear_quant: scales applied after
 * the integer accumulation; Sec. 3.2.2: the rescale is an integer dyadic
 * multiply-and-shift).  Reading: round half up, i.e.
 *   y = sat8( floor( (acc * mult + 2^(shift-1)) / 2^shift ) ).            */
int32_t orc_requant(int64_t acc, int32_t mult, int32_t shift) {
  orc_require(shift >= 1 && shift <= 62, "requant shift in [1, 62]");
  __int128 v = (__int128)acc * mult + pow2(shift - 1);
  return sat8(floor_div(v, pow2(shift)));
}

/* Two-input dyadic add onto a common output scale (Sec. 3.2.2: branches are
 * rescaled to one output scale by dyadic multiply-and-shift and summed in
 * integers).  Used for the residual connections of the encoder block. */
int32_t orc_residual(int32_t a, int32_t b, int32_t mult_a, int32_t mult_b,
                     int32_t shift) {
  orc_require(shift >= 1 && shift <= 62, "residual shift in [1, 62]");
  __int128 v = (__int128)a * mult_a + (__int128)b * mult_b + pow2(shift - 1);
  return sat8(floor_div(v, pow2(shift)));
}

/* ceil(a / b) for a >= 0, b >= 1. */
static int64_t ceil_div_nonneg(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* The sigmoid argument of eq. gelu, 1.702 x, as x + x/2 + x/8 + x/16 with
 * floor shifts (Sec. 3.3.1). */
static int64_t gelu_sigmoid_arg(int64_t x) {
  return x + (int64_t)floor_div(x, 2) + (int64_t)floor_div(x, 8) + (int64_t)floor_div(x, 16);
}

/* ShiftExp, the integer exponential of I-ViT that Sec. 3.3.1 and 3.3.2 build
 * on (its steps are spelled out in the appendix, Alg. 1).  For an input
 * I <= 0 at scale S = 1 / I0 it approximates exp(S I) = 2^(-z / I0) with
 * z = -I log2(e):
 *   - log2(e) ~ 1 + 1/2 - 1/16, applied with floor shifts to the negative
 *     input, which for the magnitude a = -I rounds the two fractions up:
 *     z = a + ceil(a / 2) - ceil(a / 16);
 *   - z is capped at k_inter I0 (the exponential is clipped below at
 *     2^-k_inter);
 *   - z = n I0 + f with 0 <= f < I0, so 2^(-z/I0) = 2^-n 2^(-f/I0), and the
 *     fractional power is the chord 1 - f / (2 I0), in units of 1/I0:
 *     I0 - ceil(f / 2);
 *   - the result carries k_inter extra bits: (I0 - ceil(f/2)) 2^(k_inter - n),
 *     at scale S / 2^k_inter. */
int64_t orc_shiftexp(int64_t I, int32_t I0, int32_t k_inter) {
  orc_require(I <= 0, "ShiftExp input must be <= 0");
  orc_require(I0 >= 1, "I0 >= 1");
  orc_require(k_inter >= 1 && k_inter <= 30, "k_inter in [1, 30]");
  const int64_t a = -I;
  int64_t z = a + ceil_div_nonneg(a, 2) - ceil_div_nonneg(a, 16);
  const int64_t z_cap = (int64_t)k_inter * I0;
  if (z > z_cap) z = z_cap;
  const int64_t n = z / I0; /* z >= 0: C division is the floor */
  const int64_t f = z - n * I0;
  orc_require(n >= 0 && n <= k_inter, "whole powers of two in [0, k_inter]");
  const int64_t chord = I0 - ceil_div_nonneg(f, 2);
  return (int64_t)((__int128)chord * pow2(k_inter - (int32_t)n));
}

/* The denominator shift of Constrained Shiftmax (Sec. 3.3.2): the division
 * needs M_req = ceil(log2 S_sum) bits, plus the margin m_p; whatever exceeds
 * the hardware precision M_hw is shifted out of the denominator:
 * s_d = max(M_req + m_p - M_hw, 0). */
int32_t orc_calibrate_shift(int64_t s_sum, int32_t m_p, int32_t M_hw) {
  orc_require(s_sum >= 1, "S_sum >= 1");
  int32_t M_req = 0; /* smallest M with 2^M >= S_sum */
  while (pow2(M_req) < s_sum) M_req++;
  const int32_t excess = M_req + m_p - M_hw;
  return excess > 0 ? excess : 0;
}

/* S_R of Sec. 3.3.2: the exponential sum reduced by s_d bits, accumulated as
 * the quotients of every term by 2^s_d plus the floor of the summed
 * remainders, which the section shows equals floor(S_sum / 2^s_d); the
 * equality is checked here. */
static int64_t reduced_denominator(const int64_t* e, int32_t d, int32_t s_d,
                                   int64_t S_sum) {
  int64_t quotients = 0, remainders = 0;
  for (int32_t i = 0; i < d; i++) {
    const int64_t Qi = (int64_t)floor_div(e[i], pow2(s_d));
    quotients += Qi;
    remainders += e[i] - (int64_t)(Qi * pow2(s_d));
  }
  const int64_t S_R = quotients + (int64_t)floor_div(remainders, pow2(s_d));
  orc_require(S_R == (int64_t)floor_div(S_sum, pow2(s_d)),
              "quotient-remainder sum equals floor(S_sum / 2^s_d)");
  return S_R;
}

/* Constrained Shiftmax over one row (Sec. 3.3.2).  The exponentials are
 * ShiftExp of the scores less the row maximum (I-ViT's Shiftmax input), their
 * sum S_sum sets s_d (or s_d_static >= 0 is used as the calibrated value; the
 * text calibrates one s_d per Shiftmax block, while -1 recomputes it from the
 * row itself), S_R is clamped to [1, 2^31 - 1], F = floor((2^31 - 1) / S_R),
 * and out_i = floor(I_exp_i F / 2^(31 - k_out + 1 + s_d)), the form the
 * section ends with.  Reading: the result is stored as a signed k_out-bit
 * integer, so it is limited to 2^(k_out-1) - 1. */
void orc_shiftmax_row(const int32_t* x, int32_t d, int32_t I0, int32_t k_inter,
                      int32_t k_out, int32_t m_p, int32_t s_d_static,
                      int32_t* out, int64_t* diag) {
  orc_require(d >= 1, "row length >= 1");
  orc_require(k_out >= 2 && k_out <= 16, "k_out in [2, 16]");
  const int32_t M_hw = 31;
  int64_t* e = (int64_t*)malloc(sizeof(int64_t) * (size_t)d);
  orc_require(e != NULL, "allocation");

  int32_t row_max = x[0];
  for (int32_t i = 1; i < d; i++) row_max = x[i] > row_max ? x[i] : row_max;
  int64_t S_sum = 0;
  for (int32_t i = 0; i < d; i++) {
    e[i] = orc_shiftexp((int64_t)x[i] - row_max, I0, k_inter);
    S_sum += e[i];
  }

  const int32_t s_d = s_d_static >= 0 ? s_d_static : orc_calibrate_shift(S_sum, m_p, M_hw);
  /* nothing bounds s_d from above (S_sum < 2^63 and m_p <= 31 keep it below
   * 64); the shifts below are taken in __int128 */
  orc_require(s_d >= 0 && s_d <= 90, "s_d in [0, 90]");

  const int64_t hw_max = 2147483647; /* 2^31 - 1 */
  int64_t S_R = reduced_denominator(e, d, s_d, S_sum);
  S_R = S_R < 1 ? 1 : (S_R > hw_max ? hw_max : S_R);
  const int64_t F = hw_max / S_R; /* both positive: C division is the floor */

  const int32_t out_shift = 31 - k_out + 1 + s_d;
  const int64_t out_cap = (int64_t)pow2(k_out - 1) - 1;
  for (int32_t i = 0; i < d; i++) {
    const __int128 v = floor_div((__int128)e[i] * F, pow2(out_shift));
    out[i] = (int32_t)(v > out_cap ? out_cap : v);
  }
  if (diag) {
    diag[0] = S_sum;
    diag[1] = s_d;
    diag[2] = S_R;
    diag[3] = F;
  }
  free(e);
}

/* I-ViT Shiftmax with a fixed division precision M (Sec. 3.3.2, eq.
 * shiftmax_original): out_i = (floor((2^M - 1) / S_sum) * I_exp_i) >>
 * (M - (k_out - 1)).  Kept as the baseline the constrained form extends. */
void orc_shiftmax_ivit_row(const int32_t* x, int32_t d, int32_t I0,
                           int32_t k_inter, int32_t k_out, int32_t M,
                           int32_t* out) {
  orc_require(d >= 1, "row length >= 1");
  int32_t I_max = x[0];
  for (int32_t i = 1; i < d; i++)
    if (x[i] > I_max) I_max = x[i];
  __int128 S_sum = 0;
  for (int32_t i = 0; i < d; i++)
    S_sum += orc_shiftexp((int64_t)x[i] - I_max, I0, k_inter);
  __int128 factor = floor_div(pow2(M) - 1, S_sum);
  for (int32_t i = 0; i < d; i++) {
    __int128 e = orc_shiftexp((int64_t)x[i] - I_max, I0, k_inter);
    out[i] = (int32_t)floor_div(factor * e, pow2(M - (k_out - 1)));
  }
}

void orc_shiftmax_ivit_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                            int32_t I0, int32_t k_inter, int32_t k_out, int32_t M) {
  orc_require(M >= k_out && M <= 32, "division precision M in [k_out, 32]");
  int32_t* in = (int32_t*)malloc(sizeof(int32_t) * (size_t)cols);
  int32_t* out = (int32_t*)malloc(sizeof(int32_t) * (size_t)cols);
  orc_require(in && out, "allocation");
  for (int64_t r = 0; r < rows; r++) {
    for (int32_t i = 0; i < cols; i++) in[i] = x[r * cols + i];
    orc_shiftmax_ivit_row(in, cols, I0, k_inter, k_out, M, out);
    for (int32_t i = 0; i < cols; i++) {
      orc_require(out[i] >= 0 && out[i] <= 127, "I-ViT Shiftmax output fits int8");
      y[r * cols + i] = (int8_t)out[i];
    }
  }
  free(in);
  free(out);
}

/* ShiftGELU of I-ViT over rows: the vector whose maximum shifts the sigmoid
 * argument is the row (one token's channels).  Reading: the maximum is
 * clamped at 0, which keeps every ShiftExp argument <= 0; a row with no
 * positive I_p then gives exactly SD-ShiftGELU. */
void orc_shiftgelu_ivit_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                             int32_t I0, int32_t k_inter, int32_t k_out,
                             int32_t out_mult, int32_t out_shift) {
  for (int64_t r = 0; r < rows; r++) {
    int64_t max_ip = 0;
    for (int32_t i = 0; i < cols; i++) {
      const int64_t Ip = gelu_sigmoid_arg(x[r * cols + i]);
      if (Ip > max_ip) max_ip = Ip;
    }
    for (int32_t i = 0; i < cols; i++)
      y[r * cols + i] = (int8_t)orc_requant(
          orc_ivit_shiftgelu(x[r * cols + i], (int32_t)max_ip, I0, k_inter, k_out),
          out_mult, out_shift);
  }
}

/* IntDiv, which the SD-ShiftGELU pseudo-code (Alg. 1) uses without defining.  Reading: the I-ViT integer
 * division of eq. shiftmax_original with M = M_hw = 31 applied to one
 * numerator, giving a k_out-bit ratio with scale 2^-(k_out-1):
 *   IntDiv(a, b) = (floor((2^31 - 1) / b) * a) >> (31 - (k_out - 1)).      */
int64_t orc_intdiv(int64_t a, int64_t b, int32_t k_out) {
  orc_require(b >= 1, "IntDiv denominator >= 1");
  orc_require(a >= 0, "IntDiv numerator >= 0");
  __int128 factor = floor_div(pow2(31) - 1, b);
  return (int64_t)floor_div(factor * a, pow2(31 - (k_out - 1)));
}

/* SD-ShiftGELU (Sec. 3.3.1): GELU(x) ~ x sigmoid(z), z = 1.702 x, with the
 * sigmoid taken in the sign-dependent form the section gives:
 *   z >= 0:  1 / (1 + exp(-z)) = exp(0) / (exp(0) + exp(-z)),
 *   z <  0:  exp(z) / (exp(z) + 1) = exp(z) / (exp(z) + exp(0)),
 * so both ShiftExp arguments are <= 0 and each element stands alone.  The
 * ratio goes through IntDiv; returns I_out = x * ratio at scale
 * S_x 2^-(k_out-1). */
int64_t orc_sdshiftgelu(int32_t x, int32_t I0, int32_t k_inter,
                        int32_t k_out) {
  const int64_t z = gelu_sigmoid_arg(x);
  const int64_t e_zero = orc_shiftexp(0, I0, k_inter);
  int64_t numer, other;
  if (z >= 0) {
    numer = e_zero;
    other = orc_shiftexp(-z, I0, k_inter);
  } else {
    numer = orc_shiftexp(z, I0, k_inter);
    other = e_zero;
  }
  return (int64_t)x * orc_intdiv(numer, numer + other, k_out);
}

/* The I-ViT ShiftGELU that SD-ShiftGELU replaces (Sec. 3.3.1): the sigmoid
 * argument is shifted by the vector maximum max_ip (>= 0) of I_p instead of
 * by ReLU(I_p) element by element. */
int64_t orc_ivit_shiftgelu(int32_t x, int32_t max_ip, int32_t I0,
                           int32_t k_inter, int32_t k_out) {
  orc_require(max_ip >= 0, "vector maximum of I_p must be >= 0");
  int64_t I = x;
  int64_t Ip = gelu_sigmoid_arg(I);
  orc_require(Ip <= max_ip, "max_ip is the vector maximum");
  int64_t a = orc_shiftexp(Ip - max_ip, I0, k_inter);
  int64_t a2 = orc_shiftexp(-(int64_t)max_ip, I0, k_inter);
  int64_t Idiv = orc_intdiv(a, a + a2, k_out);
  return I * Idiv;
}

/* Integer square root by Newton's method with a fixed iteration count
 * (Sec. 3.3: I-ViT's LayerNorm, 10 iterations, raised to 20 for the decoder).
 * Reading: the I-BERT/I-ViT form, started from the fixed estimate 2^16 and
 * iterated k <- floor((k + floor(V / k)) / 2) exactly `iters` times.  A fixed
 * start is what makes the iteration count matter.  V == 0 returns 0. */
int64_t orc_isqrt_newton(int64_t V, int32_t iters) {
  orc_require(V >= 0, "V >= 0");
  orc_require(iters >= 1 && iters <= 64, "iterations in [1, 64]");
  if (V == 0) return 0;
  int64_t k = 65536;
  for (int32_t t = 0; t < iters; t++) {
    orc_require(k >= 1, "Newton iterate stays positive for V >= 1");
    k = (int64_t)floor_div((__int128)k + floor_div(V, k), 2);
  }
  return k;
}

/* Integer LayerNorm of one row of C int8 channels (Sec. 3.3: the I-ViT
 * formulation is adopted).  The paper does not restate the formula; reading:
 *   mu  = floor((2*sum(x) + C) / (2*C))            mean, rounded half up
 *   y_i = x_i - mu;  V = sum(y_i^2)
 *   sigma = Newton isqrt of V (iters steps)
 *   F   = floor((2^31 - 1) / sigma);  n_i = floor(y_i * F / 2)
 *         (n_i has scale sqrt(C) / 2^30: it is y_i / std * 2^30 / sqrt(C))
 *   o_i = sat8(requant(n_i + beta_i; mult_i, shift_i))
 * gamma is folded into the (possibly negative) per-channel multiplier and
 * beta is an integer at the scale of n.  A constant row (V == 0) has n = 0. */
void orc_int_layernorm_row(const int8_t* x, int32_t C, const int32_t* beta,
                           const int32_t* mult, const int32_t* shift,
                           int32_t n_q, int32_t iters, int8_t* y,
                           int64_t* diag) {
  orc_require(C >= 1, "C >= 1");
  orc_require(n_q == 1 || n_q == C, "dyadic is per-tensor or per-channel");
  int64_t S = 0;
  for (int32_t i = 0; i < C; i++) S += x[i];
  int64_t mu = (int64_t)floor_div((__int128)2 * S + C, (__int128)2 * C);
  int64_t V = 0;
  for (int32_t i = 0; i < C; i++) {
    int64_t yi = x[i] - mu;
    V += yi * yi;
  }
  int64_t sigma = orc_isqrt_newton(V, iters);
  int64_t F = sigma > 0 ? (int64_t)2147483647 / sigma : 0;
  for (int32_t i = 0; i < C; i++) {
    int64_t yi = x[i] - mu;
    int64_t n = sigma > 0 ? (int64_t)floor_div((__int128)yi * F, 2) : 0;
    int32_t q = n_q == 1 ? 0 : i;
    y[i] = (int8_t)orc_requant(n + beta[i], mult[q], shift[q]);
  }
  if (diag) {
    diag[0] = mu;
    diag[1] = V;
    diag[2] = sigma;
    diag[3] = F;
  }
}

void orc_int_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                       const int32_t* beta, const int32_t* mult,
                       const int32_t* shift, int32_t n_q, int32_t iters) {
  for (int64_t r = 0; r < rows; r++)
    orc_int_layernorm_row(x + r * C, C, beta, mult, shift, n_q, iters,
                          y + r * C, NULL);
}

/* Integer linear layer (Sec. 3.2.1, eq. linear_quant): the multiply-
 * accumulate runs in integers; acc[m][n] = b[n] + sum_k x[m][k] * w[n][k].
 * x is [M, K] and w is [N, K], both row-major. */
void orc_linear_acc(const int8_t* x, const int8_t* w, const int32_t* b,
                    int64_t M, int32_t N, int32_t K, int32_t* acc) {
  for (int64_t m = 0; m < M; m++)
    for (int32_t n = 0; n < N; n++) {
      int64_t s = b ? b[n] : 0;
      for (int32_t k = 0; k < K; k++)
        s += (int32_t)x[m * K + k] * (int32_t)w[(int64_t)n * K + k];
      orc_require(s >= INT32_MIN && s <= INT32_MAX, "accumulator fits int32");
      acc[m * N + n] = (int32_t)s;
    }
}

/* Linear layer followed by the per-channel (weights) dyadic requantization to
 * a per-tensor int8 activation (Sec. 3.2.1). */
void orc_linear(const int8_t* x, const int8_t* w, const int32_t* b, int64_t M,
                int32_t N, int32_t K, const int32_t* mult, const int32_t* shift,
                int32_t n_q, int8_t* y) {
  orc_require(n_q == 1 || n_q == N, "dyadic is per-tensor or per-channel");
  int32_t* acc = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
  orc_require(acc != NULL, "allocation");
  for (int64_t m = 0; m < M; m++) {
    orc_linear_acc(x + m * K, w, b, 1, N, K, acc);
    for (int32_t n = 0; n < N; n++) {
      int32_t q = n_q == 1 ? 0 : n;
      y[m * N + n] = (int8_t)orc_requant(acc[n], mult[q], shift[q]);
    }
  }
  free(acc);
}

/* Scale-preserving split convolution (Sec. 3.2.2): the projector's
 * convolution over concatenated encoder feature maps is split into one
 * convolution per map, so that each map keeps its own activation scale S_b.
 * The int32 partial of branch b has scale S_b * S_w; it is brought to the
 * common scale S_c = max_b S_b by the dyadic m_b / 2^s_b ~ S_b / S_c (an
 * integer multiply-and-shift), and the rescaled partials are added in
 * integers.  Readings: the convolution is pointwise (a linear layer over the
 * tokens of the feature maps); the rescale rounds half up like every dyadic
 * here and does not saturate; the bias is in the common scale. */
void orc_split_conv_sum(int32_t n_branches, const int8_t* const* x,
                        const int32_t* channels, const int8_t* const* w,
                        const int32_t* const* br_mult, const int32_t* const* br_shift,
                        const int32_t* br_nq, const int32_t* bias, int64_t M,
                        int32_t N, int64_t* A) {
  orc_require(n_branches >= 1, "at least one branch");
  for (int64_t m = 0; m < M; m++)
    for (int32_t n = 0; n < N; n++) {
      __int128 total = bias ? bias[n] : 0;
      for (int32_t b = 0; b < n_branches; b++) {
        const int32_t C = channels[b];
        int64_t acc = 0;
        for (int32_t k = 0; k < C; k++)
          acc += (int32_t)x[b][m * C + k] * (int32_t)w[b][(int64_t)n * C + k];
        const int32_t q = br_nq[b] == 1 ? 0 : n;
        const int32_t s = br_shift[b][q];
        orc_require(s >= 1 && s <= 62, "branch rescale shift in [1, 62]");
        total += floor_div((__int128)acc * br_mult[b][q] + pow2(s - 1), pow2(s));
      }
      orc_require(total >= INT64_MIN && total <= INT64_MAX, "sum fits int64");
      A[m * N + n] = (int64_t)total;
    }
}

void orc_split_conv(int32_t n_branches, const int8_t* const* x,
                    const int32_t* channels, const int8_t* const* w,
                    const int32_t* const* br_mult, const int32_t* const* br_shift,
                    const int32_t* br_nq, const int32_t* bias, int64_t M, int32_t N,
                    const int32_t* out_mult, const int32_t* out_shift, int32_t out_nq,
                    int8_t* y) {
  orc_require(out_nq == 1 || out_nq == N, "dyadic is per-tensor or per-channel");
  int64_t* A = (int64_t*)malloc(sizeof(int64_t) * (size_t)N);
  orc_require(A != NULL, "allocation");
  for (int64_t m = 0; m < M; m++) {
    const int8_t* xs[64];
    orc_require(n_branches <= 64, "at most 64 branches");
    for (int32_t b = 0; b < n_branches; b++) xs[b] = x[b] + m * channels[b];
    orc_split_conv_sum(n_branches, xs, channels, w, br_mult, br_shift, br_nq, bias, 1, N,
                       A);
    for (int32_t n = 0; n < N; n++) {
      const int32_t q = out_nq == 1 ? 0 : n;
      y[m * N + n] = (int8_t)orc_requant(A[n], out_mult[q], out_shift[q]);
    }
  }
  free(A);
}

/* Patch embedding (Table mappability: patch embedding is a convolution
 * followed by an add; Sec. 3.2.1: convolutions follow the integer linear
 * formulation with per-channel weight scales).  Readings: the positional
 * embedding is an int8 table at its own scale, added to the requantized
 * convolution output with the same two-input dyadic add as the residuals. */
void orc_patch_embed(const int8_t* img, int32_t B, int32_t C_in, int32_t H, int32_t W,
                     int32_t P, const int8_t* w, const int32_t* bias, const int32_t* mult,
                     const int32_t* shift, int32_t nq, const int8_t* pos, int32_t pos_ma,
                     int32_t pos_mb, int32_t pos_shift, int32_t D, int8_t* y) {
  orc_require(P >= 1 && H % P == 0 && W % P == 0, "the patches tile the image");
  orc_require(nq == 1 || nq == D, "dyadic is per-tensor or per-channel");
  const int32_t gh = H / P, gw = W / P, T = gh * gw, K = C_in * P * P;
  for (int32_t b = 0; b < B; b++)
    for (int32_t py = 0; py < gh; py++)
      for (int32_t px = 0; px < gw; px++) {
        const int32_t t = py * gw + px;
        for (int32_t n = 0; n < D; n++) {
          int64_t acc = bias ? bias[n] : 0;
          for (int32_t c = 0; c < C_in; c++)
            for (int32_t ky = 0; ky < P; ky++)
              for (int32_t kx = 0; kx < P; kx++) {
                const int64_t pix =
                    img[(((int64_t)b * C_in + c) * H + py * P + ky) * W + px * P + kx];
                acc += pix * w[(int64_t)n * K + (c * P + ky) * P + kx];
              }
          orc_require(acc >= INT32_MIN && acc <= INT32_MAX, "accumulator fits int32");
          const int32_t q = nq == 1 ? 0 : n;
          const int32_t v = orc_requant(acc, mult[q], shift[q]);
          y[((int64_t)b * T + t) * D + n] =
              (int8_t)orc_residual(v, pos[(int64_t)t * D + n], pos_ma, pos_mb, pos_shift);
        }
      }
}

void orc_residual_tensor(const int8_t* a, const int8_t* b, int8_t* y,
                         int64_t n, int32_t mult_a, int32_t mult_b,
                         int32_t shift) {
  for (int64_t i = 0; i < n; i++)
    y[i] = (int8_t)orc_residual(a[i], b[i], mult_a, mult_b, shift);
}

void orc_shiftmax_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                       int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                       int32_t s_d_static) {
  int32_t* in = (int32_t*)malloc(sizeof(int32_t) * (size_t)cols);
  int32_t* out = (int32_t*)malloc(sizeof(int32_t) * (size_t)cols);
  orc_require(in && out, "allocation");
  for (int64_t r = 0; r < rows; r++) {
    for (int32_t i = 0; i < cols; i++) in[i] = x[r * cols + i];
    orc_shiftmax_row(in, cols, I0, k_inter, k_out, m_p, s_d_static, out, NULL);
    for (int32_t i = 0; i < cols; i++) y[r * cols + i] = (int8_t)out[i];
  }
  free(in);
  free(out);
}

/* SD-ShiftGELU over a tensor, then the dyadic requantization of I_out to the
 * int8 input of the next linear layer (activations are per-tensor int8,
 * Sec. 3.2.1; the paper's operator itself stops at (I_out, S_out)). */
void orc_sdshiftgelu_tensor(const int8_t* x, int8_t* y, int64_t n, int32_t I0,
                            int32_t k_inter, int32_t k_out, int32_t out_mult,
                            int32_t out_shift) {
  for (int64_t i = 0; i < n; i++)
    y[i] = (int8_t)orc_requant(orc_sdshiftgelu(x[i], I0, k_inter, k_out),
                               out_mult, out_shift);
}

/* Integer multi-head attention of one image (the encoder's MatMul and
 * Softmax operators, Table ablation_study; Sec. 3.2.1 for the matmuls,
 * Sec. 3.3.2 for Shiftmax).  Window attention (LW-DETR mixes window and
 * global attention) partitions the grid_h x grid_w token grid into
 * win_h x win_w windows that attend only inside themselves; global attention
 * is the single window covering the grid.  Per window and head:
 *   S = Q K^T (int32) -> per-tensor dyadic requant -> int8 scores
 *   P = ConstrainedShiftmax(row of S)        (scale 2^-(k_out-1))
 *   O = P V (int32)  -> per-tensor dyadic requant -> int8, heads concatenated */
void orc_attention(const int8_t* qkv, int32_t grid_h, int32_t grid_w,
                   int32_t win_h, int32_t win_w, int32_t D, int32_t heads,
                   int32_t head_dim, int32_t score_mult, int32_t score_shift,
                   int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                   int32_t s_d_static, int32_t pv_mult, int32_t pv_shift,
                   int8_t* out) {
  if (win_h == 0) {
    win_h = grid_h;
    win_w = grid_w;
  }
  orc_require(heads * head_dim == D, "heads * head_dim == dim");
  orc_require(grid_h % win_h == 0 && grid_w % win_w == 0,
              "windows tile the grid");
  int32_t Tw = win_h * win_w;
  int32_t D3 = 3 * D;
  int64_t* tok = (int64_t*)malloc(sizeof(int64_t) * (size_t)Tw);
  int32_t* srow = (int32_t*)malloc(sizeof(int32_t) * (size_t)Tw);
  int32_t* P = (int32_t*)malloc(sizeof(int32_t) * (size_t)Tw * Tw);
  orc_require(tok && srow && P, "allocation");
  for (int32_t wy = 0; wy < grid_h / win_h; wy++)
    for (int32_t wx = 0; wx < grid_w / win_w; wx++) {
      /* token index of each window-local position */
      for (int32_t iy = 0; iy < win_h; iy++)
        for (int32_t ix = 0; ix < win_w; ix++)
          tok[iy * win_w + ix] =
              (int64_t)(wy * win_h + iy) * grid_w + (wx * win_w + ix);
      for (int32_t h = 0; h < heads; h++) {
        int32_t qo = h * head_dim, ko = D + h * head_dim,
                vo = 2 * D + h * head_dim;
        for (int32_t i = 0; i < Tw; i++) {
          for (int32_t j = 0; j < Tw; j++) {
            int64_t s = 0;
            for (int32_t c = 0; c < head_dim; c++)
              s += (int32_t)qkv[tok[i] * D3 + qo + c] *
                   (int32_t)qkv[tok[j] * D3 + ko + c];
            srow[j] = orc_requant(s, score_mult, score_shift);
          }
          orc_shiftmax_row(srow, Tw, I0, k_inter, k_out, m_p, s_d_static,
                           P + (int64_t)i * Tw, NULL);
        }
        for (int32_t i = 0; i < Tw; i++)
          for (int32_t c = 0; c < head_dim; c++) {
            int64_t o = 0;
            for (int32_t j = 0; j < Tw; j++)
              o += (int64_t)P[(int64_t)i * Tw + j] *
                   qkv[tok[j] * D3 + vo + c];
            out[tok[i] * D + qo + c] = (int8_t)orc_requant(o, pv_mult, pv_shift);
          }
      }
    }
  free(tok);
  free(srow);
  free(P);
}

/* One integer encoder block.  The paper lists the encoder's operators
 * (Linear, MatMul, Softmax, GELU, LayerNorm; Table ablation_study) and calls
 * the encoder a plain ViT; reading: the pre-LayerNorm ViT order
 *   h  = LN1(x);  a = Attn(QKV(h));  x1 = Res(proj(a), x)
 *   h2 = LN2(x1); g = rq(SD-ShiftGELU(fc1(h2)));  y = Res(fc2(g), x1)
 * with every tensor between operators an int8 per-tensor activation. */
void orc_block_forward(const orc_block* p, const int8_t* x, int8_t* y,
                       int32_t B, int32_t grid_h, int32_t grid_w,
                       int32_t win_h, int32_t win_w) {
  const int32_t D = p->dim, Hm = p->mlp_dim;
  const int64_t T = (int64_t)grid_h * grid_w;
  int8_t* h = (int8_t*)malloc((size_t)(T * D));
  int8_t* qkv = (int8_t*)malloc((size_t)(T * 3 * D));
  int8_t* att = (int8_t*)malloc((size_t)(T * D));
  int8_t* pr = (int8_t*)malloc((size_t)(T * D));
  int8_t* x1 = (int8_t*)malloc((size_t)(T * D));
  int8_t* f1 = (int8_t*)malloc((size_t)(T * Hm));
  int8_t* g = (int8_t*)malloc((size_t)(T * Hm));
  int8_t* f2 = (int8_t*)malloc((size_t)(T * D));
  orc_require(h && qkv && att && pr && x1 && f1 && g && f2, "allocation");
  for (int32_t b = 0; b < B; b++) {
    const int8_t* xb = x + (int64_t)b * T * D;
    int8_t* yb = y + (int64_t)b * T * D;
    orc_int_layernorm(xb, h, T, D, p->ln1_beta, p->ln1_mult, p->ln1_shift,
                      p->ln1_nq, p->ln_iters);
    orc_linear(h, p->w_qkv, p->b_qkv, T, 3 * D, D, p->qkv_mult, p->qkv_shift,
               p->qkv_nq, qkv);
    orc_attention(qkv, grid_h, grid_w, win_h, win_w, D, p->heads, p->head_dim,
                  p->score_mult, p->score_shift, p->smax_I0, p->smax_k_inter,
                  p->smax_k_out, p->smax_m_p, p->smax_s_d, p->pv_mult,
                  p->pv_shift, att);
    orc_linear(att, p->w_proj, p->b_proj, T, D, D, p->proj_mult,
               p->proj_shift, p->proj_nq, pr);
    orc_residual_tensor(pr, xb, x1, T * D, p->res1_mult_a, p->res1_mult_b,
                        p->res1_shift);
    orc_int_layernorm(x1, h, T, D, p->ln2_beta, p->ln2_mult, p->ln2_shift,
                      p->ln2_nq, p->ln_iters);
    orc_linear(h, p->w_fc1, p->b_fc1, T, Hm, D, p->fc1_mult, p->fc1_shift,
               p->fc1_nq, f1);
    orc_sdshiftgelu_tensor(f1, g, T * Hm, p->gelu_I0, p->gelu_k_inter,
                           p->gelu_k_out, p->gelu_mult, p->gelu_shift);
    orc_linear(g, p->w_fc2, p->b_fc2, T, D, Hm, p->fc2_mult, p->fc2_shift,
               p->fc2_nq, f2);
    orc_residual_tensor(f2, x1, yb, T * D, p->res2_mult_a, p->res2_mult_b,
                        p->res2_shift);
  }
  free(h);
  free(qkv);
  free(att);
  free(pr);
  free(x1);
  free(f1);
  free(g);
  free(f2);
}

/* Nearest-neighbour deformable sampling location (Sec. 3.1.1: bilinear
 * interpolation is replaced by taking the nearest grid point).  Reading of
 * the fixed-point arithmetic, which the paper does not give: the reference
 * point is Q16 in [0, 1) of the map, offsets are Q8 pixels of this level;
 *   X = floor(ref_x * W / 2^8) + off_x       (Q8 pixel coordinate)
 *   ix = floor(X / 2^8)                      (pixel whose cell holds X)
 * which is the nearest pixel centre under the half-pixel convention.  A
 * sample outside the map contributes nothing (zero padding). */
/* Sampling location in Q8 pixels of a W x H level (pixel i spans
 * [256 i, 256 (i+1)), its centre at 256 i + 128).
 * Reference point (ref_dims 2: r = (x, y), Q16 fractions of the map): the
 * reference lands at floor(x W / 2^8) and the offset is added in Q8 pixels.
 * Reference box (ref_dims 4: r = (cx, cy, w, h), Q16 fractions): the offset
 * is in units of the box, as in the deformable decoder with box references,
 * location = c + (off / 2^8) / P * size / 2 as a fraction of the map; one
 * floor of the exact value in Q8 pixels:
 *   X = floor((cx * 2^9 * P + off_x * w) * W / (2^17 * P)). */
static void deform_location(const int32_t* r, int32_t ref_dims, int32_t off_x,
                            int32_t off_y, int32_t H, int32_t W, int32_t P,
                            int64_t* X, int64_t* Y) {
  if (ref_dims == 2) {
    *X = (int64_t)floor_div((__int128)r[0] * W, 256) + off_x;
    *Y = (int64_t)floor_div((__int128)r[1] * H, 256) + off_y;
  } else {
    const __int128 den = (__int128)131072 * P;
    *X = (int64_t)floor_div(((__int128)r[0] * 512 * P + (__int128)off_x * r[2]) * W, den);
    *Y = (int64_t)floor_div(((__int128)r[1] * 512 * P + (__int128)off_y * r[3]) * H, den);
  }
}

static int64_t nearest_index(int64_t X, int64_t Y, int32_t H, int32_t W) {
  int64_t ix = (int64_t)floor_div(X, 256);
  int64_t iy = (int64_t)floor_div(Y, 256);
  if (ix < 0 || ix >= W || iy < 0 || iy >= H) return -1;
  return iy * W + ix;
}

int64_t orc_deform_nearest_index(int32_t ref_x, int32_t ref_y, int32_t off_x,
                                 int32_t off_y, int32_t H, int32_t W) {
  const int32_t r[2] = {ref_x, ref_y};
  int64_t X, Y;
  deform_location(r, 2, off_x, off_y, H, W, 1, &X, &Y);
  return nearest_index(X, Y, H, W);
}

int64_t orc_deform_box_nearest_index(int32_t cx, int32_t cy, int32_t w, int32_t h,
                                     int32_t off_x, int32_t off_y, int32_t H, int32_t W,
                                     int32_t P) {
  const int32_t r[4] = {cx, cy, w, h};
  int64_t X, Y;
  deform_location(r, 4, off_x, off_y, H, W, P, &X, &Y);
  return nearest_index(X, Y, H, W);
}

/* Multi-scale deformable attention core (Sec. 3.1.1 with the decoder's
 * Softmax as Constrained Shiftmax, Sec. 3.3.2):
 *   value  int8  [B, S_total, heads, head_dim]  (levels stacked, level_start)
 *   ref    int32 [B, Q, ref_dims]               Q16 fractions of the map:
 *          points (x, y) or boxes (cx, cy, w, h)
 *   offsets int16 [B, Q, heads, L, P, 2]         (x, y): Q8 pixels for points,
 *          Q8 units of size / (2 P) for boxes (deform_location)
 *   logits int8  [B, Q, heads, L*P]  -> P = ConstrainedShiftmax per (b,q,h)
 *   out    int8  [B, Q, heads*head_dim] = sat8(rq(sum P * sampled value))
 * mode 0: nearest sampling (the paper's).  mode 1: a fixed-point bilinear
 * variant (Q8 weights on the half-pixel grid, corners outside contribute 0,
 * the 2^16 weight scale removed by 16 extra bits of the output shift). */
void orc_deform_attn(const int8_t* value, const int32_t* level_hw,
                     const int32_t* level_start, int32_t L, int32_t P,
                     const int32_t* ref, const int16_t* offsets,
                     const int8_t* logits, int8_t* out, int32_t B, int32_t Q,
                     int32_t heads, int32_t head_dim, int32_t S_total,
                     int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                     int32_t s_d_static, int32_t out_mult, int32_t out_shift,
                     int32_t mode, int32_t ref_dims) {
  orc_require(mode == 0 || mode == 1, "mode is 0 (nearest) or 1 (bilinear)");
  orc_require(ref_dims == 2 || ref_dims == 4, "references are points (2) or boxes (4)");
  const int32_t LP = L * P;
  int32_t* lg = (int32_t*)malloc(sizeof(int32_t) * (size_t)LP);
  int32_t* pw = (int32_t*)malloc(sizeof(int32_t) * (size_t)LP);
  __int128* acc = (__int128*)malloc(sizeof(__int128) * (size_t)head_dim);
  orc_require(lg && pw && acc, "allocation");
  for (int32_t b = 0; b < B; b++)
    for (int32_t q = 0; q < Q; q++)
      for (int32_t h = 0; h < heads; h++) {
        int64_t bqh = ((int64_t)b * Q + q) * heads + h;
        for (int32_t i = 0; i < LP; i++) lg[i] = logits[bqh * LP + i];
        orc_shiftmax_row(lg, LP, I0, k_inter, k_out, m_p, s_d_static, pw,
                         NULL);
        for (int32_t c = 0; c < head_dim; c++) acc[c] = 0;
        const int32_t* r = ref + ((int64_t)b * Q + q) * ref_dims;
        for (int32_t l = 0; l < L; l++) {
          int32_t Hl = level_hw[2 * l + 0], Wl = level_hw[2 * l + 1];
          for (int32_t pt = 0; pt < P; pt++) {
            int64_t oidx = ((bqh * L + l) * P + pt) * 2;
            int32_t ox = offsets[oidx + 0], oy = offsets[oidx + 1];
            int32_t wgt = pw[l * P + pt];
            int64_t X0, Y0;
            deform_location(r, ref_dims, ox, oy, Hl, Wl, P, &X0, &Y0);
            if (mode == 0) {
              int64_t idx = nearest_index(X0, Y0, Hl, Wl);
              if (idx < 0) continue;
              int64_t row = ((int64_t)b * S_total + level_start[l] + idx) *
                                heads + h;
              for (int32_t c = 0; c < head_dim; c++)
                acc[c] += (__int128)wgt * value[row * head_dim + c];
            } else {
              /* half-pixel grid: pixel centres sit at X = 256*i + 128 */
              int64_t X = X0 - 128, Y = Y0 - 128;
              int64_t x0 = (int64_t)floor_div(X, 256), fx = X - 256 * x0;
              int64_t y0 = (int64_t)floor_div(Y, 256), fy = Y - 256 * y0;
              for (int32_t dy = 0; dy < 2; dy++)
                for (int32_t dx = 0; dx < 2; dx++) {
                  int64_t xi = x0 + dx, yi = y0 + dy;
                  if (xi < 0 || xi >= Wl || yi < 0 || yi >= Hl) continue;
                  int64_t w = (dx ? fx : 256 - fx) * (dy ? fy : 256 - fy);
                  int64_t row = ((int64_t)b * S_total + level_start[l] +
                                 yi * Wl + xi) * heads + h;
                  for (int32_t c = 0; c < head_dim; c++)
                    acc[c] += (__int128)wgt * w * value[row * head_dim + c];
                }
            }
          }
        }
        int32_t sh = mode == 0 ? out_shift : out_shift + 16;
        for (int32_t c = 0; c < head_dim; c++) {
          orc_require(acc[c] >= INT64_MIN && acc[c] <= INT64_MAX,
                      "sampling accumulator fits int64");
          out[bqh * head_dim + c] = (int8_t)orc_requant((int64_t)acc[c],
                                                        out_mult, sh);
        }
      }
  free(lg);
  free(pw);
  free(acc);
}

/* Decoder layer (see the header).  Readings: post-norm sub-blocks as in the
 * deformable decoder LW-DETR uses; the positional queries are already part
 * of tgt; the offset linear yields int8 offsets in 1/16 pixel (a +-8 pixel
 * range at 8 bits), widened to the sampler's Q8 by a factor 16; the sampler's
 * Shiftmax uses k_inter = 16, k_out = 8, m_p = 4. */
void orc_decoder_forward(const orc_decoder* p, const int8_t* tgt, const int8_t* memory,
                         const int32_t* ref, const int32_t* level_hw,
                         const int32_t* level_start, int32_t B, int32_t Q, int32_t S,
                         int8_t* y) {
  const int32_t D = p->dim, H = p->heads, F = p->ffn_dim, L = p->levels, P = p->points;
  orc_require(D % H == 0, "dim is a multiple of heads");
  const int32_t hd = D / H, NO = H * L * P * 2, NW = H * L * P;
  const int64_t MQ = (int64_t)B * Q, MS = (int64_t)B * S;
  int8_t* qkv = (int8_t*)malloc((size_t)(Q * 3 * D));
  int8_t* att = (int8_t*)malloc((size_t)(MQ * D));
  int8_t* tmp = (int8_t*)malloc((size_t)(MQ * (F > D ? F : D)));
  int8_t* x = (int8_t*)malloc((size_t)(MQ * D));
  int8_t* t1 = (int8_t*)malloc((size_t)(MQ * D));
  int8_t* t2 = (int8_t*)malloc((size_t)(MQ * D));
  int8_t* v = (int8_t*)malloc((size_t)(MS * D));
  int8_t* off8 = (int8_t*)malloc((size_t)(MQ * NO));
  int16_t* off = (int16_t*)malloc(sizeof(int16_t) * (size_t)(MQ * NO));
  int8_t* lg = (int8_t*)malloc((size_t)(MQ * NW));
  int8_t* smp = (int8_t*)malloc((size_t)(MQ * D));
  int8_t* g = (int8_t*)malloc((size_t)(MQ * F));
  orc_require(qkv && att && tmp && x && t1 && t2 && v && off8 && off && lg && smp && g,
              "allocation");
  /* self-attention: one global window of Q tokens per image */
  for (int32_t b = 0; b < B; b++) {
    orc_linear(tgt + (int64_t)b * Q * D, p->w_qkv, p->b_qkv, Q, 3 * D, D, p->qkv_mult,
               p->qkv_shift, p->qkv_nq, qkv);
    orc_attention(qkv, 1, Q, 0, 0, D, H, hd, p->score_mult, p->score_shift, p->smax_I0,
                  p->smax_k_inter, p->smax_k_out, p->smax_m_p, p->smax_s_d, p->pv_mult,
                  p->pv_shift, att + (int64_t)b * Q * D);
  }
  orc_linear(att, p->w_o, p->b_o, MQ, D, D, p->o_mult, p->o_shift, p->o_nq, tmp);
  orc_residual_tensor(tmp, tgt, x, MQ * D, p->res1_mult_a, p->res1_mult_b, p->res1_shift);
  orc_int_layernorm(x, t1, MQ, D, p->ln1_beta, p->ln1_mult, p->ln1_shift, p->ln1_nq,
                    p->ln_iters);
  /* cross-attention: deformable sampling of the projected encoder maps */
  orc_linear(memory, p->w_val, p->b_val, MS, D, D, p->val_mult, p->val_shift, p->val_nq, v);
  orc_linear(t1, p->w_off, p->b_off, MQ, NO, D, p->off_mult, p->off_shift, p->off_nq, off8);
  for (int64_t i = 0; i < MQ * NO; i++) off[i] = (int16_t)(off8[i] * 16);
  orc_linear(t1, p->w_attw, p->b_attw, MQ, NW, D, p->attw_mult, p->attw_shift, p->attw_nq,
             lg);
  orc_deform_attn(v, level_hw, level_start, L, P, ref, off, lg, smp, B, Q, H, hd, S,
                  p->da_I0, 16, 8, 4, p->da_s_d, p->da_out_mult, p->da_out_shift,
                  p->da_mode, p->ref_dims);
  orc_linear(smp, p->w_co, p->b_co, MQ, D, D, p->co_mult, p->co_shift, p->co_nq, tmp);
  orc_residual_tensor(tmp, t1, x, MQ * D, p->res2_mult_a, p->res2_mult_b, p->res2_shift);
  orc_int_layernorm(x, t2, MQ, D, p->ln2_beta, p->ln2_mult, p->ln2_shift, p->ln2_nq,
                    p->ln_iters);
  /* FFN */
  orc_linear(t2, p->w_fc1, p->b_fc1, MQ, F, D, p->fc1_mult, p->fc1_shift, p->fc1_nq, tmp);
  orc_sdshiftgelu_tensor(tmp, g, MQ * F, p->gelu_I0, p->gelu_k_inter, p->gelu_k_out,
                         p->gelu_mult, p->gelu_shift);
  orc_linear(g, p->w_fc2, p->b_fc2, MQ, D, F, p->fc2_mult, p->fc2_shift, p->fc2_nq, tmp);
  orc_residual_tensor(tmp, t2, x, MQ * D, p->res3_mult_a, p->res3_mult_b, p->res3_shift);
  orc_int_layernorm(x, y, MQ, D, p->ln3_beta, p->ln3_mult, p->ln3_shift, p->ln3_nq,
                    p->ln_iters);
  free(qkv);
  free(att);
  free(tmp);
  free(x);
  free(t1);
  free(t2);
  free(v);
  free(off8);
  free(off);
  free(lg);
  free(smp);
  free(g);
}
