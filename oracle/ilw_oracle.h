/*
 * ilw_oracle.h -- CPU oracle for the integer-only I-LW-DETR operators.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * reference that the GPU path is checked against.  Only the test-suite, the
 * smoke check and the benchmark's CPU-baseline leg may load it.  It shares no
 * code, header, table or constant with the GPU library, and the GPU library
 * never calls it.
 *
 * Every function follows one statement of the paper ("Enabling Fully
 * Integer-Only Inference for Lightweight Detection Transformers"): the
 * section, equation or algorithm is named at each definition.  Where the paper
 * leaves a detail open (rounding mode, saturation range, IntDiv, the integer
 * LayerNorm formula, block order, sampling arithmetic), the reading taken is
 * stated at the definition.
 *
 * All arithmetic is integer.  Intermediates that may exceed 64 bits are done
 * in __int128 so that no overflow reasoning is needed to trust the oracle.
 */
#ifndef ILW_ORACLE_H
#define ILW_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- scalar building blocks -------------------------------------------- */
int64_t orc_floor_div_pow2(int64_t v, int32_t s);
int32_t orc_requant(int64_t acc, int32_t mult, int32_t shift);
int32_t orc_residual(int32_t a, int32_t b, int32_t mult_a, int32_t mult_b,
                     int32_t shift);
int64_t orc_shiftexp(int64_t I, int32_t I0, int32_t k_inter);
int32_t orc_calibrate_shift(int64_t s_sum, int32_t m_p, int32_t M_hw);
int64_t orc_intdiv(int64_t a, int64_t b, int32_t k_out);
int64_t orc_sdshiftgelu(int32_t x, int32_t I0, int32_t k_inter, int32_t k_out);
int64_t orc_ivit_shiftgelu(int32_t x, int32_t max_ip, int32_t I0,
                           int32_t k_inter, int32_t k_out);
int64_t orc_isqrt_newton(int64_t V, int32_t iters);

/* ---- row / tensor operators -------------------------------------------- */
/* diag (may be NULL) receives {S_sum, s_d, S_R, F}. */
void orc_shiftmax_row(const int32_t* x, int32_t d, int32_t I0, int32_t k_inter,
                      int32_t k_out, int32_t m_p, int32_t s_d_static,
                      int32_t* out, int64_t* diag);
void orc_shiftmax_ivit_row(const int32_t* x, int32_t d, int32_t I0,
                           int32_t k_inter, int32_t k_out, int32_t M,
                           int32_t* out);
void orc_shiftmax_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                       int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                       int32_t s_d_static);
/* I-ViT baselines over rows of int8 (the forms the paper's operators
 * replace): Shiftmax with a fixed division precision M (eq.
 * shiftmax_original), and ShiftGELU shifted by the row maximum of I_p
 * (clamped at 0), requantized to int8 like SD-ShiftGELU. */
void orc_shiftmax_ivit_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                            int32_t I0, int32_t k_inter, int32_t k_out, int32_t M);
void orc_shiftgelu_ivit_rows(const int8_t* x, int8_t* y, int64_t rows, int32_t cols,
                             int32_t I0, int32_t k_inter, int32_t k_out,
                             int32_t out_mult, int32_t out_shift);
void orc_sdshiftgelu_tensor(const int8_t* x, int8_t* y, int64_t n, int32_t I0,
                            int32_t k_inter, int32_t k_out, int32_t out_mult,
                            int32_t out_shift);
/* diag (may be NULL) receives {mean, V, sigma, F} for the row. */
void orc_int_layernorm_row(const int8_t* x, int32_t C, const int32_t* beta,
                           const int32_t* mult, const int32_t* shift,
                           int32_t n_q, int32_t iters, int8_t* y,
                           int64_t* diag);
void orc_int_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                       const int32_t* beta, const int32_t* mult,
                       const int32_t* shift, int32_t n_q, int32_t iters);
void orc_linear_acc(const int8_t* x, const int8_t* w, const int32_t* b,
                    int64_t M, int32_t N, int32_t K, int32_t* acc);
void orc_linear(const int8_t* x, const int8_t* w, const int32_t* b, int64_t M,
                int32_t N, int32_t K, const int32_t* mult, const int32_t* shift,
                int32_t n_q, int8_t* y);
void orc_residual_tensor(const int8_t* a, const int8_t* b, int8_t* y,
                         int64_t n, int32_t mult_a, int32_t mult_b,
                         int32_t shift);

/* Scale-preserving split convolution of the projector (Sec. 3.2.2, Fig.
 * projector_split_conv), pointwise: for each branch b (one encoder feature
 * map with its own activation scale), acc_b = x_b W_b^T over its C_b
 * channels; r_b = floor((acc_b * m_b + 2^(s_b - 1)) / 2^s_b) rescales the
 * partial to the common scale (no saturation); A = bias + sum_b r_b; the
 * output is y = sat8(rq(A; out)).  br_mult[b] / br_shift[b] hold br_nq[b]
 * entries (1 or N).  orc_split_conv_sum returns A (int64, [M, N]). */
void orc_split_conv_sum(int32_t n_branches, const int8_t* const* x,
                        const int32_t* channels, const int8_t* const* w,
                        const int32_t* const* br_mult, const int32_t* const* br_shift,
                        const int32_t* br_nq, const int32_t* bias, int64_t M,
                        int32_t N, int64_t* A);
void orc_split_conv(int32_t n_branches, const int8_t* const* x,
                    const int32_t* channels, const int8_t* const* w,
                    const int32_t* const* br_mult, const int32_t* const* br_shift,
                    const int32_t* br_nq, const int32_t* bias, int64_t M, int32_t N,
                    const int32_t* out_mult, const int32_t* out_shift, int32_t out_nq,
                    int8_t* y);

/* Patch embedding, the encoder's input layer (Table mappability: a
 * convolution and an add): a P x P stride-P convolution of the int8 image
 * [B, C_in, H, W] with weights [D, C_in * P * P] ((c, ky, kx) order), per-channel
 * requantization to int8, then the int8 positional embedding pos [T, D]
 * added with the two-input dyadic add.  Tokens are row-major over the
 * (H/P) x (W/P) patch grid: y [B, T, D]. */
void orc_patch_embed(const int8_t* img, int32_t B, int32_t C_in, int32_t H, int32_t W,
                     int32_t P, const int8_t* w, const int32_t* bias, const int32_t* mult,
                     const int32_t* shift, int32_t nq, const int8_t* pos, int32_t pos_ma,
                     int32_t pos_mb, int32_t pos_shift, int32_t D, int8_t* y);

/* One decoder layer (LW-DETR's deformable decoder made integer: Sec. 3.1.1
 * nearest sampling, Sec. 3.3.2 Constrained Shiftmax, Sec. 3.3 I-LayerNorm
 * with 20 Newton steps).  Post-norm:
 *   t1 = LN1(Res(tgt, o(Attn(QKV(tgt)))))          self-attention, global over Q
 *   v  = val(memory);  off = 16 * offl(t1);  w = attw(t1)
 *   t2 = LN2(Res(t1, co(Deform(v, ref, off, w))))  cross-attention
 *   y  = LN3(Res(t2, fc2(GELU(fc1(t2)))))          FFN
 * All pointers are host memory.  head_dim = dim / heads. */
typedef struct {
  int32_t dim, heads, ffn_dim, levels, points, ln_iters;
  const int8_t* w_qkv; const int32_t* b_qkv; const int32_t* qkv_mult;
  const int32_t* qkv_shift; int32_t qkv_nq;
  int32_t score_mult, score_shift, smax_I0, smax_k_inter, smax_k_out, smax_m_p,
      smax_s_d, pv_mult, pv_shift;
  const int8_t* w_o; const int32_t* b_o; const int32_t* o_mult;
  const int32_t* o_shift; int32_t o_nq;
  int32_t res1_mult_a, res1_mult_b, res1_shift;
  const int32_t* ln1_beta; const int32_t* ln1_mult; const int32_t* ln1_shift;
  int32_t ln1_nq;
  const int8_t* w_val; const int32_t* b_val; const int32_t* val_mult;
  const int32_t* val_shift; int32_t val_nq;
  const int8_t* w_off; const int32_t* b_off; const int32_t* off_mult;
  const int32_t* off_shift; int32_t off_nq;
  const int8_t* w_attw; const int32_t* b_attw; const int32_t* attw_mult;
  const int32_t* attw_shift; int32_t attw_nq;
  int32_t da_I0, da_s_d, da_out_mult, da_out_shift, da_mode;
  int32_t ref_dims;  /* 2: reference points (x, y); 4: reference boxes (cx, cy, w, h) */
  const int8_t* w_co; const int32_t* b_co; const int32_t* co_mult;
  const int32_t* co_shift; int32_t co_nq;
  int32_t res2_mult_a, res2_mult_b, res2_shift;
  const int32_t* ln2_beta; const int32_t* ln2_mult; const int32_t* ln2_shift;
  int32_t ln2_nq;
  const int8_t* w_fc1; const int32_t* b_fc1; const int32_t* fc1_mult;
  const int32_t* fc1_shift; int32_t fc1_nq;
  int32_t gelu_I0, gelu_k_inter, gelu_k_out, gelu_mult, gelu_shift;
  const int8_t* w_fc2; const int32_t* b_fc2; const int32_t* fc2_mult;
  const int32_t* fc2_shift; int32_t fc2_nq;
  int32_t res3_mult_a, res3_mult_b, res3_shift;
  const int32_t* ln3_beta; const int32_t* ln3_mult; const int32_t* ln3_shift;
  int32_t ln3_nq;
} orc_decoder;

void orc_decoder_forward(const orc_decoder* p, const int8_t* tgt, const int8_t* memory,
                         const int32_t* ref, const int32_t* level_hw,
                         const int32_t* level_start, int32_t B, int32_t Q, int32_t S,
                         int8_t* y);

/* Integer attention of one image: qkv is the int8 [T, 3*D] QKV output
 * (q | k | v, head-major inside each part), out is int8 [T, D]. */
void orc_attention(const int8_t* qkv, int32_t grid_h, int32_t grid_w,
                   int32_t win_h, int32_t win_w, int32_t D, int32_t heads,
                   int32_t head_dim, int32_t score_mult, int32_t score_shift,
                   int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                   int32_t s_d_static, int32_t pv_mult, int32_t pv_shift,
                   int8_t* out);

/* Parameters of one integer encoder block, host arrays. */
typedef struct {
  int32_t dim, heads, head_dim, mlp_dim, ln_iters;
  const int32_t* ln1_beta; const int32_t* ln1_mult; const int32_t* ln1_shift;
  int32_t ln1_nq;
  const int8_t* w_qkv; const int32_t* b_qkv;
  const int32_t* qkv_mult; const int32_t* qkv_shift; int32_t qkv_nq;
  int32_t score_mult, score_shift;
  int32_t smax_I0, smax_k_inter, smax_k_out, smax_m_p, smax_s_d;
  int32_t pv_mult, pv_shift;
  const int8_t* w_proj; const int32_t* b_proj;
  const int32_t* proj_mult; const int32_t* proj_shift; int32_t proj_nq;
  int32_t res1_mult_a, res1_mult_b, res1_shift;
  const int32_t* ln2_beta; const int32_t* ln2_mult; const int32_t* ln2_shift;
  int32_t ln2_nq;
  const int8_t* w_fc1; const int32_t* b_fc1;
  const int32_t* fc1_mult; const int32_t* fc1_shift; int32_t fc1_nq;
  int32_t gelu_I0, gelu_k_inter, gelu_k_out, gelu_mult, gelu_shift;
  const int8_t* w_fc2; const int32_t* b_fc2;
  const int32_t* fc2_mult; const int32_t* fc2_shift; int32_t fc2_nq;
  int32_t res2_mult_a, res2_mult_b, res2_shift;
} orc_block;

/* x, y int8 [B, grid_h*grid_w, dim]; win_h == 0 means global attention. */
void orc_block_forward(const orc_block* p, const int8_t* x, int8_t* y,
                       int32_t B, int32_t grid_h, int32_t grid_w,
                       int32_t win_h, int32_t win_w);

/* Deformable sampling location of one sample: returns the flat pixel index
 * y*W + x inside the level, or -1 when the sample falls outside the map.
 * Point reference (x, y), offsets in Q8 pixels; box reference (cx, cy, w, h),
 * offsets in Q8 units of size / (2 P) (see orc_deform_attn). */
int64_t orc_deform_nearest_index(int32_t ref_x, int32_t ref_y, int32_t off_x,
                                 int32_t off_y, int32_t H, int32_t W);
int64_t orc_deform_box_nearest_index(int32_t cx, int32_t cy, int32_t w, int32_t h,
                                     int32_t off_x, int32_t off_y, int32_t H, int32_t W,
                                     int32_t P);
void orc_deform_attn(const int8_t* value, const int32_t* level_hw,
                     const int32_t* level_start, int32_t L, int32_t P,
                     const int32_t* ref, const int16_t* offsets,
                     const int8_t* logits, int8_t* out, int32_t B, int32_t Q,
                     int32_t heads, int32_t head_dim, int32_t S_total,
                     int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                     int32_t s_d_static, int32_t out_mult, int32_t out_shift,
                     int32_t mode, int32_t ref_dims);

#ifdef __cplusplus
}
#endif
#endif
