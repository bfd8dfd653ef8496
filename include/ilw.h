/*
 * ilw.h -- C ABI of libilw.so: the integer-only I-LW-DETR encoder block and
 * deformable sampling on AMD Instinct MI355X (gfx950).
 *
 * Operators follow "Enabling Fully Integer-Only Inference for Lightweight
 * Detection Transformers" (I-LW-DETR).  Every tensor is an integer tensor;
 * float scales exist only offline, folded into the integer constants passed
 * here (I0 = round(1/S) for ShiftExp, dyadic multiplier/shift pairs for every
 * rescale).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller.  The library
 *     never allocates, frees or retains them.  Small descriptor arrays that
 *     are documented as HOST arrays are read before the call returns.
 *   - Layouts are row-major with the channel dimension contiguous.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL is the default
 *     stream) and perform no implicit synchronization.
 *   - Return ILW_OK (0) or a negative ilw_status.  Argument errors are found
 *     on the host BEFORE anything is launched, and the output is then left
 *     untouched; ilw_last_error() gives the reason.  Kernel faults surface at
 *     the caller's next synchronization.  Launch failures return ILW_E_HIP.
 *   - Rescaling is dyadic: y = sat8(floor((acc * mult + 2^(shift-1)) / 2^shift))
 *     (round half up), sat8 clamps to the symmetric int8 range [-127, 127].
 *   - int8 tensors and weights must be 16-byte aligned and their row lengths
 *     multiples of 16 where stated.
 *   - Thread-safe.  The error string is thread-local.  The rest of the
 *     process-wide state is set up once under a lock or a static
 *     initializer: the kernel-attribute cache (per device and kernel), the
 *     device address of the allocation-free scratch (per device) and the
 *     stage profiler (ilw_profile_*, guarded by a mutex).  The environment
 *     switches ILW_FUSE_LN, ILW_TAIL and ILW_GEMM_PF, which select between
 *     equivalent kernel variants for comparison runs, are read once, at the
 *     first call that needs them.
 */
#ifndef ILW_H
#define ILW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ILW_ABI_VERSION 9

typedef enum {
  ILW_OK = 0,
  ILW_E_NULL = -1,        /* a required pointer is NULL                    */
  ILW_E_SHAPE = -2,       /* sizes inconsistent or not positive             */
  ILW_E_PARAM = -3,       /* a scalar parameter is out of its range         */
  ILW_E_UNSUPPORTED = -4, /* valid but outside what the kernels implement   */
  ILW_E_WORKSPACE = -5,   /* workspace missing or smaller than required     */
  ILW_E_HIP = -6          /* the HIP runtime reported an error              */
} ilw_status;

/* Message describing the last failure on the calling thread ("" if none). */
const char* ilw_last_error(void);
/* ILW_ABI_VERSION of the loaded library. */
int ilw_abi_version(void);

/* Dyadic rescale factors as DEVICE arrays of n entries: n == 1 applies one
 * factor to every channel (per-tensor), n == channels one per channel
 * (per-channel weights, Sec. 3.2.1).  mult is any int32 except INT32_MIN
 * (negative values are allowed where gamma folds in), shift in [1, 62];
 * device-side values are the caller's responsibility. */
typedef struct {
  const int32_t* mult;
  const int32_t* shift;
  int32_t n;
} ilw_dyadic;

/* ------------------------------------------------------------------------
 * Integer linear layer with dyadic requantization (Sec. 3.2.1, eq.
 * linear_quant: integer multiply-accumulate, scales applied after it; Sec.
 * 3.2.2: rescale by dyadic multiply-and-shift).
 *   y[m][n] = sat8(rq(b[n] + sum_k x[m][k] * w[n][k]; rq.mult[n], rq.shift[n]))
 * x int8 [M, K], w int8 [N, K], b int32 [N] (may be NULL: zero bias),
 * y int8 [M, N].  K and N multiples of 16; M >= 0 (M == 0 is a no-op).
 * The accumulator must fit int32 (K * 127^2 + |b| < 2^31).  y must not alias x.
 */
int ilw_linear(const int8_t* x, const int8_t* w, const int32_t* b, ilw_dyadic rq,
               int8_t* y, int64_t M, int32_t N, int32_t K, void* stream);

/* ------------------------------------------------------------------------
 * Constrained Shiftmax (Sec. 3.3.2, Alg. 2) over `rows` contiguous rows of
 * `cols` int8 scores each.  I0 = round(1/S_x) in [1, 2^14 - 1]; k_inter in
 * [1, 16] (16 in the paper's 8/8/16 setting); k_out in [2, 8]; m_p in [0, 31]
 * (the paper uses 4); the hardware division precision is fixed to 31.
 * s_d >= 0 uses that calibrated denominator shift for every row (the text
 * calibrates one s_d per Shiftmax block); s_d == -1 derives it per row from
 * the row's exponential sum (CalibrateShift as in the algorithm listing).
 * Output in [0, 2^(k_out-1) - 1] with scale 2^-(k_out-1); a value that would
 * reach 2^(k_out-1) (possible only with an oversized static s_d) is limited
 * to 2^(k_out-1) - 1 because the output is a signed k_out-bit integer.
 * y may alias x.  cols in [1, 65536].
 */
int ilw_shiftmax(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                 int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d,
                 void* stream);

/* ------------------------------------------------------------------------
 * SD-ShiftGELU (Sec. 3.3.1, Alg. 1) element-wise over n int8 values, then the
 * dyadic requantization of I_out = I_x * I_div (scale S_x * 2^-(k_out-1)) to
 * the int8 activation of the next layer:  y = sat8(rq(I_out; out_mult,
 * out_shift)).  IntDiv, which the algorithm uses without a definition, is the
 * fixed-precision integer division of eq. shiftmax_original with M = 31.
 * I0 in [1, 2^14 - 1], k_inter in [1, 16], k_out in [2, 8], out_shift in
 * [1, 62].  y may alias x.
 */
int ilw_sdshiftgelu(const int8_t* x, int8_t* y, int64_t n, int32_t I0,
                    int32_t k_inter, int32_t k_out, int32_t out_mult,
                    int32_t out_shift, void* stream);

/* ------------------------------------------------------------------------
 * Integer LayerNorm (Sec. 3.3: I-ViT's formulation with an integer square
 * root by Newton's method; 10 iterations, 20 for the decoder) over `rows`
 * rows of C int8 channels:
 *   mu = floor((2*sum x + C) / (2C));  y_i = x_i - mu;  V = sum y_i^2
 *   sigma: k <- floor((k + floor(V/k)) / 2), newton_iters times from k = 2^16
 *   n_i = floor(y_i * floor((2^31 - 1) / sigma) / 2)     (0 when V == 0)
 *   out_i = sat8(rq(n_i + beta_i; out.mult_i, out.shift_i))
 * beta int32 [C] is at the scale of n (DEVICE array).  There is no gamma
 * argument: the affine scale is folded into the per-channel (signed) output
 * multiplier.  A model with an integer gamma_i and one output dyadic (m, s)
 * passes mult_i = gamma_i * m and beta_i = b_i / gamma_i, which equals
 * rq(n_i * gamma_i + b_i; m, s) exactly when gamma_i divides b_i (and
 * |gamma_i * m| < 2^31); a float gamma is folded when the multipliers are
 * derived, with no separate rounding of gamma.  A gamma that differs across
 * channels therefore needs a per-channel output dyadic (out.n = C): with one
 * per-tensor multiplier (out.n = 1) gamma must be uniform.  C in [4, 16384],
 * a multiple of 4; newton_iters in [1, 64].  y may alias x.
 */
int ilw_int_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                      const int32_t* beta, ilw_dyadic out, int32_t newton_iters,
                      void* stream);

/* ------------------------------------------------------------------------
 * Two-input dyadic add onto one output scale (Sec. 3.2.2: branches rescaled
 * to a common scale by dyadic multiply-and-shift and summed in integers); the
 * residual connection of the encoder block:
 *   y = sat8(floor((a * mult_a + b * mult_b + 2^(shift-1)) / 2^shift))
 * a, b, y int8 [n]; shift in [1, 62].  y may alias a or b.
 */
int ilw_residual_add(const int8_t* a, const int8_t* b, int8_t* y, int64_t n,
                     int32_t mult_a, int32_t mult_b, int32_t shift, void* stream);

/* ------------------------------------------------------------------------
 * Integer multi-head attention over window or global token groups: per
 * window and head, S = Q K^T (int32) -> per-tensor dyadic -> int8 scores;
 * P = Constrained Shiftmax of each score row; O = P V (int32) -> per-tensor
 * dyadic -> int8, heads concatenated (the encoder's MatMul and Softmax
 * operators, Table ablation_study; Sec. 3.2.1 and Sec. 3.3.2).
 *   qkv int8 [batch, grid_h*grid_w, 3*dim]: q | k | v, head h at columns
 *       h*head_dim .. of each part.
 *   out int8 [batch, grid_h*grid_w, dim].
 * win_h == win_w == 0 selects global attention; otherwise win_h x win_w
 * windows tile the grid (LW-DETR's window attention).  head_dim 32 or 64
 * (the decoder's 8 heads of 32 channels, the encoder's heads of 64);
 * dim == heads * head_dim; tokens per window in [1, 2048].  The workspace
 * (ilw_attention_workspace_bytes) holds the window-major Q, K and V^T copies,
 * rows of 64 bytes per head.
 */
typedef struct {
  int32_t score_mult, score_shift;  /* S -> int8 scores (folds 1/sqrt(d_h)) */
  int32_t I0, k_inter, k_out, m_p, s_d; /* Constrained Shiftmax, as above   */
  int32_t pv_mult, pv_shift;        /* P V -> int8                          */
} ilw_attn_params;

size_t ilw_attention_workspace_bytes(int32_t batch, int32_t grid_h, int32_t grid_w,
                                     int32_t win_h, int32_t win_w, int32_t dim,
                                     int32_t head_dim);
int ilw_attention(const int8_t* qkv, int8_t* out, int32_t batch, int32_t grid_h,
                  int32_t grid_w, int32_t win_h, int32_t win_w, int32_t dim,
                  int32_t heads, int32_t head_dim, const ilw_attn_params* ap,
                  void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * One integer pre-LayerNorm ViT encoder block (the encoder operators of
 * Table ablation_study in the plain-ViT order):
 *   h = LN1(x);  a = Attn(QKV(h));  x1 = Res(proj(a), x)
 *   h2 = LN2(x1); g = rq(SD-ShiftGELU(fc1(h2)));  y = Res(fc2(g), x1)
 * Weights are int8 [out, in] with int32 biases and per-channel dyadic
 * requantization (Sec. 3.2.1); every activation between operators is int8.
 * All pointers in the struct are DEVICE pointers; the struct itself is read
 * on the host during the call.  Residuals: y = sat8(rq2(branch * mult_a +
 * skip * mult_b; shift)).  dim and mlp_dim multiples of 16, head_dim == 64.
 */
typedef struct {
  int32_t dim, heads, head_dim, mlp_dim, ln_iters;
  const int32_t* ln1_beta; ilw_dyadic ln1_out;
  const int8_t* w_qkv; const int32_t* b_qkv; ilw_dyadic qkv;   /* [3*dim, dim] */
  ilw_attn_params attn;
  const int8_t* w_proj; const int32_t* b_proj; ilw_dyadic proj; /* [dim, dim]  */
  int32_t res1_mult_a, res1_mult_b, res1_shift;
  const int32_t* ln2_beta; ilw_dyadic ln2_out;
  const int8_t* w_fc1; const int32_t* b_fc1; ilw_dyadic fc1;   /* [mlp, dim]   */
  int32_t gelu_I0, gelu_k_inter, gelu_k_out, gelu_mult, gelu_shift;
  const int8_t* w_fc2; const int32_t* b_fc2; ilw_dyadic fc2;   /* [dim, mlp]   */
  int32_t res2_mult_a, res2_mult_b, res2_shift;
} ilw_block_params;

/* Bytes of caller-owned device workspace ilw_block_forward needs (0 on
 * invalid arguments, with ilw_last_error set). */
size_t ilw_block_workspace_bytes(const ilw_block_params* p, int32_t batch,
                                 int32_t grid_h, int32_t grid_w, int32_t win_h,
                                 int32_t win_w);
/* x, y int8 [batch, grid_h*grid_w, dim]; y may alias x (x is last read
 * before y is first written, in stream order).  The workspace must not
 * alias x or y. */
int ilw_block_forward(const ilw_block_params* p, const int8_t* x, int8_t* y,
                      int32_t batch, int32_t grid_h, int32_t grid_w, int32_t win_h,
                      int32_t win_w, void* workspace, size_t workspace_bytes,
                      void* stream);

/* Size of the library's static device scratch used by
 * ilw_block_forward_noalloc: 32 MiB on each GPU the library runs on. */
#define ILW_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
/* ilw_block_forward without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, serving loops and
 * harnesses that forbid hipMalloc.  Arguments, results and error behaviour
 * are those of ilw_block_forward; the workspace is instead a file-scope
 * device array of ILW_NOALLOC_SCRATCH_BYTES that each GPU holds from the
 * first call on it until the process ends.  Nothing is allocated or freed:
 * the first call on a device looks the array's address up once
 * (hipGetSymbolAddress) with that device current.  A call whose workspace
 * need (ilw_block_workspace_bytes) exceeds the scratch returns
 * ILW_E_WORKSPACE before any launch.  All calls on one GPU share its
 * scratch, which keeps the last call's contents: calls in stream order are
 * safe, calls that overlap in time on one GPU (several streams or threads)
 * race and give undefined results.  No byte of the scratch needs to start
 * at zero: every byte a kernel reads was written earlier in the same call.
 * The device is the caller's current device. */
int ilw_block_forward_noalloc(const ilw_block_params* p, const int8_t* x, int8_t* y,
                              int32_t batch, int32_t grid_h, int32_t grid_w,
                              int32_t win_h, int32_t win_w, void* stream);

/* ------------------------------------------------------------------------
 * Patch embedding, the encoder's input layer (Table mappability: a
 * convolution plus an add; Sec. 3.2.1 integer linear formulation): a
 * patch x patch stride-patch convolution of the int8 image, per-channel
 * requantization to int8, then the int8 positional embedding added with the
 * residual form  y = sat8(rq2(conv * pos_mult_a + pos * pos_mult_b; pos_shift)).
 *   img  int8 [batch, channels, height, width] (per-tensor scale), 16-byte
 *        aligned; height, width multiples of 16
 *   w    int8 [dim, channels * patch * patch], K order (channel, ky, kx)
 *   bias int32 [dim] or NULL; proj per-tensor or per-channel dyadic
 *   pos  int8 [T, dim], T = (height/16) * (width/16), row-major patch grid
 *   y    int8 [batch, T, dim]
 * patch == 16 (the only size implemented); channels in [1, 256].
 */
int ilw_patch_embed(const int8_t* img, int32_t batch, int32_t channels, int32_t height,
                    int32_t width, int32_t patch, const int8_t* w, const int32_t* bias,
                    ilw_dyadic proj, const int8_t* pos, int32_t pos_mult_a,
                    int32_t pos_mult_b, int32_t pos_shift, int8_t* y, int32_t dim,
                    void* stream);

/* ------------------------------------------------------------------------
 * A stack of n_blocks encoder blocks (the ViT encoder of LW-DETR, Sec. 3.1;
 * each block as ilw_block_forward), run in one call so that the LayerNorm
 * after each residual linear can be computed in that linear's epilogue
 * (dim 192 or 384; other widths run it as a separate kernel, same result).
 *   blocks  HOST array of n_blocks parameter structs (device pointers inside),
 *           all with the same dim; n_blocks in [1, 4096].
 *   windows HOST int32 [n_blocks][2] = (win_h, win_w) of each block's
 *           attention; (0, 0) = global attention.
 *   x, y    int8 [batch, grid_h*grid_w, dim]; y may alias x.  Intermediate
 *           block outputs are written to y.
 * The workspace (ilw_encoder_workspace_bytes) is the largest block
 * workspace; it must not alias x or y.  Results are bit-identical to calling
 * ilw_block_forward block by block.
 */
size_t ilw_encoder_workspace_bytes(const ilw_block_params* blocks, int32_t n_blocks,
                                   const int32_t* windows, int32_t batch, int32_t grid_h,
                                   int32_t grid_w);
int ilw_encoder_forward(const ilw_block_params* blocks, int32_t n_blocks,
                        const int32_t* windows, const int8_t* x, int8_t* y, int32_t batch,
                        int32_t grid_h, int32_t grid_w, void* workspace,
                        size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Multi-scale deformable sampling core of the decoder's cross-attention
 * (Sec. 3.1.1: bilinear interpolation replaced by nearest-neighbour
 * sampling; the attention weights come from Constrained Shiftmax, Sec. 3.3.2):
 *   value   int8  [B, S, heads, head_dim], the L levels stacked, level l at
 *           rows level_start[l] .. + H_l*W_l (row-major y, x)
 *   level_hw    HOST int32 [L][2] = (H_l, W_l), each in [1, 32767]
 *   level_start HOST int32 [L];  S = sum H_l*W_l
 *   ref     int32 [B, Q, 2]  reference point (x, y), Q16 fraction of the map
 *   offsets int16 [B, Q, heads, L, P, 2]  (x, y) in Q8 pixels of level l
 *   logits  int8  [B, Q, heads, L*P] -> Constrained Shiftmax per (b, q, h)
 *           with I0, k_inter, k_out, m_p, s_d (ranges as ilw_shiftmax; the
 *           decoder's defaults are k_inter = 16, k_out = 8, m_p = 4)
 *   out     int8  [B, Q, heads*head_dim] = sat8(rq(sum_{l,p} P * sample))
 * Location: X = floor(ref_x * W_l / 2^8) + off_x (Q8), pixel ix = floor(X/2^8);
 * samples outside the map contribute 0.  mode 0 = nearest (the paper);
 * mode 1 = a fixed-point bilinear variant on the half-pixel grid with Q8
 * weights whose 2^16 scale is removed by 16 extra bits of out_shift.
 * head_dim a multiple of 4 in [4, 256]; L in [1, 8]; L*P in [1, 64].
 */
int ilw_deform_attn(const int8_t* value, const int32_t* level_hw,
                    const int32_t* level_start, int32_t L, int32_t P,
                    const int32_t* ref, const int16_t* offsets, const int8_t* logits,
                    int8_t* out, int32_t B, int32_t Q, int32_t heads, int32_t head_dim,
                    int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d,
                    int32_t out_mult, int32_t out_shift, int32_t mode, void* stream);

/* The same sampler with reference boxes (Sec. 3.1.2: the decoder's
 * references are the encoder's top-K boxes).  The paper gives no sampling
 * rule; the one implemented takes the offsets relative to the box, as the
 * deformable decoder with box references does:
 *   ref     int32 [B, Q, 4]  (cx, cy, w, h), Q16 fractions of the map
 *   offsets int16 [B, Q, heads, L, P, 2]  (x, y) in Q8 units of size / (2 P)
 *   location = c + (off / 2^8) / P * size / 2, floored once in Q8 pixels:
 *   X = floor((cx * 2^9 * P + off_x * w) * W_l / (2^17 * P)), likewise Y with
 *   cy, h, H_l; then the nearest or bilinear rule of ilw_deform_attn.
 * Other arguments, limits and errors as for ilw_deform_attn.
 */
int ilw_deform_attn_boxes(const int8_t* value, const int32_t* level_hw,
                          const int32_t* level_start, int32_t L, int32_t P,
                          const int32_t* ref, const int16_t* offsets, const int8_t* logits,
                          int8_t* out, int32_t B, int32_t Q, int32_t heads, int32_t head_dim,
                          int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d,
                          int32_t out_mult, int32_t out_shift, int32_t mode, void* stream);

/* ------------------------------------------------------------------------
 * I-ViT baseline operators, the forms that Constrained Shiftmax and
 * SD-ShiftGELU replace (for comparisons; same layouts as the operators
 * above, one row = one contiguous run of cols int8 values, y may alias x):
 *   ilw_shiftmax_ivit   eq. shiftmax_original (Sec. 3.3.2) with a fixed
 *       division precision M in [k_out, 32]:
 *       out = (floor((2^M - 1) / S_sum) * I_exp) >> (M - (k_out - 1));
 *       the factor is 0 once S_sum >= 2^M (the collapse the paper describes)
 *   ilw_shiftgelu_ivit  ShiftGELU (Sec. 3.3.1) with the sigmoid argument
 *       shifted by the row maximum of I_p (clamped at 0) instead of
 *       element-wise, then the same int8 requantization as ilw_sdshiftgelu
 * Parameters otherwise as ilw_shiftmax / ilw_sdshiftgelu.
 */
int ilw_shiftmax_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                      int32_t k_inter, int32_t k_out, int32_t M, void* stream);
int ilw_shiftgelu_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                       int32_t k_inter, int32_t k_out, int32_t out_mult, int32_t out_shift,
                       void* stream);

/* ------------------------------------------------------------------------
 * Scale-preserving split convolution of the multi-scale projector (Sec.
 * 3.2.2, Fig. projector_split_conv), pointwise (a linear layer over the
 * tokens of the feature maps).  Branch b is one encoder feature map with its
 * own activation scale S_b; its int32 partial is brought to the common scale
 * (the largest S_b) by the branch's dyadic before the integer accumulation:
 *   acc_b[m][n] = sum_k x[b][m][k] * w[b][n][k]
 *   r_b         = floor((acc_b * m_b[n] + 2^(s_b[n]-1)) / 2^s_b[n])  (no saturation)
 *   y[m][n]     = sat8(rq(bias[n] + sum_b r_b; out))   (sum in 64 bits)
 *   n_branches  in [1, 8]
 *   x, w, branch, channels: HOST arrays of n_branches entries; x[b] DEVICE
 *               int8 [M, channels[b]], w[b] DEVICE int8 [N, channels[b]]
 *               (both 16-byte aligned), branch[b] a dyadic with n = 1 or N
 *               (m_b / 2^s_b ~ S_b / S_c), channels[b] a multiple of 64 in
 *               [64, 65536]
 *   bias        DEVICE int32 [N] in the common scale, or NULL
 *   y           DEVICE int8 [M, N]; N a multiple of 16
 */
int ilw_split_conv(int32_t n_branches, const int8_t* const* x, const int32_t* channels,
                   const int8_t* const* w, const ilw_dyadic* branch, const int32_t* bias,
                   ilw_dyadic out, int8_t* y, int64_t M, int32_t N, void* stream);

/* ------------------------------------------------------------------------
 * One integer deformable decoder layer (LW-DETR's decoder made integer:
 * Sec. 3.1.1 nearest sampling, Sec. 3.3.2 Constrained Shiftmax, Sec. 3.3
 * I-LayerNorm with 20 Newton steps), post-norm:
 *   t1 = LN1(Res1(tgt, o(Attn(QKV(tgt)))))        self-attention, one global
 *                                                  window of the queries
 *   v = val(memory); off = 16 * offl(t1) (int8 1/16 px -> Q8); w = attw(t1)
 *   t2 = LN2(Res2(t1, co(Deform(v, ref, off, w)))) cross-attention (as
 *                                                  ilw_deform_attn, mode 0/1,
 *                                                  k_inter 16, k_out 8, m_p 4)
 *   y  = LN3(Res3(t2, fc2(GELU(fc1(t2)))))         FFN
 *   tgt int8 [batch, queries, dim]; memory int8 [batch, value_tokens, dim],
 *   the levels stacked as for ilw_deform_attn (level_hw, level_start: HOST
 *   int32 [levels][2], [levels]); ref int32 Q16 [batch, queries, ref_dims];
 *   y int8 [batch, queries, dim] (must not alias tgt).
 * The struct's arrays are DEVICE pointers.  head_dim = dim / heads in
 * {32, 64}; dim, ffn_dim, heads*levels*points multiples of 16; queries in
 * [1, 2048]; levels in [1, 8], levels*points <= 64.
 */
typedef struct {
  int32_t dim, heads, ffn_dim, levels, points, ln_iters;
  const int8_t* w_qkv; const int32_t* b_qkv; ilw_dyadic qkv;     /* [3*dim, dim] */
  ilw_attn_params attn;
  const int8_t* w_o; const int32_t* b_o; ilw_dyadic o;           /* [dim, dim]   */
  int32_t res1_mult_a, res1_mult_b, res1_shift;
  const int32_t* ln1_beta; ilw_dyadic ln1_out;
  const int8_t* w_val; const int32_t* b_val; ilw_dyadic val;     /* [dim, dim]   */
  const int8_t* w_off; const int32_t* b_off; ilw_dyadic off;     /* [heads*levels*points*2, dim] */
  const int8_t* w_attw; const int32_t* b_attw; ilw_dyadic attw;  /* [heads*levels*points, dim]   */
  int32_t da_I0, da_s_d, da_out_mult, da_out_shift, da_mode;
  int32_t ref_dims;  /* 2: ref holds points (ilw_deform_attn); 4: boxes (ilw_deform_attn_boxes) */
  const int8_t* w_co; const int32_t* b_co; ilw_dyadic co;        /* [dim, dim]   */
  int32_t res2_mult_a, res2_mult_b, res2_shift;
  const int32_t* ln2_beta; ilw_dyadic ln2_out;
  const int8_t* w_fc1; const int32_t* b_fc1; ilw_dyadic fc1;     /* [ffn, dim]   */
  int32_t gelu_I0, gelu_k_inter, gelu_k_out, gelu_mult, gelu_shift;
  const int8_t* w_fc2; const int32_t* b_fc2; ilw_dyadic fc2;     /* [dim, ffn]   */
  int32_t res3_mult_a, res3_mult_b, res3_shift;
  const int32_t* ln3_beta; ilw_dyadic ln3_out;
} ilw_decoder_params;

size_t ilw_decoder_workspace_bytes(const ilw_decoder_params* p, int32_t batch,
                                   int32_t queries, int32_t value_tokens);
int ilw_decoder_layer(const ilw_decoder_params* p, const int8_t* tgt, const int8_t* memory,
                      const int32_t* ref, const int32_t* level_hw, const int32_t* level_start,
                      int8_t* y, int32_t batch, int32_t queries, int32_t value_tokens,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Per-stage kernel timing (tracing; off by default).  While enabled, every
 * kernel that ilw_block_forward, ilw_encoder_forward, ilw_attention,
 * ilw_deform_attn, ilw_split_conv, ilw_patch_embed and ilw_decoder_layer
 * launch is bracketed by a pair of HIP events recorded on the
 * caller's stream, and the launch is attributed to one of the stages below.
 * Enabling (or disabling)
 * clears the records.  ilw_profile_read waits for the last recorded event and
 * returns, per stage, the summed kernel time in milliseconds and the number of
 * launches (arrays of n_stages entries, HOST memory).  Do not enable it while
 * a stream is being captured into a graph.  Launches from several threads
 * record under one lock; each launch is attributed to the stage it belongs to.
 */
typedef enum {
  ILW_STAGE_LAYERNORM = 0,   /* stand-alone LayerNorm kernels              */
  ILW_STAGE_GEMM_QKV = 1,    /* QKV linear, window-major scatter epilogue  */
  ILW_STAGE_ATTENTION = 2,   /* fused attention (window and global)        */
  ILW_STAGE_GEMM_PROJ = 3,   /* projection + residual (+ LN2) epilogue     */
  ILW_STAGE_GEMM_FC1 = 4,    /* fc1 linear + SD-ShiftGELU epilogue         */
  ILW_STAGE_GEMM_FC2 = 5,    /* fc2 + residual (+ next LN1) epilogue       */
  ILW_STAGE_RELAYOUT = 6,    /* token-major QKV -> window-major copy       */
  ILW_STAGE_DEFORM = 7,      /* deformable sampling                        */
  ILW_STAGE_BLOCK_TAIL = 8,  /* projection ... next block's QKV, one launch */
  ILW_STAGE_SPLIT_CONV = 9,  /* scale-preserving split convolution          */
  ILW_STAGE_PATCH_EMBED = 10, /* patch embedding + positional embedding     */
  ILW_STAGE_DECODER = 11,    /* decoder linears, LayerNorms, offset widening */
  ILW_STAGE_TAIL384 = 12,    /* projection ... fc2 + residual (+ next LN1),
                                one launch (dim 384)                        */
  ILW_NUM_STAGES = 13
} ilw_stage;

int ilw_profile_enable(int enable);
int ilw_profile_read(double* total_ms, int32_t* launches, int32_t n_stages);

#ifdef __cplusplus
}
#endif
#endif /* ILW_H */
