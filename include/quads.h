/*
 * quads.h -- C ABI of libquads.so: the NVFP4 W4A4 MoE expert layer with
 * Residual Activation Compensation (QUADS, arXiv 2607.15810, rollout side)
 * as HIP kernels for AMD Instinct MI355X (gfx950).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every pointer named in a signature is a DEVICE pointer unless its
 *    comment says "host".  The caller allocates and owns every buffer,
 *    workspace included; the library allocates no device memory and keeps no
 *    pointer after a call returns.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream) and never synchronises with the host.
 *  - Arguments are validated on the host before any launch; a failed check
 *    returns a negative status and launches nothing.  QD_ERR_HIP means a
 *    launch failed (the HIP error is not cleared).
 *  - Device pointers must be 16-byte aligned; NVFP4 widths (`cols`, K) must
 *    be multiples of 16.  Zero rows is a successful no-op.
 *  - Results are deterministic: reductions use order-independent integer or
 *    max arithmetic, permutations are computed by ranks, never by atomic slot
 *    claims.  Calls running concurrently on different streams must not share
 *    output or workspace buffers.
 *
 * NVFP4 tensor (Sec. 2.2 "FP4" paragraph of the paper): E2M1 element codes,
 * one E4M3 scale per 16 consecutive elements along the contraction axis, and
 * an FP32 tensor scale pair.
 */
#ifndef QUADS_H
#define QUADS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#pragma GCC visibility push(default)
#endif

typedef int qd_status;
#define QD_OK               0
#define QD_ERR_NULL        -1  /* a required pointer is NULL                */
#define QD_ERR_SHAPE       -2  /* a size is negative, inconsistent or not a multiple of 16 */
#define QD_ERR_ALIGN       -3  /* a device pointer is not 16-byte aligned   */
#define QD_ERR_DTYPE       -4  /* unknown dtype / epilogue code             */
#define QD_ERR_WORKSPACE   -5  /* workspace NULL or smaller than required   */
#define QD_ERR_UNSUPPORTED -6  /* valid but unsupported combination         */
#define QD_ERR_HIP         -7  /* a kernel launch failed                    */

#define QD_DTYPE_BF16 0
#define QD_DTYPE_F32  1

#define QD_EPI_NONE   0   /* out[r][n] = bf16(alpha * acc)                    */
#define QD_EPI_SWIGLU 1   /* out[r][j] = bf16(silu(g_j) * u_j), N = 2I         */

/*
 * An NVFP4 tensor: `groups` matrices of [rows][cols].  The struct itself is
 * host memory; the arrays are device memory owned by the caller.
 *   codes  : uint8 [groups][rows][cols/2]; element 2i of a row in bits 3:0,
 *            element 2i+1 in bits 7:4; a code is sign<<3 | E2M1 magnitude
 *            index (magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6).
 *   scales : uint8 [groups][rows][cols/16]; E4M3FN bit patterns, sign 0.
 *   gscale : float [groups][2] = {s_enc, s_dec}, the FP32 tensor scale pair.
 * Element value: e2m1(code) * e4m3(scale) * s_dec.
 *   scales_frag : optional second copy of the scales of a weight tensor,
 *            laid out for the grouped GEMM's kernel for few rows per expert
 *            (see nvfp4_pack_frag_scales); NULL everywhere else.
 */
typedef struct {
  uint8_t *codes;
  uint8_t *scales;
  float   *gscale;
  int64_t  groups, rows, cols;
  uint8_t *scales_frag;   /* optional, weights only: NULL, or the same scales
                             in fragment order (nvfp4_pack_frag_scales) */
} qd_nvfp4;

const char *qd_status_string(qd_status s);
int         qd_version(void);

/* ---------------------------------------------------------------------
 * nvfp4_quantize_act -- Q_A, the activation QDQ of Eq. (act-error-def)
 * and Eq. (residual-def); format of Sec. 2.2.
 *   x          : [rows][cols] bf16 (x_dtype QD_DTYPE_BF16) or f32.
 *   amax_partials, n_partials : optional.  If non-NULL the tensor amax is the
 *                maximum of these n_partials non-negative floats (a static
 *                scale, or the per-block maxima another kernel produced);
 *                if NULL it is max|x|, computed here.
 *   out        : groups 1, rows, cols; written.
 *   rac_scores : optional uint64 [cols].  If non-NULL the same pass also
 *                computes the RAC channel scores of Eq. (channel-score)
 *                (fixed point: sum over rows of trunc(fl32(r*r) * 2^F),
 *                r = x_hat - x, F = 36 - 2e with amax = f*2^e) and
 *                rac_ramax (float [1]) receives max|r|.  Requires
 *                amax_partials == NULL and x_dtype bf16.  Both buffers are
 *                zeroed by this call before use.
 *   ws         : at least nvfp4_quantize_act_workspace(rows, cols) bytes.
 * ------------------------------------------------------------------- */
size_t    nvfp4_quantize_act_workspace(int64_t rows, int64_t cols);
qd_status nvfp4_quantize_act(const void *x, int x_dtype, int64_t rows, int64_t cols,
                             const float *amax_partials, int64_t n_partials,
                             const qd_nvfp4 *out, uint64_t *rac_scores, float *rac_ramax,
                             void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * nvfp4_quantize_weight -- Q_W of Eq. (weight-error-def), one tensor scale
 * per group (expert matrix).  The same quantiser feeds the trainer-side
 * fake-quant of Eq. (w4a16-qat-forward) through nvfp4_dequantize.
 *   w   : bf16 [groups][rows][cols].
 *   out : groups, rows, cols; written.
 *   ws  : at least nvfp4_quantize_weight_workspace(groups, rows, cols) bytes.
 * ------------------------------------------------------------------- */
size_t    nvfp4_quantize_weight_workspace(int64_t groups, int64_t rows, int64_t cols);
qd_status nvfp4_quantize_weight(const void *w, int64_t groups, int64_t rows, int64_t cols,
                                const qd_nvfp4 *out, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * nvfp4_dequantize -- QDQ output of Eq. (w4a16-qat-forward).
 *   unscaled 0: out = fl32(fl32(e2m1 * e4m3) * s_dec), stored as out_dtype
 *               (bf16 output rounds that float once, to nearest even);
 *   unscaled 1: out = e2m1 * e4m3 exactly (s_dec left to the caller).
 *   out : [groups][rows][cols] of out_dtype.
 * ------------------------------------------------------------------- */
qd_status nvfp4_dequantize(const qd_nvfp4 *in, int unscaled, void *out, int out_dtype,
                           void *stream);

/* ---------------------------------------------------------------------
 * moe_route_permute -- top-k routing and the grouped-GEMM row order for
 * the MoE layer (Sec. 3.3, the W13 site; Sec. 4.1 MoE model).
 *   logits         : f32 [T][E], finite.
 *   topk_ids       : int32 [T][k], experts by (logit desc, index asc).
 *   topk_w         : f32 [T][k]; renorm 1: softmax over the k selected
 *                    logits; renorm 0: full softmax probability.
 *   expert_offsets : int32 [E+1], exclusive scan of per-expert row counts.
 *   row_token      : int32 [T*k], token of each row; rows ordered by
 *                    (expert asc, token asc).
 *   inv_row        : int32 [T][k], row holding (t, topk_ids[t][s]).
 *   1 <= k <= E <= 1024.
 * ------------------------------------------------------------------- */
size_t    moe_route_permute_workspace(int64_t T, int32_t E, int32_t k);
qd_status moe_route_permute(const float *logits, int64_t T, int32_t E, int32_t k,
                            int32_t renorm, int32_t *topk_ids, float *topk_w,
                            int32_t *expert_offsets, int32_t *row_token, int32_t *inv_row,
                            void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * rac_select_channels -- online channel selection and masked residual of
 * Sec. 3.3: Eq. (channel-score), Eq. (channel-select), and the term
 * M_S (.) Q_A(dX_q) of Eq. (residual-recon).
 *   x, xq       : the bf16 activation [T][K] and its NVFP4 quantisation.
 *   Ks          : number of channels to keep, 0 <= Ks <= K (k% = Ks / K).
 *   scores      : uint64 [K]; ramax: float [1].  stats_ready 1: they hold
 *                 the values nvfp4_quantize_act produced for (x, xq);
 *                 stats_ready 0: this call computes them.
 *   sel_idx     : int32 [Ks], the selected channels in ascending order
 *                 (top Ks by score, ties to the lower index).
 *   rq          : groups 1, T, K; written: the residual quantised over all
 *                 channels with its own tensor scale, then codes outside S
 *                 set to 0 and scales of blocks without a selected channel
 *                 set to 0.
 *   ws          : at least rac_select_channels_workspace(T, K) bytes.
 *   K <= 65536.
 * ------------------------------------------------------------------- */
size_t    rac_select_channels_workspace(int64_t T, int64_t K);
qd_status rac_select_channels(const void *x, const qd_nvfp4 *xq, int32_t Ks,
                              uint64_t *scores, float *ramax, int32_t stats_ready,
                              int32_t *sel_idx, const qd_nvfp4 *rq,
                              void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * rac_select_channels_per_expert -- one channel set per expert (a variant
 * of Sec. 3.3 where Eq. (channel-score) and Eq. (channel-select) run over
 * each expert's own rows, i.e. the tokens routed to it):
 *   score_e[j] = sum over rows r of expert e of trunc(fl(r_tj^2) * 2^F),
 *   t = row_token[r], with the fixed point F of rac_select_channels (from
 *   the tensor amax of x); S_e = the Ks largest, ties to the lower channel,
 *   ascending (an expert without rows gets channels 0 .. Ks-1).
 *   x, xq          : the bf16 activation [T][K] and its NVFP4 quantisation.
 *   row_token, expert_offsets, E, rows : from moe_route_permute (rows = T*k).
 *   scores_pe      : uint64 [E][K] out; ramax: float [1] out (max |r|).
 *   sel_pe         : int32 [E][Ks] out.
 *   rq             : groups 1, T, K; written: the residual quantised over
 *                    all channels with its own tensor scale (no mask).
 *   rq_sel_rows    : f16 [rows][rac_selected_width(Ks)] out: row r holds
 *                    rq[row_token[r]] at the channels of its expert's set,
 *                    as rac_gather_selected does per token.
 *   ws             : at least rac_select_channels_per_expert_workspace(T, K, E).
 *   K <= 16384.
 * ------------------------------------------------------------------- */
size_t    rac_select_channels_per_expert_workspace(int64_t T, int64_t K, int32_t E);
qd_status rac_select_channels_per_expert(const void *x, const qd_nvfp4 *xq, int32_t Ks,
                                         const int32_t *row_token, const int32_t *expert_offsets,
                                         int32_t E, int64_t rows, uint64_t *scores_pe,
                                         float *ramax, int32_t *sel_pe, const qd_nvfp4 *rq,
                                         void *rq_sel_rows, void *ws, size_t ws_bytes,
                                         void *stream);

/* ---------------------------------------------------------------------
 * rac_gather_selected -- the masked residual restricted to the selected
 * channels S, compacted per row: the operand r_S of the residual term
 * W[:, S] r_S of Eq. (residual-recon) without its tensor scale,
 *   out[t][j] = e2m1(code of rq[t][sel_idx[j]]) * e4m3(its block scale)
 * for j < Ks (exact in f16), and 0 for Ks <= j < rac_selected_width(Ks).
 *   rq, sel_idx, Ks : from rac_select_channels.
 *   out             : f16 [rq->rows][rac_selected_width(Ks)], 16-byte aligned.
 * moe_w4a4_grouped_gemm takes it as rq_sel.
 * ------------------------------------------------------------------- */
int32_t   rac_selected_width(int32_t Ks);
qd_status rac_gather_selected(const qd_nvfp4 *rq, const int32_t *sel_idx, int32_t Ks,
                              void *out, void *stream);

/* ---------------------------------------------------------------------
 * rac_residual_gemm -- the residual contraction of Eq. (residual-recon)
 * pushed through the linear layer:
 *   out[r][n] = s_dec_r * s_dec_w[e] * sum_{j in S} rhat[src(r)][j] * what[e][n][j]
 * with rhat, what the unscaled NVFP4 values (exact), accumulated in f32.
 *   rq, sel_idx, Ks : from rac_select_channels.
 *   row_token       : int32 [rows] gather map (NULL: row r reads rq row r).
 *   expert_offsets  : int32 [E+1] (NULL: one group, all rows).
 *   w               : E groups of [N][K].
 *   out             : f32 [rows][N].
 * ------------------------------------------------------------------- */
qd_status rac_residual_gemm(const qd_nvfp4 *rq, const int32_t *sel_idx, int32_t Ks,
                            const int32_t *row_token, const int32_t *expert_offsets,
                            int64_t rows, const qd_nvfp4 *w, float *out, void *stream);

/* ---------------------------------------------------------------------
 * moe_w4a4_grouped_gemm -- the W4A4 expert GEMM of Sec. 3.3 with the RAC
 * residual fused (the main GEMM stays on NVFP4 codes, Sec. 3.3 "Targeted
 * residual compensation"):
 *   acc[r][n]  = sum_k a[src(r)][k] * w[e(r)][n][k]           (a, w NVFP4)
 *   accr[r][n] = sum_{k in S} rq[src(r)][k] * w[e(r)][n][k]   (if rq)
 *   v[r][n]    = s_dec_a*s_dec_w[e] * acc - s_dec_r*s_dec_w[e] * accr
 * Products of decoded operands are exact; accumulation is f32.
 *   a               : activations [*][K] (groups 1).
 *   row_token       : int32 [rows] gather map (NULL: row r reads a row r).
 *   expert_offsets  : int32 [E+1] row ranges per expert (NULL: E must be 1).
 *   rows            : number of grouped rows (T*k for the MoE layer).
 *   w               : E groups of [N][K]; w->scales_frag (optional) is
 *                     read by the kernel for few rows per expert.
 *   rq, sel_idx, Ks : the masked residual (NULL / 0: plain W4A4; Ks > 0
 *                     needs rq).
 *   rq_sel          : rac_gather_selected(rq, sel_idx, Ks) (f16, 16-byte
 *                     aligned).  Where moe_w4a4_grouped_gemm_residual_form
 *                     is 2 (many rows per expert, K_s small enough for the
 *                     compact weight table in LDS) the kernel contracts the
 *                     residual in this compact form and returns QD_ERR_NULL
 *                     without it; where it is 1 the kernel reads the masked
 *                     residual rq (a second pass over K for many rows) and
 *                     ignores rq_sel (NULL allowed).
 *   epilogue        : QD_EPI_NONE: out bf16 [rows][N] = bf16(v);
 *                     QD_EPI_SWIGLU: N = 2I, gate rows [0,I), up rows
 *                     [I,2I); out bf16 [rows][I] = bf16(silu(g)*u).
 *   amax_partials   : optional float [moe_w4a4_grouped_gemm_amax_count(rows, N,
 *                     K, E, Ks, epilogue)] receiving one maximum of |out| (as
 *                     stored) per workgroup; their maximum is the tensor amax
 *                     of out.  Every entry is written.
 * ------------------------------------------------------------------- */
int64_t   moe_w4a4_grouped_gemm_amax_count(int64_t rows, int64_t N, int64_t K, int32_t E,
                                           int32_t Ks, int32_t epilogue);
/* which form of the residual moe_w4a4_grouped_gemm reads for these sizes:
 * 0 none (Ks = 0 or empty), 1 the masked residual rq, 2 the compact rq_sel
 * (with rq's tensor scale).  Pure host function, no error path. */
int32_t   moe_w4a4_grouped_gemm_residual_form(int64_t rows, int64_t N, int64_t K, int32_t E,
                                              int32_t Ks, int32_t epilogue);
qd_status moe_w4a4_grouped_gemm(const qd_nvfp4 *a, const int32_t *row_token,
                                const int32_t *expert_offsets, int32_t E, int64_t rows,
                                const qd_nvfp4 *w, const qd_nvfp4 *rq,
                                const int32_t *sel_idx, int32_t Ks, const void *rq_sel,
                                int32_t epilogue, void *out, float *amax_partials,
                                void *stream);

/* ---------------------------------------------------------------------
 * moe_w4a4_grouped_gemm_per_expert -- moe_w4a4_grouped_gemm with one
 * channel set per expert (the variant of Sec. 3.3 computed by
 * rac_select_channels_per_expert): rows of expert e subtract the residual
 * at S_e,
 *   v[r][n] = s_dec_a*s_dec_w[e] * acc - s_dec_r*s_dec_w[e] * sum_{j in S_e} rhat[t][j] w[e][n][j].
 *   sel_pe          : int32 [E][Ks] (each ascending); Ks >= 1.
 *   rq              : the residual (only its tensor scale is read).
 *   rq_sel_rows     : f16 [rows][rac_selected_width(Ks)] by grouped row.
 *   amax_partials   : optional float
 *                     [moe_w4a4_grouped_gemm_per_expert_amax_count(...)].
 *   Other arguments as moe_w4a4_grouped_gemm.  Runs on the kernel for many
 *   rows per expert at every size: QD_ERR_UNSUPPORTED where it does not
 *   apply (K a multiple of 128 and >= 256, N a multiple of 128, Ks <= ~440).
 * ------------------------------------------------------------------- */
int64_t   moe_w4a4_grouped_gemm_per_expert_amax_count(int64_t rows, int64_t N, int64_t K,
                                                      int32_t E, int32_t Ks, int32_t epilogue);
qd_status moe_w4a4_grouped_gemm_per_expert(const qd_nvfp4 *a, const int32_t *row_token,
                                           const int32_t *expert_offsets, int32_t E, int64_t rows,
                                           const qd_nvfp4 *w, const qd_nvfp4 *rq,
                                           const int32_t *sel_pe, int32_t Ks,
                                           const void *rq_sel_rows, int32_t epilogue, void *out,
                                           float *amax_partials, void *stream);

/* ---------------------------------------------------------------------
 * nvfp4_pack_frag_scales -- a load-time re-layout of a weight tensor's
 * scales for the W4A4 expert GEMM of Sec. 3.3 on decode-shaped batches.
 * That kernel streams each 16-row block of weights over K in chunks of 256
 * elements; in the standard layout the 16 scale bytes a row needs per chunk
 * lie 16 bytes apart in every row's scale line, in this one the 256 bytes of
 * a block and chunk are contiguous, in the order the kernel's lanes take
 * them.  Values are not touched.
 *   w   : weights, groups E of [rows][cols]; rows % 16 == 0,
 *         cols % 256 == 0 (otherwise QD_ERR_SHAPE).
 *   out : uint8 [E][rows/16][cols/256][4][16][4] (16-byte aligned,
 *         nvfp4_frag_scales_bytes(E, rows, cols) bytes), where
 *         out[e][f][c][g][l][b] = scales[e][16 f + l][16 c + 4 g + b].
 * Set w->scales_frag = out afterwards; moe_w4a4_grouped_gemm and
 * qd_moe_layer_forward then read it instead of w->scales where it pays.
 * ------------------------------------------------------------------- */
int64_t   nvfp4_frag_scales_bytes(int64_t groups, int64_t rows, int64_t cols);
qd_status nvfp4_pack_frag_scales(const qd_nvfp4 *w, uint8_t *out, void *stream);

/* ---------------------------------------------------------------------
 * moe_unpermute_combine -- the last step of the MoE layer whose expert
 * GEMMs Sec. 3.3 quantises (the MoE model of Sec. 4.1; the paper gives no
 * router or combine details, so this is the standard top-k combine): the
 * weighted sum of the k expert outputs per token,
 *   y[t][n] = bf16( sum_{s=0..k-1} topk_w[t][s] * z[inv_row[t][s]][n] ),
 * accumulated in f32 in slot order.
 *   z : bf16 [T*k][H]; y : bf16 [T][H]; 1 <= k <= 32, H % 8 == 0.
 * ------------------------------------------------------------------- */
qd_status moe_unpermute_combine(const void *z, const int32_t *inv_row, const float *topk_w,
                                int64_t T, int32_t k, int64_t H, void *y, void *stream);

/* ---------------------------------------------------------------------
 * FP8 W8A8 comparison layer (Sec. 2.2 "FP8" paragraph: the FP8 rollout the
 * paper compares against), same routing, SwiGLU and combine, no residual.
 *
 * fp8_quantize_rows -- E4M3 codes with one f32 scale per row: for a row with
 * amax m > 0, enc = 448 / m, dec = 1 / enc (f32);
 * code = E4M3_RNE(min(|x * enc|, 448)) with the sign in bit 7; a zero row
 * takes dec = 1.  Weights [E][N][K] are E*N rows (one scale per output
 * channel), activations one scale per token.
 *   x     : bf16 (QD_DTYPE_BF16) or f32 [rows][cols].
 *   codes : u8 [rows][cols];  dec: f32 [rows].
 * ------------------------------------------------------------------- */
qd_status fp8_quantize_rows(const void *x, int32_t dtype, int64_t rows, int64_t cols,
                            uint8_t *codes, float *dec, void *stream);

/* ---------------------------------------------------------------------
 * moe_fp8_grouped_gemm -- per expert e and grouped row r:
 *   v[r][n] = a_dec[src(r)] * w_dec[e][n] * sum_k a[src(r)][k] * w[e][n][k]
 * (E4M3 products exact, f32 accumulation), epilogue as in
 * moe_w4a4_grouped_gemm (QD_EPI_NONE: bf16 [rows][N]; QD_EPI_SWIGLU: N = 2I,
 * bf16 [rows][I]).
 *   a_codes, a_dec  : u8 [a_rows][K], f32 [a_rows];  row_token / offsets as
 *                     in moe_w4a4_grouped_gemm.
 *   w_codes, w_dec  : u8 [E][N][K], f32 [E][N].
 * Sizes: K % 64 == 0, K >= 256; N % 256 == 0 (few rows per expert) or
 * N % 128 == 0 (many); otherwise QD_ERR_UNSUPPORTED.  16-byte aligned codes
 * and output.
 * ------------------------------------------------------------------- */
qd_status moe_fp8_grouped_gemm(const uint8_t *a_codes, const float *a_dec, int64_t a_rows,
                               const int32_t *row_token, const int32_t *expert_offsets,
                               int32_t E, int64_t rows, const uint8_t *w_codes,
                               const float *w_dec, int64_t N, int64_t K, int32_t epilogue,
                               void *out, void *stream);

/* qd_fp8_moe_layer_forward -- route, quantise X per token, W13 with SwiGLU,
 * quantise h per row, W2, combine: y bf16 [T][H].  w13: [E][2I][H] codes and
 * [E][2I] scales; w2: [E][H][I] and [E][H] (from fp8_quantize_rows). */
size_t    qd_fp8_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I);
qd_status qd_fp8_moe_layer_forward(const void *x, const float *logits, int64_t T, int64_t H,
                                   int32_t E, int32_t k, int64_t I, int32_t renorm,
                                   const uint8_t *w13_codes, const float *w13_dec,
                                   const uint8_t *w2_codes, const float *w2_dec, void *y,
                                   void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * MXFP4 W4A4 comparison layer: the OCP Microscaling FP4 format that CDNA4's
 * scaled MFMA reads natively (E2M1 elements, one E8M0 power-of-two scale
 * per 32 elements, no tensor scale), on the same routing, SwiGLU and combine
 * as the NVFP4 layer and without residual.  It is not the paper's format:
 * it measures what the exact NVFP4 semantics of Sec. 2.2 ("FP4" paragraph:
 * E4M3 scale per 16 elements, FP32 tensor scale) cost on this hardware.
 *
 * mxfp4_quantize_rows -- per block of 32 consecutive elements of a row,
 * with m = max |x|: s = floor(log2 m) - 2, clamped to [-127, 127] (-127 for
 * m == 0); scale byte s + 127.  code = E2M1_RNE(|x| * 2^-s) with ties to
 * even, saturating at 6, and the sign in bit 3.
 *   x      : bf16 (QD_DTYPE_BF16) or f32 [rows][cols], cols % 32 == 0,
 *            16-byte aligned.
 *   codes  : u8 [rows][cols/2], element 2i in bits 3:0 (16-byte aligned).
 *   scales : u8 [rows][cols/32].
 * ------------------------------------------------------------------- */
qd_status mxfp4_quantize_rows(const void *x, int32_t dtype, int64_t rows, int64_t cols,
                              uint8_t *codes, uint8_t *scales, void *stream);

/* ---------------------------------------------------------------------
 * moe_mxfp4_grouped_gemm -- per expert e and grouped row r:
 *   v[r][n] = sum_k a[src(r)][k] * w[e][n][k]   (MXFP4 values, f32 accumulation
 *   on v_mfma_scale_f32_32x32x64_f8f6f4), epilogue as in moe_w4a4_grouped_gemm.
 *   a_codes, a_scales : u8 [a_rows][K/2], u8 [a_rows][K/32] (4-byte aligned).
 *   w_codes, w_scales : u8 [E][N][K/2], u8 [E][N][K/32].
 *   row_token / offsets as in moe_w4a4_grouped_gemm.
 * Sizes: K % 128 == 0, K >= 256; N % 256 == 0 (few rows per expert) or
 * N % 128 == 0 (many); otherwise QD_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------- */
qd_status moe_mxfp4_grouped_gemm(const uint8_t *a_codes, const uint8_t *a_scales, int64_t a_rows,
                                 const int32_t *row_token, const int32_t *expert_offsets,
                                 int32_t E, int64_t rows, const uint8_t *w_codes,
                                 const uint8_t *w_scales, int64_t N, int64_t K, int32_t epilogue,
                                 void *out, void *stream);

/* qd_mxfp4_moe_layer_forward -- route, quantise X, W13 with SwiGLU, quantise h,
 * W2, combine: y bf16 [T][H].  w13: [E][2I][H/2] codes and [E][2I][H/32]
 * scales; w2: [E][H][I/2] and [E][H][I/32] (from mxfp4_quantize_rows). */
size_t    qd_mxfp4_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I);
qd_status qd_mxfp4_moe_layer_forward(const void *x, const float *logits, int64_t T, int64_t H,
                                     int32_t E, int32_t k, int64_t I, int32_t renorm,
                                     const uint8_t *w13_codes, const uint8_t *w13_scales,
                                     const uint8_t *w2_codes, const uint8_t *w2_scales, void *y,
                                     void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * moe_w4a16_grouped_gemm -- the trainer-side forward of Sec. 3.2, Eq.
 * (w4a16-qat-forward): bf16 activations times the NVFP4 fake-quantised
 * weights (asymmetric W4A16; the same QDQ_W as the rollout side, Eq.
 * (weight-qdq-align)), grouped over experts:
 *   v[r][n] = s_dec_w[e(r)] * sum_k a[src(r)][k] * what[e(r)][n][k]
 * with what = e2m1 * e4m3 (exact in bf16), products exact, f32 sums.
 *   a               : bf16 [a_rows][K], 16-byte aligned; row_token values
 *                     must lie in [0, a_rows).
 *   row_token       : int32 [rows] gather map (NULL: row r reads a row r).
 *   expert_offsets  : int32 [E+1] row ranges per expert (NULL: E must be 1).
 *   w               : E groups of [N][K]; K % 64 == 0, N % 32 == 0.
 *   epilogue        : QD_EPI_NONE: out bf16 [rows][N] = bf16(v);
 *                     QD_EPI_SWIGLU: gate rows [0, N/2), up rows [N/2, N);
 *                     out bf16 [rows][N/2] = bf16(silu(g) * u).
 * E <= 1024.  The backward pass (straight-through estimator) needs no
 * kernel of its own.
 * ------------------------------------------------------------------- */
qd_status moe_w4a16_grouped_gemm(const void *a, int64_t a_rows, const int32_t *row_token,
                                 const int32_t *expert_offsets, int32_t E, int64_t rows,
                                 const qd_nvfp4 *w, int32_t epilogue, void *out, void *stream);

/* ---------------------------------------------------------------------
 * qd_moe_layer_forward -- the whole rollout-side layer in one call: route,
 * quantise X with fused RAC scores, select, W13 GEMM with fused residual
 * and SwiGLU, quantise h, W2 GEMM, combine.  Same results as the seven
 * calls above in that order (bit for bit); routing and the X chain are
 * independent, so their kernels share launches here.
 *   x      : bf16 [T][H]; logits: f32 [T][E];
 *   w13    : E groups of [2I][H]; w2: E groups of [H][I];
 *   y      : bf16 [T][H];
 *   Ks     : channels of X compensated at the W13 input (0 <= Ks <= H).
 *   Ks2    : channels of h compensated at the W2 input (0 <= Ks2 <= I; 0
 *            is the paper's configuration).  With Ks2 > 0, h is quantised
 *            with its channel scores (a fresh amax pass over h), the top
 *            Ks2 channels are selected over all T*k rows (one set for all
 *            experts) and the W2 GEMM takes the masked residual as W13
 *            does, Sec. 3.3, Eq. (residual-recon).
 *   ws     : at least qd_moe_layer_workspace(T, H, E, k, I) bytes; the
 *            intermediates live there (see qd_moe_layer_views).
 * Errors: QD_ERR_SHAPE as the calls above (E <= 1024, k <= 32);
 * QD_ERR_UNSUPPORTED for Ks > 0 with H > 16384.
 * ------------------------------------------------------------------- */
size_t    qd_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I);
qd_status qd_moe_layer_forward(const void *x, const float *logits, int64_t T, int64_t H,
                               int32_t E, int32_t k, int64_t I, int32_t Ks, int32_t Ks2,
                               int32_t renorm,
                               const qd_nvfp4 *w13, const qd_nvfp4 *w2, void *y,
                               void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------
 * qd_moe_layer_forward_per_expert -- the layer with one RAC channel set per
 * expert at the W13 input (rac_select_channels_per_expert,
 * moe_w4a4_grouped_gemm_per_expert), composed of the boundary calls:
 * route, quantise X, per-expert selection and residual, W13 with SwiGLU,
 * quantise h, W2, combine.  Arguments as qd_moe_layer_forward (no W2-site
 * residual); 1 <= Ks <= H; ws at least
 * qd_moe_layer_per_expert_workspace(T, H, E, k, I, Ks) bytes.
 * ------------------------------------------------------------------- */
size_t    qd_moe_layer_per_expert_workspace(int64_t T, int64_t H, int32_t E, int32_t k,
                                            int64_t I, int32_t Ks);
qd_status qd_moe_layer_forward_per_expert(const void *x, const float *logits, int64_t T,
                                          int64_t H, int32_t E, int32_t k, int64_t I, int32_t Ks,
                                          int32_t renorm, const qd_nvfp4 *w13,
                                          const qd_nvfp4 *w2, void *y, void *ws, size_t ws_bytes,
                                          void *stream);

/*
 * Same as qd_moe_layer_forward, recording HIP events at the stage
 * boundaries: events is a host array of QD_STAGE_COUNT + 1 hipEvent_t (as
 * void*); events[i] is recorded on `stream` before stage i and
 * events[QD_STAGE_COUNT] after the last one (stages in the order below).
 * With the shared launches the first three stages are: ROUTE = routing
 * top-k with the amax pass over X; QUANT_X = routing ranks with the X
 * quantiser; SELECT = routing scatter with the channel selection, then the
 * masked residual (scatter alone when Ks == 0).  With Ks2 > 0, QUANT_H
 * also holds the W2-site selection and masked residual.  events NULL: no
 * recording.
 */
enum {
  QD_STAGE_ROUTE = 0, QD_STAGE_QUANT_X, QD_STAGE_SELECT, QD_STAGE_W13, QD_STAGE_QUANT_H,
  QD_STAGE_W2, QD_STAGE_COMBINE, QD_STAGE_COUNT
};
qd_status qd_moe_layer_forward_timed(const void *x, const float *logits, int64_t T, int64_t H,
                                     int32_t E, int32_t k, int64_t I, int32_t Ks, int32_t Ks2,
                                     int32_t renorm,
                                     const qd_nvfp4 *w13, const qd_nvfp4 *w2, void *y,
                                     void *ws, size_t ws_bytes, void *const *events,
                                     void *stream);

/*
 * Byte offsets of the layer's intermediates inside its workspace (host
 * output array `off`, QD_VIEW_COUNT entries), so a caller can inspect them
 * after qd_moe_layer_forward.
 */
enum {
  QD_VIEW_TOPK_IDS = 0, QD_VIEW_TOPK_W, QD_VIEW_OFFSETS, QD_VIEW_ROW_TOKEN, QD_VIEW_INV_ROW,
  QD_VIEW_XQ_CODES, QD_VIEW_XQ_SCALES, QD_VIEW_XQ_GSCALE, QD_VIEW_SCORES, QD_VIEW_RAMAX,
  QD_VIEW_SEL, QD_VIEW_RQ_CODES, QD_VIEW_RQ_SCALES, QD_VIEW_RQ_GSCALE, QD_VIEW_H,
  QD_VIEW_H_AMAX, QD_VIEW_HQ_CODES, QD_VIEW_HQ_SCALES, QD_VIEW_HQ_GSCALE, QD_VIEW_Z,
  QD_VIEW_RQ_SEL, QD_VIEW_H_SCORES, QD_VIEW_H_RAMAX, QD_VIEW_SEL2, QD_VIEW_HR_CODES,
  QD_VIEW_HR_SCALES, QD_VIEW_HR_GSCALE, QD_VIEW_HR_SEL, QD_VIEW_COUNT
};
qd_status qd_moe_layer_views(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I,
                             int64_t *off /* host, QD_VIEW_COUNT */);

/* ---------------------------------------------------------------------
 * qd_moe_block_forward -- the layer fed straight from the transformer's
 * hidden state: RMSNorm and the router folded into the layer's first launch
 * (the MoE block of Sec. 4.1's model; the paper names neither step, the
 * readings are: x = bf16(h / sqrt(mean_j h_j^2 + eps) * gamma), logits =
 * f32(x w_router^T)).  One pass over h gives x, the router logits (bf16
 * MFMAs, f32 accumulation), the top-k routing and the amax partials of x;
 * the rest is qd_moe_layer_forward on that x and those logits, bit for bit.
 *   h        : bf16 [T][H] (the hidden state before the norm);
 *   gamma    : bf16 [H] (the norm's gain); eps >= 0 (finite);
 *   w_router : bf16 [E][H] (row-major, one row per expert); E <= 256;
 *   other arguments as qd_moe_layer_forward; ws at least
 *   qd_moe_block_workspace(T, H, E, k, I) bytes (the layer's workspace, then
 *   x bf16 [T][H] and the logits f32 [T][E] at the offsets
 *   qd_moe_block_views gives in off[QD_BLOCK_VIEW_X] and
 *   off[QD_BLOCK_VIEW_LOGITS]; off has QD_BLOCK_VIEW_COUNT entries, the
 *   first QD_VIEW_COUNT as qd_moe_layer_views).
 * x and the logits are float32 arithmetic on the GPU (squares summed per
 * lane, then across the wave; 1 / sqrt correctly rounded): within one bf16
 * ulp of the float64 reading for x, and within float32 accumulation error
 * for the logits.
 * Errors: as qd_moe_layer_forward; QD_ERR_UNSUPPORTED for E > 256 or
 * H > 9208 (eight normalised rows must fit 144 KiB of LDS);
 * QD_ERR_SHAPE for a negative or non-finite eps.
 * ------------------------------------------------------------------- */
enum { QD_BLOCK_VIEW_X = QD_VIEW_COUNT, QD_BLOCK_VIEW_LOGITS, QD_BLOCK_VIEW_COUNT };
size_t    qd_moe_block_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I);
qd_status qd_moe_block_views(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I,
                             int64_t *off /* host, QD_BLOCK_VIEW_COUNT */);
qd_status qd_moe_block_forward(const void *h, const void *gamma, float eps, const void *w_router,
                               int64_t T, int64_t H, int32_t E, int32_t k, int64_t I, int32_t Ks,
                               int32_t Ks2, int32_t renorm, const qd_nvfp4 *w13,
                               const qd_nvfp4 *w2, void *y, void *ws, size_t ws_bytes,
                               void *stream);
/* the same with stage events as qd_moe_layer_forward_timed (ROUTE holds the
 * norm, the router and the top-k) */
qd_status qd_moe_block_forward_timed(const void *h, const void *gamma, float eps,
                                     const void *w_router, int64_t T, int64_t H, int32_t E,
                                     int32_t k, int64_t I, int32_t Ks, int32_t Ks2,
                                     int32_t renorm, const qd_nvfp4 *w13, const qd_nvfp4 *w2,
                                     void *y, void *ws, size_t ws_bytes, void *const *events,
                                     void *stream);

/* ---------------------------------------------------------------------
 * qd_moe_layer_forward_noalloc -- qd_moe_layer_forward without a caller
 * workspace, for callers that cannot allocate device memory: code under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc.
 * Same arguments (minus ws / ws_bytes), same kernels, same results bit for
 * bit.  The intermediates live in a scratch buffer of
 * QD_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds as a static
 * device array: each device the library runs on keeps its own copy until
 * the process ends.  The call allocates nothing (no hipMalloc / hipFree,
 * no allocating library routine); its first call on a device looks up that
 * device's copy (the device current at the call must be the stream's).
 *   Errors: QD_ERR_WORKSPACE if qd_moe_layer_workspace(T, H, E, k, I) exceeds
 *   qd_moe_layer_noalloc_max_bytes() (decode batches fit: 17.3 MiB for 256
 *   tokens at H = 2048, E = 128, k = 8, I = 768); otherwise as
 *   qd_moe_layer_forward.
 * Every call on one device shares that device's scratch buffer and leaves
 * the last call's intermediates in it: calls that overlap on one device
 * (several streams or host threads) race; calls on one stream are ordered.
 * ------------------------------------------------------------------- */
#define QD_NOALLOC_SCRATCH_BYTES (64u << 20)
size_t    qd_moe_layer_noalloc_max_bytes(void);
qd_status qd_moe_layer_forward_noalloc(const void *x, const float *logits, int64_t T,
                                       int64_t H, int32_t E, int32_t k, int64_t I, int32_t Ks,
                                       int32_t Ks2, int32_t renorm, const qd_nvfp4 *w13,
                                       const qd_nvfp4 *w2, void *y, void *stream);

/* ---------------------------------------------------------------------
 * Achievable-peak probes (measurement only, not part of the layer): the
 * rates the chip reaches in practice, stated beside its published peaks.
 * qd_probe_hbm_read -- streams `bytes` (a multiple of 16) of device memory
 *   `buf` once with 16-byte loads; out: uint32 [qd_probe_hbm_read_out_count()]
 *   scratch results.  Time it with events on `stream`: bytes / time is the
 *   achievable read bandwidth (use a buffer far larger than the 256 MB
 *   Infinity Cache).
 * qd_probe_mfma_f16 -- `workgroups` workgroups of four waves, each wave
 *   running `rounds` rounds of 16 independent v_mfma_f32_32x32x16_f16 on
 *   registers; qd_probe_mfma_f16_flops(rounds, workgroups) is the work in
 *   FLOP; out: float [workgroups].  random_operands = 0: slowly varying
 *   operand values (few bits toggle); 1: operands with random signs,
 *   exponents and mantissas, which draw more power and run at a lower
 *   clock -- the ceiling that GEMMs on real data see.
 * ------------------------------------------------------------------- */
int64_t   qd_probe_hbm_read_out_count(void);
qd_status qd_probe_hbm_read(const void *buf, int64_t bytes, uint32_t *out, void *stream);
double    qd_probe_mfma_f16_flops(int64_t rounds, int32_t workgroups);
qd_status qd_probe_mfma_f16(int64_t rounds, int32_t workgroups, int32_t random_operands,
                            float *out, void *stream);

#if defined(__GNUC__) || defined(__clang__)
#pragma GCC visibility pop
#endif

#ifdef __cplusplus
}
#endif
#endif /* QUADS_H */
