/*
 * flashbon_ops.h -- kernel-level entry points of the same library.
 *
 * These expose the individual HIP kernels the draft step is built from, so each can be checked
 * against the CPU oracle at the model's real shapes.  They follow the conventions of flashbon.h
 * (status codes, host validation before any device work, caller-owned device buffers, work enqueued
 * on `stream` without synchronising).  `dtype` is a flashbon_dtype: "act" below means bf16 (raw
 * 16-bit words, round-to-nearest-even from fp32) in FLASHBON_BF16 and fp32 in FLASHBON_FP32.
 */
#ifndef FLASHBON_OPS_H
#define FLASHBON_OPS_H

#include "flashbon.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FLASHBON_EPI_STORE = 0,    /* out[m][n] (act)  = acc + bias[n]                                  */
  FLASHBON_EPI_GELU = 1,     /* out[m][n] (act)  = GELU_tanh(acc + bias[n])                       */
  FLASHBON_EPI_STORE_F32 = 2,/* out[m][n] (fp32) = acc + bias[n]                                  */
  FLASHBON_EPI_RESIDUAL = 3  /* out[m][n] (fp32) += gate[n] * (acc + bias[n]) (gate NULL -> 1);
                                if cache_out != NULL also cache_out[m][n] = the updated out[m][n]  */
};

/* Linear layer: acc[m][n] = sum_k A[m][k] W[n][k] with fp32 accumulation (a DiT projection y = x W^T).
 * A: device act [M][K]; W: device act [N][K]; bias: device fp32 [N] or NULL (0);
 * out: device [M][N] (act or fp32 per epilogue); gate: device fp32 [N] or NULL; cache_out: device
 * fp32 [M][N] or NULL.  M, N >= 1, N % 4 == 0; 1 <= K <= 65536 and K % 8 == 0. */
flashbon_status flashbon_op_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                   const void *W, const float *bias, int32_t epilogue, void *out,
                                   const float *gate, float *cache_out, void *stream);

/* Residual linear layer reading the residual rows from a separate buffer:
 * out[m][n] = residual_in[m][n] + gate[n] * (acc[m][n] + bias[n]) (gate NULL -> 1), acc as in
 * flashbon_op_linear (a block's gated residual update, Eq. 7, with the input stream and the output in
 * different buffers).  residual_in: device fp32 [M][N], read only; it may be out itself (then this is
 * flashbon_op_linear with FLASHBON_EPI_RESIDUAL) and must not otherwise overlap out.  out: device
 * fp32 [M][N].  Shape rules and errors as flashbon_op_linear; residual_in and out are required. */
flashbon_status flashbon_op_linear_residual(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                            const void *W, const float *bias, const float *gate,
                                            const float *residual_in, float *out, void *stream);

/* flashbon_op_linear with a caller-owned workspace (device, workspace_bytes) for split-K partial sums,
 * as the draft and refinement steps run their linear layers: a bf16 shape whose 224 x 256 tiles would
 * fill less than half the CUs (one candidate's MLP down-projection, M = 1560, N = 1536, K = 8960) is cut
 * into K ranges of at least 16 x 64 columns, each range's fp32 partial sums stored in the workspace
 * (splits x M x N x 4 bytes, at most 48 MiB), then added in range order before the epilogue; other
 * shapes, and a workspace too small for the plan, run exactly as flashbon_op_linear.  *splits (optional)
 * receives the number of K ranges used (1 = none).  Arguments otherwise as flashbon_op_linear; the
 * workspace must not overlap any other buffer. */
flashbon_status flashbon_op_linear_ws(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                      const void *W, const float *bias, int32_t epilogue, void *out,
                                      const float *gate, float *cache_out, void *workspace,
                                      size_t workspace_bytes, int32_t *splits, void *stream);

/* The tile plan flashbon_op_linear (and every projection of the draft step) takes for this shape,
 * without launching anything or touching the GPU: *kernels = the number of kernel launches, desc =
 * a NUL-terminated one-line description of the kernels and tiles (truncated to desc_len - 1
 * characters; desc may be NULL).  Same argument rules as flashbon_op_linear; follows the
 * FLASHBON_LINEAR_TILE override like the launch does.  The plan depends on the device's CU count
 * (256 when no device is visible). */
flashbon_status flashbon_op_linear_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue,
                                        int32_t *kernels, char *desc, int32_t desc_len);

/* Multi-head softmax attention, softmax(q k^T / sqrt(head_dim)) v per (batch b, head h):
 * q row i of batch b, head h is at q + b*q_batch_stride + i*q_row_stride + h*head_dim (act);
 * k/v row j at k/v + kvb*kv_batch_stride + j*kv_row_stride + h*head_dim, where kvb = b, or
 * kv_index[b] (device int32 [batch], values clamped into [0, n_kv)) if kv_index is not NULL
 * (cross-attention to the candidate's prompt);
 * out row i at out + b*out_batch_stride + i*out_row_stride + h*head_dim (act).
 * Strides are in elements.  head_dim <= 128, multiple of 8; tq, tk >= 1. */
flashbon_status flashbon_op_attention(int32_t dtype, int32_t batch, int32_t heads, int32_t head_dim,
                                      int32_t tq, int32_t tk, const void *q, int64_t q_batch_stride,
                                      int64_t q_row_stride, const void *k, const void *v,
                                      int64_t kv_batch_stride, int64_t kv_row_stride,
                                      const int32_t *kv_index, int32_t n_kv, void *out,
                                      int64_t out_batch_stride, int64_t out_row_stride, void *stream);

/* adaLN: out[m][d] (act) = LN(x[m])[d] * (1 + scale[d]) + shift[d], LN non-affine over D with eps;
 * x device fp32 [M][D]; shift/scale device fp32 [D] or both NULL (plain LN). */
flashbon_status flashbon_op_ln_mod(int32_t dtype, int32_t M, int32_t D, float eps, const float *x,
                                   const float *shift, const float *scale, void *out, void *stream);

/* Activation proxy of Eq. 3-5 over `count` fp32 elements, computed as the draft step computes it:
 * h1, h2, h3 are the cached outputs at tau1 (most recent), tau2, tau3 (h2 unused for order 0, h3
 * unused for order < 2; may be NULL then); out = proxy at t_cur.  All device fp32. */
flashbon_status flashbon_op_proxy(int64_t count, const float *h1, const float *h2, const float *h3,
                                  int32_t order, float tau1, float tau2, float t_cur, float *out,
                                  void *stream);

/* Counter-based normals of the stochastic update (App. A.1, Eq. 20), as flashbon_step_args defines
 * them, for `count` flat elements of one candidate row at one step: words (device uint32
 * [ceil(count / 4)][4], the Philox4x32-10 outputs of counters (q, candidate, step, 0)) and normals
 * (device fp32 [count]); either may be NULL. */
flashbon_status flashbon_op_normals(int64_t count, int32_t candidate, int32_t step, uint64_t seed,
                                    uint32_t *words, float *normals, void *stream);

/* Unpatchify + stochastic update (Eq. 20) as the step performs it: v is the head output, device fp32
 * [n (H/p)(W/p)][C p p] (token i (W/p) + j of candidate b, column c p^2 + p di + dj <-> z[b][c][p i +
 * di][p j + dj]); z device fp32 [n][C][H][W] updated in place; row b draws counter row row0 + b;
 * the rest as in flashbon_step_args.
 * H, W positive multiples of p. */
flashbon_status flashbon_op_unpatch_sde(int32_t n, int32_t C, int32_t H, int32_t W, int32_t p,
                                        const float *v, float *z, float t_cur, float t_next, float a,
                                        uint64_t seed, int32_t step, int32_t row0, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBON_OPS_H */
