// Kernel-level entry points (flashbon_ops.h): validation, then one launch each.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <string>

#include "../../include/flashbon_ops.h"
#include "dispatch.h"
#include "kernels.h"
#include "model.h"

using namespace fb;

static flashbon_status launched(hipError_t e, const char *what) {
  if (e != hipSuccess) return fail(FLASHBON_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  return FLASHBON_OK;
}

extern "C" {

flashbon_status flashbon_op_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                   const void *W, const float *bias, int32_t epilogue, void *out,
                                   const float *gate, float *cache_out, void *stream) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (M < 1 || N < 1 || K < 1 || K % 8 || N % 4 || K > 65536)
    return fail(FLASHBON_ESHAPE, "need M,N,K >= 1, K <= 65536, K % 8 == 0, N % 4 == 0");
  if (!A || !W || !out) return fail(FLASHBON_EINVAL, "A, W and out are required");
  if (epilogue < FLASHBON_EPI_STORE || epilogue > FLASHBON_EPI_RESIDUAL) return fail(FLASHBON_EINVAL, "bad epilogue");
  EpiArgs e;
  e.out = out; e.ldo = N; e.bias = bias;
  if (epilogue == FLASHBON_EPI_RESIDUAL) { e.gate = gate; e.cache = cache_out; }
  ActType t = dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  return launched(launch_linear(t, epilogue, M, N, K, A, W, e, (hipStream_t)stream), "linear");
}

flashbon_status flashbon_op_linear_ws(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                      const void *W, const float *bias, int32_t epilogue, void *out,
                                      const float *gate, float *cache_out, void *workspace,
                                      size_t workspace_bytes, int32_t *splits, void *stream) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (M < 1 || N < 1 || K < 1 || K % 8 || N % 4 || K > 65536)
    return fail(FLASHBON_ESHAPE, "need M,N,K >= 1, K <= 65536, K % 8 == 0, N % 4 == 0");
  if (!A || !W || !out) return fail(FLASHBON_EINVAL, "A, W and out are required");
  if (epilogue < FLASHBON_EPI_STORE || epilogue > FLASHBON_EPI_RESIDUAL) return fail(FLASHBON_EINVAL, "bad epilogue");
  EpiArgs e;
  e.out = out; e.ldo = N; e.bias = bias;
  if (epilogue == FLASHBON_EPI_RESIDUAL) { e.gate = gate; e.cache = cache_out; }
  ActType t = dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  int sp = t == ACT_BF16 && workspace ? splitk_splits(epilogue, M, N, K) : 1;
  if (sp > 1 && (size_t)sp * M * N * 4 > workspace_bytes) sp = 1;
  if (splits) *splits = sp;
  return launched(launch_linear_ws(t, epilogue, M, N, K, A, W, e, (hipStream_t)stream, workspace, workspace_bytes),
                  "linear");
}

flashbon_status flashbon_op_linear_residual(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                                            const void *W, const float *bias, const float *gate,
                                            const float *residual_in, float *out, void *stream) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (M < 1 || N < 1 || K < 1 || K % 8 || N % 4 || K > 65536)
    return fail(FLASHBON_ESHAPE, "need M,N,K >= 1, K <= 65536, K % 8 == 0, N % 4 == 0");
  if (!A || !W || !out || !residual_in) return fail(FLASHBON_EINVAL, "A, W, residual_in and out are required");
  EpiArgs e;
  e.out = out; e.ldo = N; e.bias = bias; e.gate = gate;
  if (residual_in != out) e.res_in = residual_in;
  ActType t = dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  return launched(launch_linear(t, FLASHBON_EPI_RESIDUAL, M, N, K, A, W, e, (hipStream_t)stream), "linear");
}

flashbon_status flashbon_op_linear_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue,
                                        int32_t *kernels, char *desc, int32_t desc_len) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (M < 1 || N < 1 || K < 1 || K % 8 || N % 4 || K > 65536)
    return fail(FLASHBON_ESHAPE, "need M,N,K >= 1, K <= 65536, K % 8 == 0, N % 4 == 0");
  if (epilogue < FLASHBON_EPI_STORE || epilogue > FLASHBON_EPI_RESIDUAL) return fail(FLASHBON_EINVAL, "bad epilogue");
  if (!kernels || (desc && desc_len < 1)) return fail(FLASHBON_EINVAL, "kernels is required; desc_len >= 1 with desc");
  *kernels = describe_linear(dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32, epilogue, M, N, K, desc, desc ? desc_len : 0);
  return FLASHBON_OK;
}

flashbon_status flashbon_op_attention(int32_t dtype, int32_t batch, int32_t heads, int32_t head_dim,
                                      int32_t tq, int32_t tk, const void *q, int64_t q_batch_stride,
                                      int64_t q_row_stride, const void *k, const void *v,
                                      int64_t kv_batch_stride, int64_t kv_row_stride,
                                      const int32_t *kv_index, int32_t n_kv, void *out,
                                      int64_t out_batch_stride, int64_t out_row_stride, void *stream) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (batch < 1 || heads < 1 || tq < 1 || tk < 1) return fail(FLASHBON_ESHAPE, "batch, heads, tq, tk must be >= 1");
  if (head_dim != 8 && head_dim != 16 && head_dim != 32 && head_dim != 64 && head_dim != 128)
    return fail(FLASHBON_ESHAPE, "head_dim must be one of 8, 16, 32, 64, 128");
  if (!q || !k || !v || !out) return fail(FLASHBON_EINVAL, "q, k, v and out are required");
  if (kv_index && n_kv < 1) return fail(FLASHBON_ESHAPE, "n_kv must be >= 1 with kv_index");
  AttnArgs a;
  a.batch = batch; a.heads = heads; a.head_dim = head_dim; a.tq = tq; a.tk = tk;
  a.q = q; a.q_bs = q_batch_stride; a.q_rs = q_row_stride;
  a.k = k; a.v = v; a.kv_bs = kv_batch_stride; a.kv_rs = kv_row_stride;
  a.kv_index = kv_index; a.n_kv = kv_index ? n_kv : batch;
  a.out = out; a.o_bs = out_batch_stride; a.o_rs = out_row_stride;
  ActType t = dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  return launched(launch_attention(t, a, (hipStream_t)stream), "attention");
}

flashbon_status flashbon_op_ln_mod(int32_t dtype, int32_t M, int32_t D, float eps, const float *x,
                                   const float *shift, const float *scale, void *out, void *stream) {
  if (dtype != FLASHBON_FP32 && dtype != FLASHBON_BF16) return fail(FLASHBON_EINVAL, "bad dtype");
  if (M < 1 || D < 4 || D % 4 || D > 6144) return fail(FLASHBON_ESHAPE, "need M >= 1, 4 <= D <= 6144, D % 4 == 0");
  if (!x || !out) return fail(FLASHBON_EINVAL, "x and out are required");
  if ((shift == nullptr) != (scale == nullptr)) return fail(FLASHBON_EINVAL, "shift and scale go together");
  if (!(eps > 0.f)) return fail(FLASHBON_EINVAL, "eps must be positive");
  ActType t = dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  return launched(launch_ln_mod(t, M, D, eps, x, shift, scale, out, (hipStream_t)stream), "ln_mod");
}

flashbon_status flashbon_op_proxy(int64_t count, const float *h1, const float *h2, const float *h3,
                                  int32_t order, float tau1, float tau2, float t_cur, float *out,
                                  void *stream) {
  if (count < 1) return fail(FLASHBON_ESHAPE, "count must be >= 1");
  if (order < 0 || order > 2) return fail(FLASHBON_EINVAL, "order must be 0, 1 or 2");
  if (!h1 || !out || (order >= 1 && !h2) || (order >= 2 && !h3))
    return fail(FLASHBON_EINVAL, "missing cached entries");
  if (order >= 1 && (!(tau1 != tau2) || !std::isfinite(tau1) || !std::isfinite(tau2) || !std::isfinite(t_cur)))
    return fail(FLASHBON_EINVAL, "tau1 and tau2 must be finite and distinct");
  flashbon_cache_meta mb;
  mb.count = order + 1; mb.head = 0;
  mb.t[2] = tau1; mb.t[1] = tau2; mb.t[0] = 0.f;   // most recent = (head+2)%3, then (head+1)%3
  float ca, cb;
  taylor_coefficients(mb, t_cur, order, &ca, &cb);
  return launched(launch_proxy(count, h1, h2, h3, order, ca, cb, out, (hipStream_t)stream), "proxy");
}

flashbon_status flashbon_op_normals(int64_t count, int32_t candidate, int32_t step, uint64_t seed,
                                    uint32_t *words, float *normals, void *stream) {
  if (count < 1 || count > ((int64_t)1 << 34)) return fail(FLASHBON_ESHAPE, "count outside [1, 2^34]");
  if (candidate < 0 || step < 0) return fail(FLASHBON_EINVAL, "candidate and step must be >= 0");
  if (!words && !normals) return fail(FLASHBON_EINVAL, "words or normals is required");
  return launched(launch_normals(count, (uint32_t)candidate, (uint32_t)step, seed, words, normals,
                                 (hipStream_t)stream), "normals");
}

flashbon_status flashbon_op_unpatch_sde(int32_t n, int32_t C, int32_t H, int32_t W, int32_t p,
                                        const float *v, float *z, float t_cur, float t_next, float a,
                                        uint64_t seed, int32_t step, int32_t row0, void *stream) {
  if (n < 1 || n > 65535 || C < 1 || p < 1 || H < p || W < p || H % p || W % p)
    return fail(FLASHBON_ESHAPE, "need 1 <= n <= 65535, C >= 1, H and W positive multiples of p");
  if ((int64_t)C * H * W > INT32_MAX) return fail(FLASHBON_ESHAPE, "C H W must fit in int32");
  if (!v || !z) return fail(FLASHBON_EINVAL, "v and z are required");
  if (step < 0 || row0 < 0) return fail(FLASHBON_EINVAL, "step and row0 must be >= 0");
  SdeArgs s;
  if (!sde_coefficients(t_cur, t_next, a, seed, step, row0, &s))
    return fail(FLASHBON_EINVAL, "need a >= 0, finite, and 0 < t_cur <= 1 (t_next < 1 when t_cur = 1)");
  return launched(launch_head_update(n, C, H, W, p, v, false, 0.f, z, s, nullptr, 0.f, (hipStream_t)stream),
                  "unpatch_sde");
}

}  // extern "C"
