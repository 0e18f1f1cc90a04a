// Softmax attention of the DiT block: self-attention over image tokens and cross-attention to the
// candidate's prompt tokens, softmax(q k^T / sqrt(dh)) v per (candidate, head).
//   * k_attn_valu: one lane per query, online softmax over 16-key sub-tiles staged in LDS as fp32;
//     any head_dim <= 128 (multiple of 8); fp32 or bf16 operands.  Used by the fp32 mode and for
//     head dims the MFMA kernel does not take.
#include "common.h"
#include "kernels.h"

namespace fb {

struct AttnP {
  int batch, heads, tq, tk;
  const void *q; int64_t q_bs, q_rs;
  const void *k; const void *v; int64_t kv_bs, kv_rs;
  const int32_t *kv_index; int n_kv;
  void *out; int64_t o_bs, o_rs;
  float qscale;  // log2(e) / sqrt(head_dim)
};

__device__ __forceinline__ int kv_batch(const AttnP &p, int b) {
  if (!p.kv_index) return b;
  int c = p.kv_index[b];
  return c < 0 ? 0 : (c >= p.n_kv ? p.n_kv - 1 : c);
}

template <typename T, int DH>
__global__ __launch_bounds__(64) void k_attn_valu(AttnP p) {
  constexpr int KT = 16;
  __shared__ float sK[KT][DH];
  __shared__ float sV[KT][DH];
  const int b = blockIdx.z, h = blockIdx.y;
  const int i = blockIdx.x * 64 + threadIdx.x;
  const bool active = i < p.tq;
  const T *Q = (const T *)p.q + (int64_t)b * p.q_bs + (int64_t)(active ? i : 0) * p.q_rs + h * DH;
  const int kb = kv_batch(p, b);
  const T *Kp = (const T *)p.k + (int64_t)kb * p.kv_bs + h * DH;
  const T *Vp = (const T *)p.v + (int64_t)kb * p.kv_bs + h * DH;

  float q[DH], o[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    q[d] = to_f32(Q[d]) * p.qscale;
    o[d] = 0.f;
  }
  float mrun = -INFINITY, lrun = 0.f;
  for (int j0 = 0; j0 < p.tk; j0 += KT) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < KT * DH; idx += 64) {
      int j = idx / DH, d = idx % DH;
      bool ok = (j0 + j) < p.tk;
      sK[j][d] = ok ? to_f32(Kp[(int64_t)(j0 + j) * p.kv_rs + d]) : 0.f;
      sV[j][d] = ok ? to_f32(Vp[(int64_t)(j0 + j) * p.kv_rs + d]) : 0.f;
    }
    __syncthreads();
    float s[KT];
    float tmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float a = 0.f;
#pragma unroll
      for (int d = 0; d < DH; ++d) a = fmaf(q[d], sK[j][d], a);
      s[j] = (j0 + j) < p.tk ? a : -INFINITY;
      tmax = fmaxf(tmax, s[j]);
    }
    const float mnew = fmaxf(mrun, tmax);
    const float corr = exp2f(mrun - mnew);
    lrun *= corr;
#pragma unroll
    for (int d = 0; d < DH; ++d) o[d] *= corr;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float pj = exp2f(s[j] - mnew);
      lrun += pj;
#pragma unroll
      for (int d = 0; d < DH; ++d) o[d] = fmaf(pj, sV[j][d], o[d]);
    }
    mrun = mnew;
  }
  if (!active) return;
  const float inv = 1.0f / lrun;
  T *O = (T *)p.out + (int64_t)b * p.o_bs + (int64_t)i * p.o_rs + h * DH;
#pragma unroll
  for (int d = 0; d < DH; ++d) O[d] = from_f32<T>(o[d] * inv);
}

template <typename T>
static hipError_t launch_valu(const AttnP &p, int dh, hipStream_t s) {
  dim3 grid((p.tq + 63) / 64, p.heads, p.batch), block(64);
  switch (dh) {
    case 8: hipLaunchKernelGGL((k_attn_valu<T, 8>), grid, block, 0, s, p); break;
    case 16: hipLaunchKernelGGL((k_attn_valu<T, 16>), grid, block, 0, s, p); break;
    case 32: hipLaunchKernelGGL((k_attn_valu<T, 32>), grid, block, 0, s, p); break;
    case 64: hipLaunchKernelGGL((k_attn_valu<T, 64>), grid, block, 0, s, p); break;
    case 128: hipLaunchKernelGGL((k_attn_valu<T, 128>), grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(ActType t, const AttnArgs &a, hipStream_t s) {
  AttnP p;
  p.batch = a.batch; p.heads = a.heads; p.tq = a.tq; p.tk = a.tk;
  p.q = a.q; p.q_bs = a.q_bs; p.q_rs = a.q_rs;
  p.k = a.k; p.v = a.v; p.kv_bs = a.kv_bs; p.kv_rs = a.kv_rs;
  p.kv_index = a.kv_index; p.n_kv = a.n_kv;
  p.out = a.out; p.o_bs = a.o_bs; p.o_rs = a.o_rs;
  p.qscale = (float)(1.4426950408889634 / sqrt((double)a.head_dim));
  if (t == ACT_BF16) return launch_valu<bf16>(p, a.head_dim, s);
  return launch_valu<float>(p, a.head_dim, s);
}

}  // namespace fb
