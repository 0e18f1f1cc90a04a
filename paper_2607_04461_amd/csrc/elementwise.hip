// HBM-bound kernels of the draft step: adaLN normalisation, the activation proxy (Eq. 3-5),
// patchify, the timestep path and dtype conversion.
#include "common.h"
#include "kernels.h"

namespace fb {

// ------------------------------------------------------------------------------------------ adaLN
// One wave per row; the row stays in registers between the two statistics passes.  NV = float4s
// per lane, a compile-time bound (D <= 256 NV), so register use matches the row length.  NT: the rows
// are read non-temporally (launches reading at least kNTLoadBytes), so that the stream's lines, read once
// here, do not push this kernel's output (the next linear layer's operand) out of the caches: the
// 1.3B-shaped pool's draft measured 238.2 -> 237.3 and 244.9 -> 243.5 ms (two boxes, alternating, latents
// bit-identical); one candidate's refinement (9.6 MB rows) keeps cached loads.
template <typename T, int NV, bool NT>
__global__ __launch_bounds__(256) void k_ln_mod(int M, int D, float eps, const float *__restrict__ x,
                                                const float *__restrict__ shift,
                                                const float *__restrict__ scale, T *__restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float4 *xr = reinterpret_cast<const float4 *>(x + row * D);
  const int nv = D >> 2;
  float4 v[NV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    int c = lane + i * 64;
    if (c >= nv) {
      v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    } else if constexpr (NT) {
      const f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(xr) + c);
      v[i] = make_float4(t[0], t[1], t[2], t[3]);
    } else {
      v[i] = xr[c];
    }
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  const float mean = wave_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    int c = lane + i * 64;
    if (c < nv) {
      float a = v[i].x - mean, b = v[i].y - mean, cc = v[i].z - mean, d = v[i].w - mean;
      q += (a * a + b * b) + (cc * cc + d * d);
    }
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + eps);
  T *orow = out + row * D;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    int c = lane + i * 64;
    if (c < nv) {
      float r[4] = {(v[i].x - mean) * rstd, (v[i].y - mean) * rstd, (v[i].z - mean) * rstd,
                    (v[i].w - mean) * rstd};
      if (shift) {
        float4 sh = reinterpret_cast<const float4 *>(shift)[c];
        float4 sc = reinterpret_cast<const float4 *>(scale)[c];
        r[0] = r[0] * (1.0f + sc.x) + sh.x;
        r[1] = r[1] * (1.0f + sc.y) + sh.y;
        r[2] = r[2] * (1.0f + sc.z) + sh.z;
        r[3] = r[3] * (1.0f + sc.w) + sh.w;
      }
      if constexpr (sizeof(T) == 4) {
        reinterpret_cast<float4 *>(orow)[c] = make_float4(r[0], r[1], r[2], r[3]);
      } else {
        bf16x4 o4 = {(bf16)r[0], (bf16)r[1], (bf16)r[2], (bf16)r[3]};
        reinterpret_cast<bf16x4 *>(orow)[c] = o4;
      }
    }
  }
}

constexpr size_t kNTLoadBytes = (size_t)128 << 20;

template <typename T, bool NT>
static hipError_t launch_ln_t(int M, int D, float eps, const float *x, const float *shift,
                              const float *scale, void *out, hipStream_t s) {
  dim3 grid((M + 3) / 4), block(256);
  const int nv = (D / 4 + 63) / 64;
#define FB_LN(NVC)                                                                                      \
  case NVC:                                                                                             \
    hipLaunchKernelGGL((k_ln_mod<T, NVC, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); \
    break;
  switch (nv) {
    FB_LN(1) FB_LN(2) FB_LN(3) FB_LN(4) FB_LN(5) FB_LN(6) FB_LN(8) FB_LN(12) FB_LN(16) FB_LN(20) FB_LN(24)
    default:
      if (nv <= 8) { hipLaunchKernelGGL((k_ln_mod<T, 8, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); }
      else if (nv <= 12) { hipLaunchKernelGGL((k_ln_mod<T, 12, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); }
      else if (nv <= 16) { hipLaunchKernelGGL((k_ln_mod<T, 16, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); }
      else if (nv <= 20) { hipLaunchKernelGGL((k_ln_mod<T, 20, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); }
      else { hipLaunchKernelGGL((k_ln_mod<T, 24, NT>), grid, block, 0, s, M, D, eps, x, shift, scale, (T *)out); }
  }
#undef FB_LN
  return hipGetLastError();
}

hipError_t launch_ln_mod(ActType t, int M, int D, float eps, const float *x, const float *shift,
                         const float *scale, void *out, hipStream_t s) {
  if (t == ACT_BF16) {
    if ((size_t)M * (size_t)D * sizeof(float) >= kNTLoadBytes)
      return launch_ln_t<bf16, true>(M, D, eps, x, shift, scale, out, s);
    return launch_ln_t<bf16, false>(M, D, eps, x, shift, scale, out, s);
  }
  return launch_ln_t<float, false>(M, D, eps, x, shift, scale, out, s);
}

// ------------------------------------------------------------------------------ activation proxy
// Difference form h1 + ca (h1 - h2) + cb (h1 - 2 h2 + h3): a constant cache reproduces itself
// exactly, whatever the coefficients.
template <int ORDER, bool ACC>
__global__ __launch_bounds__(256) void k_proxy(int64_t n4, const float4 *__restrict__ h1,
                                               const float4 *__restrict__ h2,
                                               const float4 *__restrict__ h3, float ca, float cb,
                                               float4 *__restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x) {
    float4 a = h1[i];
    if constexpr (ORDER == 0) {
      if constexpr (ACC) {
        float4 o = out[i];
        a = make_float4(o.x + a.x, o.y + a.y, o.z + a.z, o.w + a.w);
      }
      out[i] = a;
    } else {
      float4 b = h2[i];
      float4 d1 = make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w);
      float4 r = make_float4(a.x + ca * d1.x, a.y + ca * d1.y, a.z + ca * d1.z, a.w + ca * d1.w);
      if constexpr (ORDER == 2) {
        float4 c = h3[i];
        r.x += cb * ((a.x - b.x) - (b.x - c.x));
        r.y += cb * ((a.y - b.y) - (b.y - c.y));
        r.z += cb * ((a.z - b.z) - (b.z - c.z));
        r.w += cb * ((a.w - b.w) - (b.w - c.w));
      }
      if constexpr (ACC) {
        float4 o = out[i];
        r = make_float4(o.x + r.x, o.y + r.y, o.z + r.z, o.w + r.w);
      }
      out[i] = r;
    }
  }
}

__global__ void k_proxy_tail(int64_t start, int64_t count, const float *h1, const float *h2,
                             const float *h3, int order, float ca, float cb, float *out, int acc) {
  int64_t i = start + threadIdx.x;
  if (i >= count) return;
  float a = h1[i];
  float r = a;
  if (order >= 1) r = a + ca * (a - h2[i]);
  if (order >= 2) r += cb * ((a - h2[i]) - (h2[i] - h3[i]));
  out[i] = acc ? out[i] + r : r;
}

template <bool ACC>
static void proxy_body(int64_t n4, dim3 g, dim3 b, hipStream_t s, int order, const float4 *a, const float4 *bb,
                       const float4 *c, float ca, float cb, float4 *o) {
  if (order == 0) hipLaunchKernelGGL((k_proxy<0, ACC>), g, b, 0, s, n4, a, bb, c, ca, cb, o);
  else if (order == 1) hipLaunchKernelGGL((k_proxy<1, ACC>), g, b, 0, s, n4, a, bb, c, ca, cb, o);
  else hipLaunchKernelGGL((k_proxy<2, ACC>), g, b, 0, s, n4, a, bb, c, ca, cb, o);
}

hipError_t launch_proxy(int64_t count, const float *h1, const float *h2, const float *h3, int order,
                        float ca, float cb, float *out, hipStream_t s, bool accumulate) {
  int64_t n4 = count / 4;
  if (n4 > 0) {
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 256 * 16) blocks = 256 * 16;
    dim3 g((unsigned)blocks), b(256);
    auto *o = (float4 *)out;
    auto *a = (const float4 *)h1, *bb = (const float4 *)h2, *c = (const float4 *)h3;
    if (accumulate) proxy_body<true>(n4, g, b, s, order, a, bb, c, ca, cb, o);
    else proxy_body<false>(n4, g, b, s, order, a, bb, c, ca, cb, o);
  }
  if (count % 4)
    hipLaunchKernelGGL(k_proxy_tail, dim3(1), dim3(64), 0, s, n4 * 4, count, h1, h2, h3, order, ca,
                       cb, out, accumulate ? 1 : 0);
  return hipGetLastError();
}

// -------------------------------------------------------------------------------------- patchify
template <typename T>
__global__ __launch_bounds__(256) void k_patchify(int n, int zrows, int C, int H, int W, int p,
                                                  const float *__restrict__ z, T *__restrict__ tok) {
  const int P = C * p * p, wp = W / p, T_ = (H / p) * wp;
  const int64_t total = (int64_t)n * T_ * P;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int f = (int)(idx % P);
    int64_t m = idx / P;
    int t = (int)(m % T_), b = (int)(m / T_) % zrows;
    int i = t / wp, j = t % wp;
    int c = f / (p * p), r = f % (p * p), di = r / p, dj = r % p;
    tok[idx] = from_f32<T>(z[(((int64_t)b * C + c) * H + (p * i + di)) * W + (p * j + dj)]);
  }
}

hipError_t launch_patchify(ActType t, int n, int zrows, int C, int H, int W, int p, const float *z, void *tok,
                           hipStream_t s) {
  int64_t total = (int64_t)n * C * H * W;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (t == ACT_BF16)
    hipLaunchKernelGGL(k_patchify<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, n, zrows, C, H, W, p, z,
                       (bf16 *)tok);
  else
    hipLaunchKernelGGL(k_patchify<float>, dim3((unsigned)blocks), dim3(256), 0, s, n, zrows, C, H, W, p, z,
                       (float *)tok);
  return hipGetLastError();
}

// ------------------------------------------------------------------ qk RMSNorm + 3-D rotary table
// (cos, sin) per (token, pair): token t = i wp + j sits at (frame 0, row i, column j); pair k of the
// head dim falls in the frame, height or width band (widths dh - 4 (dh/6), 2 (dh/6), 2 (dh/6)) and
// turns by position * 10000^(-2 k' / width), k' its index inside the band.  Computed in double.
__global__ void k_rope_table(int T, int wp, int dh, float2 *__restrict__ tab) {
  const int half = dh / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)T * half) return;
  const int t = (int)(idx / half), k = (int)(idx % half);
  const int q6 = dh / 6, fw = dh - 4 * q6, bw = 2 * q6;
  int pos, kb, width;
  if (2 * k < fw) { pos = 0; kb = k; width = fw; }
  else if (2 * k < fw + bw) { pos = t / wp; kb = k - fw / 2; width = bw; }
  else { pos = t % wp; kb = k - (fw + bw) / 2; width = bw; }
  const double ang = (double)pos * pow(10000.0, -2.0 * (double)kb / (double)width);
  double sn, cs;
  sincos(ang, &sn, &cs);
  tab[idx] = make_float2((float)cs, (float)sn);
}

hipError_t launch_rope_table(int T, int wp, int dh, float2 *tab, hipStream_t s) {
  const int64_t n = (int64_t)T * (dh / 2);
  hipLaunchKernelGGL(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, T, wp, dh, tab);
  return hipGetLastError();
}

template <typename T> __device__ __forceinline__ void load8(const T *p, float v[8]);
template <> __device__ __forceinline__ void load8<float>(const float *p, float v[8]) {
  const float4 a = reinterpret_cast<const float4 *>(p)[0], b = reinterpret_cast<const float4 *>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <> __device__ __forceinline__ void load8<bf16>(const bf16 *p, float v[8]) {
  const bf16x8 a = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
}
template <typename T> __device__ __forceinline__ void store8(T *p, const float v[8]);
template <> __device__ __forceinline__ void store8<float>(float *p, const float v[8]) {
  reinterpret_cast<float4 *>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4 *>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
template <> __device__ __forceinline__ void store8<bf16>(bf16 *p, const float v[8]) {
  bf16x8 a;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (bf16)v[i];
  *reinterpret_cast<bf16x8 *>(p) = a;
}

// In place on rows of x (stride rs): x <- RMSNorm(x) * gain over D, then, with a table, every pair
// (2k, 2k+1) of each head rotated by the table entry of (row % T, k).  One wave per row, two passes
// over the row (statistics, then normalise + rotate), 8 elements per lane per load.
template <typename T>
__global__ __launch_bounds__(256) void k_qk_norm(int M, int D, int dh, T *__restrict__ x, int64_t rs,
                                                 const float *__restrict__ gain, float eps,
                                                 const float2 *__restrict__ tab, int tokens) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  T *xr = x + row * rs;
  const int chunks = D >> 3;
  float ss = 0.f;
  for (int c = lane; c < chunks; c += 64) {
    float v[8];
    load8<T>(xr + 8 * c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[i], v[i], ss);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)D + eps);
  const float2 *tr = tab ? tab + (row % tokens) * (dh >> 1) : nullptr;
  for (int c = lane; c < chunks; c += 64) {
    float v[8];
    load8<T>(xr + 8 * c, v);
    const float4 g0 = reinterpret_cast<const float4 *>(gain + 8 * c)[0];
    const float4 g1 = reinterpret_cast<const float4 *>(gain + 8 * c)[1];
    const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v[i] * rstd * g[i];
    if (tr) {
#pragma unroll
      for (int pr = 0; pr < 4; ++pr) {
        const int d = (8 * c + 2 * pr) % dh;
        const float2 cs = tr[d >> 1];
        const float a = v[2 * pr], b = v[2 * pr + 1];
        v[2 * pr] = a * cs.x - b * cs.y;
        v[2 * pr + 1] = a * cs.y + b * cs.x;
      }
    }
    store8<T>(xr + 8 * c, v);
  }
}

hipError_t launch_qk_norm(ActType t, int M, int D, int dh, void *x, int64_t rs, const float *gain, float eps,
                          const float2 *tab, int tokens, hipStream_t s) {
  dim3 g((unsigned)((M + 3) / 4)), b(256);
  if (t == ACT_BF16)
    hipLaunchKernelGGL(k_qk_norm<bf16>, g, b, 0, s, M, D, dh, (bf16 *)x, rs, gain, eps, tab, tokens);
  else
    hipLaunchKernelGGL(k_qk_norm<float>, g, b, 0, s, M, D, dh, (float *)x, rs, gain, eps, tab, tokens);
  return hipGetLastError();
}

// --------------------------------------------------------------------------------- timestep path
__global__ void k_time_features(double t, int half, float *f) {
  int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= half) return;
  double w = pow(10000.0, -(double)j / (double)half);
  double a = 1000.0 * t * w;
  f[j] = (float)cos(a);
  f[half + j] = (float)sin(a);
}

hipError_t launch_time_features(double t, int freq_dim, float *f, hipStream_t s) {
  int half = freq_dim / 2;
  hipLaunchKernelGGL(k_time_features, dim3((half + 255) / 256), dim3(256), 0, s, t, half, f);
  return hipGetLastError();
}

// One wave per output row; lanes stride over the row with float4 loads.
__global__ __launch_bounds__(256) void k_gemv(int out, int in, const float *__restrict__ W,
                                              const float *__restrict__ b,
                                              const float *__restrict__ x, float *__restrict__ y,
                                              int act_in, int act_out) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= out) return;
  const float *wr = W + (int64_t)o * in;
  float acc = 0.f;
  for (int k = lane; k < in; k += 64) {
    float xv = x[k];
    if (act_in == 1) xv = silu(xv);
    acc += wr[k] * xv;
  }
  acc = wave_sum(acc);
  if (lane == 0) {
    float r = acc + (b ? b[o] : 0.f);
    if (act_out == 1) r = silu(r);
    y[o] = r;
  }
}

// The same with 16-byte loads (in % 4 == 0, 16-byte aligned rows): each lane keeps four row chunks
// in flight, so a wave streams its row at the memory rate rather than one dependent 4-byte load at a
// time (the 6D x D modulation matrix, 56.6 MB in fp32 at D = 1536, is read once per step).
__global__ __launch_bounds__(256) void k_gemv4(int out, int in, const float *__restrict__ W,
                                               const float *__restrict__ b,
                                               const float *__restrict__ x, float *__restrict__ y,
                                               int act_in, int act_out) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= out) return;
  const float4 *wr = reinterpret_cast<const float4 *>(W + (int64_t)o * in);
  const float4 *xr = reinterpret_cast<const float4 *>(x);
  const int n4 = in >> 2;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = lane; k0 < n4; k0 += 256) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = k0 + 64 * u;
      if (k < n4) {
        const float4 w = wr[k];
        float4 xv = xr[k];
        if (act_in == 1) xv = make_float4(silu(xv.x), silu(xv.y), silu(xv.z), silu(xv.w));
        acc[u] += (w.x * xv.x + w.y * xv.y) + (w.z * xv.z + w.w * xv.w);
      }
    }
  }
  float a = wave_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
  if (lane == 0) {
    float r = a + (b ? b[o] : 0.f);
    if (act_out == 1) r = silu(r);
    y[o] = r;
  }
}

hipError_t launch_gemv(int out, int in, const float *W, const float *b, const float *x, float *y,
                       int act_in, int act_out, hipStream_t s) {
  if (in % 4 == 0 && (((uintptr_t)W | (uintptr_t)x) & 15) == 0)
    hipLaunchKernelGGL(k_gemv4, dim3((out + 3) / 4), dim3(256), 0, s, out, in, W, b, x, y, act_in, act_out);
  else
    hipLaunchKernelGGL(k_gemv, dim3((out + 3) / 4), dim3(256), 0, s, out, in, W, b, x, y, act_in,
                       act_out);
  return hipGetLastError();
}

__global__ void k_block_mods(int L, int width, const float *__restrict__ m,
                             const float *__restrict__ tables, int64_t stride,
                             float *__restrict__ mods) {
  int j = blockIdx.x * blockDim.x + threadIdx.x;
  int l = blockIdx.y;
  if (j >= width) return;
  mods[(int64_t)l * width + j] = m[j] + tables[l * stride + j];
}

hipError_t launch_block_mods(int L, int width, const float *m, const float *tables,
                             int64_t table_stride, float *mods, hipStream_t s) {
  hipLaunchKernelGGL(k_block_mods, dim3((width + 255) / 256, L), dim3(256), 0, s, L, width, m,
                     tables, table_stride, mods);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------ conversion
// up to 128 int32 values carried in the kernel arguments, written to dst[0 .. n)
struct I32Args {
  int32_t n;
  int32_t v[128];
};
__global__ __launch_bounds__(128) void k_store_i32(I32Args args, int32_t *__restrict__ dst) {
  const int i = threadIdx.x;
  if (i < args.n) dst[i] = args.v[i];
}

hipError_t launch_store_i32(int n, const int32_t *vals, int32_t *dst, hipStream_t s) {
  if (n < 0 || n > 128) return hipErrorInvalidValue;
  I32Args args{};
  args.n = n;
  for (int i = 0; i < n; ++i) args.v[i] = vals[i];
  hipLaunchKernelGGL(k_store_i32, dim3(1), dim3(128), 0, s, args, dst);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_f32_to_bf16(int64_t n, const float *__restrict__ x,
                                                     bf16 *__restrict__ y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    y[i] = (bf16)x[i];
}

hipError_t launch_f32_to_bf16(int64_t count, const float *x, void *y, hipStream_t s) {
  int64_t blocks = (count + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_f32_to_bf16, dim3((unsigned)blocks), dim3(256), 0, s, count, x, (bf16 *)y);
  return hipGetLastError();
}

}  // namespace fb
