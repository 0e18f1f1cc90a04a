// Head update of the latents outside the head GEMM's epilogue: unpatchify, optional classifier-free
// guidance, and the stochastic flow update of App. A.1 (Eq. 20) with its counter-based normals (or
// the Euler update, a = 0).
//
//   z <- z + dt [v + k (z + (1 - t) v)] + g eps,   k = sigma_t^2 / (2 t),  g = sigma_t sqrt(|dt|),
//   sigma_t = a sqrt(t / (1 - t))  (1 - t_next in the denominator when t = 1).
//
// eps for flat element e of candidate b's latent [C][H][W] at step s is normal e % 4 of one
// Philox4x32-10 block (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as easy as 1, 2, 3",
// SC'11) with key (seed low word, seed high word) and counter (e / 4, row0 + b, s, 0), where row0 is
// the pool index of the launch's first row; the four 32-bit words become four normals by the
// Box-Muller transform, computed in double:
// u1 = (w0 + 1) 2^-32, u2 = w1 2^-32, r = sqrt(-2 ln u1), normals r cos(2 pi u2), r sin(2 pi u2);
// (w2, w3) likewise.  One thread owns one counter, i.e. four consecutive latent elements, so every
// generated normal is used once.  The kernel is HBM-bound: per element it reads z and v and writes z.
#include <cmath>

#include "common.h"
#include "kernels.h"

namespace fb {

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  constexpr uint32_t kMul0 = 0xD2511F53u, kMul1 = 0xCD9E8D57u;   // round multipliers
  constexpr uint32_t kBump0 = 0x9E3779B9u, kBump1 = 0xBB67AE85u; // key schedule increments
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(kMul0, c[0]), lo0 = kMul0 * c[0];
    const uint32_t hi1 = __umulhi(kMul1, c[2]), lo1 = kMul1 * c[2];
    const uint32_t x0 = hi1 ^ c[1] ^ k0, x2 = hi0 ^ c[3] ^ k1;
    c[0] = x0; c[1] = lo1; c[2] = x2; c[3] = lo0;
    k0 += kBump0; k1 += kBump1;
  }
}

__device__ __forceinline__ void box_muller(uint32_t w0, uint32_t w1, float &z0, float &z1) {
  const double u1 = ((double)w0 + 1.0) * 0x1p-32, u2 = (double)w1 * 0x1p-32;
  const double r = sqrt(-2.0 * log(u1));
  double sn, cs;
  sincospi(2.0 * u2, &sn, &cs);
  z0 = (float)(r * cs);
  z1 = (float)(r * sn);
}

__device__ __forceinline__ void normals4(uint32_t quad, uint32_t cand, uint32_t step, uint32_t k0,
                                         uint32_t k1, uint32_t w[4], float z[4]) {
  w[0] = quad; w[1] = cand; w[2] = step; w[3] = 0u;
  philox4x32_10(w, k0, k1);
  box_muller(w[0], w[1], z[0], z[1]);
  box_muller(w[2], w[3], z[2], z[3]);
}

// grid (ceil(quads / 256), n); v: head output [(n or 2n) T][C p p] fp32 (bias included); z: [n][C][H][W].
// Guided (vu != null): the unconditional twin of candidate b is token row block n + b, and the
// velocity is v_u + scale (v_c - v_u).  s.g == 0 (no noise) skips the normals.
__global__ __launch_bounds__(256) void k_head_update(int C, int H, int W, int p,
                                                     const float *__restrict__ v, int guided, float scale,
                                                     float *__restrict__ z, SdeArgs s,
                                                     float *__restrict__ preview, float t_cur) {
  const int64_t chw = (int64_t)C * H * W, quads = (chw + 3) >> 2;
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int b = blockIdx.y, n = gridDim.y;
  if (q >= quads) return;
  uint32_t w[4];
  float eps[4] = {0.f, 0.f, 0.f, 0.f};
  if (s.g != 0.f) normals4((uint32_t)q, s.row0 + (uint32_t)b, s.step, s.key0, s.key1, w, eps);
  const int hw = H * W, wp = W / p, pp = p * p;
  const int64_t T = (int64_t)(H / p) * wp, P = (int64_t)C * pp;
  float *zb = z + (int64_t)b * chw;
  const float *vb = v + (int64_t)b * T * P;
  const float *vu = guided ? v + (int64_t)(n + b) * T * P : nullptr;
  // (c, y, x) of the quad's first element by one 32-bit division each (a candidate's latent holds
  // fewer than 2^31 elements), then carried element by element
  const int e0 = (int)(4 * q);
  int c = e0 / hw, y = (e0 - c * hw) / W, x = e0 - c * hw - y * W;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t e = 4 * q + i;
    if (e >= chw) break;
    if (i > 0 && ++x == W) {
      x = 0;
      if (++y == H) {
        y = 0;
        ++c;
      }
    }
    const int ti = y / p, di = y - ti * p, tj = x / p, dj = x - tj * p;
    const int64_t vi = (int64_t)(ti * wp + tj) * P + c * pp + di * p + dj;
    float vv = vb[vi];
    if (vu) vv = fmaf(scale, vv - vu[vi], vu[vi]);
    const float zz = zb[e];
    if (preview) preview[(int64_t)b * chw + e] = zz - t_cur * vv;
    const float drift = fmaf(s.k, fmaf(s.omt, vv, zz), vv);
    const float zn = fmaf(s.dt, drift, zz);
    zb[e] = s.g != 0.f ? fmaf(s.g, eps[i], zn) : zn;
  }
}

__global__ __launch_bounds__(256) void k_normals(int64_t count, uint32_t cand, uint32_t step,
                                                 uint32_t k0, uint32_t k1, uint32_t *__restrict__ words,
                                                 float *__restrict__ normals) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= (count + 3) >> 2) return;
  uint32_t w[4];
  float z[4];
  normals4((uint32_t)q, cand, step, k0, k1, w, z);
  if (words) {
#pragma unroll
    for (int i = 0; i < 4; ++i) words[4 * q + i] = w[i];
  }
  if (normals) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * q + i < count) normals[4 * q + i] = z[i];
  }
}

bool sde_coefficients(float t_cur, float t_next, float a, uint64_t seed, int32_t step, int32_t row0,
                      SdeArgs *out) {
  const double tc = t_cur, tn = t_next, dt = tn - tc;
  if (!(a >= 0.f) || !std::isfinite(a) || !(tc > 0.0) || !(tc <= 1.0)) return false;
  const double one_minus = tc < 1.0 ? 1.0 - tc : 1.0 - tn;
  if (!(one_minus > 0.0)) return false;
  const double sigma = (double)a * std::sqrt(tc / one_minus);
  out->dt = (float)dt;
  out->k = (float)(sigma * sigma / (2.0 * tc));
  out->omt = (float)(1.0 - tc);
  out->g = (float)(sigma * std::sqrt(std::fabs(dt)));
  out->key0 = (uint32_t)(seed & 0xFFFFFFFFu);
  out->key1 = (uint32_t)(seed >> 32);
  out->step = (uint32_t)step;
  out->row0 = (uint32_t)row0;
  return std::isfinite(out->k) && std::isfinite(out->g);
}

hipError_t launch_head_update(int n, int C, int H, int W, int p, const float *v, bool guided, float scale,
                              float *z, const SdeArgs &a, float *preview, float t_cur, hipStream_t s) {
  const int64_t quads = ((int64_t)C * H * W + 3) / 4;
  hipLaunchKernelGGL(k_head_update, dim3((unsigned)((quads + 255) / 256), (unsigned)n), dim3(256), 0, s,
                     C, H, W, p, v, guided ? 1 : 0, scale, z, a, preview, t_cur);
  return hipGetLastError();
}

hipError_t launch_normals(int64_t count, uint32_t cand, uint32_t step, uint64_t seed, uint32_t *words,
                          float *normals, hipStream_t s) {
  const int64_t quads = (count + 3) / 4;
  hipLaunchKernelGGL(k_normals, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, s, count, cand, step,
                     (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), words, normals);
  return hipGetLastError();
}

}  // namespace fb
