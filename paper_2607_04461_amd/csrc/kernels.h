// Internal launcher interface between the host-side step driver and the HIP kernels.
// Every launcher enqueues on `s` and returns hipGetLastError() of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fb {

enum ActType { ACT_F32 = 0, ACT_BF16 = 1 };

enum Epilogue {
  EPI_STORE = 0,      // out act  = acc + bias
  EPI_GELU = 1,       // out act  = gelu(acc + bias)
  EPI_STORE_F32 = 2,  // out fp32 = acc + bias
  EPI_RESIDUAL = 3,   // out fp32 = (res_in or out) + gate * (acc + bias); optional cache copy of the result
  EPI_EULER = 4       // latent z[scatter(m, n)] += dt * (acc + bias)   (head + unpatchify + Euler)
};

struct EpiArgs {
  void *out = nullptr;         // [M][ldo] (act or fp32)
  int64_t ldo = 0;
  const float *bias = nullptr; // [N] or null
  const float *gate = nullptr; // [N] or null (RESIDUAL)
  const float *res_in = nullptr; // RESIDUAL: [M][ldo] fp32 rows added to (out = res_in + ...), or null:
                                 // out is updated in place.  Read only; equal to out or disjoint from it.
  float *cache = nullptr;      // [M][ldo] fp32 or null (RESIDUAL)
  bool cache_delta = false;    // RESIDUAL: cache = updated out - cache (the cache held the block input)
  // EULER: z [n][C][H][W] fp32, tokens per candidate T = (H/p)(W/p), N = C p p
  float *z = nullptr;
  float dt = 0.f;
  float *preview = nullptr;    // EULER: optional [n][C][H][W] fp32 output z - t_cur v (before the update)
  float t_cur = 0.f;
  int C = 0, H = 0, W = 0, p = 0, T = 0;
};

// C[m][n] = sum_k A[m][k] * Wt[n][k] (+ epilogue).  K % 8 == 0.
hipError_t launch_linear(ActType t, int epi, int M, int N, int K, const void *A, const void *Wt,
                         const EpiArgs &e, hipStream_t s);
// As launch_linear, given a workspace of ws_bytes for split-K partial sums: shapes whose tiles would
// leave most CUs idle (splitk_splits > 1) then run as a split-K launch plus an in-order reduction that
// applies the epilogue (needs splits x M x N x 4 bytes, at most kSplitBytes); else as launch_linear.
constexpr size_t kSplitBytes = (size_t)48 << 20;
int splitk_splits(int epi, int M, int N, int K);
hipError_t launch_linear_ws(ActType t, int epi, int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e,
                            hipStream_t s, void *ws, size_t ws_bytes);
// The kernels launch_linear would use for this shape, without launching: returns the number of
// launches and writes a NUL-terminated description (truncated to len - 1 characters) into buf.
int describe_linear(ActType t, int epi, int M, int N, int K, char *buf, int len);

struct AttnArgs {
  int batch, heads, head_dim, tq, tk;
  const void *q; int64_t q_bs, q_rs;
  const void *k; const void *v; int64_t kv_bs, kv_rs;
  const int32_t *kv_index; int n_kv;   // device, or null (kv batch = q batch)
  void *out; int64_t o_bs, o_rs;
};
hipError_t launch_attention(ActType t, const AttnArgs &a, hipStream_t s);

hipError_t launch_ln_mod(ActType t, int M, int D, float eps, const float *x, const float *shift,
                         const float *scale, void *out, hipStream_t s);

// out = h1 + ca (h1 - h2) + cb (h1 - 2 h2 + h3)   (order 2; order 1 drops cb, order 0 copies h1);
// accumulate: out += that forecast instead
hipError_t launch_proxy(int64_t count, const float *h1, const float *h2, const float *h3, int order,
                        float ca, float cb, float *out, hipStream_t s, bool accumulate = false);

// tokens [n*T][C p p] (act) from z [zrows][C][H][W] fp32; token row block b reads latent b % zrows
hipError_t launch_patchify(ActType t, int n, int zrows, int C, int H, int W, int p, const float *z, void *tok,
                           hipStream_t s);

// sinusoidal features of 1000 t, computed in double: f[j] = cos, f[half + j] = sin
hipError_t launch_time_features(double t, int freq_dim, float *f, hipStream_t s);

// y[o] = act_out(sum_k W[o][k] act_in(x[k]) + b[o]); act: 0 none, 1 SiLU.  fp32.
hipError_t launch_gemv(int out, int in, const float *W, const float *b, const float *x, float *y,
                       int act_in, int act_out, hipStream_t s);

// mods[l][j] = m[j] + table_l[j], table_l = tables + l * table_stride, j < width
hipError_t launch_block_mods(int L, int width, const float *m, const float *tables,
                             int64_t table_stride, float *mods, hipStream_t s);

hipError_t launch_f32_to_bf16(int64_t count, const float *x, void *y, hipStream_t s);

// dst[i] = vals[i], i < n <= 128, the values travelling in the kernel's arguments (nothing on the host
// has to outlive the call)
hipError_t launch_store_i32(int n, const int32_t *vals, int32_t *dst, hipStream_t s);

// qk RMSNorm + 3-D rotary embedding: (cos, sin) table [T][dh/2] for a token grid of width wp; and the
// in-place normalisation (gain over D, eps) of M rows of x (act, row stride rs), rotated by the table
// (row % tokens) when tab is not null.  D % 8 == 0.
hipError_t launch_rope_table(int T, int wp, int dh, float2 *tab, hipStream_t s);
hipError_t launch_qk_norm(ActType t, int M, int D, int dh, void *x, int64_t rs, const float *gain, float eps,
                          const float2 *tab, int tokens, hipStream_t s);

// Stochastic update (App. A.1, Eq. 20): z <- z + dt [v + k (z + omt v)] + g eps, eps from Philox4x32-10
// with key (key0, key1) and counter (element / 4, candidate, step, 0) through Box-Muller.
struct SdeArgs {
  float dt, k, omt, g;
  uint32_t key0, key1, step, row0;
};
// Host: coefficients for noise level a at (t_cur, t_next); false if a < 0, t_cur outside (0, 1] or
// sigma_t is not finite.  Row b of a launch draws counter row row0 + b.
bool sde_coefficients(float t_cur, float t_next, float a, uint64_t seed, int32_t step, int32_t row0,
                      SdeArgs *out);
// z [n][C][H][W] fp32 updated in place from v = head output [n T][C p p] fp32 (unpatchified here).
// guided: v holds 2n token rows, the unconditional twins after the n conditional ones, and the
// velocity is v_u + scale (v_c - v_u).  a.g == 0 skips the normals (the Euler update when a.k == 0).
// preview (optional, same layout as z) receives z - t_cur v before the update.
hipError_t launch_head_update(int n, int C, int H, int W, int p, const float *v, bool guided, float scale,
                              float *z, const SdeArgs &a, float *preview, float t_cur, hipStream_t s);
// the words (uint32 [ceil(count/4)][4], or null) and normals (fp32 [count], or null) of one candidate
hipError_t launch_normals(int64_t count, uint32_t cand, uint32_t step, uint64_t seed, uint32_t *words,
                          float *normals, hipStream_t s);

}  // namespace fb
