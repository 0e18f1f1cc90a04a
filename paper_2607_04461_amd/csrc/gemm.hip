// Linear layers of the DiT step: C[m][n] = sum_k A[m][k] Wt[n][k] with fused epilogues.
//   * k_linear_dma8 / k_linear_dma / k_linear_mfma: bf16 operands on gfx950 matrix cores
//     (v_mfma_f32_16x16x32_bf16), fp32 accumulation.  Workgroup tiles of 160..256 rows x 256 columns
//     (k_linear_dma8: 8 waves, two per SIMD, LDS filled by buffer loads that write LDS themselves,
//     K % 64 == 0 -- the default; k_linear_dma: the same tiles on 4 waves, one per SIMD, for forced
//     plans; k_linear_mfma<8,4,2,4>: 8 waves of 128x64 with register-staged loads for other K) or
//     128x128 (4 waves of 64x64, two workgroups per CU), chosen per shape by a round-count model;
//     k_linear_deep: the 8-wave tile at 128 or 160 rows x 128 or 256 columns with a three-stage LDS
//     ring, for launches that fit one round of workgroups one per CU (one or two candidates); K
//     tiles of 64 in double-buffered, XOR-swizzled LDS; XCD-aware grouped tile order.  Operands are swapped (the weight tile feeds the MFMA "A" side) and the weight rows
//     permuted so that every lane owns 8 consecutive output columns of one row.  Every kernel
//     accumulates K in the same order, so an output element does not depend on the tiling.  The
//     8-wave tiles' epilogues (bf16 store and GELU of 256-column tiles, residual updates, split-K
//     partial sums) pass each wave's block through the freed LDS ring so that every global access
//     covers whole 128-byte rows.
//   * k_linear_valu: fp32 (or bf16) operands on the vector ALUs, 64x64 tiles; used by the fp32 mode
//     and for shapes the MFMA tiling does not take.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <string>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace fb {

// ---------------------------------------------------------------------------------- epilogues
template <int EPI, typename TO>
__device__ __forceinline__ void epilogue4(const EpiArgs &e, int m, int n, float v0, float v1,
                                          float v2, float v3) {
  float v[4] = {v0, v1, v2, v3};
  if (e.bias) {
    float4 b = *reinterpret_cast<const float4 *>(e.bias + n);
    v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
  }
  if constexpr (EPI == EPI_STORE || EPI == EPI_GELU) {
    if constexpr (EPI == EPI_GELU) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = gelu_tanh(v[i]);
    }
    TO *o = reinterpret_cast<TO *>(e.out) + (int64_t)m * e.ldo + n;
    if constexpr (sizeof(TO) == 4) {
      *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
      bf16x4 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
      *reinterpret_cast<bf16x4 *>(o) = w;
    }
  } else if constexpr (EPI == EPI_STORE_F32) {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)m * e.ldo + n;
    *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
  } else if constexpr (EPI == EPI_RESIDUAL) {
    float *o = reinterpret_cast<float *>(e.out) + (int64_t)m * e.ldo + n;
    float4 h = *reinterpret_cast<const float4 *>(e.res_in ? e.res_in + (int64_t)m * e.ldo + n : o);
    if (e.gate) {
      float4 g = *reinterpret_cast<const float4 *>(e.gate + n);
      h.x += g.x * v[0]; h.y += g.y * v[1]; h.z += g.z * v[2]; h.w += g.w * v[3];
    } else {
      h.x += v[0]; h.y += v[1]; h.z += v[2]; h.w += v[3];
    }
    *reinterpret_cast<float4 *>(o) = h;
    if (e.cache) {
      float4 *cp = reinterpret_cast<float4 *>(e.cache + (int64_t)m * e.ldo + n);
      if (e.cache_delta) {
        const float4 c0 = *cp;
        *cp = make_float4(h.x - c0.x, h.y - c0.y, h.z - c0.z, h.w - c0.w);
      } else {
        *cp = h;
      }
    }
  } else if constexpr (EPI == EPI_EULER) {
    // m = candidate * T + token, token = i * (W/p) + j; n = c p^2 + p di + dj
    const int b = m / e.T, t = m % e.T, wp = e.W / e.p;
    const int i = t / wp, j = t % wp, pp = e.p * e.p;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int nn = n + q;
      int c = nn / pp, r = nn % pp, di = r / e.p, dj = r % e.p;
      const int64_t zi = (((int64_t)b * e.C + c) * e.H + (e.p * i + di)) * e.W + (e.p * j + dj);
      const float z0 = e.z[zi];
      if (e.preview) e.preview[zi] = z0 - e.t_cur * v[q];   // clean-latent estimate z - t v
      e.z[zi] = z0 + e.dt * v[q];
    }
  }
}

// Eight consecutive output columns n .. n+7 of row m: one 16-byte bf16 store or two 16-byte fp32
// stores per lane.
template <int EPI, typename TO>
__device__ __forceinline__ void epilogue8(const EpiArgs &e, int m, int n, const float *v_in) {
  if constexpr (EPI == EPI_EULER) {
    epilogue4<EPI, TO>(e, m, n, v_in[0], v_in[1], v_in[2], v_in[3]);
    epilogue4<EPI, TO>(e, m, n + 4, v_in[4], v_in[5], v_in[6], v_in[7]);
  } else {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = v_in[q];
    if (e.bias) {
      float4 b0 = *reinterpret_cast<const float4 *>(e.bias + n);
      float4 b1 = *reinterpret_cast<const float4 *>(e.bias + n + 4);
      v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
      v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
    }
    if constexpr (EPI == EPI_STORE || EPI == EPI_GELU) {
      if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = gelu_tanh(v[q]);
      }
      TO *o = reinterpret_cast<TO *>(e.out) + (int64_t)m * e.ldo + n;
      if constexpr (sizeof(TO) == 4) {
        reinterpret_cast<float4 *>(o)[0] = make_float4(v[0], v[1], v[2], v[3]);
        reinterpret_cast<float4 *>(o)[1] = make_float4(v[4], v[5], v[6], v[7]);
      } else {
        bf16x8 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
                    (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
        *reinterpret_cast<bf16x8 *>(o) = w;
      }
    } else if constexpr (EPI == EPI_STORE_F32) {
      float *o = reinterpret_cast<float *>(e.out) + (int64_t)m * e.ldo + n;
      reinterpret_cast<float4 *>(o)[0] = make_float4(v[0], v[1], v[2], v[3]);
      reinterpret_cast<float4 *>(o)[1] = make_float4(v[4], v[5], v[6], v[7]);
    } else if constexpr (EPI == EPI_RESIDUAL) {
      float *o = reinterpret_cast<float *>(e.out) + (int64_t)m * e.ldo + n;
      const float4 *hi = reinterpret_cast<const float4 *>(e.res_in ? e.res_in + (int64_t)m * e.ldo + n : o);
      float4 h0 = hi[0], h1 = hi[1];
      if (e.gate) {
        float4 g0 = *reinterpret_cast<const float4 *>(e.gate + n);
        float4 g1 = *reinterpret_cast<const float4 *>(e.gate + n + 4);
        h0.x += g0.x * v[0]; h0.y += g0.y * v[1]; h0.z += g0.z * v[2]; h0.w += g0.w * v[3];
        h1.x += g1.x * v[4]; h1.y += g1.y * v[5]; h1.z += g1.z * v[6]; h1.w += g1.w * v[7];
      } else {
        h0.x += v[0]; h0.y += v[1]; h0.z += v[2]; h0.w += v[3];
        h1.x += v[4]; h1.y += v[5]; h1.z += v[6]; h1.w += v[7];
      }
      reinterpret_cast<float4 *>(o)[0] = h0;
      reinterpret_cast<float4 *>(o)[1] = h1;
      if (e.cache) {
        float4 *c = reinterpret_cast<float4 *>(e.cache + (int64_t)m * e.ldo + n);
        if (e.cache_delta) {
          const float4 c0 = c[0], c1 = c[1];
          c[0] = make_float4(h0.x - c0.x, h0.y - c0.y, h0.z - c0.z, h0.w - c0.w);
          c[1] = make_float4(h1.x - c1.x, h1.y - c1.y, h1.z - c1.z, h1.w - c1.w);
        } else {
          c[0] = h0;
          c[1] = h1;
        }
      }
    }
  }
}

// ------------------------------------------------------------- whole-tile epilogue of the MFMA kernels
// A wave's accumulators acc[i][j] (i over 16-column W fragments, permuted so that fragments 2a and
// 2a+1 give a lane 8 consecutive columns; j over 16-row A fragments) hold rows mbase + 16 j + fr and
// columns nbase + 32 a + 8 fq .. + 7.  On gfx9 one counter tracks vector loads and stores in issue
// order, so a load issued after stores cannot be waited for without waiting for those stores too.
// The epilogue therefore loads the per-column bias and gate once, before any store, and fetches the
// residual rows one column group ahead of the stores that use them.  Rows past M and columns past N
// go through buffer instructions whose offset is pushed out of the resource's range (loads read
// zero, stores are dropped), so the memory instructions are issued unconditionally.
namespace epi {
constexpr uint32_t OUT_OF_RANGE = 0x80000000u;   // past every resource below (each < 2^31 bytes)

// The arguments are wave-uniform (kernel arguments and workgroup/wave indices); readfirstlane states
// it, so the resource lives in scalar registers rather than behind a per-lane waterfall loop.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  const uint64_t p = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
__device__ __forceinline__ f32x4 ld4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// POL: the cache-policy bits of the store (0, or kStoreNT below)
template <int POL = 0>
__device__ __forceinline__ void st4(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, POL);
}
// Non-temporal (the nt bit): the 8-wave kernel's bf16 output stores (store and GELU epilogues) when the
// launch's output is at least kNTBytes (64 MiB), so that a round's burst of output lines does not push the
// next tiles' operands out of L2.  Measured on the 1.3B-shaped pool of 16 (same box, alternating, latents
// bit-identical): draft 240.7 -> 238.4 ms at a 128 MiB threshold (QKV and MLP up), 247.1 -> 245.7 ms on
// another box when the threshold also takes cross q's 77 MB; with the residual epilogues' fp32 stores
// non-temporal too 238.9 (the residual projection alone 168 -> 146 us, but the next LayerNorm then reads
// its rows from further out); with non-temporal stores at every size, one candidate's refinement step
// (outputs of 10-28 MB, read back from the caches by the next kernel) measured 7.53 -> 7.78 ms, hence the
// size threshold.
constexpr int kStoreNT = 2;
constexpr size_t kNTBytes = (size_t)64 << 20;
}  // namespace epi

// A wave's output, whatever the MFMA shape, is walked as NCG column groups x NRB row blocks: in row
// block rb the lane owns row mbase + RS rb + r0 and, in column group cg, the 8 consecutive columns
// nbase + col(cg) .. + 7 with values val(cg, rb, q), q = 0..7 (two 4-column halves).

// Residual update out = in + gate (acc + bias), in = e.res_in or out itself, optional cache write
// (CM 1: copy of the new row, CM 2: new row minus what the cache held).  Batches of JB row blocks of one column group; a column group's
// bias and gate come with its first batch.  PIPE 2: the loads of batch x + 1 are issued before the
// stores of batch x.
template <int NCG, int NRB, int RS, int CM, int PIPE, int JB, int POL = 0, typename Col, typename Val>
__device__ __forceinline__ void residual_tile(const EpiArgs &e, int M, int N, int mbase, int nbase, int r0,
                                              Col col, Val val) {
  using namespace epi;
  constexpr int NJ = NRB / JB, NB = NCG * NJ;
  static_assert(NRB % JB == 0, "row blocks per batch");
  const int rows = max(0, min(M - mbase, RS * NRB));
  const uint32_t bytes = (uint32_t)rows * (uint32_t)e.ldo * 4u;
  const __amdgpu_buffer_rsrc_t rsO = rsrc((float *)e.out + (int64_t)mbase * e.ldo, bytes);
  const __amdgpu_buffer_rsrc_t rsI = rsrc((e.res_in ? e.res_in : (const float *)e.out) + (int64_t)mbase * e.ldo, bytes);
  const __amdgpu_buffer_rsrc_t rsC = rsrc(CM ? e.cache + (int64_t)mbase * e.ldo : nullptr, CM ? bytes : 0u);
  const __amdgpu_buffer_rsrc_t rsB = rsrc(e.bias, e.bias ? (uint32_t)N * 4u : 0u);
  const __amdgpu_buffer_rsrc_t rsG = rsrc(e.gate, e.gate ? (uint32_t)N * 4u : 0u);
  const bool has_gate = e.gate != nullptr;
  uint32_t c0[NCG], c1[NCG];   // byte offsets of the two 4-column halves, or out of range
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    const int n = nbase + col(cg);
    c0[cg] = n < N ? (uint32_t)n * 4u : OUT_OF_RANGE;
    c1[cg] = n + 4 < N ? (uint32_t)(n + 4) * 4u : OUT_OF_RANGE;
  }
  const uint32_t ro = (uint32_t)r0 * (uint32_t)e.ldo * 4u, rstep = (uint32_t)RS * (uint32_t)e.ldo * 4u;
  f32x4 h[PIPE][JB][2], c[CM == 2 ? PIPE : 1][JB][2], b[NCG][2], g[NCG][2];
  auto fetch = [&](int x, int buf) {   // batch x: column group x / NJ, row blocks JB (x % NJ) ..
    const int cg = x / NJ, j0 = JB * (x % NJ);
    if (x % NJ == 0) {
      b[cg][0] = ld4(rsB, c0[cg]);
      b[cg][1] = ld4(rsB, c1[cg]);
      if (has_gate) {
        g[cg][0] = ld4(rsG, c0[cg]);
        g[cg][1] = ld4(rsG, c1[cg]);
      } else {
        g[cg][0] = g[cg][1] = f32x4{1.f, 1.f, 1.f, 1.f};
      }
    }
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const uint32_t r = ro + (uint32_t)(j0 + jj) * rstep;
      h[buf][jj][0] = ld4(rsI, r + c0[cg]);
      h[buf][jj][1] = ld4(rsI, r + c1[cg]);
      if constexpr (CM == 2) {
        c[buf][jj][0] = ld4(rsC, r + c0[cg]);
        c[buf][jj][1] = ld4(rsC, r + c1[cg]);
      }
    }
  };
  if constexpr (PIPE == 2) fetch(0, 0);
#pragma unroll
  for (int x = 0; x < NB; ++x) {
    const int cg = x / NJ, j0 = JB * (x % NJ);
    const int buf = PIPE == 2 ? (x & 1) : 0;
    if constexpr (PIPE == 2) {
      if (x + 1 < NB) fetch(x + 1, (x + 1) & 1);
    } else {
      fetch(x, 0);
    }
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        f32x4 o = h[buf][jj][hf];
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] += g[cg][hf][q] * (val(cg, j0 + jj, 4 * hf + q) + b[cg][hf][q]);
        const uint32_t off = ro + (uint32_t)(j0 + jj) * rstep + (hf ? c1[cg] : c0[cg]);
        st4<POL>(rsO, off, o);
        if constexpr (CM == 1) st4<POL>(rsC, off, o);
        if constexpr (CM == 2) st4<POL>(rsC, off, o - c[buf][jj][hf]);
      }
    }
  }
}

// Residual update of the 8-wave tile (NCG column groups of 32 per wave, 16 WTA rows) through LDS: for each
// column group the wave writes its (16 WTA) x 32 fp32 block to a region of its own (16-byte chunk k of
// row r at k ^ (r & 7)) and reads it back row by row, so that every load of the residual rows, store of
// the updated rows and cache write covers 8 whole rows x 128 bytes per instruction instead of 16-byte
// pieces of 16 rows.  Arithmetic as residual_tile (out = in + gate (acc + bias), the same expression per
// element).  lds: the K-loop's ring, free once every wave is past its last fragment reads (the barrier);
// a wave reuses its region for the next column group without one, its LDS accesses completing in order.
// Batches of B read-back rows, the residual loads of batch b + 1 issued before the stores of batch b.
template <int NCG, int WTA, int CM, int POL>
__device__ __forceinline__ void residual_staged(const EpiArgs &e, const f32x4 (&acc)[2 * NCG][WTA], int M, int N,
                                                int mbase, int nbase, int fr, int fq, int lane, int wave,
                                                char *lds) {
  using namespace epi;
  constexpr int R = 16 * WTA;              // rows of the wave's block
  constexpr int NT = R / 8;                // read-back instructions per column group
  constexpr int B = NT % 4 == 0 ? 4 : 2;   // rows-sets per batch
  constexpr int NB = NT / B;
  char *wl = lds + wave * (R * 32 * 4);
  const int rows = max(0, min(M - mbase, R));
  const uint32_t bytes = (uint32_t)rows * (uint32_t)e.ldo * 4u;
  const __amdgpu_buffer_rsrc_t rsO = rsrc((float *)e.out + (int64_t)mbase * e.ldo, bytes);
  const __amdgpu_buffer_rsrc_t rsI = rsrc((e.res_in ? e.res_in : (const float *)e.out) + (int64_t)mbase * e.ldo, bytes);
  const __amdgpu_buffer_rsrc_t rsC = rsrc(CM ? e.cache + (int64_t)mbase * e.ldo : nullptr, CM ? bytes : 0u);
  const __amdgpu_buffer_rsrc_t rsB = rsrc(e.bias, e.bias ? (uint32_t)N * 4u : 0u);
  const __amdgpu_buffer_rsrc_t rsG = rsrc(e.gate, e.gate ? (uint32_t)N * 4u : 0u);
  const bool has_gate = e.gate != nullptr;
  const int k = lane & 7, rr = lane >> 3;   // read-back: columns 4 k .. + 3 of row 8 t + rr
  const uint32_t rstep = 8u * (uint32_t)e.ldo * 4u, r0 = (uint32_t)rr * (uint32_t)e.ldo * 4u;
  __syncthreads();   // every wave is past its last fragment reads: the ring is free
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
    for (int rb = 0; rb < WTA; ++rb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int r = 16 * rb + fr, kk = 2 * fq + hf;   // the lane's columns 8 fq + 4 hf .. + 3 of row r
        *reinterpret_cast<f32x4 *>(wl + r * 128 + ((kk ^ (r & 7)) << 4)) = acc[2 * cg + hf][rb];
      }
    const int n = nbase + 32 * cg + 4 * k;
    const uint32_t cn = n < N ? (uint32_t)n * 4u : OUT_OF_RANGE;
    const f32x4 bb = ld4(rsB, cn);
    const f32x4 gg = has_gate ? ld4(rsG, cn) : f32x4{1.f, 1.f, 1.f, 1.f};
    f32x4 h[2][B], c[CM == 2 ? 2 : 1][B];
    auto fetch = [&](int bt, int buf) {
#pragma unroll
      for (int i = 0; i < B; ++i) {
        const uint32_t off = r0 + (uint32_t)(B * bt + i) * rstep + cn;
        h[buf][i] = ld4(rsI, off);
        if constexpr (CM == 2) c[buf][i] = ld4(rsC, off);
      }
    };
    fetch(0, 0);
#pragma unroll
    for (int bt = 0; bt < NB; ++bt) {
      const int buf = bt & 1;
      if (bt + 1 < NB) fetch(bt + 1, buf ^ 1);
#pragma unroll
      for (int i = 0; i < B; ++i) {
        const int t = B * bt + i, r = 8 * t + rr;
        const f32x4 a = *reinterpret_cast<const f32x4 *>(wl + r * 128 + ((k ^ (r & 7)) << 4));
        f32x4 o = h[buf][i];
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] += gg[q] * (a[q] + bb[q]);
        const uint32_t off = r0 + (uint32_t)t * rstep + cn;
        st4<POL>(rsO, off, o);
        if constexpr (CM == 1) st4<POL>(rsC, off, o);
        if constexpr (CM == 2) st4<POL>(rsC, off, o - c[buf][i]);
      }
    }
  }
}

// Store (bf16 or fp32), GELU-and-store, or fp32 store; bias loaded first, no load between the
// stores.  WHOLE8: N % 8 == 0, one 16-byte store per 8 bf16 values; else two 8-byte stores.
template <int EPI, typename TO, int NCG, int NRB, int RS, bool WHOLE8, int POL = 0, typename Col, typename Val>
__device__ __forceinline__ void store_tile(const EpiArgs &e, int M, int N, int mbase, int nbase, int r0, Col col,
                                           Val val) {
  using namespace epi;
  constexpr bool F32 = EPI == EPI_STORE_F32 || sizeof(TO) == 4;
  constexpr uint32_t ES = F32 ? 4u : 2u;
  const int rows = max(0, min(M - mbase, RS * NRB));
  const __amdgpu_buffer_rsrc_t rsO = rsrc((char *)e.out + (int64_t)mbase * e.ldo * ES, (uint32_t)rows * (uint32_t)e.ldo * ES);
  const __amdgpu_buffer_rsrc_t rsB = rsrc(e.bias, e.bias ? (uint32_t)N * 4u : 0u);
  uint32_t c0[NCG], c1[NCG];
  f32x4 b[NCG][2];
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    const int n = nbase + col(cg);
    c0[cg] = n < N ? (uint32_t)n : OUT_OF_RANGE;
    c1[cg] = n + 4 < N ? (uint32_t)(n + 4) : OUT_OF_RANGE;
    b[cg][0] = ld4(rsB, n < N ? (uint32_t)n * 4u : OUT_OF_RANGE);
    b[cg][1] = ld4(rsB, n + 4 < N ? (uint32_t)(n + 4) * 4u : OUT_OF_RANGE);
  }
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      const uint32_t ro = (uint32_t)(RS * rb + r0) * (uint32_t)e.ldo;
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = val(cg, rb, q) + b[cg][q >> 2][q & 3];
      if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = gelu_tanh(v[q]);
      }
      // an out-of-range column offset stays out of range after the row offset and scaling are added
      const uint32_t o0 = c0[cg] == OUT_OF_RANGE ? OUT_OF_RANGE : (ro + c0[cg]) * ES;
      const uint32_t o1 = c1[cg] == OUT_OF_RANGE ? OUT_OF_RANGE : (ro + c1[cg]) * ES;
      if constexpr (F32) {
        st4<POL>(rsO, o0, f32x4{v[0], v[1], v[2], v[3]});
        st4<POL>(rsO, o1, f32x4{v[4], v[5], v[6], v[7]});
      } else {
        const bf16x4 w0 = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
        const bf16x4 w1 = {(bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
        if constexpr (WHOLE8) {
          const bf16x8 w = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, w), rsO, o0, 0, POL);
        } else {
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, w0), rsO, o0, 0, POL);
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, w1), rsO, o1, 0, POL);
        }
      }
    }
  }
}

// bf16 store or GELU-and-store of the 8-wave tile with 256-column tiles (2 column groups of 32 per wave)
// through LDS: the wave writes its (16 WTA) x 64 bf16 block to a region of its own (16-byte chunk k of
// row r at k ^ (r & 7), rows of 128 bytes) and reads it back so that each store instruction writes 8
// whole rows x 128 bytes instead of 16 rows x 64 bytes.  Values as store_tile (bias added, GELU, rounded
// to bf16 before staging).  lds: the K-loop's ring, free once every wave is past its last fragment reads.
template <int EPI, int WTA, int POL>
__device__ __forceinline__ void store_staged(const EpiArgs &e, const f32x4 (&acc)[4][WTA], int M, int N, int mbase,
                                             int nbase, int fr, int fq, int lane, int wave, char *lds) {
  using namespace epi;
  constexpr int R = 16 * WTA;
  char *wl = lds + wave * (R * 128);
  const int rows = max(0, min(M - mbase, R));
  const __amdgpu_buffer_rsrc_t rsO = rsrc((bf16 *)e.out + (int64_t)mbase * e.ldo, (uint32_t)rows * (uint32_t)e.ldo * 2u);
  const __amdgpu_buffer_rsrc_t rsB = rsrc(e.bias, e.bias ? (uint32_t)N * 4u : 0u);
  f32x4 b[2][2];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    const int n = nbase + 32 * cg + 8 * fq;
    b[cg][0] = ld4(rsB, n < N ? (uint32_t)n * 4u : OUT_OF_RANGE);
    b[cg][1] = ld4(rsB, n + 4 < N ? (uint32_t)(n + 4) * 4u : OUT_OF_RANGE);
  }
  __syncthreads();   // every wave is past its last fragment reads: the ring is free
#pragma unroll
  for (int cg = 0; cg < 2; ++cg)
#pragma unroll
    for (int rb = 0; rb < WTA; ++rb) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = acc[2 * cg + (q >> 2)][rb][q & 3] + b[cg][q >> 2][q & 3];
      if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = gelu_tanh(v[q]);
      }
      const bf16x8 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3], (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
      const int r = 16 * rb + fr, kk = 4 * cg + fq;   // columns 8 kk .. + 7 of row r
      *reinterpret_cast<bf16x8 *>(wl + r * 128 + ((kk ^ (r & 7)) << 4)) = w;
      // GELU on 256-row tiles: without a fence the scheduler overlaps enough chunks to spill
    }
  const int k = lane & 7, rr = lane >> 3;   // read-back: columns 8 k .. + 7 of row 8 t + rr
  const int n = nbase + 8 * k;
  const uint32_t cn = n < N ? (uint32_t)n * 2u : OUT_OF_RANGE;   // N % 8 == 0: a chunk is in or out whole
  const uint32_t rstep = 8u * (uint32_t)e.ldo * 2u, r0 = (uint32_t)rr * (uint32_t)e.ldo * 2u;
#pragma unroll
  for (int t = 0; t < R / 8; ++t) {
    const int r = 8 * t + rr;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(wl + r * 128 + ((k ^ (r & 7)) << 4));
    __builtin_amdgcn_raw_buffer_store_b128(v, rsO, cn == OUT_OF_RANGE ? OUT_OF_RANGE : r0 + (uint32_t)t * rstep + cn, 0,
                                           POL);
  }
}

// fp32 store of the 8-wave tile (the K ranges' partial sums of a split-K launch) through LDS, as
// residual_staged without the residual: per column group the wave's (16 WTA) x 32 block goes to its LDS
// region and back so that each store instruction writes 8 whole rows x 128 bytes.  out = acc + bias.
template <int NCG, int WTA, int POL>
__device__ __forceinline__ void store_staged_f32(const EpiArgs &e, const f32x4 (&acc)[2 * NCG][WTA], int M, int N,
                                                 int mbase, int nbase, int fr, int fq, int lane, int wave,
                                                 char *lds) {
  using namespace epi;
  constexpr int R = 16 * WTA;
  char *wl = lds + wave * (R * 32 * 4);
  const int rows = max(0, min(M - mbase, R));
  const __amdgpu_buffer_rsrc_t rsO = rsrc((float *)e.out + (int64_t)mbase * e.ldo, (uint32_t)rows * (uint32_t)e.ldo * 4u);
  const __amdgpu_buffer_rsrc_t rsB = rsrc(e.bias, e.bias ? (uint32_t)N * 4u : 0u);
  const int k = lane & 7, rr = lane >> 3;   // read-back: columns 4 k .. + 3 of row 8 t + rr
  const uint32_t rstep = 8u * (uint32_t)e.ldo * 4u, r0 = (uint32_t)rr * (uint32_t)e.ldo * 4u;
  __syncthreads();   // every wave is past its last fragment reads: the ring is free
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
    for (int rb = 0; rb < WTA; ++rb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int r = 16 * rb + fr, kk = 2 * fq + hf;
        *reinterpret_cast<f32x4 *>(wl + r * 128 + ((kk ^ (r & 7)) << 4)) = acc[2 * cg + hf][rb];
      }
    const int n = nbase + 32 * cg + 4 * k;
    const uint32_t cn = n < N ? (uint32_t)n * 4u : OUT_OF_RANGE;
    const f32x4 bb = ld4(rsB, cn);
#pragma unroll
    for (int t = 0; t < R / 8; ++t) {
      const int r = 8 * t + rr;
      const f32x4 a = *reinterpret_cast<const f32x4 *>(wl + r * 128 + ((k ^ (r & 7)) << 4));
      f32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = a[q] + bb[q];
      st4<POL>(rsO, cn == OUT_OF_RANGE ? OUT_OF_RANGE : r0 + (uint32_t)t * rstep + cn, o);
    }
  }
}

// The epilogue of a wave's output for every epilogue kind, on the group/block walk above.  PIPE:
// residual rows fetched one batch ahead (2) or per batch (1), by the kernel's register budget.
template <int EPI, typename TO, int NCG, int NRB, int RS, int PIPE, bool WHOLE8, int POL = 0, typename Col, typename Val>
__device__ __forceinline__ void wave_epilogue(const EpiArgs &e, int M, int N, int mbase, int nbase, int r0, Col col,
                                              Val val) {
  if constexpr (EPI == EPI_RESIDUAL) {
    constexpr int JB = PIPE == 2 ? (NRB % 2 == 0 ? 2 : 1) : (NRB % 4 == 0 ? 4 : (NRB % 2 == 0 ? 2 : 1));
    if (!e.cache) residual_tile<NCG, NRB, RS, 0, PIPE, JB, POL>(e, M, N, mbase, nbase, r0, col, val);
    else if (!e.cache_delta) residual_tile<NCG, NRB, RS, 1, PIPE, JB, POL>(e, M, N, mbase, nbase, r0, col, val);
    else residual_tile<NCG, NRB, RS, 2, 1, JB, POL>(e, M, N, mbase, nbase, r0, col, val);
  } else if constexpr (EPI == EPI_EULER) {
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
      const int n = nbase + col(cg);
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        const int m = mbase + RS * rb + r0;
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = val(cg, rb, q);
        if (m < M && n < N) {
          if (n + 8 <= N) epilogue8<EPI, TO>(e, m, n, v);
          else epilogue4<EPI, TO>(e, m, n, v[0], v[1], v[2], v[3]);   // N % 8 == 4 edge
        }
      }
    }
  } else {
    store_tile<EPI, TO, NCG, NRB, RS, WHOLE8, POL>(e, M, N, mbase, nbase, r0, col, val);
  }
}

// 16x16 MFMA tiles: acc[i][j] (i over 16-column W fragments, permuted so that fragments 2a and 2a+1
// give a lane 8 consecutive columns; j over 16-row A fragments) holds rows mbase + 16 j + fr and
// columns nbase + 32 a + 8 fq .. + 7 (fr = lane & 15, fq = lane >> 4).
template <int EPI, typename TO, int WTN, int WTM, int PIPE, bool WHOLE8, int POL = 0>
__device__ __forceinline__ void tile_epilogue(const EpiArgs &e, const f32x4 (&acc)[WTN][WTM], int M, int N,
                                              int mbase, int nbase, int fr, int fq) {
  wave_epilogue<EPI, TO, WTN / 2, WTM, 16, PIPE, WHOLE8, POL>(
      e, M, N, mbase, nbase, fr, [&](int cg) { return 32 * cg + 8 * fq; },
      [&](int cg, int rb, int q) { return acc[2 * cg + (q >> 2)][rb][q & 3]; });
}

// ---------------------------------------------------------------------------------- MFMA path
namespace mf {
constexpr int BK = 64;
// A workgroup is a WGM x WGN grid of waves, each computing a (16 WTM) x (16 WTN) tile of C.
// LDS tile: [rows][64] bf16 = 8 chunks of 16 B per row, chunk c of row r stored at c ^ swz(r).  The
// 16 lanes of one ds_read_b128 phase read one chunk of 16 rows and must land in 16 distinct 16-byte
// slots of the 256-byte bank window, slot = (r & 1) 8 + (c ^ swz(r)).  With swz bits (r1, r2 ^ r4, r3)
// that holds both for 16 consecutive rows (the A fragments) and for the permuted W fragment rows
// {0..3, 8..11, 16..19, 24..27} (+ 4) of a 32-row group.
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 5) | (((r >> 1) ^ (r >> 3)) & 2); }
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ swz(r)) << 3); }

// Raw buffer resource over `rows` rows of K bf16; loads whose VGPR offset lies past the range return
// zero.  The entry points bound K by 65536, so 256 rows span at most 32 MiB, well inside 32 bits.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const bf16 *base, int rows, int K) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16 *>(base), (short)0, rows * K * 2, 0x00020000);
}

// Workgroup id -> (m tile, n tile).  Workgroups are dispatched round-robin over the 8 XCDs; each XCD
// is given a contiguous range of tiles, and tiles are ordered in groups of `group` m-tiles sweeping
// all n-tiles, so the workgroups resident on one XCD share A rows and W rows in that XCD's L2
// (group 1: every n-tile of one row block before the next row block).
constexpr int GROUP_M = 8;
__device__ __forceinline__ void tile_of(int bid, int MT, int NT, int &mt, int &nt, int group_m = GROUP_M) {
  const int total = MT * NT;
  const int xcd = bid & 7, local = bid >> 3;
  const int base = total >> 3, rem = total & 7;
  const int t = xcd * base + min(xcd, rem) + local;
  const int per_group = group_m * NT;
  const int group = t / per_group, first_m = group * group_m;
  const int gm = min(MT - first_m, group_m);
  const int r = t - group * per_group;
  mt = first_m + r % gm;
  nt = r / gm;
}
}  // namespace mf

// A 4-wave workgroup must leave room for a second one on the CU (2 waves per SIMD, <= 256 registers).
template <int WTM, int WTN, int WGM, int WGN, int DEPTH, bool KTAIL, int EPI, typename TO>
__global__ __launch_bounds__(64 * WGM * WGN, WGM * WGN <= 4 ? 2 : 1) void k_linear_mfma(int M, int N, int K,
                                                                   const bf16 *__restrict__ A,
                                                                   const bf16 *__restrict__ Wt,
                                                                   EpiArgs e, int MT, int NT) {
  using namespace mf;
  constexpr int THREADS = 64 * WGM * WGN, ROWS = THREADS / 8;  // rows covered per load pass
  constexpr int BM = 16 * WTM * WGM, BN = 16 * WTN * WGN;
  constexpr int LA = BM / ROWS, LW = BN / ROWS;  // 16-byte chunks per thread per K tile
  constexpr int STAGE = (BM + BN) * BK;          // elements of one LDS stage: A tile then W tile
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int total = MT * NT;
  const int ld_r = tid >> 3, ld_c = tid & 7;  // row 0..ROWS-1 (+ROWS i), chunk 0..7

  // Per-tile load addressing (rows past the edge are clamped; their results are never stored).
  int m0 = 0, n0 = 0;
  const bf16 *Ab = A, *Wb = Wt;
  uint32_t oa[LA], ow[LW];
  auto setup_tile = [&](int t) {
    int mt, nt;
    tile_of(t, MT, NT, mt, nt);
    m0 = mt * BM;
    n0 = nt * BN;
    Ab = A + (int64_t)m0 * K + ld_c * 8;
    Wb = Wt + (int64_t)n0 * K + ld_c * 8;
#pragma unroll
    for (int i = 0; i < LA; ++i) oa[i] = (uint32_t)(min(ld_r + ROWS * i, M - 1 - m0) * K);
#pragma unroll
    for (int i = 0; i < LW; ++i) ow[i] = (uint32_t)(min(ld_r + ROWS * i, N - 1 - n0) * K);
  };

  // Staging registers: DEPTH sets, so that a K tile's global loads are issued DEPTH tiles before
  // they are stored to LDS.  K tail: chunks past K are loaded from a valid address and zeroed at
  // store time (a select, so freshly issued loads are never waited on early).
  u32x4 ra[DEPTH][LA], rw[DEPTH][LW];
  bool okk[DEPTH];
  auto load_tile = [&](int k0, int set) {
    okk[set] = !KTAIL || (k0 + ld_c * 8) < K;
    const int kk = okk[set] ? k0 : K - 8 - ld_c * 8;
#pragma unroll
    for (int i = 0; i < LA; ++i) ra[set][i] = *reinterpret_cast<const u32x4 *>(Ab + oa[i] + kk);
#pragma unroll
    for (int i = 0; i < LW; ++i) rw[set][i] = *reinterpret_cast<const u32x4 *>(Wb + ow[i] + kk);
  };
  auto store_tile = [&](bf16 *sA, int set) {
    bf16 *sW = sA + BM * BK;
    const u32x4 z = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < LA; ++i) *reinterpret_cast<u32x4 *>(&sA[lds_off(ld_r + ROWS * i, ld_c)]) = (!KTAIL || okk[set]) ? ra[set][i] : z;
#pragma unroll
    for (int i = 0; i < LW; ++i) *reinterpret_cast<u32x4 *>(&sW[lds_off(ld_r + ROWS * i, ld_c)]) = (!KTAIL || okk[set]) ? rw[set][i] : z;
  };

  f32x4 acc[WTN][WTM];
  const int fr = lane & 15, fq = lane >> 4;
  const int rowA = 16 * WTM * wm + fr;
  // MFMA tile i takes W rows 32 (i/2) + 8 (fr/4) + 4 (i%2) + fr%4, so a lane's outputs of tiles 2a
  // and 2a+1 are 8 consecutive columns (WTN is even)
  auto w_row = [&](int i) { return 16 * WTN * wn + 32 * (i >> 1) + 8 * (fr >> 2) + 4 * (i & 1) + (fr & 3); };
  // All fragments of a 32-wide K substep are requested before its MFMA chain starts, so the LDS
  // latency is paid once per substep rather than once per few MFMAs.
  auto compute = [&](const bf16 *sA) {
    const bf16 *sW = sA + BM * BK;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 fw[WTN], fa[WTM];
#pragma unroll
      for (int i = 0; i < WTN; ++i)
        fw[i] = *reinterpret_cast<const bf16x8 *>(&sW[lds_off(w_row(i), fq + 4 * ks)]);
#pragma unroll
      for (int j = 0; j < WTM; ++j)
        fa[j] = *reinterpret_cast<const bf16x8 *>(&sA[lds_off(rowA + 16 * j, fq + 4 * ks)]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < WTM; ++j)
#pragma unroll
        for (int i = 0; i < WTN; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // acc[i][j] (C^T tile 16x16): lane column = m index (lane & 15), rows = 4 consecutive n.
  auto epilogue = [&](int em0, int en0) {
    tile_epilogue<EPI, TO, WTN, WTM, 1, false>(e, acc, M, N, em0 + 16 * WTM * wm, en0 + 16 * WTN * wn, fr, fq);
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
      for (int j = 0; j < WTM; ++j) acc[i][j] = f32x4{0, 0, 0, 0};
  };

  const int ktiles = (K + BK - 1) / BK;
  if constexpr (DEPTH == 1) {
    setup_tile(blockIdx.x);
    zero_acc();
    load_tile(0, 0);
    store_tile(smem, 0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
      const bool more = kt + 1 < ktiles;
      if (more) load_tile((kt + 1) * BK, 0);
      compute(smem + (kt & 1) * STAGE);
      if (more) store_tile(smem + ((kt + 1) & 1) * STAGE, 0);
      __syncthreads();
    }
    epilogue(m0, n0);
  } else {
    // tile t is loaded into register set t % 2 during iteration t - 2 and stored during t - 1
    setup_tile(blockIdx.x);
    zero_acc();
    load_tile(0, 0);
    if (ktiles > 1) load_tile(BK, 1);
    store_tile(smem, 0);
    __syncthreads();
    auto iter = [&](int kt, int set_next) {   // set_next = (kt + 1) % 2, compile-time per call site
      if (kt + 2 < ktiles) load_tile((kt + 2) * BK, set_next ^ 1);
      compute(smem + (kt & 1) * STAGE);
      if (kt + 1 < ktiles) store_tile(smem + ((kt + 1) & 1) * STAGE, set_next);
      __syncthreads();
    };
    int kt = 0;
    for (; kt + 1 < ktiles; kt += 2) {
      iter(kt, 1);
      iter(kt + 1, 0);
    }
    if (kt < ktiles) iter(kt, 1);
    epilogue(m0, n0);
  }
}

// ------------------------------------------------- MFMA path, 4 waves, LDS filled directly
// (32 WTA)x256 workgroup tile (WTA = 4..8; the plan uses 8 and 7), 4 waves in a 2x2 grid, each (16 WTA) (m) x 128 (n) with up
// to 256 accumulators (one wave per SIMD; the compiler holds them in AGPRs); K tiles of 64 (K % 64 ==
// 0, K >= 128).  The tile height lets a launch fill whole rounds of the chip (at M = 24960, N = 1536:
// 672 tiles of 224 rows fill three rounds, where 588 tiles of 256 rows leave the third 30% full).
// Global -> LDS by buffer loads that write LDS themselves (no staging registers, no ds_write): one
// load instruction fills 1 KB = 8 rows of the swizzled layout, lane l writing 16-byte slot l, so each
// lane fetches the chunk that belongs in its slot.  Two LDS stages.  Per K tile: substep 0's MFMAs
// while substep 1's fragments are read; wait for the next tile's loads and barrier; the loads of the
// tile after next go into the stage just finished; substep 1's MFMAs while the next tile's substep-0
// fragments are read.
__host__ __device__ constexpr int vmcnt_imm(int n) {   // s_waitcnt vmcnt(n), expcnt and lgkmcnt open
  return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xF00;
}

// One (32 WTA)x256 tile at rows m0.., columns n0.. (the body of k_linear_dma).
template <int EPI, typename TO, int WTA>
__device__ __forceinline__ void dma_tile(int M, int N, int K, const bf16 *__restrict__ A, const bf16 *__restrict__ Wt,
                                         const EpiArgs &e, int m0, int n0, bf16 *smem) {
  using namespace mf;
  static_assert(WTA >= 4 && WTA <= 8, "tile height 128..256");
  constexpr int BM = 32 * WTA, BN = 256, WT = 8;
  constexpr int STAGE = (BM + BN) * BK;
  constexpr int NL = WTA + 8;      // load instructions per wave per K tile (A rows, then W rows)
  constexpr int NR = WTA + 8;      // fragment reads per wave per substep (W, then A)
  constexpr int NS = 2 * WTA;      // MFMA groups of 4 per substep, the slots the reads and loads ride in
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const __amdgpu_buffer_rsrc_t rsA = tile_rsrc(A + (int64_t)m0 * K, min(M - m0, BM), K);
  const __amdgpu_buffer_rsrc_t rsW = tile_rsrc(Wt + (int64_t)n0 * K, min(N - n0, BN), K);
  // load x of this wave: x < WTA -> A rows 8 WTA wave + 8 x .. + 7, else W rows 64 wave + 8 (x - WTA)
  // .. + 7; lane l -> row + (l >> 3), slot l & 7
  int voffA[8], voffW[8];   // voffA: first WTA used
#pragma unroll
  for (int x = 0; x < WTA; ++x) {
    const int r = 8 * WTA * wave + 8 * x + (lane >> 3);
    voffA[x] = (r * K + (((lane & 7) ^ swz(r)) << 3)) * 2;
  }
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int r = 64 * wave + 8 * x + (lane >> 3);
    voffW[x] = (r * K + (((lane & 7) ^ swz(r)) << 3)) * 2;
  }
  auto dma_one = [&](int kt, int st, int x) {
    const int soff = kt * BK * 2;
    bf16 *sA = smem + st * STAGE;
    if (x < WTA)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (__attribute__((address_space(3))) void *)(sA + (8 * WTA * wave + 8 * x) * BK),
                                               16, voffA[x], soff, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (__attribute__((address_space(3))) void *)(sA + BM * BK + (64 * wave + 8 * (x - WTA)) * BK),
                                               16, voffW[x - WTA], soff, 0, 0);
  };
  auto dma_all = [&](int kt, int st) {
#pragma unroll
    for (int x = 0; x < NL; ++x) dma_one(kt, st, x);
  };
  f32x4 acc[WT][WTA];
  const int fr = lane & 15, fq = lane >> 4;
  // Fragment x of substep ks: x < 8 -> W fragment i = x, rows 128 wn + 32 (i/2) + 8 (fr/4) + 4 (i%2) +
  // fr%4 (a lane's outputs of tiles 2a, 2a+1 are then 8 consecutive columns); x >= 8 -> A fragment
  // j = x - 8, rows 16 WTA wm + 16 j + fr.  Rows 32 apart share the swizzle, so each fragment is one of
  // four per-lane byte offsets ([ks][parity], W and A) plus an immediate.
  uint32_t offW[2][2], offA[2][2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      offW[ks][q] = 2 * (BM * BK + lds_off(128 * wn + 8 * (fr >> 2) + 4 * q + (fr & 3), fq + 4 * ks));
      offA[ks][q] = 2 * lds_off(16 * WTA * wm + 16 * q + fr, fq + 4 * ks);
    }
  const char *lds = reinterpret_cast<const char *>(smem);
  bf16x8 fw0[WT], fa0[WTA], fw1[WT], fa1[WTA];
  auto rd = [&](int st, int ks, bf16x8 *fw, bf16x8 *fa, int x) {
    const char *base = lds + st * (STAGE * 2);
    if (x < WT) fw[x] = *reinterpret_cast<const bf16x8 *>(base + offW[ks][x & 1] + 4096 * (x >> 1));
    else fa[x - WT] = *reinterpret_cast<const bf16x8 *>(base + offA[ks][x & 1] + 4096 * ((x - WT) >> 1));
  };
  // The 8 WTA MFMAs of one substep in NS groups of 4, the NR fragment reads of the next substep (READ)
  // and the NL loads of a later tile (LOAD) spread over the groups; fences pin the interleaving.  The
  // MFMAs are builtins so the compiler sees their latency and covers it wherever it copies an
  // accumulator.
  auto substep = [&](auto READ, auto LOAD, const bf16x8 *fw, const bf16x8 *fa, int nst, int nks, bf16x8 *nfw,
                     bf16x8 *nfa, int dma_kt, int dma_st) {
#pragma unroll
    for (int j = 0; j < WTA; ++j) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int slot = 2 * j + h;
#pragma unroll
        for (int i = 4 * h; i < 4 * h + 4; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
        if constexpr (decltype(READ)::value) {
#pragma unroll
          for (int x = slot * NR / NS; x < (slot + 1) * NR / NS; ++x) rd(nst, nks, nfw, nfa, x);
        }
        if constexpr (decltype(LOAD)::value) {
#pragma unroll
          for (int x = slot * NL / NS; x < (slot + 1) * NL / NS; ++x) dma_one(dma_kt, dma_st, x);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  const int KT = K / BK;   // >= 2
  dma_all(0, 0);
  dma_all(1, 1);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(NL));   // tile 0 has landed (tile 1's NL loads may be in flight)
  __syncthreads();
#pragma unroll
  for (int x = 0; x < NR; ++x) rd(0, 0, fw0, fa0, x);
#pragma unroll
  for (int i = 0; i < WT; ++i)
#pragma unroll
    for (int j = 0; j < WTA; ++j) acc[i][j] = f32x4{0, 0, 0, 0};
  // K tile kt sits in stage kt & 1; tile kt+1 is in flight into the other stage
  int kt = 0;
  for (; kt + 2 < KT; ++kt) {
    substep(T_{}, F_{}, fw0, fa0, kt & 1, 1, fw1, fa1, 0, 0);
    // tile kt+1 has landed (the LDS-writing loads count in vmcnt, which the barrier alone does not
    // wait for); after the barrier nobody reads stage kt & 1 any more
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    substep(T_{}, T_{}, fw1, fa1, (kt + 1) & 1, 0, fw0, fa0, kt + 2, kt & 1);
  }
  substep(T_{}, F_{}, fw0, fa0, kt & 1, 1, fw1, fa1, 0, 0);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // the last K tile has landed
  __syncthreads();
  substep(T_{}, F_{}, fw1, fa1, (kt + 1) & 1, 0, fw0, fa0, 0, 0);
  ++kt;
  substep(T_{}, F_{}, fw0, fa0, kt & 1, 1, fw1, fa1, 0, 0);
  substep(F_{}, F_{}, fw1, fa1, 0, 0, fw0, fa0, 0, 0);
  tile_epilogue<EPI, TO, WT, WTA, 2, true>(e, acc, M, N, m0 + 16 * WTA * wm, n0 + 128 * wn, fr, fq);
}

// ------------------------------------------------- MFMA path, 8 waves, LDS filled directly
// (32 WTA)x256 workgroup tile (WTA = 6..8), 8 waves in a 2 (m) x 4 (n) grid, each (16 WTA) x 64 (4 WTA
// MFMAs of 16x16x32 per K substep, 16 WTA accumulators), two waves per SIMD: one wave alone issues
// these MFMAs well below the matrix cores' rate (about 1.46 of 1.9 PFLOP/s in an MFMA-only loop), two
// alternating waves keep them busy.  Same LDS layout, LDS-writing loads (waves 0-3 fill the A rows,
// WTA instructions each per K tile, waves 4-7 the W rows, 8 each), two stages of K = 64 and the same
// interleaving of fragment reads and loads with the MFMA groups as dma_tile.
// s_waitcnt until at most n (wave-uniform, 0..4) K tiles of PER loads each are in flight
template <int PER>
__device__ __forceinline__ void wait_tiles(int n) {
  static_assert(4 * PER < 64, "vmcnt holds 6 bits");
  switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;
    case 1: __builtin_amdgcn_s_waitcnt(vmcnt_imm(PER)); break;
    case 2: __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * PER)); break;
    case 3: __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * PER)); break;
    default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * PER)); break;
  }
}

// One (32 WTA) x (64 WT) tile on 8 waves in a 2 (m) x 4 (n) grid of (16 WTA) x (16 WT) wave tiles, K tiles
// of 64 through an LDS ring of NST stages, each K tile's loads issued NST - 1 tiles ahead.
template <int EPI, typename TO, int WTA, int WT = 4, int NST = 2, int POL = 0>
__device__ __forceinline__ void dma8_tile(int M, int N, int K, const bf16 *__restrict__ A, const bf16 *__restrict__ Wt,
                                          const EpiArgs &e, int m0, int n0, bf16 *smem, int ldk) {
  // K: columns accumulated (K % 64 == 0, K >= 128); ldk: row stride of A and Wt in elements (ldk >= K;
  // larger for one K range of a split-K launch, whose A and Wt point at the range's first column)
  using namespace mf;
  static_assert(WTA >= 4 && WTA <= 8, "tile height 128..256");
  static_assert(WT == 2 || WT == 4, "tile width 128 or 256");
  static_assert(NST >= 2 && NST * (32 * WTA + 64 * WT) * BK * 2 <= 160 * 1024, "LDS ring within 160 KB");
  constexpr int BM = 32 * WTA, BN = 64 * WT;
  constexpr int STAGE = (BM + BN) * BK;
  // load slots per K tile: WTA for an A wave (8 WTA rows), 2 WT for a W wave (16 WT rows)
  constexpr int NL = WTA > 2 * WT ? WTA : 2 * WT;
  constexpr int NR = WT + WTA;     // fragment reads per wave per substep (W, then A)
  constexpr int NS = WTA;          // MFMA groups of WT per substep
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const bool loads_a = wave < 4;
  const __amdgpu_buffer_rsrc_t rsA = tile_rsrc(A + (int64_t)m0 * ldk, min(M - m0, BM), ldk);
  const __amdgpu_buffer_rsrc_t rsW = tile_rsrc(Wt + (int64_t)n0 * ldk, min(N - n0, BN), ldk);
  // load x of this wave: rows 8 WTA wave + 8 x .. + 7 of A (waves 0-3, x < WTA) or 16 WT (wave - 4) +
  // 8 x .. + 7 of W (waves 4-7, x < 2 WT); lane l -> row + (l >> 3), slot l & 7
  static_assert(NL <= 8, "load slots");
  uint32_t voff[8];   // a fixed size: hipcc's host pass rejects one that depends on the template arguments
  const int row0 = loads_a ? 8 * WTA * wave : 16 * WT * (wave - 4);
#pragma unroll
  for (int x = 0; x < NL; ++x) {
    const int r = row0 + 8 * x + (lane >> 3);
    voff[x] = (uint32_t)((r * ldk + (((lane & 7) ^ swz(r)) << 3)) * 2);
  }
  const uint32_t lds_row0 = (uint32_t)((loads_a ? 0 : BM * BK) + row0 * BK) * 2u;
  auto dma_one = [&](int kt, int st, int x) {
    if (loads_a ? x >= WTA : x >= 2 * WT) return;
    char *dst = reinterpret_cast<char *>(smem) + st * (STAGE * 2) + lds_row0 + x * (8 * BK * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(loads_a ? rsA : rsW, (__attribute__((address_space(3))) void *)dst, 16,
                                             voff[x], kt * BK * 2, 0, 0);
  };
  auto dma_all = [&](int kt, int st) {
#pragma unroll
    for (int x = 0; x < NL; ++x) dma_one(kt, st, x);
  };
  f32x4 acc[WT][WTA];
  const int fr = lane & 15, fq = lane >> 4;
  // Fragment x of substep ks: x < WT -> W fragment i = x, rows 16 WT wn + 32 (i/2) + 8 (fr/4) + 4 (i%2) +
  // fr%4; x >= WT -> A fragment j = x - WT, rows 16 WTA wm + 16 j + fr.  Rows 32 apart share the swizzle.
  uint32_t offW[2][2], offA[2][2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      offW[ks][q] = 2 * (BM * BK + lds_off(16 * WT * wn + 8 * (fr >> 2) + 4 * q + (fr & 3), fq + 4 * ks));
      offA[ks][q] = 2 * lds_off(16 * WTA * wm + 16 * q + fr, fq + 4 * ks);
    }
  const char *lds = reinterpret_cast<const char *>(smem);
  bf16x8 fw0[WT], fa0[WTA], fw1[WT], fa1[WTA];
  auto rd = [&](int st, int ks, bf16x8 *fw, bf16x8 *fa, int x) {
    const char *base = lds + st * (STAGE * 2);
    if (x < WT) fw[x] = *reinterpret_cast<const bf16x8 *>(base + offW[ks][x & 1] + 4096 * (x >> 1));
    else fa[x - WT] = *reinterpret_cast<const bf16x8 *>(base + offA[ks][x & 1] + 4096 * ((x - WT) >> 1));
  };
  auto substep = [&](auto READ, auto LOAD, const bf16x8 *fw, const bf16x8 *fa, int nst, int nks, bf16x8 *nfw,
                     bf16x8 *nfa, int dma_kt, int dma_st) {
#pragma unroll
    for (int j = 0; j < NS; ++j) {
#pragma unroll
      for (int i = 0; i < WT; ++i)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
      if constexpr (decltype(READ)::value) {
#pragma unroll
        for (int x = j * NR / NS; x < (j + 1) * NR / NS; ++x) rd(nst, nks, nfw, nfa, x);
      }
      if constexpr (decltype(LOAD)::value) {
#pragma unroll
        for (int x = j * NL / NS; x < (j + 1) * NL / NS; ++x) dma_one(dma_kt, dma_st, x);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  const int KT = K / BK;   // >= 2
  if constexpr (NST == 2) {
    dma_all(0, 0);
    dma_all(1, 1);
    // tile 0 has landed once only this wave's loads of tile 1 may be in flight
    if (loads_a) __builtin_amdgcn_s_waitcnt(vmcnt_imm(WTA));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * WT));
  } else {
    // tiles 0 .. min(NST, KT) - 1 into stages 0 ..; tile 0 has landed once the others alone may be in flight
#pragma unroll
    for (int t = 0; t < NST; ++t)
      if (t < KT) dma_all(t, t);
    if (loads_a) wait_tiles<WTA>(min(NST, KT) - 1);
    else wait_tiles<2 * WT>(min(NST, KT) - 1);
  }
  __syncthreads();
#pragma unroll
  for (int x = 0; x < NR; ++x) rd(0, 0, fw0, fa0, x);
#pragma unroll
  for (int i = 0; i < WT; ++i)
#pragma unroll
    for (int j = 0; j < WTA; ++j) acc[i][j] = f32x4{0, 0, 0, 0};
  int kt = 0, last;   // last: the stage of the last K tile
  if constexpr (NST == 2) {
    for (; kt + 2 < KT; ++kt) {
      substep(T_{}, F_{}, fw0, fa0, kt & 1, 1, fw1, fa1, 0, 0);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // tile kt+1 has landed
      __syncthreads();                            // nobody reads stage kt & 1 any more
      substep(T_{}, T_{}, fw1, fa1, (kt + 1) & 1, 0, fw0, fa0, kt + 2, kt & 1);
    }
    substep(T_{}, F_{}, fw0, fa0, kt & 1, 1, fw1, fa1, 0, 0);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // the last K tile has landed
    __syncthreads();
    substep(T_{}, F_{}, fw1, fa1, (kt + 1) & 1, 0, fw0, fa0, 0, 0);
    last = (kt + 1) & 1;
  } else {
    // stage of tile t: t % NST.  Iteration kt loads tile kt + NST into the stage of tile kt, which every
    // wave has finished reading by the barrier.
    int st = 0;
    for (; kt + NST < KT; ++kt) {
      const int nx = st + 1 == NST ? 0 : st + 1;
      substep(T_{}, F_{}, fw0, fa0, st, 1, fw1, fa1, 0, 0);
      if (loads_a) wait_tiles<WTA>(NST - 2);   // tile kt+1 has landed
      else wait_tiles<2 * WT>(NST - 2);
      __syncthreads();
      substep(T_{}, T_{}, fw1, fa1, nx, 0, fw0, fa0, kt + NST, st);
      st = nx;
    }
    for (; kt + 1 < KT; ++kt) {   // no loads left to issue; tiles kt+2 .. KT-1 may still be in flight
      const int nx = st + 1 == NST ? 0 : st + 1;
      substep(T_{}, F_{}, fw0, fa0, st, 1, fw1, fa1, 0, 0);
      if (loads_a) wait_tiles<WTA>(KT - 2 - kt);
      else wait_tiles<2 * WT>(KT - 2 - kt);
      __syncthreads();
      substep(T_{}, F_{}, fw1, fa1, nx, 0, fw0, fa0, 0, 0);
      st = nx;
    }
    last = st;
  }
  substep(T_{}, F_{}, fw0, fa0, last, 1, fw1, fa1, 0, 0);
  substep(F_{}, F_{}, fw1, fa1, 0, 0, fw0, fa0, 0, 0);
  if constexpr (EPI == EPI_RESIDUAL && 8 * 16 * WTA * 32 * 4 <= NST * STAGE * 2) {
    // the ring (NST stages of (32 WTA + 64 WT) x 64 bf16) holds the 8 waves' (16 WTA) x 32 fp32 blocks
    // (all tiles but 160 x 128 with 2 stages)
    char *lw = reinterpret_cast<char *>(smem);
    const int mb = m0 + 16 * WTA * wm, nb = n0 + 16 * WT * wn;
    if (!e.cache) residual_staged<WT / 2, WTA, 0, POL>(e, acc, M, N, mb, nb, fr, fq, lane, wave, lw);
    else if (!e.cache_delta) residual_staged<WT / 2, WTA, 1, POL>(e, acc, M, N, mb, nb, fr, fq, lane, wave, lw);
    else residual_staged<WT / 2, WTA, 2, POL>(e, acc, M, N, mb, nb, fr, fq, lane, wave, lw);
  } else if constexpr ((EPI == EPI_STORE || EPI == EPI_GELU) && sizeof(TO) == 2 && WT == 4 &&
                       8 * 16 * WTA * 128 <= NST * STAGE * 2) {
    store_staged<EPI, WTA, POL>(e, acc, M, N, m0 + 16 * WTA * wm, n0 + 16 * WT * wn, fr, fq, lane, wave,
                                reinterpret_cast<char *>(smem));
  } else if constexpr (EPI == EPI_STORE_F32 && 8 * 16 * WTA * 32 * 4 <= NST * STAGE * 2) {
    store_staged_f32<WT / 2, WTA, POL>(e, acc, M, N, m0 + 16 * WTA * wm, n0 + 16 * WT * wn, fr, fq, lane, wave,
                                       reinterpret_cast<char *>(smem));
  } else {
    tile_epilogue<EPI, TO, WT, WTA, 2, true, POL>(e, acc, M, N, m0 + 16 * WTA * wm, n0 + 16 * WT * wn, fr, fq);
  }
}

// MT row blocks x NT column tiles of 256 on the 8-wave tile; row blocks of two heights as in
// k_linear_dma.
template <int EPI, typename TO, int WTA, int POL = 0>
__global__ __launch_bounds__(512, 1) void k_linear_dma8(int M, int N, int K, const bf16 *__restrict__ A,
                                                 const bf16 *__restrict__ Wt, EpiArgs e, int MT, int NT, int tall,
                                                 int group_m) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  int mt, nt;
  mf::tile_of(blockIdx.x, MT, NT, mt, nt, group_m);
  const int before = (int)((int64_t)mt * tall / MT), upto = (int)((int64_t)(mt + 1) * tall / MT);
  const int m0 = 32 * ((WTA - 1) * mt + before), n0 = nt * 256;
  if (m0 >= M) return;   // a block past the last row (a forced plan with more blocks than M needs)
  if constexpr (WTA > 5) {
    if (upto == before) {
      dma8_tile<EPI, TO, WTA - 1, 4, 2, POL>(M, N, K, A, Wt, e, m0, n0, smem, K);
      return;
    }
  }
  dma8_tile<EPI, TO, WTA, 4, 2, POL>(M, N, K, A, Wt, e, m0, n0, smem, K);
}

// MT x NT tiles of (32 WTA) x (64 WT) on the 8-wave tile with an LDS ring of NST stages: for launches with
// no more tiles than CUs, where each workgroup's K loop waits on load latency rather than on the matrix
// cores (one candidate's projections, M = 1560).
template <int EPI, typename TO, int WTA, int WT, int NST>
__global__ __launch_bounds__(512, 1) void k_linear_deep(int M, int N, int K, const bf16 *__restrict__ A,
                                                 const bf16 *__restrict__ Wt, EpiArgs e, int MT, int NT,
                                                 int group_m) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  int mt, nt;
  mf::tile_of(blockIdx.x, MT, NT, mt, nt, group_m);
  const int m0 = 32 * WTA * mt, n0 = 64 * WT * nt;
  if (m0 >= M) return;
  dma8_tile<EPI, TO, WTA, WT, NST>(M, N, K, A, Wt, e, m0, n0, smem, K);
}

// Split-K: MT x NT tiles of (32 WTA) x (64 WT) on the 8-wave tile with an LDS ring of NST stages, each
// tile's K range cut into `splits` ranges of ks columns (the last one shorter); workgroup (tile, split)
// accumulates its range and stores the fp32 partial sums into part + split M N ([M][N] per split, no
// bias).  k_splitk_reduce then adds the splits in order and applies the epilogue.  For launches whose
// tiles alone would leave most CUs idle (one candidate's MLP down-projection, K = 8960).
template <int WTA, int WT, int NST>
__global__ __launch_bounds__(512, 1) void k_linear_splitk(int M, int N, int K, const bf16 *__restrict__ A,
                                                   const bf16 *__restrict__ Wt, float *__restrict__ part,
                                                   int MT, int NT, int ks, int group_m) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  const int tiles = MT * NT;
  const int split = blockIdx.x / tiles;
  int mt, nt;
  mf::tile_of(blockIdx.x - split * tiles, MT, NT, mt, nt, group_m);
  const int m0 = 32 * WTA * mt, n0 = 64 * WT * nt, k0 = split * ks;
  if (m0 >= M || k0 >= K) return;
  EpiArgs e;
  e.out = part + (int64_t)split * M * N;
  e.ldo = N;
  dma8_tile<EPI_STORE_F32, float, WTA, WT, NST>(M, N, min(ks, K - k0), A + k0, Wt + k0, e, m0, n0, smem, K);
}

// out = epilogue(sum over s of part[s] + bias), the splits added in order s = 0, 1, ..; one thread per 8
// consecutive columns of a row (N % 8 == 0).
template <int EPI>
__global__ __launch_bounds__(256) void k_splitk_reduce(int M, int N, int splits, const float *__restrict__ part,
                                                       EpiArgs e) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n8 = N / 8;
  if (i >= (int64_t)M * n8) return;
  const int m = (int)(i / n8), n = (int)(i % n8) * 8;
  const int64_t plane = (int64_t)M * N, at = (int64_t)m * N + n;
  float v[8];
  {
    const float4 a = *reinterpret_cast<const float4 *>(part + at), b = *reinterpret_cast<const float4 *>(part + at + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  for (int sp = 1; sp < splits; ++sp) {
    const float *p = part + sp * plane + at;
    const float4 a = *reinterpret_cast<const float4 *>(p), b = *reinterpret_cast<const float4 *>(p + 4);
    v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w; v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
  }
  epilogue8<EPI, bf16>(e, m, n, v);
}

// MT row blocks x NT column tiles of 256.  Row blocks come in two heights: `tall` of them 32 WTA rows
// high and the rest 32 (WTA - 1), the tall ones spread evenly over the block index (block i is tall
// when floor((i + 1) tall / MT) > floor(i tall / MT)), so that every XCD's range of tiles holds its
// share.  tall == MT is a launch of one height.  Mixing two heights lets a launch fill whole rounds
// of the chip with tiles of nearly equal duration.
template <int EPI, typename TO, int WTA>
__global__ __launch_bounds__(256, 1) void k_linear_dma(int M, int N, int K, const bf16 *__restrict__ A,
                                                const bf16 *__restrict__ Wt, EpiArgs e, int MT, int NT, int tall,
                                                int group_m) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  int mt, nt;
  mf::tile_of(blockIdx.x, MT, NT, mt, nt, group_m);
  const int before = (int)((int64_t)mt * tall / MT), upto = (int)((int64_t)(mt + 1) * tall / MT);
  const int m0 = 32 * ((WTA - 1) * mt + before), n0 = nt * 256;
  if (m0 >= M) return;   // a block past the last row (a forced plan with more blocks than M needs)
  if constexpr (WTA > 4) {
    if (upto == before) {
      dma_tile<EPI, TO, WTA - 1>(M, N, K, A, Wt, e, m0, n0, smem);
      return;
    }
  }
  dma_tile<EPI, TO, WTA>(M, N, K, A, Wt, e, m0, n0, smem);
}
// ---------------------------------------------------------------------------------- VALU path
template <typename TI, int EPI, typename TO>
__global__ __launch_bounds__(256) void k_linear_valu(int M, int N, int K, const TI *__restrict__ A,
                                                     const TI *__restrict__ Wt, EpiArgs e) {
  constexpr int T = 64, TK = 16;
  __shared__ float sA[TK][T + 4];
  __shared__ float sW[TK][T + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.x * T, n0 = blockIdx.y * T;
  float acc[4][4] = {};
  const int lr = tid >> 2, lk = (tid & 3) * 4;  // loader: row 0..63, 4 consecutive k
  for (int k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int k = k0 + lk + q;
      int ma = m0 + lr, nw = n0 + lr;
      sA[lk + q][lr] = (ma < M && k < K) ? to_f32(A[(int64_t)ma * K + k]) : 0.f;
      sW[lk + q][lr] = (nw < N && k < K) ? to_f32(Wt[(int64_t)nw * K + k]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = sW[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
  const int n = n0 + tx * 4;
  if (n >= N) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int m = m0 + ty * 4 + i;
    if (m < M) epilogue4<EPI, TO>(e, m, n, acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
  }
}

// Tile choice for bf16 operands.  The 256x256 kernel runs one workgroup per CU, the 128x128 kernel
// two; a launch takes ceil(tiles / slots) rounds.  Measured on MI355X, a round of 128x128 tiles
// costs 0.64 of a round of 256x256 tiles at the same K (so the small tile does 0.78 of the big
// tile's work per CU).  Candidates: all 256x256; all 128x128; the whole rows of 256x256 tiles that
// fill complete rounds plus the remaining rows as 128x128 tiles (a second launch), which trims a
// last round that would leave most CUs idle; and row blocks of two adjacent heights (32 w and
// 32 (w - 1) rows), as many blocks as fill whole rounds.  Where the LDS-writing loads apply (K % 64
// == 0, K >= 128, N % 8 == 0) the 256-column tiles run on the 8-wave kernel, which measured 6-7%
// faster than the 4-wave kernel on the same tiles at every projection of the draft; the 4-wave
// kernel is kept for forced plans.
enum TilePlan { PLAN_BIG, PLAN_SMALL, PLAN_SPLIT, PLAN_MIX, PLAN_DEEP };
struct TileChoice {
  TilePlan plan;
  int wta;    // PLAN_MIX: the taller height, 32 wta rows
  int rows;   // PLAN_SPLIT: rows on 256x256 tiles
  int mb;     // PLAN_MIX: row blocks
  int tall;   // PLAN_MIX: row blocks of the taller height (the others are 32 (wta - 1) rows)
  int waves = 4;   // PLAN_MIX: the 4-wave (k_linear_dma) or the 8-wave (k_linear_dma8) kernel
  int wt = 4, nst = 2;   // PLAN_DEEP: (32 wta) x (64 wt) tiles, nst LDS stages
};
static int cu_count();
// The deep-ring tiles (wta, wt) in the order the plans try them: 128 x 128, 160 x 128, 128 x 256, 160 x 256.
static constexpr int kDeepTiles[4][2] = {{4, 2}, {5, 2}, {4, 4}, {5, 4}};
// The deep-ring instantiations: 128 or 160 rows x 128 or 256 columns, 2 or 3 LDS stages.
static bool deep_ok(int wta, int wt, int nst) {
  return (wta == 4 || wta == 5) && (wt == 2 || wt == 4) && (nst == 2 || nst == 3);
}

// Round-count model, in units of one K step of a 256x256 round: a launch takes ceil(tiles / slots)
// rounds; a round of 4-wave tiles 32 w rows high costs kF[w] K + kG (the constant: per-tile prologue
// and epilogue), of 128x128 tiles (two per CU) kSmallA K + kSmallFix.  Measured on MI355X at
// M = 24960, K = 1536 and 8960: per round, 224-row tiles take 0.85 of the time of 256-row tiles
// (for 0.875 of the rows), 192-row tiles 0.82, 160-row tiles 0.79.  The plans of one height are
// compared first.  A launch of two heights spreads its taller tiles over all rounds and lets CUs
// that finish a shorter tile early take the next one; it is costed at the block-weighted mean of
// the two heights, and taken only when that beats the best one-height plan by more than kMixGain
// (mixed launches measured a few percent slower than this estimate at wide N).
static constexpr double kF[9] = {0, 0, 0, 0, 0, 0.79, 0.82, 0.85, 1.0};
// The same for the 8-wave kernel (M = 24960, K = 1536): 224-row rounds 0.885 and 192-row rounds
// 0.826 of a 256-row round, 160 rows estimated; a 128x128 round costs kSmall8 more in these units
// than in the 4-wave kernel's (its 256-row round is that much faster); its two-height launches are
// taken when kMixGain8 better than the best one-height plan.
static constexpr double kF8[9] = {0, 0, 0, 0, 0, 0.78, 0.826, 0.885, 1.0};
static constexpr double kSmall8 = 1.064, kMixGain8 = 0.01;
static constexpr double kG = 130.0, kMixGain = 0.02;
static TileChoice pick_tiles(int M, int N, int K, bool dma_ok) {
  // FLASHBON_LINEAR_TILE (tests and tuning): "256x256", "128x128", "bm:<rows>" (4-wave kernel, one
  // tile height: rows 160, 192 or 224), "mix:<w>:<blocks>:<tall>" (4-wave kernel, `blocks` row blocks,
  // `tall` of them 32 w rows high and the rest 32 (w - 1), w in 6..8, covering M), or
  // "split:<rows>" (rows a multiple of 256 with 0 < rows < M: the first rows on 256x256 tiles, the
  // rest on 128x128 tiles); "w8" (the 8-wave kernel, 256x256 tiles), "w8:bm:<rows>" and
  // "w8:mix:<w>:<blocks>:<tall>" (the 8-wave kernel with those row blocks); "deep:<rows>:<cols>:<stages>"
  // (k_linear_deep: rows 128 or 160, cols 128 or 256, 2 or 3 LDS stages)
  const char *force = getenv("FLASHBON_LINEAR_TILE");
  if (force) {
    if (dma_ok && !strncmp(force, "deep:", 5)) {
      int rows = 0, cols = 0, nst = 0;
      if (sscanf(force + 5, "%d:%d:%d", &rows, &cols, &nst) == 3 && deep_ok(rows / 32, cols / 64, nst) &&
          rows % 32 == 0 && cols % 64 == 0) {
        TileChoice c = {PLAN_DEEP, rows / 32, 0, 0, 0, 8};
        c.wt = cols / 64;
        c.nst = nst;
        return c;
      }
    }
    if (!strncmp(force, "split:", 6)) {
      const int rows = atoi(force + 6);
      if (rows > 0 && rows % 256 == 0 && rows < M && K % mf::BK == 0) return {PLAN_SPLIT, 8, rows, 0, 0};
      return {PLAN_BIG, 8, 0, 0, 0};
    }
    int waves = 4;
    if (dma_ok && !strncmp(force, "w8", 2)) {
      waves = 8;
      force += force[2] == ':' ? 3 : 2;
      if (!*force) {
        const int mb = (M + 255) / 256;
        return {PLAN_MIX, 8, 0, mb, mb, 8};
      }
    }
    if (dma_ok && !strncmp(force, "bm:", 3)) {
      const int rows = atoi(force + 3);
      if (rows == 160 || rows == 192 || rows == 224) {
        const int w = rows / 32, mb = (M + rows - 1) / rows;
        return {PLAN_MIX, w + 1, 0, mb, 0, waves};   // all blocks of the shorter height of the w + 1 kernel
      }
    }
    if (dma_ok && !strncmp(force, "mix:", 4)) {
      int w = 0, mb = 0, tall = 0;
      if (sscanf(force + 4, "%d:%d:%d", &w, &mb, &tall) == 3 && w >= 6 && w <= 8 && mb > 0 && tall >= 0 &&
          tall <= mb && 32 * ((int64_t)(w - 1) * mb + tall) >= M)
        return {PLAN_MIX, w, 0, mb, tall, waves};
    }
    return {strcmp(force, "128x128") ? PLAN_BIG : PLAN_SMALL, 8, 0, 0, 0};
  }
  constexpr double kSmallA = 0.704, kSmallFix = 604.0;
  const int cus = cu_count();
  auto rounds = [&](int64_t tiles, int per_cu) { return (double)((tiles + per_cu * cus - 1) / (per_cu * cus)); };
  const double *F = dma_ok ? kF8 : kF;
  auto cost = [&](int w) { return F[w] * K + kG; };
  const int64_t NT = (N + 255) / 256, T = (int64_t)((M + 255) / 256) * NT, NT2 = (N + 127) / 128;
  const double big = cost(8), small = (kSmallA * K + kSmallFix) * (dma_ok ? kSmall8 : 1.0);
  TileChoice best = {PLAN_BIG, 8, 0, 0, 0};
  double t_best = rounds(T, 1) * big;
  if (dma_ok) {
    for (int w = 7; w >= 5; --w) {   // one height, 32 w rows: the kernel for w + 1 with no tall blocks
      const int mb = (M + 32 * w - 1) / (32 * w);
      const double t = rounds((int64_t)mb * NT, 1) * cost(w);
      if (t < t_best) { t_best = t; best = {PLAN_MIX, w + 1, 0, mb, 0, 8}; }
    }
  }
  // a 128x128 launch with no more tiles than CUs runs one workgroup per CU, each faster than when
  // two share the CU: costed at kAlone of a shared round (the refinement of one candidate, M = 1560,
  // has its N = 1536 projections here: 156 tiles)
  constexpr double kAlone = 0.6;
  auto rounds_small = [&](int64_t tiles) { return tiles <= cus ? kAlone : rounds(tiles, 2); };
  const double t_small = rounds_small((int64_t)((M + 127) / 128) * NT2) * small;
  if (t_small < t_best) { t_best = t_small; best = {PLAN_SMALL, 8, 0, 0, 0}; }
  const int64_t mt_big = (T - T % cus) / NT;
  const int rows = (int)(mt_big * 256);
  if (K % mf::BK == 0 && rows > 0 && rows < M) {
    const double t_split = rounds(mt_big * NT, 1) * big + rounds_small(((M - rows + 127) / 128) * NT2) * small;
    if (t_split < t_best) { t_best = t_split; best = {PLAN_SPLIT, 8, rows, 0, 0}; }
  }
  if (dma_ok) {
    // two heights, 32 w and 32 (w - 1) rows.  The 8-wave kernel also mixes 256- with 224-row blocks:
    // at M = 24960 that fills whole rounds for MLP up (102 blocks, 66 of 256 rows: 579 -> 567 us) and
    // QKV (99 blocks, 87 of 256: 292.5 -> 286.9 us), where the 4-wave kernel measured such mixes slower
    const double t_pure = t_best, gain = kMixGain8;
    for (int w = 8; w >= 6; --w) {
      const int lo = 32 * (w - 1);
      const int mb_min = (M + 32 * w - 1) / (32 * w), mb_max = (M + lo - 1) / lo;
      for (int mb = mb_min; mb <= mb_max; ++mb) {
        const int tall = max(0, (int)(((int64_t)M - (int64_t)lo * mb + 31) / 32));
        if (tall == 0 || tall == mb) continue;
        const double t = rounds((int64_t)mb * NT, 1) * ((double)tall * cost(w) + (double)(mb - tall) * cost(w - 1)) / mb;
        if (t < (1.0 - gain) * t_pure && t < t_best) { t_best = t; best = {PLAN_MIX, w, 0, mb, tall, 8}; }
      }
    }
    // Where a launch fits in one round of workgroups one per CU (one or two candidates' projections,
    // M = 1560 or 3120), every workgroup's K loop waits on load latency: there the 8-wave tile with a
    // third LDS stage (loads two K tiles ahead) runs instead, on whichever of 128 x 128, 160 x 128,
    // 128 x 256 and 160 x 256 gives the most tiles within one round.  Measured at M = 1560, K = 1536:
    // QKV (128 x 256, 234 tiles) 28.3 -> 26.6 us, the N = 1536 projections (128 x 128, 156 tiles)
    // 21.0 -> 14.0 us (store) and 24.6 -> 18.2 us (residual); at M = 3120 (160 x 128, 240 tiles) the
    // N = 1536 residual projection 37.2 -> 22.4 us and MLP down 104.3 -> 83.5 us.  Four or five stages
    // measured no faster than three.
    TileChoice deep = {PLAN_DEEP, 0, 0, 0, 0, 8};
    deep.nst = 3;
    int64_t most = 0;
    for (const auto &d : kDeepTiles) {
      const int64_t t = (int64_t)((M + 32 * d[0] - 1) / (32 * d[0])) * ((N + 64 * d[1] - 1) / (64 * d[1]));
      if (t <= cus && t > most) {
        most = t;
        deep.wta = d[0];
        deep.wt = d[1];
      }
    }
    if (most > 0) return deep;
  }
  return best;
}

template <int WTM, int WTN, int WGM, int WGN, int EPI, int DEPTH>
static hipError_t launch_mfma(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e,
                              hipStream_t s) {
  constexpr int BM = 16 * WTM * WGM, BN = 16 * WTN * WGN;
  const size_t lds = (size_t)2 * (BM + BN) * mf::BK * sizeof(bf16);
  auto kern = K % mf::BK ? k_linear_mfma<WTM, WTN, WGM, WGN, DEPTH, true, EPI, bf16>
                          : k_linear_mfma<WTM, WTN, WGM, WGN, DEPTH, false, EPI, bf16>;
  static bool attr_set[2] = {false, false};
  if (!attr_set[K % mf::BK ? 1 : 0]) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set[K % mf::BK ? 1 : 0] = true;
  }
  const int MT = (M + BM - 1) / BM, NT = (N + BN - 1) / BN;
  hipLaunchKernelGGL(kern, dim3(MT * NT), dim3(64 * WGM * WGN), lds, s, M, N, K, (const bf16 *)A,
                     (const bf16 *)Wt, e, MT, NT);
  return hipGetLastError();
}

// Row blocks per tile group of the linear kernels' order (see mf::tile_of).  Narrow outputs (at most
// 8 column tiles) take groups of 1, so an XCD runs every column tile of a row block together and each
// A row block (3.4 MB at K = 8960) is fetched once rather than again in a later round; up to 24 column
// tiles groups of 8 (the 32 tiles an XCD runs at once then span 8 row blocks x 4 column tiles), wider
// outputs groups of 6.  Swept in the 1.3B-shaped draft (M = 24960) on the 8-wave kernel: MLP down
// (N = 1536, K = 8960) best at 1 (61.2 ms per draft against 65.0 at 8), the K = 1536, N = 1536
// projections at 1 (about 1% ahead of 4), QKV (18 column tiles) at 8, MLP up (35) at 6 (55.8 against
// 56.5 ms at 8).  The order does not change any output.  FLASHBON_LINEAR_GROUP (tuning): a fixed
// group height.
static int group_rows(int MT, int NT, int K) {
  const char *force = getenv("FLASHBON_LINEAR_GROUP");
  if (force && atoi(force) > 0) return atoi(force);
  (void)MT; (void)K;
  if (NT <= 8) return 1;
  return NT <= 24 ? mf::GROUP_M : 6;
}

// The 4-wave kernel over mb row blocks, `tall` of them 32 WTA rows high, the rest 32 (WTA - 1).
template <int EPI, int WTA>
static hipError_t launch_dma(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e,
                             hipStream_t s, int mb, int tall) {
  constexpr int BM = 32 * WTA;
  const size_t lds = (size_t)2 * (BM + 256) * mf::BK * sizeof(bf16);
  auto kern = k_linear_dma<EPI, bf16, WTA>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int NT = (N + 255) / 256;
  hipLaunchKernelGGL(kern, dim3(mb * NT), dim3(256), lds, s, M, N, K, (const bf16 *)A, (const bf16 *)Wt, e,
                     mb, NT, tall, group_rows(mb, NT, K));
  return hipGetLastError();
}

// The 8-wave kernel over mb row blocks, `tall` of them 32 WTA rows high, the rest 32 (WTA - 1).
template <int EPI, int WTA>
static hipError_t launch_dma8(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e, hipStream_t s,
                              int mb, int tall) {
  const size_t lds = (size_t)2 * (32 * WTA + 256) * mf::BK * sizeof(bf16);
  // the store policy of a bf16 output by its size (epi::kNTBytes); the fp32 outputs (residual stream and
  // cache, read back by the next LayerNorm or proxy) keep the default
  bool nt = false;
  auto kern = k_linear_dma8<EPI, bf16, WTA, 0>;
  if constexpr (EPI == EPI_STORE || EPI == EPI_GELU) {
    nt = (size_t)M * (size_t)e.ldo * sizeof(bf16) >= epi::kNTBytes;
    if (nt) kern = k_linear_dma8<EPI, bf16, WTA, epi::kStoreNT>;
  }
  static bool attr_set[2] = {false, false};
  if (!attr_set[nt]) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set[nt] = true;
  }
  const int NT = (N + 255) / 256;
  hipLaunchKernelGGL(kern, dim3(mb * NT), dim3(512), lds, s, M, N, K, (const bf16 *)A, (const bf16 *)Wt, e, mb, NT,
                     tall, group_rows(mb, NT, K));
  return hipGetLastError();
}

// The deep-ring 8-wave kernel: (32 WTA) x (64 WT) tiles, NST LDS stages.
template <int EPI, int WTA, int WT, int NST>
static hipError_t launch_deep(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e, hipStream_t s) {
  const size_t lds = (size_t)NST * (32 * WTA + 64 * WT) * mf::BK * sizeof(bf16);
  auto kern = k_linear_deep<EPI, bf16, WTA, WT, NST>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int MT = (M + 32 * WTA - 1) / (32 * WTA), NT = (N + 64 * WT - 1) / (64 * WT);
  hipLaunchKernelGGL(kern, dim3(MT * NT), dim3(512), lds, s, M, N, K, (const bf16 *)A, (const bf16 *)Wt, e, MT, NT,
                     group_rows(MT, NT, K));
  return hipGetLastError();
}

static int cu_count() {
  static int n = 0;
  if (!n) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

// The rows [m, M) of a problem: operand and output pointers moved down by m rows.
template <int EPI>
static EpiArgs rows_from(const EpiArgs &e, int m) {
  EpiArgs r = e;
  const size_t osz = (EPI == EPI_STORE || EPI == EPI_GELU) ? sizeof(bf16) : sizeof(float);
  r.out = (char *)e.out + (size_t)m * e.ldo * osz;
  if (r.cache) r.cache = e.cache + (size_t)m * e.ldo;
  if (r.res_in) r.res_in = e.res_in + (size_t)m * e.ldo;
  return r;
}

// 256x256 tiles: the 8-wave kernel with LDS-writing loads when it takes the shape, else the generic
// 8-wave kernel with register-staged loads (K % 64 != 0, K < 128 or N % 8 != 0, and the latent
// scatter).
template <int EPI>
static hipError_t launch_big(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e, hipStream_t s) {
  if constexpr (EPI != EPI_EULER) {
    if (K % mf::BK == 0 && K >= 2 * mf::BK && N % 8 == 0) {
      const int mb = (M + 255) / 256;
      return launch_dma8<EPI, 8>(M, N, K, A, Wt, e, s, mb, mb);
    }
  }
  return launch_mfma<8, 4, 2, 4, EPI, 1>(M, N, K, A, Wt, e, s);
}

template <int EPI>
static hipError_t launch_epi(ActType t, int M, int N, int K, const void *A, const void *Wt,
                             const EpiArgs &e, hipStream_t s) {
  if (t == ACT_BF16) {
    const bool dma_ok = EPI != EPI_EULER && K % mf::BK == 0 && K >= 2 * mf::BK && N % 8 == 0;
    TileChoice c = pick_tiles(M, N, K, dma_ok);
    if (c.plan == PLAN_SPLIT && EPI == EPI_EULER) c = {PLAN_BIG, 8, 0, 0, 0};   // the latent scatter needs whole rows
    if (c.plan == PLAN_SMALL) return launch_mfma<4, 4, 2, 2, EPI, 2>(M, N, K, A, Wt, e, s);
    if (c.plan == PLAN_BIG) return launch_big<EPI>(M, N, K, A, Wt, e, s);
    if constexpr (EPI != EPI_EULER) {
      if (c.plan == PLAN_DEEP) {
        const int key = 100 * c.wta + 10 * c.wt + c.nst;
        switch (key) {
          case 422: return launch_deep<EPI, 4, 2, 2>(M, N, K, A, Wt, e, s);
          case 423: return launch_deep<EPI, 4, 2, 3>(M, N, K, A, Wt, e, s);
          case 522: return launch_deep<EPI, 5, 2, 2>(M, N, K, A, Wt, e, s);
          case 523: return launch_deep<EPI, 5, 2, 3>(M, N, K, A, Wt, e, s);
          case 442: return launch_deep<EPI, 4, 4, 2>(M, N, K, A, Wt, e, s);
          case 443: return launch_deep<EPI, 4, 4, 3>(M, N, K, A, Wt, e, s);
          case 542: return launch_deep<EPI, 5, 4, 2>(M, N, K, A, Wt, e, s);
          case 543: return launch_deep<EPI, 5, 4, 3>(M, N, K, A, Wt, e, s);
          default: return hipErrorInvalidValue;
        }
      }
      if (c.plan == PLAN_MIX && c.waves == 8) {
        if (c.wta == 8) return launch_dma8<EPI, 8>(M, N, K, A, Wt, e, s, c.mb, c.tall);
        if (c.wta == 7) return launch_dma8<EPI, 7>(M, N, K, A, Wt, e, s, c.mb, c.tall);
        return launch_dma8<EPI, 6>(M, N, K, A, Wt, e, s, c.mb, c.tall);
      }
      if (c.plan == PLAN_MIX) {
        if (c.wta == 8) return launch_dma<EPI, 8>(M, N, K, A, Wt, e, s, c.mb, c.tall);
        if (c.wta == 7) return launch_dma<EPI, 7>(M, N, K, A, Wt, e, s, c.mb, c.tall);
        return launch_dma<EPI, 6>(M, N, K, A, Wt, e, s, c.mb, c.tall);
      }
    }
    hipError_t err = launch_big<EPI>(c.rows, N, K, A, Wt, e, s);
    if (err != hipSuccess) return err;
    return launch_mfma<4, 4, 2, 2, EPI, 2>(M - c.rows, N, K, (const bf16 *)A + (size_t)c.rows * K, Wt,
                                           rows_from<EPI>(e, c.rows), s);
  }
  dim3 grid((M + 63) / 64, (N + 63) / 64);
  hipLaunchKernelGGL((k_linear_valu<float, EPI, float>), grid, dim3(256), 0, s, M, N, K,
                     (const float *)A, (const float *)Wt, e);
  return hipGetLastError();
}

int describe_linear(ActType t, int epi, int M, int N, int K, char *buf, int len) {
  std::string d;
  int kernels = 1;
  auto rows_of = [](int w) { return std::to_string(32 * w); };
  if (t != ACT_BF16) {
    d = "k_linear_valu: 64x64 tiles, fp32 vector ALUs";
  } else {
    const bool dma_ok = epi != EPI_EULER && K % mf::BK == 0 && K >= 2 * mf::BK && N % 8 == 0;
    TileChoice c = pick_tiles(M, N, K, dma_ok);
    if (c.plan == PLAN_SPLIT && epi == EPI_EULER) c = {PLAN_BIG, 8, 0, 0, 0};
    const std::string nt = std::to_string((N + 255) / 256);
    if (c.plan == PLAN_DEEP) {
      d = "k_linear_deep (8 waves): " + rows_of(c.wta) + "x" + std::to_string(64 * c.wt) + " tiles, " +
          std::to_string(c.nst) + " LDS stages";
    } else if (c.plan == PLAN_SMALL) {
      d = "k_linear_mfma: 128x128 tiles, 4 waves, two workgroups per CU";
    } else if (c.plan == PLAN_BIG) {
      d = dma_ok ? "k_linear_dma8 (8 waves): 256x256 tiles, " + std::to_string((M + 255) / 256) + " row blocks x " + nt
                 : std::string("k_linear_mfma: 256x256 tiles, 8 waves");
    } else if (c.plan == PLAN_MIX) {
      const std::string blocks = std::to_string(c.mb) + " row blocks x " + nt;
      const std::string kn = c.waves == 8 ? "k_linear_dma8 (8 waves): " : "k_linear_dma: ";
      if (c.tall == c.mb) d = kn + rows_of(c.wta) + "x256 tiles, " + blocks;
      else if (c.tall == 0) d = kn + rows_of(c.wta - 1) + "x256 tiles, " + blocks;
      else
        d = kn + blocks + ", " + std::to_string(c.tall) + " of " + rows_of(c.wta) + " rows and " +
            std::to_string(c.mb - c.tall) + " of " + rows_of(c.wta - 1);
    } else {
      kernels = 2;
      d = std::string(dma_ok ? "k_linear_dma8" : "k_linear_mfma") + ": 256x256 tiles on rows 0.." + std::to_string(c.rows - 1) +
          " + k_linear_mfma: 128x128 tiles on the remaining " + std::to_string(M - c.rows) + " rows";
    }
  }
  if (buf && len > 0) {
    const size_t n = std::min((size_t)len - 1, d.size());
    memcpy(buf, d.data(), n);
    buf[n] = 0;
  }
  return kernels;
}

// The split-K plan of a shape: the tile (32 wta) x (64 wt) with nst LDS stages, cut into `splits` K
// ranges (1 = none).  Only bf16 shapes the 8-wave kernel takes, whose 224 x 256 tiles fill less than half
// the CUs, with at least 16 K tiles per split and the partial sums within kSplitBytes.  Among the
// deep-ring tiles (three LDS stages) and split counts, the plan with the most workgroups within one
// round of the CUs (on a tie, the first tile in kDeepTiles order and the fewest splits).  Measured for one
// candidate's MLP down-projection (M = 1560, N = 1536, K = 8960, residual epilogue; reduction included):
// 160 x 128 x 2 ranges (240 workgroups) 53 us, against 62 us for 224 x 256 x 5 ranges on two stages,
// 56 us for 128 x 256 x 3, 60 us for 160 x 256 x 4 and 63 us unsplit (128 x 128, 156 workgroups).  A
// function of the shape alone, so every caller with a workspace gets the same plan (and the same bits).
// FLASHBON_SPLITK (tuning): "<rows>:<cols>:<stages>:<splits>" forces a plan on the shapes that split.
struct SplitPlan {
  int splits, wta, wt, nst;
};
static SplitPlan splitk_plan(int epi, int M, int N, int K) {
  SplitPlan none = {1, 7, 4, 2};
  if (epi == EPI_EULER || K % mf::BK || N % 8 || K < 2 * mf::BK) return none;
  const int64_t tiles = (int64_t)((M + 223) / 224) * ((N + 255) / 256);
  const int cus = cu_count();
  if (2 * tiles > cus) return none;
  const int kt = K / mf::BK;
  // the launch gives each split ceil(kt / sp) K tiles: a count is usable when every split is non-empty
  // and the last has at least the two K tiles the tile loop needs
  auto usable = [&](int sp) {
    const int ks = (kt + sp - 1) / sp;
    return sp >= 2 && (kt + ks - 1) / ks == sp && kt - (sp - 1) * ks >= 2 &&
           (size_t)sp * M * N * 4 <= kSplitBytes;
  };
  const char *force = getenv("FLASHBON_SPLITK");
  if (force) {
    int rows = 0, cols = 0, nst = 0, sp = 0;
    if (sscanf(force, "%d:%d:%d:%d", &rows, &cols, &nst, &sp) == 4 && usable(sp) &&
        ((rows == 224 && cols == 256 && nst == 2) || (deep_ok(rows / 32, cols / 64, nst) && rows % 32 == 0 &&
                                                       cols % 64 == 0)))
      return {sp, rows / 32, cols / 64, nst};
  }
  SplitPlan best = none;
  int64_t most = 0;
  for (const auto &d : kDeepTiles) {
    const int64_t t = (int64_t)((M + 32 * d[0] - 1) / (32 * d[0])) * ((N + 64 * d[1] - 1) / (64 * d[1]));
    for (int sp = 2; sp <= K / (16 * mf::BK) && t * sp <= cus; ++sp)
      if (usable(sp) && t * sp > most) {
        most = t * sp;
        best = {sp, d[0], d[1], 3};
      }
  }
  return best;
}

int splitk_splits(int epi, int M, int N, int K) { return splitk_plan(epi, M, N, K).splits; }

template <int WTA, int WT, int NST>
static hipError_t launch_splitk(int M, int N, int K, const void *A, const void *Wt, float *part, int sp,
                                hipStream_t s) {
  const int ks = (K / mf::BK + sp - 1) / sp * mf::BK;
  const size_t lds = (size_t)NST * (32 * WTA + 64 * WT) * mf::BK * sizeof(bf16);
  auto kern = k_linear_splitk<WTA, WT, NST>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int MT = (M + 32 * WTA - 1) / (32 * WTA), NT = (N + 64 * WT - 1) / (64 * WT);
  hipLaunchKernelGGL(kern, dim3(MT * NT * sp), dim3(512), lds, s, M, N, K, (const bf16 *)A, (const bf16 *)Wt, part,
                     MT, NT, ks, group_rows(MT, NT, K));
  return hipGetLastError();
}

hipError_t launch_linear_ws(ActType t, int epi, int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e,
                            hipStream_t s, void *ws, size_t ws_bytes) {
  const SplitPlan pl = t == ACT_BF16 && ws ? splitk_plan(epi, M, N, K) : SplitPlan{1, 7, 4, 2};
  const int sp = pl.splits;
  if (sp < 2 || (size_t)sp * M * N * 4 > ws_bytes) return launch_linear(t, epi, M, N, K, A, Wt, e, s);
  float *part = (float *)ws;
  hipError_t err;
  switch (100 * pl.wta + 10 * pl.wt + pl.nst) {
    case 742: err = launch_splitk<7, 4, 2>(M, N, K, A, Wt, part, sp, s); break;
    case 422: err = launch_splitk<4, 2, 2>(M, N, K, A, Wt, part, sp, s); break;
    case 423: err = launch_splitk<4, 2, 3>(M, N, K, A, Wt, part, sp, s); break;
    case 522: err = launch_splitk<5, 2, 2>(M, N, K, A, Wt, part, sp, s); break;
    case 523: err = launch_splitk<5, 2, 3>(M, N, K, A, Wt, part, sp, s); break;
    case 442: err = launch_splitk<4, 4, 2>(M, N, K, A, Wt, part, sp, s); break;
    case 443: err = launch_splitk<4, 4, 3>(M, N, K, A, Wt, part, sp, s); break;
    case 542: err = launch_splitk<5, 4, 2>(M, N, K, A, Wt, part, sp, s); break;
    case 543: err = launch_splitk<5, 4, 3>(M, N, K, A, Wt, part, sp, s); break;
    default: return hipErrorInvalidValue;
  }
  if (err != hipSuccess) return err;
  const int64_t threads = (int64_t)M * (N / 8);
  const dim3 grid((unsigned)((threads + 255) / 256));
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL(k_splitk_reduce<EPI_STORE>, grid, dim3(256), 0, s, M, N, sp, part, e); break;
    case EPI_GELU: hipLaunchKernelGGL(k_splitk_reduce<EPI_GELU>, grid, dim3(256), 0, s, M, N, sp, part, e); break;
    case EPI_STORE_F32: hipLaunchKernelGGL(k_splitk_reduce<EPI_STORE_F32>, grid, dim3(256), 0, s, M, N, sp, part, e); break;
    case EPI_RESIDUAL: hipLaunchKernelGGL(k_splitk_reduce<EPI_RESIDUAL>, grid, dim3(256), 0, s, M, N, sp, part, e); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_linear(ActType t, int epi, int M, int N, int K, const void *A, const void *Wt,
                         const EpiArgs &e, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch_epi<EPI_STORE>(t, M, N, K, A, Wt, e, s);
    case EPI_GELU: return launch_epi<EPI_GELU>(t, M, N, K, A, Wt, e, s);
    case EPI_STORE_F32: return launch_epi<EPI_STORE_F32>(t, M, N, K, A, Wt, e, s);
    case EPI_RESIDUAL: return launch_epi<EPI_RESIDUAL>(t, M, N, K, A, Wt, e, s);
    case EPI_EULER: return launch_epi<EPI_EULER>(t, M, N, K, A, Wt, e, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fb
