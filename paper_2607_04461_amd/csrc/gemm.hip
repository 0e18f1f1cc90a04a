// Linear layers of the DiT step: C[m][n] = sum_k A[m][k] Wt[n][k] with fused epilogues.
//   * k_linear_mfma: bf16 operands on gfx950 matrix cores (v_mfma_f32_16x16x32_bf16), fp32
//     accumulation, LDS-staged 128x128x64 tiles with an XOR swizzle, register prefetch of the next
//     K tile.  Operands are swapped (the weight tile feeds the MFMA "A" side) so that every lane
//     ends up owning four consecutive output columns of one row, which the epilogues store as one
//     vector.
//   * k_linear_valu: fp32 (or bf16) operands on the vector ALUs, 64x64 tiles; used by the fp32 mode
//     and for shapes the MFMA tiling does not take.
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
    float4 h = *reinterpret_cast<float4 *>(o);
    if (e.gate) {
      float4 g = *reinterpret_cast<const float4 *>(e.gate + n);
      h.x += g.x * v[0]; h.y += g.y * v[1]; h.z += g.z * v[2]; h.w += g.w * v[3];
    } else {
      h.x += v[0]; h.y += v[1]; h.z += v[2]; h.w += v[3];
    }
    *reinterpret_cast<float4 *>(o) = h;
    if (e.cache) *reinterpret_cast<float4 *>(e.cache + (int64_t)m * e.ldo + n) = h;
  } else if constexpr (EPI == EPI_EULER) {
    // m = candidate * T + token, token = i * (W/p) + j; n = c p^2 + p di + dj
    const int b = m / e.T, t = m % e.T, wp = e.W / e.p;
    const int i = t / wp, j = t % wp, pp = e.p * e.p;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int nn = n + q;
      int c = nn / pp, r = nn % pp, di = r / e.p, dj = r % e.p;
      float *zp = e.z + (((int64_t)b * e.C + c) * e.H + (e.p * i + di)) * e.W + (e.p * j + dj);
      *zp = *zp + e.dt * v[q];
    }
  }
}

// ---------------------------------------------------------------------------------- MFMA path
namespace mf {
constexpr int BM = 128;  // activation rows per workgroup
constexpr int BN = 128;  // weight rows (output columns) per workgroup
constexpr int BK = 64;
constexpr int THREADS = 256;
// LDS tile: [rows][64] bf16 = 8 chunks of 16 B per row, chunk c of row r stored at c ^ swz(r).
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int lds_off(int r, int c) { return r * 64 + ((c ^ swz(r)) << 3); }
}  // namespace mf

template <int EPI, typename TO>
__global__ __launch_bounds__(256) void k_linear_mfma(int M, int N, int K,
                                                     const bf16 *__restrict__ A,
                                                     const bf16 *__restrict__ Wt, EpiArgs e) {
  using namespace mf;
  __shared__ __attribute__((aligned(16))) bf16 sA[BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sW[BN * BK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // wave tile: rows 64*wm.., cols 64*wn..
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;

  // global -> register staging: each thread moves 4 chunks of A and 4 of W per K tile
  const int ld_r = tid >> 3, ld_c = tid & 7;  // row 0..31 (+32 i), chunk 0..7
  const bf16 *pa[4];
  const bf16 *pw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int ra = min(m0 + ld_r + 32 * i, M - 1);
    int rw = min(n0 + ld_r + 32 * i, N - 1);
    pa[i] = A + (int64_t)ra * K + ld_c * 8;
    pw[i] = Wt + (int64_t)rw * K + ld_c * 8;
  }
  u32x4 ra[4], rw[4];
  auto load_tile = [&](int k0) {
    const bool ok = (k0 + ld_c * 8) < K;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = ok ? *reinterpret_cast<const u32x4 *>(pa[i] + k0) : u32x4{0, 0, 0, 0};
      rw[i] = ok ? *reinterpret_cast<const u32x4 *>(pw[i] + k0) : u32x4{0, 0, 0, 0};
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = ld_r + 32 * i;
      *reinterpret_cast<u32x4 *>(&sA[lds_off(r, ld_c)]) = ra[i];
      *reinterpret_cast<u32x4 *>(&sW[lds_off(r, ld_c)]) = rw[i];
    }
  };

  f32x4 acc[4][4];  // [n tile i][m tile j]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0, 0, 0, 0};

  const int fr = lane & 15, fq = lane >> 4;  // fragment row within 16, k-chunk quarter
  const int ktiles = (K + BK - 1) / BK;
  load_tile(0);
  for (int kt = 0; kt < ktiles; ++kt) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kt + 1 < ktiles) load_tile((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 fw[4], fa[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int r = 64 * wn + 16 * i + fr;
        fw[i] = *reinterpret_cast<const bf16x8 *>(&sW[lds_off(r, fq + 4 * ks)]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int r = 64 * wm + 16 * j + fr;
        fa[j] = *reinterpret_cast<const bf16x8 *>(&sA[lds_off(r, fq + 4 * ks)]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
    }
  }

  // acc[i][j] lane layout (C^T tile 16x16): column = m index (lane & 15), rows = 4 consecutive n.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + 64 * wn + 16 * i + 4 * fq;
    if (n >= N) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + 64 * wm + 16 * j + fr;
      if (m < M) epilogue4<EPI, TO>(e, m, n, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
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

template <int EPI>
static hipError_t launch_epi(ActType t, int M, int N, int K, const void *A, const void *Wt,
                             const EpiArgs &e, hipStream_t s) {
  if (t == ACT_BF16) {
    dim3 grid((M + mf::BM - 1) / mf::BM, (N + mf::BN - 1) / mf::BN);
    hipLaunchKernelGGL((k_linear_mfma<EPI, bf16>), grid, dim3(mf::THREADS), 0, s, M, N, K,
                       (const bf16 *)A, (const bf16 *)Wt, e);
  } else {
    dim3 grid((M + 63) / 64, (N + 63) / 64);
    hipLaunchKernelGGL((k_linear_valu<float, EPI, float>), grid, dim3(256), 0, s, M, N, K,
                       (const float *)A, (const float *)Wt, e);
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
