// Linear layers of the DiT step: C[m][n] = sum_k A[m][k] Wt[n][k] with fused epilogues.
//   * k_linear_ilv / k_linear_mfma: bf16 operands on gfx950 matrix cores (v_mfma_f32_16x16x32_bf16),
//     fp32 accumulation.  Workgroup tiles of 256x256 (8 waves of 128x64; explicitly interleaved
//     schedule when K % 64 == 0) or 128x128 (4 waves of 64x64, loads two K tiles ahead), chosen per
//     shape; K tiles of 64 staged through double-buffered, XOR-swizzled LDS (one barrier per K
//     tile); XCD-aware grouped tile order.  Operands are swapped (the weight tile feeds the MFMA "A" side) so that every lane ends
//     up owning four consecutive output columns of one row, which the epilogues store as one vector.
//   * k_linear_valu: fp32 (or bf16) operands on the vector ALUs, 64x64 tiles; used by the fp32 mode
//     and for shapes the MFMA tiling does not take.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>

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
      float4 h0 = reinterpret_cast<float4 *>(o)[0], h1 = reinterpret_cast<float4 *>(o)[1];
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
// is given a contiguous range of tiles, and tiles are ordered in groups of GROUP_M m-tiles sweeping
// all n-tiles, so the workgroups resident on one XCD share A rows and W rows in that XCD's L2.
constexpr int GROUP_M = 8;
__device__ __forceinline__ void tile_of(int bid, int MT, int NT, int &mt, int &nt) {
  const int total = MT * NT;
  const int xcd = bid & 7, local = bid >> 3;
  const int base = total >> 3, rem = total & 7;
  const int t = xcd * base + min(xcd, rem) + local;
  const int per_group = GROUP_M * NT;
  const int group = t / per_group, first_m = group * GROUP_M;
  const int gm = min(MT - first_m, GROUP_M);
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
#pragma unroll
    for (int pa = 0; pa < WTN / 2; ++pa) {
      const int n = en0 + 16 * WTN * wn + 32 * pa + 8 * fq;
#pragma unroll
      for (int j = 0; j < WTM; ++j) {
        const int m = em0 + 16 * WTM * wm + 16 * j + fr;
        const float v[8] = {acc[2 * pa][j][0], acc[2 * pa][j][1], acc[2 * pa][j][2], acc[2 * pa][j][3],
                            acc[2 * pa + 1][j][0], acc[2 * pa + 1][j][1], acc[2 * pa + 1][j][2],
                            acc[2 * pa + 1][j][3]};
        if (m < M && n < N) {
          if (n + 8 <= N) epilogue8<EPI, TO>(e, m, n, v);
          else epilogue4<EPI, TO>(e, m, n, v[0], v[1], v[2], v[3]);   // N % 8 == 4 edge
        }
      }
    }
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

// ------------------------------------------------------- MFMA path, explicitly interleaved 256x256
// 8 waves of 128 (m) x 64 (n), K tiles of 64 (K % 64 == 0), register-staged double-buffered LDS.
// The instruction order inside a K tile is pinned: the next tile's global loads first; substep-1 W
// fragments; substep 0's MFMAs with substep-1 A fragments read in place between MFMA groups (so
// each fragment register is refilled right after its last use); half of substep 1; the staged
// stores and the barrier; the next tile's substep-0 fragments, again refilled in place, overlapping
// the second half of substep 1.  LDS latency is then hidden behind MFMA groups instead of exposed
// at each substep, and the barrier drain overlaps 16 MFMAs.
template <int EPI, typename TO>
__global__ __launch_bounds__(512, 1) void k_linear_ilv(int M, int N, int K, const bf16 *__restrict__ A,
                                                const bf16 *__restrict__ Wt, EpiArgs e, int MT, int NT) {
  using namespace mf;
  constexpr int BM = 256, BN = 256, WTM = 8, WTN = 4, ROWS = 64, LA = 4, LW = 4;
  constexpr int STAGE = (BM + BN) * BK;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  int mt, nt;
  tile_of(blockIdx.x, MT, NT, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int ld_r = tid >> 3, ld_c = tid & 7;
  // Buffer loads over the workgroup's rows: rows past M (N) fall outside the buffer's range and read
  // as zero.  The range check covers the VGPR offset only (not the scalar one), so each row's offset
  // is a VGPR and only the K position (inside every row) rides in the scalar offset.
  const __amdgpu_buffer_rsrc_t rsA = tile_rsrc(A + (int64_t)m0 * K, min(M - m0, BM), K);
  const __amdgpu_buffer_rsrc_t rsW = tile_rsrc(Wt + (int64_t)n0 * K, min(N - n0, BN), K);
  static_assert(LA == LW, "A and W share the row offsets");
  int voff[LA];
#pragma unroll
  for (int i = 0; i < LA; ++i) voff[i] = ((ld_r + ROWS * i) * K + ld_c * 8) * 2;
  u32x4 ra[LA], rw[LW];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < LA; ++i) ra[i] = __builtin_amdgcn_raw_buffer_load_b128(rsA, voff[i], k0 * 2, 0);
#pragma unroll
    for (int i = 0; i < LW; ++i) rw[i] = __builtin_amdgcn_raw_buffer_load_b128(rsW, voff[i], k0 * 2, 0);
  };
  auto lstore = [&](bf16 *sA) {
    bf16 *sW = sA + BM * BK;
#pragma unroll
    for (int i = 0; i < LA; ++i) *reinterpret_cast<u32x4 *>(&sA[lds_off(ld_r + ROWS * i, ld_c)]) = ra[i];
#pragma unroll
    for (int i = 0; i < LW; ++i) *reinterpret_cast<u32x4 *>(&sW[lds_off(ld_r + ROWS * i, ld_c)]) = rw[i];
  };
  f32x4 acc[WTN][WTM];
#pragma unroll
  for (int i = 0; i < WTN; ++i)
#pragma unroll
    for (int j = 0; j < WTM; ++j) acc[i][j] = f32x4{0, 0, 0, 0};
  const int fr = lane & 15, fq = lane >> 4;
  // MFMA tile i of this wave takes W rows 32 (i/2) + 8 (fr/4) + 4 (i%2) + fr%4 (fr = lane & 15), so
  // the C^T rows a lane ends up with for tiles 2a and 2a+1 are 8 consecutive output columns
  const int rowA = 16 * WTM * wm + fr;
  auto w_row = [&](int i) { return 16 * WTN * wn + 32 * (i >> 1) + 8 * (fr >> 2) + 4 * (i & 1) + (fr & 3); };
  bf16x8 fw0[WTN], fw1[WTN], fa[WTM];
  auto rd_w = [&](const bf16 *st, int ks, bf16x8 *fw) {
    const bf16 *sW = st + BM * BK;
#pragma unroll
    for (int i = 0; i < WTN; ++i) fw[i] = *reinterpret_cast<const bf16x8 *>(&sW[lds_off(w_row(i), fq + 4 * ks)]);
  };
  auto rd_a = [&](const bf16 *st, int ks, int j) {
    fa[j] = *reinterpret_cast<const bf16x8 *>(&st[lds_off(rowA + 16 * j, fq + 4 * ks)]);
  };
  auto mm = [&](const bf16x8 *fw, int j) {
#pragma unroll
    for (int i = 0; i < WTN; ++i) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
  };
  const int KT = K / BK;
  gload(0);
  lstore(smem);
  __syncthreads();
  rd_w(smem, 0, fw0);
#pragma unroll
  for (int j = 0; j < WTM; ++j) rd_a(smem, 0, j);
  for (int kt = 0; kt < KT; ++kt) {
    const bool more = kt + 1 < KT;
    const bf16 *cur = smem + (kt & 1) * STAGE;
    bf16 *nxt = smem + ((kt + 1) & 1) * STAGE;
    if (more) gload((kt + 1) * BK);
    rd_w(cur, 1, fw1);
    __builtin_amdgcn_sched_barrier(0);
    // substep 0; substep-1 A fragments replace substep-0 ones in place
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
      mm(fw0, j);
      rd_a(cur, 1, j);
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // substep 1, first half
#pragma unroll
    for (int j = 0; j < WTM / 2; ++j) mm(fw1, j);
    __builtin_amdgcn_sched_barrier(0);
    if (more) lstore(nxt);
    __syncthreads();
    if (more) {
      rd_w(nxt, 0, fw0);
#pragma unroll
      for (int j = 0; j < WTM / 2; ++j) rd_a(nxt, 0, j);
    }
    __builtin_amdgcn_sched_barrier(0);
    // substep 1, second half; next tile's A fragments replace these in place
#pragma unroll
    for (int j = WTM / 2; j < WTM; ++j) {
      mm(fw1, j);
      if (more) rd_a(nxt, 0, j);
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int pa = 0; pa < WTN / 2; ++pa) {
    const int n = n0 + 16 * WTN * wn + 32 * pa + 8 * fq;
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
      const int m = m0 + 16 * WTM * wm + 16 * j + fr;
      const float v[8] = {acc[2 * pa][j][0], acc[2 * pa][j][1], acc[2 * pa][j][2], acc[2 * pa][j][3],
                          acc[2 * pa + 1][j][0], acc[2 * pa + 1][j][1], acc[2 * pa + 1][j][2],
                          acc[2 * pa + 1][j][3]};
      if (m < M && n < N) {
        if (n + 8 <= N) epilogue8<EPI, TO>(e, m, n, v);
        else epilogue4<EPI, TO>(e, m, n, v[0], v[1], v[2], v[3]);   // N % 8 == 4 edge
      }
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

// Tile choice for bf16 operands.  The 256x256 kernel runs one workgroup per CU, the 128x128 kernel
// two; a launch takes ceil(tiles / slots) rounds.  Measured on MI355X, a round of 128x128 tiles
// costs 0.64 of a round of 256x256 tiles at the same K (so the small tile does 0.78 of the big
// tile's work per CU).  Candidates: all 256x256; all 128x128; or the whole rows of 256x256 tiles
// that fill complete rounds plus the remaining rows as 128x128 tiles (a second launch), which
// trims a last round that would leave most CUs idle.
enum TilePlan { PLAN_BIG, PLAN_SMALL, PLAN_SPLIT };
static int cu_count();

static TilePlan pick_tiles(int M, int N, int K, int *split_rows) {
  const char *force = getenv("FLASHBON_LINEAR_TILE");  // "256x256" or "128x128": tests and tuning
  if (force) return strcmp(force, "128x128") ? PLAN_BIG : PLAN_SMALL;
  constexpr double kSmallRound = 0.64;
  const int cus = cu_count();
  const int64_t NT = (N + 255) / 256, T = (int64_t)((M + 255) / 256) * NT, NT2 = (N + 127) / 128;
  const double t_big = (double)((T + cus - 1) / cus);
  const double t_small = (double)((((M + 127) / 128) * NT2 + 2 * cus - 1) / (2 * cus)) * kSmallRound;
  double t_split = 1e30;
  const int64_t mt_big = (T - T % cus) / NT;
  const int rows = (int)(mt_big * 256);
  if (K % mf::BK == 0 && rows > 0 && rows < M) {
    const int64_t T2 = ((M - rows + 127) / 128) * NT2;
    t_split = (double)((mt_big * NT + cus - 1) / cus) + (double)((T2 + 2 * cus - 1) / (2 * cus)) * kSmallRound;
  }
  *split_rows = rows;
  if (t_split < t_big && t_split < t_small) return PLAN_SPLIT;
  return t_big <= t_small ? PLAN_BIG : PLAN_SMALL;
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

template <int EPI>
static hipError_t launch_ilv(int M, int N, int K, const void *A, const void *Wt, const EpiArgs &e,
                             hipStream_t s) {
  const size_t lds = (size_t)2 * (256 + 256) * mf::BK * sizeof(bf16);
  auto kern = k_linear_ilv<EPI, bf16>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int MT = (M + 255) / 256, NT = (N + 255) / 256;
  hipLaunchKernelGGL(kern, dim3(MT * NT), dim3(512), lds, s, M, N, K, (const bf16 *)A, (const bf16 *)Wt, e,
                     MT, NT);
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
  return r;
}

template <int EPI>
static hipError_t launch_epi(ActType t, int M, int N, int K, const void *A, const void *Wt,
                             const EpiArgs &e, hipStream_t s) {
  if (t == ACT_BF16) {
    int rows = 0;
    TilePlan plan = pick_tiles(M, N, K, &rows);
    if (plan == PLAN_SPLIT && EPI == EPI_EULER) plan = PLAN_BIG;   // the latent scatter needs whole rows
    if (plan == PLAN_SMALL) return launch_mfma<4, 4, 2, 2, EPI, 2>(M, N, K, A, Wt, e, s);
    if (K % mf::BK) return launch_mfma<8, 4, 2, 4, EPI, 1>(M, N, K, A, Wt, e, s);
    if (plan == PLAN_BIG) return launch_ilv<EPI>(M, N, K, A, Wt, e, s);
    hipError_t err = launch_ilv<EPI>(rows, N, K, A, Wt, e, s);
    if (err != hipSuccess) return err;
    return launch_mfma<4, 4, 2, 2, EPI, 2>(M - rows, N, K, (const bf16 *)A + (size_t)rows * K, Wt,
                                           rows_from<EPI>(e, rows), s);
  }
  dim3 grid((M + 63) / 64, (N + 63) / 64);
  hipLaunchKernelGGL((k_linear_valu<float, EPI, float>), grid, dim3(256), 0, s, M, N, K,
                     (const float *)A, (const float *)Wt, e);
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
