// Softmax attention of the DiT block: self-attention over image tokens and cross-attention to the
// candidate's prompt tokens, softmax(q k^T / sqrt(dh)) v per (candidate, head).
//   * k_attn_valu: one lane per query, online softmax over 16-key sub-tiles staged in LDS as fp32;
//     any head_dim <= 128 (multiple of 8); fp32 or bf16 operands.  Used by the fp32 mode and for
//     head dims the MFMA kernel does not take.
//   * k_attn_mfma: bf16, head_dim 128, gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).  Each wave owns
//     32 queries.  Scores are formed transposed, S^T = K Q^T, so every lane holds 16 scores of one
//     query (its partner lane l^32 holds the other 16 of a 32-key slab): the online-softmax max is a
//     single cross-lane exchange and the running sum stays per lane until the end.  The output is
//     accumulated transposed as well, O^T += V^T P^T: the probabilities feed the second MFMA straight
//     from the first one's accumulator registers (the key order inside each 16-key chunk is permuted
//     identically on both operands), and every lane rescales only its own query.  K and V tiles are
//     staged in LDS row-major with 16-byte stores and XOR swizzles; V^T fragments come from gfx950's
//     LDS transpose read (ds_read_b64_tr_b16): in each group of 16 lanes, lane j addresses 4
//     consecutive head dims of one key and lane 4a + b receives element b of the pieces addressed by
//     lanes a, a + 4, a + 8, a + 12 -- i.e. one head dim across four keys.
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace fb {

struct AttnP {
  int batch, heads, tq, tk;
  int nqb;       // query blocks per (candidate, head) (k_attn_fa's 1-D grid)
  const void *q; int64_t q_bs, q_rs;
  const void *k; const void *v; int64_t kv_bs, kv_rs;
  const int32_t *kv_index; int n_kv;
  void *out; int64_t o_bs, o_rs;
  float qscale;  // log2(e) / sqrt(head_dim)
  float lazy_thr;  // k_attn_fa: how far a tile maximum may pass the running one before O is rescaled
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

namespace fa {
constexpr int DH = 128;
constexpr int KT = 64;          // keys per LDS tile
constexpr int QW = 32;          // queries per wave
constexpr int WAVES = 4;
constexpr int QB = QW * WAVES;  // queries per workgroup
__device__ __forceinline__ int k_off(int r, int c) { return r * DH + ((c ^ (r & 15)) << 3); }
// V rows: 16-byte chunk c of key r at c ^ 4 (r mod 4).  A transpose read serves 32 lanes a cycle:
// four keys r..r+3 (r a multiple of 4) times chunks 4 dt .. 4 dt + 3, whose positions then differ in
// bits 2-3 per key, so the 32 eight-byte pieces fill the 256-byte bank window once.
__device__ __forceinline__ int v_off(int r, int c) { return r * DH + ((c ^ ((r & 3) << 2)) << 3); }
}  // namespace fa

__global__ __launch_bounds__(256, 2) void k_attn_mfma(AttnP p) {
  using namespace fa;
  __shared__ __attribute__((aligned(16))) bf16 sKV[2][2][KT * DH];  // [stage][K, V]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 5, li = lane & 31;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q0 = blockIdx.x * QB + w * QW;
  const int kb = kv_batch(p, b);
  const bf16 *Q = (const bf16 *)p.q + (int64_t)b * p.q_bs + h * DH;
  const bf16 *K = (const bf16 *)p.k + (int64_t)kb * p.kv_bs + h * DH;
  const bf16 *V = (const bf16 *)p.v + (int64_t)kb * p.kv_bs + h * DH;

  // this lane's query row, as the B operand of S^T = K Q^T: 8 k-steps of 16 head dims
  const int qi = min(q0 + li, p.tq - 1);
  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8 *>(Q + (int64_t)qi * p.q_rs + 16 * ks + 8 * g);

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[dt][j] = 0.f;
  float mrun = -INFINITY, lsum = 0.f;

  // global -> LDS staging: 64 keys x 16 chunks of 8 head dims; 4 chunks per thread for K and for V
  const int lr = tid >> 4, lc = tid & 15;
  u32x4 rk[4], rv[4];
  auto gload = [&](int j0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int key = min(j0 + lr + 16 * i, p.tk - 1);
      rk[i] = *reinterpret_cast<const u32x4 *>(K + (int64_t)key * p.kv_rs + 8 * lc);
      rv[i] = *reinterpret_cast<const u32x4 *>(V + (int64_t)key * p.kv_rs + 8 * lc);
    }
  };
  auto lstore = [&](int stage) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = lr + 16 * i;
      *reinterpret_cast<u32x4 *>(&sKV[stage][0][k_off(r, lc)]) = rk[i];
      *reinterpret_cast<u32x4 *>(&sKV[stage][1][v_off(r, lc)]) = rv[i];
    }
  };

  // two LDS stages: tile t+1 is loaded into registers while tile t is consumed, then stored to the
  // other stage; one barrier per tile
  gload(0);
  lstore(0);
  __syncthreads();
  for (int j0 = 0, it = 0; j0 < p.tk; j0 += KT, ++it) {
    const int st = it & 1;
    const bf16 *sK = sKV[st][0], *sV = sKV[st][1];
    const bool more = j0 + KT < p.tk;
    if (more) gload(j0 + KT);

    // S^T for two 32-key slabs: lane holds query li, keys 32 st + (j/4)*8 + 4 g + (j%4)
    f32x16 sc[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int j = 0; j < 16; ++j) sc[st][j] = 0.f;
      const int r = 32 * st + li;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        bf16x8 kf = *reinterpret_cast<const bf16x8 *>(&sK[k_off(r, 2 * ks + g)]);
        sc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc[st], 0, 0, 0);
      }
    }
    // online softmax in base 2: running max of the raw scores (the scale is positive), exponent
    // argument formed by one FMA; keys past tk are masked only on the ragged last tile; the
    // accumulators are rescaled only when some lane's maximum moved
    if (j0 + KT > p.tk) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          int key = j0 + 32 * st + (j >> 2) * 8 + 4 * g + (j & 3);
          if (key >= p.tk) sc[st][j] = -INFINITY;
        }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int j = 0; j < 16; ++j) tmax = fmaxf(tmax, sc[st][j]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(mrun, tmax);
    if (__any(mnew > mrun)) {
      const float corr = __builtin_amdgcn_exp2f((mrun - mnew) * p.qscale);
      lsum *= corr;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[dt][j] *= corr;
      mrun = mnew;
    }
    const float mb = mrun * p.qscale;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float e = __builtin_amdgcn_exp2f(fmaf(sc[st][j], p.qscale, -mb));
        lsum += e;
        sc[st][j] = e;
      }
    // O^T += V^T P^T over four 16-key chunks; k-slot i of group g <-> key 16c + (i/4)*8 + 4g + i%4.
    // Transpose-read addressing: lane (16-lane group h = bit 4, q = low 4 bits) addresses key
    // 16c + 4g + (q >> 2) (+8 for k-slots 4..7) at head dims 32 dt + 16 h + 4 (q & 3) .. + 3, so lane l
    // receives head dim 32 dt + (l & 31) for those four keys.
    const int tq = lane & 15, th = (lane >> 4) & 1;
    const int tkey = 4 * g + (tq >> 2), tdim = 16 * th + 4 * (tq & 3);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      bf16x8 pf;
#pragma unroll
      for (int i = 0; i < 8; ++i) pf[i] = (bf16)sc[c >> 1][8 * (c & 1) + i];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int d = 32 * dt + tdim, k0 = 16 * c + tkey;
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4 *)&sV[v_off(k0, d >> 3) + (d & 7)]);
        s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4 *)&sV[v_off(k0 + 8, d >> 3) + (d & 7)]);
        bf16x4 w0 = __builtin_bit_cast(bf16x4, v0), w1 = __builtin_bit_cast(bf16x4, v1);
        bf16x8 vf = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[dt], 0, 0, 0);
      }
    }
    if (more) lstore(st ^ 1);
    __syncthreads();
  }
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / ltot;
  if (q0 + li >= p.tq) return;
  bf16 *O = (bf16 *)p.out + (int64_t)b * p.o_bs + (int64_t)(q0 + li) * p.o_rs + h * DH;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      bf16x4 w4 = {(bf16)(o[dt][4 * jq] * inv), (bf16)(o[dt][4 * jq + 1] * inv),
                   (bf16)(o[dt][4 * jq + 2] * inv), (bf16)(o[dt][4 * jq + 3] * inv)};
      *reinterpret_cast<bf16x4 *>(O + 32 * dt + 8 * jq + 4 * g) = w4;
    }
}

// ---------------------------------------------------------------- pipelined MFMA attention (dh 128)
// Same fragment layouts as k_attn_mfma (S^T = K Q^T per 32-key slab, O^T += V^T P^T per 16-key chunk,
// one lane per query), reorganised so that matrix cores and vector ALUs of a wave work at the same
// time: while the VALUs turn the scores of key tile j into probabilities, the MFMAs already form the
// scores of tile j + 1; the V^T P^T products of tile j follow.  K and V tiles reach LDS through
// buffer loads that write LDS themselves (no staging registers): K tiles in a ring of two one tile
// ahead, V tiles in their own ring of two; one barrier per tile.  Keys past tk read as zero (the
// buffer range ends at the last key) and are masked on the ragged last tile.  LDS offsets are
// per-lane bases plus immediates (stage, slab, chunk).
namespace fa2 {
constexpr int DH = 128, KT = 64, QW = 32, WAVES = 4, QB = QW * WAVES;
constexpr int TILE_B = KT * DH * 2;   // bytes of one K or V tile
// LDS: K stage 0, K stage 1, V stage 0, V stage 1
constexpr int K_OFF = 0, V_OFF = 2 * TILE_B;
}  // namespace fa2

__global__ __launch_bounds__(256, 2) void k_attn_fa(AttnP p) {
  using namespace fa2;
  __shared__ __attribute__((aligned(16))) bf16 sm[4 * KT * DH];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, li = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // 1-D grid, XCD-aware: workgroups go to the 8 XCDs round-robin by id, so id -> (unit u = head *
  // batch + candidate, query block) keeps every query block of a unit on XCD u % 8, where its K and V
  // stay in that XCD's L2 (and the text K/V of one head is shared by the candidates on that XCD)
  const int id = blockIdx.x, rest = id >> 3;
  const int u = (rest / p.nqb) * 8 + (id & 7), qblk = rest % p.nqb;
  if (u >= p.batch * p.heads) return;
  const int h = u / p.batch, b = u % p.batch;
  const int q0 = qblk * QB + w * QW;
  // a wave whose 32 queries all lie past tq (the last query block of a unit) still loads its share
  // of every K/V tile and meets every barrier, but forms no scores, probabilities or outputs, leaving
  // its SIMD's issue slots to the co-resident workgroup's wave
  const bool idle = q0 >= p.tq;
  const int kb = kv_batch(p, b);
  const bf16 *Q = (const bf16 *)p.q + (int64_t)b * p.q_bs + h * DH;
  const bf16 *Kb = (const bf16 *)p.k + (int64_t)kb * p.kv_bs + h * DH;
  const bf16 *Vb = (const bf16 *)p.v + (int64_t)kb * p.kv_bs + h * DH;
  const int nt = (p.tk + KT - 1) / KT;
  char *lds = reinterpret_cast<char *>(sm);

  // this lane's query row, as the B operand of S^T = K Q^T: 8 k-steps of 16 head dims
  const int qi = min(q0 + li, p.tq - 1);
  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8 *>(Q + (int64_t)qi * p.q_rs + 16 * ks + 8 * g);

  // ---- tile loads: wave w fills rows 16 w + 4 x + (lane >> 4), x = 0..3, one 1 KiB load each; lane
  // l writes 16-byte slot l & 15 of its row, so it fetches the chunk the swizzle puts there
  auto tile_rsrc = [&](const bf16 *base, int j) {
    const int valid = min(KT, p.tk - j * KT);
    const uint64_t a = (uint64_t)(base + (int64_t)j * KT * p.kv_rs);
    const uint32_t bytes = (uint32_t)((valid - 1) * p.kv_rs + DH) * 2u;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0,
                                             (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
  };
  auto load_k = [&](int j, int st) {
    const __amdgpu_buffer_rsrc_t r = tile_rsrc(Kb, j);
#pragma unroll
    for (int x = 0; x < 4; ++x)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (__attribute__((address_space(3))) void *)(lds + K_OFF + st * TILE_B + (16 * w + 4 * x) * DH * 2), 16,
          (uint32_t)((16 * w + 4 * x + (lane >> 4)) * p.kv_rs + 8 * ((lane & 15) ^ ((4 * x + (lane >> 4)) & 15))) * 2u, 0, 0, 0);
  };
  auto load_v = [&](int j, int st) {
    const __amdgpu_buffer_rsrc_t r = tile_rsrc(Vb, j);
#pragma unroll
    for (int x = 0; x < 4; ++x)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (__attribute__((address_space(3))) void *)(lds + V_OFF + st * TILE_B + (16 * w + 4 * x) * DH * 2), 16,
          (uint32_t)((16 * w + 4 * x + (lane >> 4)) * p.kv_rs + 8 * ((lane & 15) ^ (((lane >> 4) & 3) << 2))) * 2u, 0, 0, 0);
  };

  // ---- fragment offsets.  K fragment (slab sl, k-step ks): key 32 sl + li, chunk 2 ks + g at
  // chunk ^ (key & 15).  V^T fragment (chunk c, dims 32 dt ..): transpose read of key 16 c + tkey
  // (+ 8), head dims 32 dt + tdim .. + 3, chunk (d >> 3) ^ 4 (key & 3).
  uint32_t ko[8], vo[4];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) ko[ks] = (uint32_t)(li * DH * 2 + (((2 * ks + g) ^ (li & 15)) << 4));
  const int tq = lane & 15, th = (lane >> 4) & 1;
  const int tkey = 4 * g + (tq >> 2), tdim = 16 * th + 4 * (tq & 3);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    const int d = 32 * dt + tdim;
    vo[dt] = (uint32_t)(tkey * DH * 2 + (((d >> 3) ^ ((tkey & 3) << 2)) << 4) + (d & 7) * 2);
  }

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[dt][j] = 0.f;
  float mrun = -INFINITY, lsum = 0.f;

  // S^T of the tile in K stage st: lane holds query li, keys 32 sl + (j/4)*8 + 4 g + (j%4).  The two
  // slabs' accumulations alternate, so consecutive MFMAs never wait on each other's result.
  auto scores = [&](int st, f32x16 (&sc)[2]) {
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int j = 0; j < 16; ++j) sc[sl][j] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(lds + K_OFF + st * TILE_B + sl * 32 * DH * 2 + ko[ks]);
        sc[sl] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc[sl], 0, 0, 0);
      }
    }
  };
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  auto vread = [&](int st, int c, int dt, int hh) {
    return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4 *)(lds + V_OFF + st * TILE_B + (16 * c + 8 * hh) * DH * 2 + vo[dt])));
  };

  // One key tile j (K of j in stage j & 1, V of j in stage j & 1): probabilities from sc, interleaved
  // with the scores of tile j + 1 into sn when there is one, then O^T += V^T P^T.
  auto tile = [&](auto STAGE, int j, f32x16 (&sc)[2], f32x16 (&sn)[2]) {
    constexpr int st = decltype(STAGE)::value;
    // K of j + 1 and V of j have landed; every wave is done with K of j (read one tile ago) and V of
    // j - 1, so those stages take K of j + 2 and V of j + 1
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    __syncthreads();
    if (j + 2 < nt) load_k(j + 2, st);
    if (j + 1 < nt) load_v(j + 1, st ^ 1);
    if (idle) return;
    if ((j + 1) * KT > p.tk) {   // ragged last tile: keys at or past tk get -inf
      const int lim = p.tk - j * KT - 4 * g;
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int q = 0; q < 16; ++q) sc[sl][q] = 32 * sl + (q >> 2) * 8 + (q & 3) < lim ? sc[sl][q] : -INFINITY;
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int q = 0; q < 16; ++q) tmax = fmaxf(tmax, sc[sl][q]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    // Lazy rescaling: the running maximum moves only once some row's tile maximum passes it by more
    // than 8 / qscale (a factor 2^8 after exp2).  Until then the probabilities stay at most 256, well
    // inside bf16 (P) and fp32 (O, l), and O / l is the same quotient, so the wave skips the O rescale
    // on almost every tile.  The first tile always moves it (mrun = -inf, tile maxima are finite).
    if (__any(tmax > mrun + p.lazy_thr)) {
      const float mnew = fmaxf(mrun, tmax);
      const float corr = __builtin_amdgcn_exp2f((mrun - mnew) * p.qscale);
      lsum *= corr;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int q = 0; q < 16; ++q) o[dt][q] *= corr;
      mrun = mnew;
    }
    const float mb = mrun * p.qscale;
    // the next tile's scores (after the last tile: from a stale stage, unused), this tile's
    // probabilities and its V^T P^T products in one block, chunk by chunk (16 keys), with the V
    // fragments of chunk c + 1 read while chunk c is in flight
    scores(st ^ 1, sn);
    bf16x8 vf[2][4];
    auto vload = [&](int c, bf16x8 (&v)[4]) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x4 w0 = vread(st, c, dt, 0), w1 = vread(st, c, dt, 1);
        v[dt] = bf16x8{w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
      }
    };
    vload(0, vf[0]);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      bf16x8 pc;
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        const float e0 = __builtin_amdgcn_exp2f(fmaf(sc[c >> 1][8 * (c & 1) + i], p.qscale, -mb));
        const float e1 = __builtin_amdgcn_exp2f(fmaf(sc[c >> 1][8 * (c & 1) + i + 1], p.qscale, -mb));
        lsum += e0 + e1;
        const bf16x2 pr = __builtin_convertvector((float __attribute__((ext_vector_type(2)))){e0, e1}, bf16x2);
        pc[i] = pr[0];
        pc[i + 1] = pr[1];
      }
      if (c + 1 < 4) vload(c + 1, vf[(c + 1) & 1]);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[c & 1][dt], pc, o[dt], 0, 0, 0);
    }
  };

  load_k(0, 0);
  if (nt > 1) load_k(1, 1);
  load_v(0, 0);
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  f32x16 s0[2], s1[2];
  if (!idle) scores(0, s0);
  for (int j = 0; j < nt; j += 2) {
    tile(std::integral_constant<int, 0>{}, j, s0, s1);
    if (j + 1 >= nt) break;
    tile(std::integral_constant<int, 1>{}, j + 1, s1, s0);
  }
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / ltot;
  if (q0 + li >= p.tq) return;
  bf16 *O = (bf16 *)p.out + (int64_t)b * p.o_bs + (int64_t)(q0 + li) * p.o_rs + h * DH;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      bf16x4 w4 = {(bf16)(o[dt][4 * jq] * inv), (bf16)(o[dt][4 * jq + 1] * inv),
                   (bf16)(o[dt][4 * jq + 2] * inv), (bf16)(o[dt][4 * jq + 3] * inv)};
      *reinterpret_cast<bf16x4 *>(O + 32 * dt + 8 * jq + 4 * g) = w4;
    }
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
  p.nqb = 0;
  p.batch = a.batch; p.heads = a.heads; p.tq = a.tq; p.tk = a.tk;
  p.q = a.q; p.q_bs = a.q_bs; p.q_rs = a.q_rs;
  p.k = a.k; p.v = a.v; p.kv_bs = a.kv_bs; p.kv_rs = a.kv_rs;
  p.kv_index = a.kv_index; p.n_kv = a.n_kv;
  p.out = a.out; p.o_bs = a.o_bs; p.o_rs = a.o_rs;
  p.qscale = (float)(1.4426950408889634 / sqrt((double)a.head_dim));
  // FLASHBON_ATTN_LAZY=0 (tests and tuning): rescale whenever a row maximum grows
  const char *lazy = getenv("FLASHBON_ATTN_LAZY");
  p.lazy_thr = lazy && !strcmp(lazy, "0") ? 0.0f : 8.0f / p.qscale;
  if (t == ACT_BF16 && a.head_dim == fa::DH) {
    dim3 grid((p.tq + fa::QB - 1) / fa::QB, p.heads, p.batch);
    const char *sel = getenv("FLASHBON_ATTN");   // "mfma": the unpipelined kernel (tuning)
    if (sel && !strcmp(sel, "mfma")) {
      hipLaunchKernelGGL(k_attn_mfma, grid, dim3(256), 0, s, p);
    } else {
      p.nqb = (p.tq + fa2::QB - 1) / fa2::QB;
      const int64_t units8 = ((int64_t)p.batch * p.heads + 7) / 8 * 8;
      hipLaunchKernelGGL(k_attn_fa, dim3((unsigned)(units8 * p.nqb)), dim3(256), 0, s, p);
    }
    return hipGetLastError();
  }
  if (t == ACT_BF16) return launch_valu<bf16>(p, a.head_dim, s);
  return launch_valu<float>(p, a.head_dim, s);
}

}  // namespace fb
