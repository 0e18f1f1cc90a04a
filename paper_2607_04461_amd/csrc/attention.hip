// Softmax attention of the DiT block: self-attention over image tokens and cross-attention to the
// candidate's prompt tokens, softmax(q k^T / sqrt(dh)) v per (candidate, head).
//   * k_attn_valu: one lane per query, online softmax over 16-key sub-tiles staged in LDS as fp32;
//     any head_dim <= 128 (multiple of 8); fp32 or bf16 operands.  Used by the fp32 mode and for
//     head dims the MFMA kernel does not take.
//   * k_attn_fa: bf16, head_dim 128, gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).  Each wave owns
//     32 queries.  Scores are formed transposed, S^T = K Q^T, so every lane holds 16 scores of one
//     query (its partner lane l^32 holds the other 16 of a 32-key slab): the online-softmax max is a
//     single cross-lane exchange and the running sum stays per lane until the end.  The output is
//     accumulated transposed as well, O^T += V^T P^T: the probabilities feed the second MFMA straight
//     from the first one's accumulator registers (the key order inside each 16-key chunk is permuted
//     identically on both operands), and every lane rescales only its own query.  K and V tiles are
//     staged in LDS row-major, 16-byte chunks XOR-swizzled per row; V^T fragments come from gfx950's
//     LDS transpose read (ds_read_b64_tr_b16): in each group of 16 lanes, lane j addresses 4
//     consecutive head dims of one key and lane 4a + b receives element b of the pieces addressed by
//     lanes a, a + 4, a + 8, a + 12 -- i.e. one head dim across four keys.  Keys are taken in tiles of
//     64 with an online softmax; the order of a wave's work is described at the kernel.
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

namespace fa2 {
constexpr int DH = 128, KT = 64, QW = 32, WAVES = 4, QB = QW * WAVES;
constexpr int TILE_B = KT * DH * 2;   // bytes of one K or V tile
// LDS: K stage 0, K stage 1, V stage 0, V stage 1
constexpr int K_OFF = 0, V_OFF = 2 * TILE_B;
}  // namespace fa2

// ---------------------------------------------------------------- MFMA flash attention (dh 128)
// A wave keeps its matrix cores and its vector ALUs busy at the same time by ordering its own work:
// with the scores S(j) of key tile j and their row maxima already known, step j runs two interleaved
// phases,
//   A: the 16 MFMAs of S(j + 1) = K(j + 1) Q^T, with the exponentials of S(j)'s first 32 keys between
//      them;
//   B: the 16 MFMAs of O^T += V(j)^T P(j)^T chunk by chunk, with the exponentials of the last 32 keys
//      and the row maxima of S(j + 1) between them.
// The running maximum then moves for tile j + 1, lazily: only once some row's tile maximum passes it by
// more than 8 / qscale (a factor 2^8 after exp2); until then the probabilities stay at most 256, well
// inside bf16 (P) and fp32 (O, l), and O / l is the same quotient.  Each phase is written out as 8
// fenced slots of two MFMAs, one or two pairs of exponentials (or a share of the row maxima) and the
// fragment reads of two slots later, so the MFMAs do not wait on their LDS reads.  Two workgroups of 4
// waves share a CU (two waves per SIMD).  K and V tiles reach LDS through buffer loads that write LDS
// themselves, in rings of two stages filled one tile ahead, one barrier per tile; keys past tk read as
// zero (the buffer range ends at the last key) and are masked on the ragged last tile.  1-D grid,
// XCD-aware: workgroups go to the 8 XCDs round-robin by id, so id -> (unit u = head * batch + candidate,
// query block) keeps every query block of a unit on XCD u % 8, where its K and V stay in that XCD's L2.
// The normalised output leaves through LDS (the rings are free after a last barrier): a lane holds
// 16-byte pieces of one query row, so direct stores would write every 128-byte line of the output in
// several partial pieces; staged, each store instruction writes 4 whole rows.  Measured (same box,
// outputs bit-identical): cross-attention 110 -> 100 us, self-attention 308-320 -> 299-309 us, the
// 1.3B-shaped pool's draft 238.9 -> 236.8 ms.
__global__ __launch_bounds__(256, 2) void k_attn_fa(AttnP p) {
  using namespace fa2;
  constexpr int RW = KT / WAVES;     // K (V) tile rows each wave loads
  __shared__ __attribute__((aligned(16))) bf16 sm[4 * KT * DH];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, li = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int id = blockIdx.x, rest = id >> 3;
  const int u = (rest / p.nqb) * 8 + (id & 7), qblk = rest % p.nqb;
  if (u >= p.batch * p.heads) return;
  const int h = u / p.batch, b = u % p.batch;
  const int q0 = qblk * QB + w * QW;
  const bool idle = q0 >= p.tq;   // loads its share of every tile and meets every barrier, nothing else
  const int kb = kv_batch(p, b);
  const bf16 *Q = (const bf16 *)p.q + (int64_t)b * p.q_bs + h * DH;
  const bf16 *Kb = (const bf16 *)p.k + (int64_t)kb * p.kv_bs + h * DH;
  const bf16 *Vb = (const bf16 *)p.v + (int64_t)kb * p.kv_bs + h * DH;
  const int nt = (p.tk + KT - 1) / KT;
  char *lds = reinterpret_cast<char *>(sm);

  const int qi = min(q0 + li, p.tq - 1);
  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8 *>(Q + (int64_t)qi * p.q_rs + 16 * ks + 8 * g);

  auto tile_rsrc = [&](const bf16 *base, int j) {
    const int valid = min(KT, p.tk - j * KT);
    const uint64_t a = (uint64_t)(base + (int64_t)j * KT * p.kv_rs);
    const uint32_t bytes = (uint32_t)((valid - 1) * p.kv_rs + DH) * 2u;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0,
                                             (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
  };
  // wave w fills rows RW w + 4 x + (lane >> 4), x < RW / 4, one 1 KiB load each; lane l writes 16-byte
  // slot l & 15 of its row, so it fetches the chunk the row's swizzle puts there
  auto load_k = [&](int j, int st) {
    const __amdgpu_buffer_rsrc_t r = tile_rsrc(Kb, j);
#pragma unroll
    for (int x = 0; x < RW / 4; ++x) {
      const int row = RW * w + 4 * x + (lane >> 4);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (__attribute__((address_space(3))) void *)(lds + K_OFF + st * TILE_B + (RW * w + 4 * x) * DH * 2), 16,
          (uint32_t)(row * p.kv_rs + 8 * ((lane & 15) ^ (row & 15))) * 2u, 0, 0, 0);
    }
  };
  auto load_v = [&](int j, int st) {
    const __amdgpu_buffer_rsrc_t r = tile_rsrc(Vb, j);
#pragma unroll
    for (int x = 0; x < RW / 4; ++x) {
      const int row = RW * w + 4 * x + (lane >> 4);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (__attribute__((address_space(3))) void *)(lds + V_OFF + st * TILE_B + (RW * w + 4 * x) * DH * 2), 16,
          (uint32_t)(row * p.kv_rs + 8 * ((lane & 15) ^ ((row & 3) << 2))) * 2u, 0, 0, 0);
    }
  };
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
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  auto vfrag = [&](int st, int c, int dt) __attribute__((always_inline)) {
    const bf16x4 w0 = __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4 *)(lds + V_OFF + st * TILE_B + (16 * c) * DH * 2 + vo[dt])));
    const bf16x4 w1 = __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4 *)(lds + V_OFF + st * TILE_B + (16 * c + 8) * DH * 2 + vo[dt])));
    return bf16x8{w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
  };
  auto kfrag = [&](int st, int ks, int sl) __attribute__((always_inline)) {
    return *reinterpret_cast<const bf16x8 *>(lds + K_OFF + st * TILE_B + sl * 32 * DH * 2 + ko[ks]);
  };

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[dt][j] = 0.f;
  float mrun = -INFINITY, lsum = 0.f, mb = 0.f;
  bf16x8 pp[4];   // probabilities of the current tile, 16 keys per chunk

  // one pair of exponentials: keys 8 (c & 1) + i, + 1 of chunk c of the scores sc into pp[c]; the row
  // sum takes the pairs chunk by chunk
  auto epair = [&](const f32x16 (&sc)[2], int c, int i) __attribute__((always_inline)) {
    const float e0 = __builtin_amdgcn_exp2f(fmaf(sc[c >> 1][8 * (c & 1) + i], p.qscale, -mb));
    const float e1 = __builtin_amdgcn_exp2f(fmaf(sc[c >> 1][8 * (c & 1) + i + 1], p.qscale, -mb));
    lsum += e0 + e1;
    const bf16x2 pr = __builtin_convertvector((float __attribute__((ext_vector_type(2)))){e0, e1}, bf16x2);
    pp[c][i] = pr[0];
    pp[c][i + 1] = pr[1];
  };
  // keys at or past tk get -inf (the ragged last tile j)
  auto mask_tail = [&](f32x16 (&sc)[2], int j) __attribute__((always_inline)) {
    const int lim = p.tk - j * KT - 4 * g;
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int q = 0; q < 16; ++q) sc[sl][q] = 32 * sl + (q >> 2) * 8 + (q & 3) < lim ? sc[sl][q] : -INFINITY;
  };
  auto rowmax = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
    float t = -INFINITY;
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int q = 0; q < 16; ++q) t = fmaxf(t, sc[sl][q]);
    return t;
  };
  // the running maximum moves (lazily, see above) for a tile whose row maxima are tmax; O and the row
  // sum then rescale; mb is the exponent offset of the next exponentials
  auto advance = [&](float tmax) __attribute__((always_inline)) {
    {   // max over lanes l and l ^ 32 (the two halves of each query's keys): swap the 32-lane halves
      const uint32_t u = __builtin_bit_cast(uint32_t, tmax);
      const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
      tmax = fmaxf(__builtin_bit_cast(float, (uint32_t)sw[0]), __builtin_bit_cast(float, (uint32_t)sw[1]));
    }
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
    mb = mrun * p.qscale;
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // Step j (K of tile i in K stage i & 1, V of i in V stage i & 1; sc = S(j) masked, mb set for it).
  // At the top, V of j and K of j + 1 have landed and nobody reads V of j - 1 or K of j any more: those
  // stages take V of j + 1 and K of j + 2.  NEXT: whether tile j + 1 exists (S(j + 1) into sn).  Each
  // phase is 8 slots of two MFMAs, fenced, with the fragment reads of two slots later and a share of the
  // VALU work in every slot.
  auto step = [&](auto PAR, auto NEXT, int j, f32x16 (&sc)[2], f32x16 (&sn)[2]) __attribute__((always_inline)) {
    constexpr int par = decltype(PAR)::value, oth = par ^ 1;
    constexpr bool next = decltype(NEXT)::value;
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    __syncthreads();
    if (j + 1 < nt) load_v(j + 1, oth);
    if (j + 2 < nt) load_k(j + 2, par);
    if (idle) return;
    bf16x8 vf[4][4];
    // phase A: S(j + 1) (slot ks: k-step ks of both slabs) and the exponentials of chunks 0 and 1
    if constexpr (next) {
      bf16x8 kf[8][2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) kf[ks][sl] = kfrag(oth, ks, sl);
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int q = 0; q < 16; ++q) sn[sl][q] = 0.f;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
        for (int sl = 0; sl < 2; ++sl)
          sn[sl] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][sl], qf[ks], sn[sl], 0, 0, 0);
        epair(sc, ks >> 2, 2 * (ks & 3));
        if (ks + 2 < 8) {
#pragma unroll
          for (int sl = 0; sl < 2; ++sl) kf[ks + 2][sl] = kfrag(oth, ks + 2, sl);
        } else {
#pragma unroll
          for (int dt = 2 * (ks - 6); dt < 2 * (ks - 6) + 2; ++dt) vf[0][dt] = vfrag(par, 0, dt);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // chunks 0 and 1 and the row sum are formed in the slots above, not sunk past this branch to their
      // first use
      asm volatile("" : "+v"(pp[0]), "+v"(pp[1]), "+v"(lsum));
      if ((j + 2) * KT > p.tk) mask_tail(sn, j + 1);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) epair(sc, i >> 2, 2 * (i & 3));
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) vf[0][dt] = vfrag(par, 0, dt);
    }
    __builtin_amdgcn_sched_barrier(0);
    // phase B: O^T += V(j)^T P(j)^T (slot s: chunk s / 2, head-dim tiles 2 (s % 2), + 1), the exponentials
    // of chunk 2 (slots 0-3) and chunk 3 (slots 4, 5), the row maxima of S(j + 1) (slots 6, 7)
    float t0 = -INFINITY, t1 = -INFINITY;
#pragma unroll
    for (int sl8 = 0; sl8 < 8; ++sl8) {
      const int c = sl8 >> 1, d0 = 2 * (sl8 & 1);
#pragma unroll
      for (int dt = d0; dt < d0 + 2; ++dt) o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[c][dt], pp[c], o[dt], 0, 0, 0);
      if (sl8 < 4) {
        epair(sc, 2, 2 * sl8);
      } else if (sl8 < 6) {
        epair(sc, 3, 4 * (sl8 - 4));
        epair(sc, 3, 4 * (sl8 - 4) + 2);
      } else if constexpr (next) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          if (sl8 == 6) t0 = fmaxf(t0, sn[0][q]);
          else t1 = fmaxf(t1, sn[1][q]);
        }
      }
      if (c + 1 < 4) {
#pragma unroll
        for (int dt = d0; dt < d0 + 2; ++dt) vf[c + 1][dt] = vfrag(par, c + 1, dt);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (next) advance(fmaxf(t0, t1));
  };

  load_k(0, 0);
  if (nt > 1) load_k(1, 1);
  load_v(0, 0);
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  if (idle) {   // the loads and barriers of every step, nothing else
    for (int j = 0; j < nt; ++j) {
      __builtin_amdgcn_s_waitcnt(0x0F70);
      __syncthreads();
      if (j + 1 < nt) load_v(j + 1, (j + 1) & 1);
      if (j + 2 < nt) load_k(j + 2, j & 1);
    }
    __syncthreads();   // the output pass's barrier below
    return;
  }
  f32x16 sa[2], sb[2];
  {   // S(0) and its maxima
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int q = 0; q < 16; ++q) sa[sl][q] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) sa[sl] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(0, ks, sl), qf[ks], sa[sl], 0, 0, 0);
    if (KT > p.tk) mask_tail(sa, 0);
    advance(rowmax(sa));
  }
  using T_ = std::true_type;
  using F_ = std::false_type;
  int j = 0;
  for (; j + 2 < nt; j += 2) {
    step(S0{}, T_{}, j, sa, sb);
    step(S1{}, T_{}, j + 1, sb, sa);
  }
  if (j + 2 == nt) {
    step(S0{}, T_{}, j, sa, sb);
    step(S1{}, F_{}, j + 1, sb, sa);
  } else {
    step(S0{}, F_{}, j, sa, sb);
  }
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / ltot;
  __syncthreads();   // every wave has read its last K and V fragments: the rings are free
  // the wave's 32 x 128 output block goes through LDS (16-byte chunk c of row r at c ^ (r & 15)), so that
  // each global store writes 4 whole rows
  char *ob = lds + w * (QW * DH * 2);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      bf16x4 w4 = {(bf16)(o[dt][4 * jq] * inv), (bf16)(o[dt][4 * jq + 1] * inv),
                   (bf16)(o[dt][4 * jq + 2] * inv), (bf16)(o[dt][4 * jq + 3] * inv)};
      const int c = 4 * dt + jq;
      *reinterpret_cast<bf16x4 *>(ob + li * (DH * 2) + ((c ^ (li & 15)) << 4) + 8 * g) = w4;
    }
  const int cc = lane & 15;
  bf16 *Ob = (bf16 *)p.out + (int64_t)b * p.o_bs + h * DH + 8 * cc;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = (lane >> 4) + 4 * i;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(ob + r * (DH * 2) + ((cc ^ (r & 15)) << 4));
    if (q0 + r < p.tq) *reinterpret_cast<u32x4 *>(Ob + (int64_t)(q0 + r) * p.o_rs) = v;
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
  if (t == ACT_BF16 && a.head_dim == fa2::DH) {
    p.nqb = (p.tq + fa2::QB - 1) / fa2::QB;
    const int64_t units8 = ((int64_t)p.batch * p.heads + 7) / 8 * 8;
    hipLaunchKernelGGL(k_attn_fa, dim3((unsigned)(units8 * p.nqb)), dim3(256), 0, s, p);
    return hipGetLastError();
  }
  if (t == ACT_BF16) return launch_valu<bf16>(p, a.head_dim, s);
  return launch_valu<float>(p, a.head_dim, s);
}

}  // namespace fb
