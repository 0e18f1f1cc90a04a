/*
 * flashbon.h -- C ABI of the MI355X (gfx950) batched draft-generation library for Flash-BoN
 * (arXiv 2607.04461).
 *
 * The library runs one denoising step of a DiT over a pool of N candidates with the paper's three
 * draft knobs (Sec. 4.1):
 *   (1) timestep truncation   -- the caller loops over the first S' steps of the schedule (Eq. 2);
 *   (2) activation proxies    -- a proxied block's output is the second-order Taylor forecast of
 *                                Eq. 3-5 from that block's cached outputs;
 *   (3) layer skipping        -- a skipped block is the identity on the residual stream (Eq. 6);
 * a computed block is h = B_l(h, x, t) (Eq. 7).  The latent update is the flow-matching Euler step
 * (App. A.1, Eq. 20 with a = 0): z <- z + (t_next - t_cur) v.  Refinement (Sec. 4.2 Stage 3,
 * Eq. 13) is the same step with every knob off.
 *
 * Conventions shared by every call:
 *   - Every call returns flashbon_status (0 = OK).  Validation errors return before any device
 *     write and before any change to host-side state (meta, trace, text_kv_valid).  A HIP failure
 *     returns FLASHBON_EHIP; the device state of the caller's buffers is then undefined and the
 *     caller must re-zero `meta` and `text_kv_valid`.  flashbon_last_error() describes the last
 *     failure of the calling thread.  Nothing throws or aborts across this boundary.
 *   - "device" pointers are HIP device allocations on the current device; "host" pointers are
 *     ordinary host memory.  The caller owns every buffer it passes; the library owns only the
 *     model (weights + workspace).  The library keeps no pointer to caller buffers after a call
 *     returns, except that work enqueued on `stream` keeps reading/writing them until it completes.
 *   - Device work is enqueued on `stream` (a hipStream_t passed as void*; NULL = default stream) and
 *     the call returns without synchronising.  Host outputs (trace, meta, text_kv_valid) are final
 *     at return, since dispatch is decided on the host.
 *   - Calls on one model must be serialised (the workspace is shared); overlapping calls race.
 *   - Row-major layouts throughout; tensors are dense (no padding between rows).
 */
#ifndef FLASHBON_H
#define FLASHBON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque handle of a model (weights + workspace), created by flashbon_init_model. */
typedef struct flashbon_model flashbon_model;

typedef enum {
  FLASHBON_OK = 0,
  FLASHBON_EINVAL = -1, /* NULL where a pointer is required, bad enum, non-finite or unordered t */
  FLASHBON_ESHAPE = -2, /* a size is zero/negative, inconsistent, or above the configured maxima */
  FLASHBON_ENOMEM = -3, /* a device or pinned-host allocation failed (init only) */
  FLASHBON_EHIP = -4,   /* a HIP runtime call or kernel launch failed */
  FLASHBON_ESTATE = -5  /* cache metadata out of range (count > 3, head > 2, ...) */
} flashbon_status;

typedef enum {
  FLASHBON_FP32 = 0, /* all GEMM operands, attention and activations in fp32 */
  FLASHBON_BF16 = 1  /* bf16 GEMM/attention operands with fp32 accumulation; residual stream,
                        cache, latents and normalisation statistics stay fp32 */
} flashbon_dtype;

/* Model shape.  The DiT block is a Wan-shaped block (the paper does not describe one):
 *   a = LN(h)(1+scale1)+shift1; h += gate1 * SelfAttn(a)
 *   c = LN(h);                  h += CrossAttn(c, text)
 *   a = LN(h)(1+scale2)+shift2; h += gate2 * MLP(a), MLP = W2 GELU_tanh(W1 a + b1) + b2
 * LN is non-affine over `hidden`; head_dim = hidden / heads. */
typedef struct {
  int32_t num_blocks;      /* L */
  int32_t hidden;          /* D, multiple of 8, <= 6144 */
  int32_t heads;           /* H; hidden % heads == 0, head_dim in {8, 16, 32, 64, 128} */
  int32_t mlp_hidden;      /* F, multiple of 8, <= 65536 */
  int32_t latent_channels; /* C */
  int32_t patch;           /* p (2): token = p x p patch of every channel */
  int32_t freq_dim;        /* width of the sinusoidal timestep features (even) */
  int32_t text_dim;        /* width of the text-conditioning tokens, multiple of 8, <= 65536 */
  int32_t dtype;           /* flashbon_dtype */
  float ln_eps;            /* LayerNorm epsilon (1e-6) */
  int32_t max_n;           /* largest pool size a step may use */
  int32_t max_tokens;      /* largest T = (latent_h/p)(latent_w/p) */
  int32_t max_text_len;    /* largest text_len */
  int32_t max_cond;        /* largest n_cond */
  int32_t qk_norm_rope;    /* 0 or 1: RMSNorm (eps = ln_eps, per-block gains) on q and k of both attentions
                              -- the text keys once, when text_kv is made -- and 3-D rotary position
                              embedding on self-attention: head_dim splits into frame, height and width
                              bands of dh - 4 (dh/6), 2 (dh/6), 2 (dh/6) dims; a token at (frame 0, row i,
                              column j) turns pair k of a band of width d by p 10000^(-2k/d), p its
                              position along the band's axis, pairs (2k, 2k+1) of each head */
} flashbon_model_config;

/* Per-block activation-cache metadata, host side (one per block).  The cache of a block is a ring of
 * three slots.  A computed block writes slot `head`, stores t_cur in t[head], advances
 * head = (head+1) % 3 and saturates count at 3.  The most recent entry is slot (head+2) % 3, then
 * (head+1) % 3, then head.  The caller zeroes it at the start of a pool. */
typedef struct {
  int32_t count; /* valid entries, 0..3 */
  int32_t head;  /* next slot to write, 0..2 */
  float t[3];    /* timestep of the entry in each slot */
} flashbon_cache_meta;

enum { FLASHBON_COMPUTE = 0, FLASHBON_SKIP = 1, FLASHBON_PROXY = 2 };

/* What one block did at one step (bit-exact, host-decided):
 *   COMPUTE: order -1, slot = cache slot written, live 1
 *   SKIP   : order -1, slot -1, live 0
 *   PROXY  : order 0..2 (Taylor order = min(count,3)-1), slot = most recent entry's slot,
 *            live = 1 iff the next non-skipped block is computed or there is none (otherwise the
 *            proxy's output would be overwritten unread, and nothing is launched for it). */
typedef struct {
  int8_t action;
  int8_t order;
  int8_t slot;
  int8_t live;
} flashbon_trace_entry;

typedef struct {
  int32_t n;        /* candidates in this call, 1..max_n */
  int32_t latent_h; /* H, multiple of patch */
  int32_t latent_w; /* W, multiple of patch; T = (H/p)(W/p) <= max_tokens */

  float *latents; /* device [n, C, H, W] fp32: z_{t_cur} in, z_{t_next} out (in place) */
  float t_cur;    /* current timestep t_k (host scalar from the caller's schedule) */
  float t_next;   /* next timestep t_{k+1}; the update adds (t_next - t_cur) * v */

  const float *text;         /* device [n_cond, text_len, text_dim] fp32 conditioning tokens */
  int32_t n_cond;            /* prompts in the pool, 1..max_cond */
  int32_t text_len;          /* tokens per prompt, 1..max_text_len */
  const int32_t *cond_index; /* host [n]: prompt of each candidate, values in [0, n_cond) */
  void *text_kv;             /* device scratch of flashbon_text_kv_bytes() bytes, caller-owned:
                                per-block cross-attention K/V of every prompt */
  int32_t *text_kv_valid;    /* host flag in/out: 0 -> the call first computes text_kv from `text`
                                and sets it to 1; 1 -> text_kv is reused as is.  The caller resets it
                                to 0 whenever `text` changes. */

  const uint8_t *skip;  /* host [num_blocks]: 1 = skip block l at this step (draft only) */
  const uint8_t *proxy; /* host [num_blocks]: 1 = proxy block l at this step (draft only);
                           skip wins over proxy; a proxy with an empty cache computes */
  float *cache;         /* device fp32 [num_blocks][3][n][T][hidden] (flashbon_cache_bytes());
                           draft only: computed block outputs, proxy inputs */
  flashbon_cache_meta *meta;   /* host [num_blocks] in/out (draft only) */
  flashbon_trace_entry *trace; /* host [num_blocks] out, optional (NULL = not reported) */

  float *hidden_dump; /* optional debug output, device fp32 [num_blocks+1][rows][T][hidden] (rows = n, or
                         2n with guidance): the residual stream after the patch embedding (index 0) and
                         after block l (index l+1).  Entries whose value the step never forms are left
                         untouched: the embedding when the first non-skipped block is a proxy, a dead
                         proxy, and a skipped block whose input was not formed (it follows one of
                         those with no launched block in between).  NULL = off. */
  void *stream;       /* hipStream_t */

  /* Stochastic update (App. A.1, Eq. 20) in place of the Euler one; sde_a = 0 (a zero-initialised
   * struct) keeps the Euler update bit for bit.  With sde_a > 0 the step computes
   *   z <- z + dt [v + sigma^2 / (2 t) (z + (1 - t) v)] + sigma sqrt(|dt|) eps,
   *   t = t_cur, dt = t_next - t_cur, sigma = sde_a sqrt(t / (1 - t)) (1 - t_next when t = 1),
   * eps[b][e] (flat element e of candidate row b of this call) = normal e % 4 of Philox4x32-10 with
   * key (sde_seed low 32 bits, high 32 bits) and counter (e / 4, sde_row0 + b, sde_step, 0), through Box-Muller
   * (u1 = (w0 + 1) 2^-32, u2 = w1 2^-32; r = sqrt(-2 ln u1); r cos 2 pi u2, r sin 2 pi u2; then w2, w3).
   * Requires 0 < t_cur <= 1 (t_next < 1 if t_cur = 1); else FLASHBON_EINVAL before any device work. */
  float sde_a;       /* noise level a >= 0 */
  int32_t sde_step;  /* third counter word: a distinct value per step keeps draws independent */
  uint64_t sde_seed; /* Philox key */
  int32_t sde_row0;  /* candidate index of row 0 in the counter (>= 0): a slice of a larger pool, or a
                        single refined candidate, draws the normals of its place in the pool */

  float *preview; /* optional device fp32 [n, C, H, W] output, NULL = off: the clean-latent estimate
                     z - t_cur v of this step's state (rectified flow x_t = (1 - t) x_0 + t x_1, so
                     x_0 = x_t - t v), i.e. one Euler jump of the step's output to t = 0 -- the
                     draft preview a verifier scores (Sec. 4.2 Stage 1).  Must not alias latents. */

  /* Classifier-free guidance, off when cfg == 0.  On, the step runs 2n token rows through the
   * network: rows [0, n) with prompts cond_index, rows [n, 2n) -- the unconditional twins of the same
   * n latents -- with prompts uncond_index (host [n], values in [0, n_cond), typically a null
   * prompt), and steps candidate b with v = v_u + cfg_scale (v_c - v_u).  2n <= max_n; cache and
   * hidden_dump then hold 2n rows (flashbon_cache_bytes(model, 2n, T)). */
  int32_t cfg;
  float cfg_scale;
  const int32_t *uncond_index;

  /* Reading of the activation proxy (draft only): 0 (FLASHBON_PROXY_OUTPUT) -- h^(l) of Eq. 3-5 is
   * the block's output, cached by computed blocks and forecast by proxies; 1
   * (FLASHBON_PROXY_RESIDUAL) -- h^(l) is the block's residual delta B_l(h) - h: computed blocks cache
   * their delta and a proxy adds the forecast delta to its input (every proxy is then live and the
   * patch embedding always runs).  The cache holds one reading's entries: switching between calls
   * needs a reset cache (meta count 0). */
  int32_t proxy_mode;
} flashbon_step_args;

/* Number of floats `host_weights` must hold for `cfg`. Returns 0 if cfg is invalid. */
size_t flashbon_weight_count(const flashbon_model_config *cfg);

/* Create a model: validates cfg, allocates device weights (fp32 for small vectors and the timestep
 * path, plus a bf16 copy of every matrix in BF16 mode) and a workspace sized for the maxima,
 * copies `host_weights` (fp32, `n_weights` floats, packed as below) and synchronises.
 * Packing order, every matrix [out][in] row-major:
 *   t_w1[D][freq] t_b1[D] t_w2[D][D] t_b2[D] mod_w[6D][D] mod_b[6D] head_mod_w[2D][D] head_mod_b[2D]
 *   pe_w[D][C p p] pe_b[D] txt_w[D][text_dim] txt_b[D]
 *   per block l: mod[6][D] wq wk wv[D][D each] bq bk bv[D each] wo[D][D] bo[D] wqc[D][D] bqc[D]
 *                wkc wvc[D][D each] bkc bvc[D each] woc[D][D] boc[D] w1[F][D] b1[F] w2[D][F] b2[D]
 *                and, with qk_norm_rope, the RMSNorm gains nq nk nqc nkc[D each]
 *   head_w[C p p][D] head_b[C p p]
 * Timestep conditioning: f = [cos(1000 t w_j) | sin(1000 t w_j)], w_j = 10000^(-j/(freq/2));
 * e = t_w2 SiLU(t_w1 f + t_b1) + t_b2; m = mod_w SiLU(e) + mod_b; block l uses m + mod_l split as
 * (shift1, scale1, gate1, shift2, scale2, gate2); the head uses head_mod_w SiLU(e) + head_mod_b split
 * as (shift, scale).  On success *out owns the model; free it with flashbon_free. */
flashbon_status flashbon_init_model(const flashbon_model_config *cfg, const float *host_weights,
                                    size_t n_weights, flashbon_model **out);

/* Bytes of the caller-owned cross-attention K/V scratch for n_cond prompts of text_len tokens. */
size_t flashbon_text_kv_bytes(const flashbon_model *model, int32_t n_cond, int32_t text_len);

/* Bytes of the caller-owned activation cache for n candidates of `tokens` tokens. */
size_t flashbon_cache_bytes(const flashbon_model *model, int32_t n, int32_t tokens);

/* One draft step (Sec. 4.2 Stage 1, Eq. 8) over the pool with the step's skip/proxy masks: plans
 * every block on the host (trace, meta), then enqueues the step.  Skipped blocks and dead proxies
 * launch nothing. */
flashbon_status flashbon_draft_step(flashbon_model *model, const flashbon_step_args *args);

/* One full-quality step (Sec. 4.2 Stage 3, Eq. 13): as flashbon_draft_step with every mask zero;
 * skip, proxy, cache and meta are ignored (may be NULL).  trace, if given, reports all COMPUTE. */
flashbon_status flashbon_refine_step(flashbon_model *model, const flashbon_step_args *args);

/* Refinement step that allocates nothing and touches no model workspace -- for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it), and for refining one pool's winner on one stream while the same model drafts on another.
 * Same arguments, results (bit for bit) and validation as flashbon_refine_step.  The step's working
 * buffers (residual stream, activations, timestep path, text projection when *text_kv_valid is 0,
 * prompt indices, rotary table) come from a static device array of FLASHBON_NOALLOC_SCRATCH_BYTES that
 * the library holds on every GPU it runs on until the process ends; nothing in it has to start at
 * zero.  FLASHBON_ESHAPE, before any device work, if a call needs more (about 121 MB for one candidate
 * of the 1.3B-shaped model at 1560 tokens in bf16 mode, 48 MiB of it the split-K partial sums of the
 * linear layers; 118 MB in fp32 mode) or more than 128 token-row
 * blocks; FLASHBON_EINVAL if the current device is not the model's.  Every call on a GPU shares that
 * GPU's array: calls of this entry point that overlap on one GPU (other streams, other threads, other
 * models) race.  No timing sites are recorded. */
#define FLASHBON_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
flashbon_status flashbon_refine_step_noalloc(flashbon_model *model, const flashbon_step_args *args);

/* Release the model.  NULL is a no-op.  Synchronises the device before freeing. */
void flashbon_free(flashbon_model *model);

enum { FLASHBON_PROXY_OUTPUT = 0, FLASHBON_PROXY_RESIDUAL = 1 };

/* Host-only dispatch of one step, as flashbon_draft_step performs it (Eq. 3-6 plus the cache
 * ring): fills trace[num_blocks] and advances meta[num_blocks] in place.  proxy_mode as in
 * flashbon_step_args.  No device work. */
flashbon_status flashbon_plan_step(int32_t num_blocks, const uint8_t *skip, const uint8_t *proxy,
                                   flashbon_cache_meta *meta, float t_cur,
                                   flashbon_trace_entry *trace, int32_t proxy_mode);

/* Verifier callback of flashbon_select: judge candidate a (ranked above b) against candidate b.
 * Returns the winner (a or b) and writes the verifier's confidence to *confidence: 0 high, 1 medium,
 * 2 low.  Any other result aborts the selection with FLASHBON_EINVAL. */
typedef int32_t (*flashbon_judge_fn)(void *ctx, int32_t a, int32_t b, int32_t *confidence);

/* Multi-stage selection with Elo ratings (Sec. 4.2 Stage 2, Eq. 9-12), host only:
 *   1. rating r_j = 1500 + 100 (scores[j] - 5) from the integer pointwise scores (1..10, host [m]);
 *      keep the top ceil(rho1 m) -> M1 survivors;
 *   2. ceil(kappa M1) verifier matches between neighbours of the rating order (sweeps over the
 *      neighbour pairs, re-ordered by rating after each sweep; none if M1 < 2); keep the top
 *      ceil(rho2 M1) -> M2 survivors;
 *   3. every pair of the M2 survivors plays once (rating order at the stage's start, pairs (i, j),
 *      i < j, lexicographically); *winner = the highest rating.
 * Each match updates both ratings zero-sum by K c (S_a - E_a), E_a = 1 / (1 + 10^((r_b - r_a) / 400)),
 * K = 32, c = 1.2 / 1.0 / 0.7 for high / medium / low confidence.  Orders break rating ties by the
 * smaller index; ceil(x) is ceil(x - 1e-9).  rho1, rho2 in (0, 1], kappa >= 0 (paper: 0.5, 0.5, 1.5).
 * ratings (host [m], final ratings) and pairwise_calls may be NULL.  Outputs are written only on
 * success. */
flashbon_status flashbon_select(int32_t m, const int32_t *scores, double rho1, double rho2, double kappa,
                                flashbon_judge_fn judge, void *ctx, int32_t *winner, double *ratings,
                                int32_t *pairwise_calls);

/* Launch sites of the draft step whose device time can be measured (bit i of a site mask). */
enum {
  FLASHBON_SITE_QKV = 0,        /* self-attention q/k/v projection        */
  FLASHBON_SITE_ATTN_SELF = 1,  /* self-attention                         */
  FLASHBON_SITE_OUT = 2,        /* self-attention output projection       */
  FLASHBON_SITE_CROSS_Q = 3,    /* cross-attention query projection       */
  FLASHBON_SITE_ATTN_CROSS = 4, /* cross-attention                        */
  FLASHBON_SITE_OUT_CROSS = 5,  /* cross-attention output projection      */
  FLASHBON_SITE_MLP_UP = 6,     /* MLP up projection + GELU               */
  FLASHBON_SITE_MLP_DOWN = 7,   /* MLP down projection + gate + residual + cache store */
  FLASHBON_SITE_NORM = 8,       /* the three adaLN / LN launches of a block and the head's */
  FLASHBON_SITE_PROXY = 9,      /* activation proxy                       */
  FLASHBON_SITE_EMBED = 10,     /* patchify + patch embedding             */
  FLASHBON_SITE_HEAD = 11,      /* head projection + unpatchify + Euler   */
  FLASHBON_SITE_TIME = 12,      /* timestep conditioning                  */
  FLASHBON_SITE_TEXT = 13,      /* text projection and per-block cross K/V */
  FLASHBON_NUM_SITES = 14
};

/* Enable device timing of the sites in `site_mask` for later calls on this model: the library then
 * records a HIP event pair on the step's stream around every launch at those sites (a few
 * microseconds of host time per launch; 0 disables).  Accumulated results are read, and reset, by
 * flashbon_read_timing. */
flashbon_status flashbon_set_timing(flashbon_model *model, uint32_t site_mask);

/* Synchronise on the recorded events and return, for one site, the summed device time (ms) and the
 * number of launches timed since the last read; resets that site's record. */
flashbon_status flashbon_read_timing(flashbon_model *model, int32_t site, double *total_ms, int64_t *launches);

/* Description of the calling thread's last failure ("" if none).  Valid until the next call. */
const char *flashbon_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBON_H */
