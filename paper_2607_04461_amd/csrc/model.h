// Internal model state of the draft-step library.
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "../../include/flashbon.h"
#include "kernels.h"

namespace fb {

// Element offsets of every tensor in the packed weight blob (same offsets in the fp32 and bf16 copies).
struct BlockOff {
  size_t mod, wqkv, bqkv, wo, bo, wqc, bqc, wkvc, bkvc, woc, boc, w1, b1, w2, b2;
  size_t nq = 0, nk = 0, nqc = 0, nkc = 0;   // RMSNorm gains (qk_norm_rope)
};
struct Layout {
  size_t t_w1, t_b1, t_w2, t_b2, mod_w, mod_b, hmod_w, hmod_b, pe_w, pe_b, txt_w, txt_b;
  std::vector<BlockOff> blk;
  size_t head_w, head_b, total, block_stride;
};

struct Model {
  flashbon_model_config c;
  Layout lay;
  ActType act;
  size_t asz;
  int D, H, dh, F, C, p, P, fd, Dt, L;
  int64_t maxM;
  int device = 0;
  float *w32 = nullptr;  // every weight, fp32
  void *w16 = nullptr;   // every weight, bf16 (BF16 mode)
  void *ws = nullptr;    // workspace
  size_t ws_bytes = 0;
  float *h;              // residual stream [maxM][D] fp32
  void *a, *qkv, *o, *u, *tok, *txt, *ctx;  // act buffers
  float *vtok;           // head output [maxM][C p p] fp32 (stochastic update only)
  float2 *rope = nullptr;  // (cos, sin) per token and pair [max_tokens][head_dim/2] (qk_norm_rope)
  int rope_h = -1, rope_w = -1;   // latent size the table was made for
  float *tf, *e1, *e, *m6, *bmods, *hmod;   // timestep path (fp32)
  int32_t *d_cond;
  std::vector<int32_t> last_cond;
  // device timing of launch sites (flashbon_set_timing)
  uint32_t timing_mask = 0;
  struct Site {
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
    double total_ms = 0;
    int64_t launches = 0;
  } sites[FLASHBON_NUM_SITES];
  std::vector<hipEvent_t> spare_events;
};

flashbon_status fail(flashbon_status st, const std::string &msg);
bool config_ok(const flashbon_model_config *c, std::string *why);
Layout make_layout(const flashbon_model_config &c);

}  // namespace fb
