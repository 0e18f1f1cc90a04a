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

// Working buffers of one step: the residual stream, activations, text projection, timestep path and
// the device copy of the prompt indices.  Carved from the model workspace, or from the per-device
// scratch array for the allocation-free refinement step.
struct StepBufs {
  float *h = nullptr;          // residual stream [M][D] fp32
  void *a = nullptr, *qkv = nullptr, *o = nullptr, *u = nullptr, *tok = nullptr;  // act [M][D|3D|D|F|P]
  void *txt = nullptr, *ctx = nullptr;  // text tokens (act copy, bf16 mode) and projected context
  float *vtok = nullptr;       // head output [M][C p p] fp32 (stochastic update / guidance)
  float2 *rope = nullptr;      // (cos, sin) per token and pair [T][head_dim/2] (qk_norm_rope)
  float *tf = nullptr, *e1 = nullptr, *e = nullptr, *m6 = nullptr, *bmods = nullptr, *hmod = nullptr;
  int32_t *d_cond = nullptr;   // prompt of each token-row block
  void *part = nullptr;        // split-K partial sums of the linear layers (bf16 mode), kSplitBytes
  size_t part_bytes = 0;
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
  StepBufs bufs;          // carved from ws, sized for the maxima
  int rope_h = -1, rope_w = -1;   // latent size the workspace rotary table was made for
  std::vector<int32_t> last_cond; // prompt indices last uploaded to bufs.d_cond
  // device timing of launch sites (flashbon_set_timing)
  uint32_t timing_mask = 0;
  struct Site {
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
    double total_ms = 0;
    int64_t launches = 0;
  } sites[FLASHBON_NUM_SITES];
  std::vector<hipEvent_t> spare_events;
};

// Scratch of the allocation-free refinement step: one static device array per GPU.
constexpr size_t kScratchBytes = (size_t)128 << 20;
constexpr int kMaxDevices = 64;
constexpr int kMaxScratchRows = 128;   // token-row blocks (candidates, twice with guidance) per call
// Device address of this GPU's scratch array (taken once per device, with that device current).
hipError_t scratch_base(int device, char **out);
// Bytes the step's buffers take in scratch for `rows` candidate rows of `tokens` tokens and `text_rows`
// text tokens to project (0 when text_kv is valid); with base != null also fills B.
size_t scratch_layout(const Model *m, int rows, int tokens, int text_rows, char *base, StepBufs *B);

flashbon_status fail(flashbon_status st, const std::string &msg);
bool config_ok(const flashbon_model_config *c, std::string *why);
Layout make_layout(const flashbon_model_config &c);

}  // namespace fb
