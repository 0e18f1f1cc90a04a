// C ABI of the draft-step library: model creation, the draft / refine step driver, and helpers.
// Host code only: validates, plans (dispatch.cpp), then enqueues the kernels of kernels.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/flashbon.h"
#include "dispatch.h"
#include "kernels.h"
#include "model.h"

namespace fb {

thread_local std::string g_err;

flashbon_status fail(flashbon_status st, const std::string &msg) {
  g_err = msg;
  return st;
}

bool config_ok(const flashbon_model_config *c, std::string *why) {
  auto bad = [&](const char *m) { if (why) *why = m; return false; };
  if (!c) return bad("config is NULL");
  if (c->num_blocks < 1) return bad("num_blocks must be >= 1");
  if (c->hidden < 8 || c->hidden % 8) return bad("hidden must be a positive multiple of 8");
  if (c->hidden > 6144) return bad("hidden must be <= 6144");
  if (c->heads < 1 || c->hidden % c->heads) return bad("heads must divide hidden");
  int dh = c->hidden / c->heads;
  if (dh != 8 && dh != 16 && dh != 32 && dh != 64 && dh != 128)
    return bad("head_dim must be one of 8, 16, 32, 64, 128");
  if (c->mlp_hidden < 8 || c->mlp_hidden % 8 || c->mlp_hidden > 65536)
    return bad("mlp_hidden must be a positive multiple of 8, <= 65536");
  if (c->latent_channels < 1 || c->patch < 1) return bad("latent_channels and patch must be >= 1");
  if ((c->latent_channels * c->patch * c->patch) % 8) return bad("latent_channels*patch^2 must be a multiple of 8");
  if (c->freq_dim < 2 || c->freq_dim % 8) return bad("freq_dim must be a positive multiple of 8");
  if (c->text_dim < 8 || c->text_dim % 8 || c->text_dim > 65536)
    return bad("text_dim must be a positive multiple of 8, <= 65536");
  if (c->dtype != FLASHBON_FP32 && c->dtype != FLASHBON_BF16) return bad("dtype must be FP32 or BF16");
  if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps)) return bad("ln_eps must be positive");
  if (c->qk_norm_rope != 0 && c->qk_norm_rope != 1) return bad("qk_norm_rope must be 0 or 1");
  if (c->max_n < 1 || c->max_tokens < 1 || c->max_text_len < 1 || c->max_cond < 1)
    return bad("max_n, max_tokens, max_text_len, max_cond must be >= 1");
  if ((int64_t)c->max_n * c->max_tokens > (int64_t)1 << 30) return bad("max_n * max_tokens too large");
  return true;
}

Layout make_layout(const flashbon_model_config &c) {
  Layout L;
  size_t o = 0;
  auto take = [&](size_t n) { size_t r = o; o += n; return r; };
  const size_t D = c.hidden, F = c.mlp_hidden, P = (size_t)c.latent_channels * c.patch * c.patch;
  const size_t fd = c.freq_dim, Dt = c.text_dim;
  L.t_w1 = take(D * fd); L.t_b1 = take(D); L.t_w2 = take(D * D); L.t_b2 = take(D);
  L.mod_w = take(6 * D * D); L.mod_b = take(6 * D);
  L.hmod_w = take(2 * D * D); L.hmod_b = take(2 * D);
  L.pe_w = take(D * P); L.pe_b = take(D);
  L.txt_w = take(D * Dt); L.txt_b = take(D);
  L.blk.resize(c.num_blocks);
  for (int l = 0; l < c.num_blocks; ++l) {
    BlockOff &b = L.blk[l];
    b.mod = take(6 * D);
    b.wqkv = take(3 * D * D); b.bqkv = take(3 * D);
    b.wo = take(D * D); b.bo = take(D);
    b.wqc = take(D * D); b.bqc = take(D);
    b.wkvc = take(2 * D * D); b.bkvc = take(2 * D);
    b.woc = take(D * D); b.boc = take(D);
    b.w1 = take(F * D); b.b1 = take(F);
    b.w2 = take(D * F); b.b2 = take(D);
    if (c.qk_norm_rope) { b.nq = take(D); b.nk = take(D); b.nqc = take(D); b.nkc = take(D); }
  }
  L.block_stride = c.num_blocks > 1 ? L.blk[1].mod - L.blk[0].mod : 0;
  L.head_w = take(P * D); L.head_b = take(P);
  L.total = o;
  return L;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---------------------------------------------------------------- scratch of the allocation-free step
// One array per GPU, loaded with the library's code object and held until the process ends.  In host
// code its name is only a stand-in: the device address comes from hipGetSymbolAddress, taken once per
// device with that device current, and only that address is handed to kernels.
static __device__ __align__(256) char scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static char *g_scratch_ptr[kMaxDevices] = {};

hipError_t scratch_base(int device, char **out) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = (char *)p;
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

size_t scratch_layout(const Model *m, int rows, int tokens, int text_rows, char *base, StepBufs *B) {
  const size_t D = m->D, F = m->F, P = m->P, M = (size_t)rows * tokens, a = m->asz;
  size_t off = 0;
  auto carve = [&](size_t bytes) { size_t r = off; off += align256(bytes); return base ? base + r : nullptr; };
  char *h = carve(M * D * 4), *act = carve(M * D * a), *qkv = carve(M * 3 * D * a), *o = carve(M * D * a),
       *u = carve(M * F * a), *tok = carve(M * P * a), *vtok = carve(M * P * 4),
       *txt = carve(m->act == ACT_BF16 ? (size_t)text_rows * m->Dt * a : 0), *ctx = carve((size_t)text_rows * D * a),
       *tf = carve(m->fd * 4), *e1 = carve(D * 4), *e = carve(D * 4), *m6 = carve(6 * D * 4),
       *bm = carve((size_t)m->L * 6 * D * 4), *hm = carve(2 * D * 4), *cond = carve((size_t)rows * 4),
       *rope = carve(m->c.qk_norm_rope ? (size_t)tokens * (m->dh / 2) * 8 : 0),
       *part = carve(m->act == ACT_BF16 ? kSplitBytes : 0);
  if (B) {
    B->h = (float *)h; B->a = act; B->qkv = qkv; B->o = o; B->u = u; B->tok = tok; B->vtok = (float *)vtok;
    B->txt = txt; B->ctx = ctx; B->tf = (float *)tf; B->e1 = (float *)e1; B->e = (float *)e; B->m6 = (float *)m6;
    B->bmods = (float *)bm; B->hmod = (float *)hm; B->d_cond = (int32_t *)cond;
    B->rope = m->c.qk_norm_rope ? (float2 *)rope : nullptr;
    B->part = m->act == ACT_BF16 ? part : nullptr;
    B->part_bytes = m->act == ACT_BF16 ? kSplitBytes : 0;
  }
  return off;
}

}  // namespace fb

using namespace fb;

#define HIPCHK(expr, what)                                                                       \
  do {                                                                                           \
    hipError_t _e = (expr);                                                                      \
    if (_e != hipSuccess) return fail(FLASHBON_EHIP, std::string(what) + ": " + hipGetErrorString(_e)); \
  } while (0)

extern "C" {

const char *flashbon_last_error(void) { return g_err.c_str(); }

size_t flashbon_weight_count(const flashbon_model_config *cfg) {
  if (!config_ok(cfg, nullptr)) return 0;
  return make_layout(*cfg).total;
}

flashbon_status flashbon_plan_step(int32_t num_blocks, const uint8_t *skip, const uint8_t *proxy,
                                   flashbon_cache_meta *meta, float t_cur,
                                   flashbon_trace_entry *trace, int32_t proxy_mode) {
  if (num_blocks < 1) return fail(FLASHBON_ESHAPE, "num_blocks must be >= 1");
  if (!meta || !trace) return fail(FLASHBON_EINVAL, "meta and trace are required");
  if (!std::isfinite(t_cur)) return fail(FLASHBON_EINVAL, "t_cur must be finite");
  for (int l = 0; l < num_blocks; ++l)
    if (!meta_valid(meta[l])) return fail(FLASHBON_ESTATE, "cache meta out of range at block " + std::to_string(l));
  if (proxy_mode != FLASHBON_PROXY_OUTPUT && proxy_mode != FLASHBON_PROXY_RESIDUAL)
    return fail(FLASHBON_EINVAL, "proxy_mode must be 0 or 1");
  plan_step(num_blocks, skip, proxy, meta, t_cur, trace, proxy_mode == FLASHBON_PROXY_RESIDUAL);
  g_err.clear();
  return FLASHBON_OK;
}

flashbon_status flashbon_init_model(const flashbon_model_config *cfg, const float *host_weights,
                                    size_t n_weights, flashbon_model **out) {
  std::string why;
  if (!out) return fail(FLASHBON_EINVAL, "out is NULL");
  *out = nullptr;
  if (!config_ok(cfg, &why)) return fail(cfg ? FLASHBON_ESHAPE : FLASHBON_EINVAL, why);
  if (!host_weights) return fail(FLASHBON_EINVAL, "host_weights is NULL");
  Model *m = new Model();
  m->c = *cfg;
  m->lay = make_layout(*cfg);
  if (n_weights != m->lay.total) {
    size_t want = m->lay.total;
    delete m;
    return fail(FLASHBON_ESHAPE, "n_weights " + std::to_string(n_weights) + " != expected " + std::to_string(want));
  }
  m->act = cfg->dtype == FLASHBON_BF16 ? ACT_BF16 : ACT_F32;
  m->asz = m->act == ACT_BF16 ? 2 : 4;
  m->D = cfg->hidden; m->H = cfg->heads; m->dh = cfg->hidden / cfg->heads; m->F = cfg->mlp_hidden;
  m->C = cfg->latent_channels; m->p = cfg->patch; m->P = m->C * m->p * m->p;
  m->fd = cfg->freq_dim; m->Dt = cfg->text_dim; m->L = cfg->num_blocks;
  m->maxM = (int64_t)cfg->max_n * cfg->max_tokens;
  if (hipGetDevice(&m->device) != hipSuccess) { delete m; return fail(FLASHBON_EHIP, "hipGetDevice"); }

  auto cleanup = [&](flashbon_status st, const std::string &msg) {
    flashbon_free(reinterpret_cast<flashbon_model *>(m));
    // a failed allocation is also recorded as the thread's last HIP error, which the next launch check
    // (hipGetLastError after a launch) would report as that launch's failure: clear it
    if (st == FLASHBON_ENOMEM) (void)hipGetLastError();
    return fail(st, msg);
  };
  const size_t total = m->lay.total;
  if (hipMalloc(&m->w32, total * 4) != hipSuccess) return cleanup(FLASHBON_ENOMEM, "weights (fp32)");
  if (m->act == ACT_BF16 && hipMalloc(&m->w16, total * 2) != hipSuccess)
    return cleanup(FLASHBON_ENOMEM, "weights (bf16)");

  // workspace carve-out
  const size_t D = m->D, F = m->F, P = m->P, M = m->maxM, a = m->asz;
  const size_t txt_rows = (size_t)cfg->max_cond * cfg->max_text_len;
  size_t off = 0;
  auto carve = [&](size_t bytes) { size_t r = off; off += align256(bytes); return r; };
  size_t o_h = carve(M * D * 4), o_a = carve(M * D * a), o_qkv = carve(M * 3 * D * a),
         o_o = carve(M * D * a), o_u = carve(M * F * a), o_tok = carve(M * P * a),
         o_txt = carve(m->act == ACT_BF16 ? txt_rows * m->Dt * a : 0), o_ctx = carve(txt_rows * D * a),
         o_tf = carve(m->fd * 4), o_e1 = carve(D * 4), o_e = carve(D * 4), o_m6 = carve(6 * D * 4),
         o_bm = carve((size_t)m->L * 6 * D * 4), o_hm = carve(2 * D * 4), o_cond = carve(cfg->max_n * 4),
         o_v = carve(M * P * 4),
         o_rope = carve(cfg->qk_norm_rope ? (size_t)cfg->max_tokens * (D / cfg->heads / 2) * 8 : 0),
         o_part = carve(m->act == ACT_BF16 ? kSplitBytes : 0);
  if (hipMalloc(&m->ws, off) != hipSuccess) return cleanup(FLASHBON_ENOMEM, "workspace of " + std::to_string(off) + " bytes");
  m->ws_bytes = off;
  char *w = (char *)m->ws;
  StepBufs &B = m->bufs;
  B.h = (float *)(w + o_h); B.a = w + o_a; B.qkv = w + o_qkv; B.o = w + o_o; B.u = w + o_u;
  B.tok = w + o_tok; B.txt = w + o_txt; B.ctx = w + o_ctx;
  B.tf = (float *)(w + o_tf); B.e1 = (float *)(w + o_e1); B.e = (float *)(w + o_e);
  B.m6 = (float *)(w + o_m6); B.bmods = (float *)(w + o_bm); B.hmod = (float *)(w + o_hm);
  B.d_cond = (int32_t *)(w + o_cond); B.vtok = (float *)(w + o_v);
  if (cfg->qk_norm_rope) B.rope = (float2 *)(w + o_rope);
  if (m->act == ACT_BF16) { B.part = w + o_part; B.part_bytes = kSplitBytes; }
  // the allocation-free step's scratch array of this device: its address, once per device
  {
    char *base = nullptr;
    hipError_t e = scratch_base(m->device, &base);
    if (e != hipSuccess) return cleanup(FLASHBON_EHIP, std::string("scratch address: ") + hipGetErrorString(e));
  }

  if (hipMemcpy(m->w32, host_weights, total * 4, hipMemcpyHostToDevice) != hipSuccess)
    return cleanup(FLASHBON_EHIP, "weight upload");
  if (m->act == ACT_BF16) {
    if (launch_f32_to_bf16((int64_t)total, m->w32, m->w16, 0) != hipSuccess)
      return cleanup(FLASHBON_EHIP, "weight conversion");
  }
  if (hipDeviceSynchronize() != hipSuccess) return cleanup(FLASHBON_EHIP, "init synchronise");
  *out = reinterpret_cast<flashbon_model *>(m);
  g_err.clear();
  return FLASHBON_OK;
}

void flashbon_free(flashbon_model *model) {
  if (!model) return;
  Model *m = reinterpret_cast<Model *>(model);
  (void)hipDeviceSynchronize();
  for (auto &site : m->sites)
    for (auto &pr : site.pending) { (void)hipEventDestroy(pr.first); (void)hipEventDestroy(pr.second); }
  for (hipEvent_t e : m->spare_events) (void)hipEventDestroy(e);
  if (m->w32) (void)hipFree(m->w32);
  if (m->w16) (void)hipFree(m->w16);
  if (m->ws) (void)hipFree(m->ws);
  delete m;
}

size_t flashbon_text_kv_bytes(const flashbon_model *model, int32_t n_cond, int32_t text_len) {
  if (!model || n_cond < 1 || text_len < 1) return 0;
  const Model *m = reinterpret_cast<const Model *>(model);
  return (size_t)m->L * n_cond * text_len * 2 * m->D * m->asz;
}

size_t flashbon_cache_bytes(const flashbon_model *model, int32_t n, int32_t tokens) {
  if (!model || n < 1 || tokens < 1) return 0;
  const Model *m = reinterpret_cast<const Model *>(model);
  return (size_t)m->L * 3 * n * tokens * m->D * 4;
}

}  // extern "C"

namespace fb {

static hipError_t take_event(Model *m, hipEvent_t *e) {
  if (!m->spare_events.empty()) {
    *e = m->spare_events.back();
    m->spare_events.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}

// Drain the finished event pairs of one site into its totals.
static hipError_t harvest(Model *m, int site) {
  Model::Site &st = m->sites[site];
  for (auto &pr : st.pending) {
    hipError_t e = hipEventSynchronize(pr.second);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, pr.first, pr.second);
    if (e != hipSuccess) return e;
    st.total_ms += ms;
    st.launches += 1;
    m->spare_events.push_back(pr.first);
    m->spare_events.push_back(pr.second);
  }
  st.pending.clear();
  return hipSuccess;
}

// Run `launch` (returning hipError_t), bracketed by events when the site is timed.
template <typename F>
static hipError_t timed(Model *m, uint32_t mask, int site, hipStream_t s, F &&launch) {
  if (!(mask & (1u << site))) return launch();
  hipEvent_t e0, e1;
  hipError_t e = take_event(m, &e0);
  if (e == hipSuccess) e = take_event(m, &e1);
  if (e != hipSuccess) return e;
  if ((e = hipEventRecord(e0, s)) != hipSuccess) return e;
  if ((e = launch()) != hipSuccess) return e;
  if ((e = hipEventRecord(e1, s)) != hipSuccess) return e;
  m->sites[site].pending.emplace_back(e0, e1);
  if (m->sites[site].pending.size() > 65536) return harvest(m, site);
  return hipSuccess;
}

static flashbon_status run_step(Model *m, const flashbon_step_args *a, bool draft, bool noalloc = false) {
  if (!m) return fail(FLASHBON_EINVAL, "model is NULL");
  if (!a) return fail(FLASHBON_EINVAL, "args is NULL");
  const flashbon_model_config &c = m->c;
  const int L = m->L, D = m->D, F = m->F, P = m->P, p = m->p;
  // ---------------------------------------------------------------- validation (no side effects)
  const bool guided = a->cfg != 0;
  const int R = guided ? 2 * a->n : a->n;   // token rows through the network (twins when guided)
  if (a->n < 1 || R > c.max_n) return fail(FLASHBON_ESHAPE, guided ? "2n outside [2, max_n]" : "n outside [1, max_n]");
  if (guided && (!a->uncond_index || !std::isfinite(a->cfg_scale)))
    return fail(FLASHBON_EINVAL, "guidance needs uncond_index and a finite cfg_scale");
  if (a->latent_h < p || a->latent_w < p || a->latent_h % p || a->latent_w % p)
    return fail(FLASHBON_ESHAPE, "latent_h/latent_w must be positive multiples of patch");
  const int64_t T64 = (int64_t)(a->latent_h / p) * (a->latent_w / p);
  if (T64 > c.max_tokens) return fail(FLASHBON_ESHAPE, "tokens exceed max_tokens");
  const int T = (int)T64;
  const int64_t M = (int64_t)R * T;
  if (!a->latents) return fail(FLASHBON_EINVAL, "latents is NULL");
  if (a->preview && a->preview == a->latents) return fail(FLASHBON_EINVAL, "preview must not alias latents");
  if (!std::isfinite(a->t_cur) || !std::isfinite(a->t_next)) return fail(FLASHBON_EINVAL, "t_cur/t_next must be finite");
  if (!a->text || !a->cond_index || !a->text_kv || !a->text_kv_valid)
    return fail(FLASHBON_EINVAL, "text, cond_index, text_kv and text_kv_valid are required");
  if (a->n_cond < 1 || a->n_cond > c.max_cond) return fail(FLASHBON_ESHAPE, "n_cond outside [1, max_cond]");
  if (a->text_len < 1 || a->text_len > c.max_text_len) return fail(FLASHBON_ESHAPE, "text_len outside [1, max_text_len]");
  for (int i = 0; i < a->n; ++i)
    if (a->cond_index[i] < 0 || a->cond_index[i] >= a->n_cond)
      return fail(FLASHBON_EINVAL, "cond_index[" + std::to_string(i) + "] outside [0, n_cond)");
  if (guided)
    for (int i = 0; i < a->n; ++i)
      if (a->uncond_index[i] < 0 || a->uncond_index[i] >= a->n_cond)
        return fail(FLASHBON_EINVAL, "uncond_index[" + std::to_string(i) + "] outside [0, n_cond)");
  if (a->proxy_mode != FLASHBON_PROXY_OUTPUT && a->proxy_mode != FLASHBON_PROXY_RESIDUAL)
    return fail(FLASHBON_EINVAL, "proxy_mode must be 0 or 1");
  const bool residual = draft && a->proxy_mode == FLASHBON_PROXY_RESIDUAL;
  if (draft) {
    if (!a->meta) return fail(FLASHBON_EINVAL, "draft step needs meta");
    if (!a->cache) return fail(FLASHBON_EINVAL, "draft step needs cache");
    for (int l = 0; l < L; ++l)
      if (!meta_valid(a->meta[l])) return fail(FLASHBON_ESTATE, "cache meta out of range at block " + std::to_string(l));
  }
  std::vector<flashbon_cache_meta> meta_new(L);
  std::vector<flashbon_trace_entry> trace(L);
  if (draft) {
    std::memcpy(meta_new.data(), a->meta, sizeof(flashbon_cache_meta) * L);
    plan_step(L, a->skip, a->proxy, meta_new.data(), a->t_cur, trace.data(), residual);
  } else {
    std::vector<flashbon_cache_meta> z(L);
    std::memset(z.data(), 0, sizeof(flashbon_cache_meta) * L);
    plan_step(L, nullptr, nullptr, z.data(), a->t_cur, trace.data());
  }
  std::vector<float> ca(L, 0.f), cb(L, 0.f);
  for (int l = 0; l < L; ++l) {
    if (trace[l].action != FLASHBON_PROXY || !trace[l].live) continue;
    const flashbon_cache_meta &mb = a->meta[l];
    if (trace[l].order >= 1) {
      float t1 = mb.t[(mb.head + 2) % 3], t2 = mb.t[(mb.head + 1) % 3];
      if (!(t1 != t2) || !std::isfinite(t1) || !std::isfinite(t2))
        return fail(FLASHBON_ESTATE, "cached timesteps of block " + std::to_string(l) + " coincide or are not finite");
    }
    taylor_coefficients(mb, a->t_cur, trace[l].order, &ca[l], &cb[l]);
  }
  SdeArgs sde;
  const bool stochastic = a->sde_a != 0.f;
  if (stochastic && (a->sde_step < 0 || a->sde_row0 < 0))
    return fail(FLASHBON_EINVAL, "sde_step and sde_row0 must be >= 0");
  if (stochastic && !sde_coefficients(a->t_cur, a->t_next, a->sde_a, a->sde_seed, a->sde_step, a->sde_row0, &sde))
    return fail(FLASHBON_EINVAL, "stochastic update needs sde_a >= 0, finite, and 0 < t_cur <= 1 (t_next < 1 when t_cur = 1)");

  // the step's working buffers: the model workspace, or this device's scratch array (sized for this call)
  StepBufs B = m->bufs;
  const uint32_t tmask = noalloc ? 0u : m->timing_mask;
  if (noalloc) {
    if (R > kMaxScratchRows) return fail(FLASHBON_ESHAPE, "allocation-free step: more than 128 token rows of candidates");
    const size_t need = scratch_layout(m, R, T, *a->text_kv_valid ? 0 : a->n_cond * a->text_len, nullptr, nullptr);
    if (need > kScratchBytes)
      return fail(FLASHBON_ESHAPE, "allocation-free step needs " + std::to_string(need) + " bytes of scratch, the limit is " +
                                       std::to_string(kScratchBytes));
    int dev = -1;
    HIPCHK(hipGetDevice(&dev), "hipGetDevice");
    if (dev != m->device) return fail(FLASHBON_EINVAL, "allocation-free step: the model's device must be current");
    char *base = nullptr;
    HIPCHK(scratch_base(dev, &base), "scratch address");
    scratch_layout(m, R, T, *a->text_kv_valid ? 0 : a->n_cond * a->text_len, base, &B);
  }

  // linear layers: split-K (with its partial sums in this step's buffers) where the plan asks for it
  auto lin = [&](ActType t_, int epi_, int M_, int N_, int K_, const void *A_, const void *W_, const EpiArgs &e_,
                 hipStream_t s_) { return launch_linear_ws(t_, epi_, M_, N_, K_, A_, W_, e_, s_, B.part, B.part_bytes); };

  // ---------------------------------------------------------------- enqueue
  hipStream_t s = (hipStream_t)a->stream;
  const ActType act = m->act;
  const size_t asz = m->asz;
  auto Wp = [&](size_t off) -> const void * {
    return act == ACT_BF16 ? (const void *)((const char *)m->w16 + off * 2) : (const void *)(m->w32 + off);
  };
  auto Bp = [&](size_t off) -> const float * { return m->w32 + off; };

  // cond_index -> device.  Model workspace: only when it changed (the previous step may still read the
  // old copy).  Scratch: every call, as kernel arguments (no host memory outlives the call).
  std::vector<int32_t> cond(a->cond_index, a->cond_index + a->n);
  if (guided) cond.insert(cond.end(), a->uncond_index, a->uncond_index + a->n);
  if (noalloc) {
    HIPCHK(launch_store_i32((int)cond.size(), cond.data(), B.d_cond, s), "cond_index upload");
  } else if (cond != m->last_cond) {
    HIPCHK(hipStreamSynchronize(s), "synchronise before cond_index upload");
    HIPCHK(hipMemcpy(B.d_cond, cond.data(), sizeof(int32_t) * cond.size(), hipMemcpyHostToDevice), "cond_index upload");
    m->last_cond = cond;
  }

  const int Lt = a->text_len, NC = a->n_cond;
  const int64_t kv_block = (int64_t)NC * Lt * 2 * D;  // elements per block in text_kv
  if (*a->text_kv_valid == 0) {
    const void *txt = a->text;
    if (act == ACT_BF16) {
      HIPCHK(timed(m, tmask, FLASHBON_SITE_TEXT, s, [&] { return launch_f32_to_bf16((int64_t)NC * Lt * m->Dt, a->text, B.txt, s); }), "text convert");
      txt = B.txt;
    }
    EpiArgs e;
    e.out = B.ctx; e.ldo = D; e.bias = Bp(m->lay.txt_b);
    HIPCHK(timed(m, tmask, FLASHBON_SITE_TEXT, s, [&] { return lin(act, EPI_STORE, NC * Lt, D, m->Dt, txt, Wp(m->lay.txt_w), e, s); }), "text projection");
    for (int l = 0; l < L; ++l) {
      EpiArgs k;
      k.out = (char *)a->text_kv + (size_t)l * kv_block * asz; k.ldo = 2 * D; k.bias = Bp(m->lay.blk[l].bkvc);
      HIPCHK(timed(m, tmask, FLASHBON_SITE_TEXT, s, [&] { return lin(act, EPI_STORE, NC * Lt, 2 * D, D, B.ctx, Wp(m->lay.blk[l].wkvc), k, s); }), "text K/V");
      if (c.qk_norm_rope)
        HIPCHK(timed(m, tmask, FLASHBON_SITE_TEXT, s, [&] { return launch_qk_norm(act, NC * Lt, D, m->dh, k.out, 2 * D, Bp(m->lay.blk[l].nkc), c.ln_eps, nullptr, 1, s); }),
               "text key RMSNorm");
    }
  }

  // timestep conditioning, shared by all candidates
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_time_features((double)a->t_cur, m->fd, B.tf, s); }), "time features");
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_gemv(D, m->fd, m->w32 + m->lay.t_w1, Bp(m->lay.t_b1), B.tf, B.e1, 0, 1, s); }), "time mlp 1");
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_gemv(D, D, m->w32 + m->lay.t_w2, Bp(m->lay.t_b2), B.e1, B.e, 0, 0, s); }), "time mlp 2");
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_gemv(6 * D, D, m->w32 + m->lay.mod_w, Bp(m->lay.mod_b), B.e, B.m6, 1, 0, s); }), "modulation");
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_gemv(2 * D, D, m->w32 + m->lay.hmod_w, Bp(m->lay.hmod_b), B.e, B.hmod, 1, 0, s); }), "head modulation");
  HIPCHK(timed(m, tmask, FLASHBON_SITE_TIME, s, [&] { return launch_block_mods(L, 6 * D, B.m6, m->w32 + m->lay.blk[0].mod, (int64_t)m->lay.block_stride, B.bmods, s); }),
         "block modulation");

  // rotary table of this latent size (kept in the model workspace while the size does not change; made
  // on every call in scratch)
  if (c.qk_norm_rope && (noalloc || m->rope_h != a->latent_h || m->rope_w != a->latent_w)) {
    HIPCHK(launch_rope_table(T, a->latent_w / p, m->dh, B.rope, s), "rotary table");
    if (!noalloc) {
      m->rope_h = a->latent_h;
      m->rope_w = a->latent_w;
    }
  }

  const int64_t MD = M * D;
  // Where the residual stream currently lives.  A computed block of a draft step (output reading of
  // the proxy) writes its new rows only into its cache slot, which then serves as the stream until the
  // next block writes: the next computed block reads it there and its self-attention output
  // projection writes the updated rows back into B.h; a proxy writes B.h; a skip leaves it.  This
  // saves the second copy of every computed block's output.
  const float *hcur = B.h;
  auto dump = [&](int idx) -> flashbon_status {
    if (!a->hidden_dump) return FLASHBON_OK;
    HIPCHK(hipMemcpyAsync(a->hidden_dump + (int64_t)idx * MD, hcur, MD * 4, hipMemcpyDeviceToDevice, s), "hidden dump");
    return FLASHBON_OK;
  };
  flashbon_status st;

  // patch embedding, unless the first non-skipped block is a proxy (its input is then never read)
  bool embed_live = true;
  for (int l = 0; l < L && !residual; ++l)
    if (trace[l].action != FLASHBON_SKIP) { embed_live = trace[l].action == FLASHBON_COMPUTE; break; }
  // `formed`: the stream buffer holds this step's value at the current point of the block loop.  It is
  // false from an elided embedding or a dead proxy up to the next launched proxy, and the hidden-state
  // dump then leaves those entries untouched (their values are never formed).
  bool formed = embed_live;
  if (embed_live) {
    HIPCHK(timed(m, tmask, FLASHBON_SITE_EMBED, s, [&] { return launch_patchify(act, R, a->n, m->C, a->latent_h, a->latent_w, p, a->latents, B.tok, s); }), "patchify");
    EpiArgs e;
    e.out = B.h; e.ldo = D; e.bias = Bp(m->lay.pe_b);
    HIPCHK(timed(m, tmask, FLASHBON_SITE_EMBED, s, [&] { return lin(act, EPI_STORE_F32, (int)M, D, P, B.tok, Wp(m->lay.pe_w), e, s); }), "patch embed");
    if ((st = dump(0)) != FLASHBON_OK) return st;
  }

  const int H = m->H, dh = m->dh;
  for (int l = 0; l < L; ++l) {
    const flashbon_trace_entry &tr = trace[l];
    const BlockOff &b = m->lay.blk[l];
    const float *mod = B.bmods + (int64_t)l * 6 * D;
    if (tr.action == FLASHBON_SKIP) {
      if (formed && (st = dump(l + 1)) != FLASHBON_OK) return st;
      continue;
    }
    if (tr.action == FLASHBON_PROXY) {
      if (!tr.live) {
        formed = false;
        continue;
      }
      const flashbon_cache_meta &mb = a->meta[l];
      const int s1 = (mb.head + 2) % 3, s2 = (mb.head + 1) % 3, s3 = mb.head;
      auto slot_ptr = [&](int sl) { return a->cache + ((int64_t)l * 3 + sl) * MD; };
      HIPCHK(timed(m, tmask, FLASHBON_SITE_PROXY, s, [&] { return launch_proxy(MD, slot_ptr(s1), slot_ptr(s2), slot_ptr(s3), tr.order, ca[l], cb[l], B.h, s, residual); }),
             "activation proxy");
      hcur = B.h;
      formed = true;
      if ((st = dump(l + 1)) != FLASHBON_OK) return st;
      continue;
    }
    // COMPUTE (Eq. 7); the residual reading first keeps the block input in its cache slot, which the
    // down-projection epilogue turns into the block's delta
    if (residual)
      HIPCHK(hipMemcpyAsync(a->cache + ((int64_t)l * 3 + tr.slot) * MD, B.h, MD * 4, hipMemcpyDeviceToDevice, s),
             "block input to cache");
    HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_ln_mod(act, (int)M, D, c.ln_eps, hcur, mod + 0 * D, mod + 1 * D, B.a, s); }), "adaLN 1");
    {
      EpiArgs e; e.out = B.qkv; e.ldo = 3 * D; e.bias = Bp(b.bqkv);
      HIPCHK(timed(m, tmask, FLASHBON_SITE_QKV, s, [&] { return lin(act, EPI_STORE, (int)M, 3 * D, D, B.a, Wp(b.wqkv), e, s); }), "qkv projection");
    }
    if (c.qk_norm_rope) {
      void *kp = (char *)B.qkv + (size_t)D * asz;
      HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_qk_norm(act, (int)M, D, dh, B.qkv, 3 * D, Bp(b.nq), c.ln_eps, B.rope, T, s); }), "q RMSNorm + rotary");
      HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_qk_norm(act, (int)M, D, dh, kp, 3 * D, Bp(b.nk), c.ln_eps, B.rope, T, s); }), "k RMSNorm + rotary");
    }
    {
      AttnArgs at;
      at.batch = R; at.heads = H; at.head_dim = dh; at.tq = T; at.tk = T;
      at.q = B.qkv; at.q_bs = (int64_t)T * 3 * D; at.q_rs = 3 * D;
      at.k = (const char *)B.qkv + (size_t)D * asz; at.v = (const char *)B.qkv + (size_t)2 * D * asz;
      at.kv_bs = (int64_t)T * 3 * D; at.kv_rs = 3 * D; at.kv_index = nullptr; at.n_kv = R;
      at.out = B.o; at.o_bs = (int64_t)T * D; at.o_rs = D;
      HIPCHK(timed(m, tmask, FLASHBON_SITE_ATTN_SELF, s, [&] { return launch_attention(act, at, s); }), "self-attention");
    }
    {
      EpiArgs e; e.out = B.h; e.ldo = D; e.bias = Bp(b.bo); e.gate = mod + 2 * D;
      if (hcur != B.h) e.res_in = hcur;
      HIPCHK(timed(m, tmask, FLASHBON_SITE_OUT, s, [&] { return lin(act, EPI_RESIDUAL, (int)M, D, D, B.o, Wp(b.wo), e, s); }), "self-attn out projection");
      hcur = B.h;
    }
    HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_ln_mod(act, (int)M, D, c.ln_eps, B.h, nullptr, nullptr, B.a, s); }), "cross LN");
    {
      EpiArgs e; e.out = B.qkv; e.ldo = D; e.bias = Bp(b.bqc);
      HIPCHK(timed(m, tmask, FLASHBON_SITE_CROSS_Q, s, [&] { return lin(act, EPI_STORE, (int)M, D, D, B.a, Wp(b.wqc), e, s); }), "cross q projection");
    }
    if (c.qk_norm_rope)
      HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_qk_norm(act, (int)M, D, dh, B.qkv, D, Bp(b.nqc), c.ln_eps, nullptr, T, s); }), "cross q RMSNorm");
    {
      const char *kv = (const char *)a->text_kv + (size_t)l * kv_block * asz;
      AttnArgs at;
      at.batch = R; at.heads = H; at.head_dim = dh; at.tq = T; at.tk = Lt;
      at.q = B.qkv; at.q_bs = (int64_t)T * D; at.q_rs = D;
      at.k = kv; at.v = kv + (size_t)D * asz; at.kv_bs = (int64_t)Lt * 2 * D; at.kv_rs = 2 * D;
      at.kv_index = B.d_cond; at.n_kv = NC;
      at.out = B.o; at.o_bs = (int64_t)T * D; at.o_rs = D;
      HIPCHK(timed(m, tmask, FLASHBON_SITE_ATTN_CROSS, s, [&] { return launch_attention(act, at, s); }), "cross-attention");
    }
    {
      EpiArgs e; e.out = B.h; e.ldo = D; e.bias = Bp(b.boc);
      HIPCHK(timed(m, tmask, FLASHBON_SITE_OUT_CROSS, s, [&] { return lin(act, EPI_RESIDUAL, (int)M, D, D, B.o, Wp(b.woc), e, s); }), "cross out projection");
    }
    HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_ln_mod(act, (int)M, D, c.ln_eps, B.h, mod + 3 * D, mod + 4 * D, B.a, s); }), "adaLN 2");
    {
      EpiArgs e; e.out = B.u; e.ldo = F; e.bias = Bp(b.b1);
      HIPCHK(timed(m, tmask, FLASHBON_SITE_MLP_UP, s, [&] { return lin(act, EPI_GELU, (int)M, F, D, B.a, Wp(b.w1), e, s); }), "mlp up");
    }
    {
      EpiArgs e; e.out = B.h; e.ldo = D; e.bias = Bp(b.b2); e.gate = mod + 5 * D;
      float *slot = draft ? a->cache + ((int64_t)l * 3 + tr.slot) * MD : nullptr;
      if (slot && !residual) {   // the new rows go to the cache slot only, which becomes the stream
        e.out = slot;
        e.res_in = B.h;
      } else {
        e.cache = slot;
        e.cache_delta = residual;
      }
      HIPCHK(timed(m, tmask, FLASHBON_SITE_MLP_DOWN, s, [&] { return lin(act, EPI_RESIDUAL, (int)M, D, F, B.u, Wp(b.w2), e, s); }), "mlp down");
      hcur = (const float *)e.out;
    }
    if ((st = dump(l + 1)) != FLASHBON_OK) return st;
  }

  // head + unpatchify + Euler update of the latents (or the stochastic update of Eq. 20)
  HIPCHK(timed(m, tmask, FLASHBON_SITE_NORM, s, [&] { return launch_ln_mod(act, (int)M, D, c.ln_eps, hcur, B.hmod, B.hmod + D, B.a, s); }), "head adaLN");
  if (stochastic || guided) {
    if (!stochastic) {                      // Euler update through the same kernel: no drift term, no noise
      sde = SdeArgs{};
      sde.dt = a->t_next - a->t_cur;
    }
    EpiArgs e;
    e.out = B.vtok; e.ldo = P; e.bias = Bp(m->lay.head_b);
    HIPCHK(timed(m, tmask, FLASHBON_SITE_HEAD, s, [&] { return lin(act, EPI_STORE_F32, (int)M, P, D, B.a, Wp(m->lay.head_w), e, s); }), "head");
    HIPCHK(timed(m, tmask, FLASHBON_SITE_HEAD, s, [&] { return launch_head_update(a->n, m->C, a->latent_h, a->latent_w, p, B.vtok, guided, a->cfg_scale, a->latents, sde, a->preview, a->t_cur, s); }),
           "unpatchify + guidance + update");
  } else {
    EpiArgs e;
    e.bias = Bp(m->lay.head_b); e.z = a->latents; e.dt = a->t_next - a->t_cur;
    e.preview = a->preview; e.t_cur = a->t_cur;
    e.C = m->C; e.H = a->latent_h; e.W = a->latent_w; e.p = p; e.T = T;
    HIPCHK(timed(m, tmask, FLASHBON_SITE_HEAD, s, [&] { return lin(act, EPI_EULER, (int)M, P, D, B.a, Wp(m->lay.head_w), e, s); }), "head + Euler");
  }

  // ---------------------------------------------------------------- commit host state
  if (draft) std::memcpy(a->meta, meta_new.data(), sizeof(flashbon_cache_meta) * L);
  if (a->trace) std::memcpy(a->trace, trace.data(), sizeof(flashbon_trace_entry) * L);
  *a->text_kv_valid = 1;
  g_err.clear();
  return FLASHBON_OK;
}

}  // namespace fb

extern "C" {

flashbon_status flashbon_draft_step(flashbon_model *model, const flashbon_step_args *args) {
  return run_step(reinterpret_cast<Model *>(model), args, true);
}

flashbon_status flashbon_refine_step(flashbon_model *model, const flashbon_step_args *args) {
  return run_step(reinterpret_cast<Model *>(model), args, false);
}

flashbon_status flashbon_refine_step_noalloc(flashbon_model *model, const flashbon_step_args *args) {
  return run_step(reinterpret_cast<Model *>(model), args, false, true);
}

flashbon_status flashbon_set_timing(flashbon_model *model, uint32_t site_mask) {
  if (!model) return fail(FLASHBON_EINVAL, "model is NULL");
  if (site_mask >> FLASHBON_NUM_SITES) return fail(FLASHBON_EINVAL, "unknown site in mask");
  reinterpret_cast<Model *>(model)->timing_mask = site_mask;
  g_err.clear();
  return FLASHBON_OK;
}

flashbon_status flashbon_read_timing(flashbon_model *model, int32_t site, double *total_ms, int64_t *launches) {
  if (!model || !total_ms || !launches) return fail(FLASHBON_EINVAL, "model, total_ms and launches are required");
  if (site < 0 || site >= FLASHBON_NUM_SITES) return fail(FLASHBON_EINVAL, "unknown site");
  Model *m = reinterpret_cast<Model *>(model);
  HIPCHK(harvest(m, site), "timing events");
  *total_ms = m->sites[site].total_ms;
  *launches = m->sites[site].launches;
  m->sites[site].total_ms = 0;
  m->sites[site].launches = 0;
  g_err.clear();
  return FLASHBON_OK;
}

}  // extern "C"
