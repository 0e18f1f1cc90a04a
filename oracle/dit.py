"""Oracle: a plain fp64 CPU implementation of one masked/proxied DiT denoising step of Flash-BoN.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never links, imports or calls it, and it
shares no code with the HIP path; both take their inputs from the seeded generators.

What it follows:
  * the denoising recursion z_{t_{i-1}} = f_theta(z_{t_i}, x, t_i) and its truncation to the first S'
    steps (Sec. 4.1 (1), Eq. 2);
  * activation proxies by second-order Taylor expansion with finite-difference derivatives from cached
    block outputs (Sec. 4.1 (2), Eq. 3-5), computed exactly as printed;
  * layer skipping: a skipped block is the identity on the residual stream (Sec. 4.1 (3), Eq. 6);
    a computed block is h = B_l(h, x, t) (Eq. 7);
  * the flow-matching update: the Euler-Maruyama rule of App. A.1 (Eq. 20) with a = 0, i.e.
    z <- z + (t_next - t_cur) * v; optionally the stochastic rule with a > 0 (oracle/sde.py);
  * refinement resumes from the draft's latent with every knob off (Sec. 4.2, Stage 3, Eq. 13).

The paper does not describe the DiT block.  The block used here (and by the library) is a Wan-shaped
DiT block -- our reading: adaLN-modulated self-attention with a gate, cross-attention to projected
text tokens, and an adaLN-modulated tanh-GELU MLP with a gate; non-affine LayerNorm (eps 1e-6);
sinusoidal timestep features of 1000 t; no positional encoding.

Parity pins: every function here is checked in ``tests/test_oracle_*.py`` against closed forms,
invariants, brute force on tiny inputs or values fixed by the paper.  The block's internal algebra
(LayerNorm, GELU, modulation, projections) is pinned only by textbook definitions, since the paper
gives none.

Precision: float64 everywhere; float32 inputs are widened, never narrowed.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .dispatch import COMPUTE, PROXY, SKIP, plan_step, recent_slots
from . import sde

f64 = np.float64


# ----------------------------------------------------------------------------- elementary operations

def linear(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y = x W^T + b with W stored [out, in]."""
    return x @ np.asarray(w, f64).T + np.asarray(b, f64)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """tanh approximation of GELU."""
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """Non-affine LayerNorm over the last axis (biased variance)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Single-head softmax(q k^T / sqrt(d)) v, with the row maximum subtracted before exp."""
    d = q.shape[-1]
    s = (q @ k.T) / np.sqrt(d)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def multi_head_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """q [Tq, D], k/v [Tk, D]; head h uses columns h*dh .. (h+1)*dh - 1."""
    D = q.shape[-1]
    dh = D // heads
    out = np.empty((q.shape[0], D), f64)
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        out[:, sl] = attention(q[:, sl], k[:, sl], v[:, sl])
    return out


def timestep_features(t: float, freq_dim: int) -> np.ndarray:
    """[cos(1000 t w_j) | sin(1000 t w_j)], w_j = 10000^(-j/half), j < half = freq_dim / 2."""
    half = freq_dim // 2
    tau = 1000.0 * f64(t)
    w = np.power(10000.0, -np.arange(half, dtype=f64) / half)
    return np.concatenate([np.cos(tau * w), np.sin(tau * w)])


# ----------------------------------------------------------------------------- model pieces

def modulations(W: Dict[str, np.ndarray], num_blocks: int, freq_dim: int, t: float
                ) -> Tuple[np.ndarray, np.ndarray]:
    """Timestep conditioning shared by every candidate.

    Returns (block_mod [L, 6, D], head_mod [2, D]); block_mod[l] = (shift1, scale1, gate1, shift2,
    scale2, gate2), head_mod = (shift, scale).
    """
    f = timestep_features(t, freq_dim)
    e = linear(silu(linear(f, W["t_w1"], W["t_b1"])), W["t_w2"], W["t_b2"])
    m = linear(silu(e), W["mod_w"], W["mod_b"])
    D = e.shape[0]
    block_mod = np.stack([(m + np.asarray(W[f"blk{l}.mod"], f64).reshape(-1)).reshape(6, D)
                          for l in range(num_blocks)])
    head_mod = linear(silu(e), W["head_mod_w"], W["head_mod_b"]).reshape(2, D)
    return block_mod, head_mod


def patchify(z: np.ndarray, p: int) -> np.ndarray:
    """One candidate's latent [C, H, W] -> tokens [(H/p)(W/p), C p p].

    Token i*(W/p) + j takes the p x p patch at rows p i.., cols p j..; feature c p^2 + p di + dj holds
    z[c, p i + di, p j + dj].
    """
    C, H, Wd = z.shape
    x = z.reshape(C, H // p, p, Wd // p, p)          # c, i, di, j, dj
    x = x.transpose(1, 3, 0, 2, 4)                   # i, j, c, di, dj
    return x.reshape((H // p) * (Wd // p), C * p * p)


def unpatchify(tok: np.ndarray, C: int, H: int, Wd: int, p: int) -> np.ndarray:
    """Inverse of :func:`patchify`: tokens [T, C p p] -> [C, H, W]."""
    x = tok.reshape(H // p, Wd // p, C, p, p)        # i, j, c, di, dj
    x = x.transpose(2, 0, 3, 1, 4)                   # c, i, di, j, dj
    return x.reshape(C, H, Wd)


def text_kv(W: Dict[str, np.ndarray], num_blocks: int, text: np.ndarray, eps: float = 1e-6
            ) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Per-block cross-attention keys/values of one prompt: ctx = text W_txt^T + b; K, V = ctx W^T + b
    (K RMS-normalised with its gain when the model has qk RMSNorm, reading R26)."""
    ctx = linear(np.asarray(text, f64), W["txt_w"], W["txt_b"])
    out = []
    for l in range(num_blocks):
        k = linear(ctx, W[f"blk{l}.wkc"], W[f"blk{l}.bkc"])
        if f"blk{l}.nkc" in W:
            k = rms_norm(k, W[f"blk{l}.nkc"], eps)
        out.append((k, linear(ctx, W[f"blk{l}.wvc"], W[f"blk{l}.bvc"])))
    return out


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis (textbook RMSNorm)."""
    x = np.asarray(x, f64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + f64(eps)) * np.asarray(g, f64)


def rope_bands(dh: int) -> Tuple[int, int, int]:
    """Head-dim split of the 3-D rotary embedding: (frame, height, width) bands; reading R26."""
    q = dh // 6
    return dh - 4 * q, 2 * q, 2 * q


def rope_angles(hp: int, wp: int, dh: int, theta: float = 10000.0) -> np.ndarray:
    """[T, dh/2] rotation angles of tokens t = i wp + j at position (frame 0, row i, column j): pair k of
    a band of width d at position p turns by p theta^(-2k/d); bands in frame, height, width order."""
    fb_, hb, wb = rope_bands(dh)
    T = hp * wp
    pos = np.stack([np.zeros(T), np.arange(T) // wp, np.arange(T) % wp], axis=1).astype(f64)
    cols = []
    for band, d in enumerate((fb_, hb, wb)):
        freq = f64(theta) ** (-np.arange(0, d, 2, dtype=f64) / d)
        cols.append(pos[:, band:band + 1] * freq[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(x: np.ndarray, angles: np.ndarray, heads: int) -> np.ndarray:
    """Rotate consecutive pairs (2k, 2k + 1) of every head of x [T, D] by angles [T, dh/2]."""
    x = np.asarray(x, f64)
    T, D = x.shape
    dh = D // heads
    xr = x.reshape(T, heads, dh // 2, 2)
    c, s = np.cos(angles)[:, None, :], np.sin(angles)[:, None, :]
    out = np.empty_like(xr)
    out[..., 0] = xr[..., 0] * c - xr[..., 1] * s
    out[..., 1] = xr[..., 0] * s + xr[..., 1] * c
    return out.reshape(T, D)


def block_forward(W: Dict[str, np.ndarray], l: int, h: np.ndarray, mod: np.ndarray,
                  kv: Tuple[np.ndarray, np.ndarray], heads: int, eps: float,
                  angles: Optional[np.ndarray] = None) -> np.ndarray:
    """B_l(h, x, t) (Eq. 7) for one candidate; h [T, D], mod [6, D] -> new residual stream [T, D].

    With qk RMSNorm weights in W (reading R26): q and k of both attentions are RMS-normalised over D
    with their gains, and self-attention's q and k are then rotated by ``angles`` (3-D RoPE); the text
    keys in ``kv`` are normalised where they are made (``text_kv``)."""
    b = f"blk{l}."
    qkn = (b + "nq") in W
    sh1, sc1, g1, sh2, sc2, g2 = mod
    a = layer_norm(h, eps) * (1.0 + sc1) + sh1
    q = linear(a, W[b + "wq"], W[b + "bq"])
    k = linear(a, W[b + "wk"], W[b + "bk"])
    v = linear(a, W[b + "wv"], W[b + "bv"])
    if qkn:
        q = apply_rope(rms_norm(q, W[b + "nq"], eps), angles, heads)
        k = apply_rope(rms_norm(k, W[b + "nk"], eps), angles, heads)
    o = multi_head_attention(q, k, v, heads)
    h = h + g1 * linear(o, W[b + "wo"], W[b + "bo"])
    c = layer_norm(h, eps)
    qc = linear(c, W[b + "wqc"], W[b + "bqc"])
    if qkn:
        qc = rms_norm(qc, W[b + "nqc"], eps)
    oc = multi_head_attention(qc, kv[0], kv[1], heads)
    h = h + linear(oc, W[b + "woc"], W[b + "boc"])
    a = layer_norm(h, eps) * (1.0 + sc2) + sh2
    u = gelu_tanh(linear(a, W[b + "w1"], W[b + "b1"]))
    h = h + g2 * linear(u, W[b + "w2"], W[b + "b2"])
    return h


def taylor_proxy(entries: Sequence[Tuple[np.ndarray, float]], t_cur: float, order: int) -> np.ndarray:
    """Activation proxy of Eq. 3-5.

    ``entries`` are (h, tau) of the block's cached outputs, most recent first, so tau_1 < tau_2 < ...
    (denoising runs from high to low t).  With Delta = t_cur - tau_1:
      hdot  = (h1 - h2) / (tau_1 - tau_2)                        (Eq. 3)
      hddot = (h1 - 2 h2 + h3) / (tau_1 - tau_2)^2               (Eq. 4)
      proxy = h1 + Delta hdot + 1/2 Delta^2 hddot                (Eq. 5)
    Lower orders drop the trailing terms (order 0: proxy = h1).
    """
    h1, tau1 = np.asarray(entries[0][0], f64), f64(entries[0][1])
    out = h1.copy()
    if order >= 1:
        h2, tau2 = np.asarray(entries[1][0], f64), f64(entries[1][1])
        delta = f64(t_cur) - tau1
        hdot = (h1 - h2) / (tau1 - tau2)
        out = out + delta * hdot
        if order >= 2:
            h3 = np.asarray(entries[2][0], f64)
            hddot = (h1 - 2.0 * h2 + h3) / (tau1 - tau2) ** 2
            out = out + 0.5 * delta ** 2 * hddot
    return out


# ----------------------------------------------------------------------------- one step

class PoolCache:
    """Activation cache of a candidate pool: block l, slot s -> [T, D] fp64 per candidate.

    Slots follow the 3-slot ring of the cache metadata (see ``oracle.dispatch``).
    """

    def __init__(self, num_blocks: int):
        self.meta = [{"count": 0, "head": 0, "t": [0.0, 0.0, 0.0]} for _ in range(num_blocks)]
        self.data: Dict[Tuple[int, int, int], np.ndarray] = {}   # (candidate, block, slot) -> h


def candidate_velocity(W: Dict[str, np.ndarray], shape, z: np.ndarray, t_cur: float,
                       kv: List[Tuple[np.ndarray, np.ndarray]], block_mod: np.ndarray,
                       head_mod: np.ndarray, trace, meta_before: List[Dict], cache: Optional[PoolCache],
                       row: int, hidden: Optional[List[np.ndarray]] = None,
                       residual: bool = False) -> np.ndarray:
    """The network's velocity v [C, H, W] for one candidate under an already-planned trace; computed
    block outputs are cached under key ``row``.

    ``residual``: the alternative reading of the proxy in which h^(l) of Eq. 3-5 is the block's
    residual delta B_l(h) - h (as in TaylorSeer-style feature forecasting): a computed block caches its
    delta, a proxied block adds the forecast delta to its input."""
    C, H, Wd = z.shape
    p = shape.patch
    angles = rope_angles(H // p, Wd // p, shape.head_dim) if getattr(shape, "qk_norm_rope", False) else None
    tok = patchify(np.asarray(z, f64), p)
    h = linear(tok, W["pe_w"], W["pe_b"])
    if hidden is not None:
        hidden.append(h.copy())
    for l, (action, order, slot, live) in enumerate(trace):
        if action == SKIP:                                    # Eq. 6: identity
            pass
        elif action == PROXY:                                 # Eq. 3-5
            m = meta_before[l]
            slots = recent_slots(m)
            entries = [(cache.data[(row, l, s)], m["t"][s]) for s in slots]
            h = h + taylor_proxy(entries, t_cur, order) if residual else taylor_proxy(entries, t_cur, order)
        else:                                                 # Eq. 7
            h_in = h
            h = block_forward(W, l, h, block_mod[l], kv[l], shape.heads, shape.ln_eps, angles)
            if cache is not None:
                cache.data[(row, l, slot)] = (h - h_in) if residual else h.copy()
        if hidden is not None:
            hidden.append(h.copy())
    sh, sc = head_mod
    a = layer_norm(h, shape.ln_eps) * (1.0 + sc) + sh
    out = linear(a, W["head_w"], W["head_b"])
    return unpatchify(out, C, H, Wd, p)


def update(z: np.ndarray, v: np.ndarray, t_cur: float, t_next: float,
           noise: Optional[Tuple[float, int, int, int]] = None) -> np.ndarray:
    """Euler update z + (t_next - t_cur) v (Eq. 20 with a = 0), or with ``noise = (a, seed, step, row)``
    the stochastic update of App. A.1 (Eq. 20) with the normals of counter row ``row``."""
    if noise is not None:
        a, seed, step, row = noise
        eps = sde.latent_normals(z.shape, row, step, seed)
        return sde.sde_update(z, v, t_cur, t_next, a, eps)
    return np.asarray(z, f64) + (f64(t_next) - f64(t_cur)) * v


def guided(v_cond: np.ndarray, v_uncond: np.ndarray, scale: float) -> np.ndarray:
    """Classifier-free guidance: v = v_u + s (v_c - v_u)."""
    return np.asarray(v_uncond, f64) + f64(scale) * (np.asarray(v_cond, f64) - np.asarray(v_uncond, f64))


def candidate_step(W: Dict[str, np.ndarray], shape, z: np.ndarray, t_cur: float, t_next: float,
                   kv: List[Tuple[np.ndarray, np.ndarray]], block_mod: np.ndarray,
                   head_mod: np.ndarray, trace, meta_before: List[Dict], cache: Optional[PoolCache],
                   cand: int, hidden: Optional[List[np.ndarray]] = None,
                   noise: Optional[Tuple[float, int, int, int]] = None) -> np.ndarray:
    """One denoising step of one candidate under an already-planned trace; returns z_next [C, H, W].

    ``noise = (a, seed, step, row)`` replaces the Euler update by the stochastic one of App. A.1
    (Eq. 20) with the normals of counter row ``row`` at counter ``step`` (oracle/sde.py).
    """
    v = candidate_velocity(W, shape, z, t_cur, kv, block_mod, head_mod, trace, meta_before, cache, cand,
                           hidden)
    return update(z, v, t_cur, t_next, noise)


def _noise(sde_args, n: int):
    """(a, seed, step[, row0]) -> the noise tuple of candidate row n, or None."""
    if sde_args is None:
        return None
    a, seed, step = sde_args[:3]
    row0 = sde_args[3] if len(sde_args) > 3 else 0
    return a, seed, step, row0 + n


def clean_estimate(z: np.ndarray, v: np.ndarray, t: float) -> np.ndarray:
    """Preview of the clean latent from state z at time t with velocity v: x_t = (1 - t) x_0 + t x_1
    and v = x_1 - x_0 give x_0 = x_t - t v (rectified flow, App. A.1); the draft a verifier scores
    (Sec. 4.2 Stage 1) is this estimate at the truncation point."""
    return np.asarray(z, f64) - f64(t) * np.asarray(v, f64)


def draft_step(W: Dict[str, np.ndarray], shape, z: np.ndarray, t_cur: float, t_next: float,
               kv_per_cond: List[List[Tuple[np.ndarray, np.ndarray]]], cond_index: np.ndarray,
               skip: np.ndarray, proxy: np.ndarray, cache: PoolCache,
               candidates: Optional[Sequence[int]] = None,
               hidden: Optional[Dict[int, List[np.ndarray]]] = None,
               sde_args: Optional[Tuple[float, int, int]] = None,
               cfg: Optional[Tuple[float, np.ndarray]] = None, residual: bool = False):
    """One draft step over the pool (Eq. 2 with the knobs of Sec. 4.1).

    z [N, C, H, W]; returns (z_next [N, C, H, W] fp64 -- rows not in ``candidates`` are left as z --,
    trace).  The cache metadata advances once per step, as all candidates share the masks.
    ``sde_args = (a, seed, step[, row0])`` selects the stochastic update (Eq. 20), candidate n
    drawing the normals of counter row row0 + n (row0 = 0 by default) at ``step``.
    ``cfg = (scale, uncond_index)``: classifier-free guidance; candidate n also runs with prompt
    uncond_index[n] (cache key N + n) and steps with v_u + scale (v_c - v_u).
    ``residual``: proxies forecast residual deltas (see ``candidate_velocity``).
    """
    trace, new_meta = plan_step(skip, proxy, cache.meta, t_cur, residual)
    block_mod, head_mod = modulations(W, shape.num_blocks, shape.freq_dim, t_cur)
    out = np.asarray(z, f64).copy()
    N = z.shape[0]
    for n in (range(N) if candidates is None else candidates):
        hid = None if hidden is None else hidden.setdefault(n, [])
        v = candidate_velocity(W, shape, z[n], t_cur, kv_per_cond[int(cond_index[n])], block_mod, head_mod,
                               trace, cache.meta, cache, n, hid, residual)
        if cfg is not None:
            v_u = candidate_velocity(W, shape, z[n], t_cur, kv_per_cond[int(cfg[1][n])], block_mod, head_mod,
                                     trace, cache.meta, cache, N + n, None, residual)
            v = guided(v, v_u, cfg[0])
        out[n] = update(z[n], v, t_cur, t_next, _noise(sde_args, n))
    cache.meta = new_meta
    return out, trace


def refine_step(W: Dict[str, np.ndarray], shape, z: np.ndarray, t_cur: float, t_next: float,
                kv_per_cond, cond_index: np.ndarray, candidates: Optional[Sequence[int]] = None,
                sde_args: Optional[Tuple[float, int, int]] = None,
                cfg: Optional[Tuple[float, np.ndarray]] = None):
    """Full-quality step (phi_full of Eq. 13): no skipping, no proxies, no cache.

    ``sde_args`` and ``cfg`` as in ``draft_step``."""
    L = shape.num_blocks
    zeros = np.zeros(L, np.uint8)
    trace, _ = plan_step(zeros, zeros, [{"count": 0, "head": 0, "t": [0.0] * 3} for _ in range(L)],
                         t_cur)
    block_mod, head_mod = modulations(W, L, shape.freq_dim, t_cur)
    out = np.asarray(z, f64).copy()
    for n in (range(z.shape[0]) if candidates is None else candidates):
        v = candidate_velocity(W, shape, z[n], t_cur, kv_per_cond[int(cond_index[n])], block_mod, head_mod,
                               trace, None, None, n)
        if cfg is not None:
            v_u = candidate_velocity(W, shape, z[n], t_cur, kv_per_cond[int(cfg[1][n])], block_mod, head_mod,
                                     trace, None, None, n)
            v = guided(v, v_u, cfg[0])
        out[n] = update(z[n], v, t_cur, t_next, _noise(sde_args, n))
    return out


def prepare_text(W: Dict[str, np.ndarray], shape, text: np.ndarray):
    """Per-prompt cross-attention keys/values for every block."""
    return [text_kv(W, shape.num_blocks, text[c], shape.ln_eps) for c in range(text.shape[0])]


def run_draft(W, shape, z0, schedule, steps_draft: int, masks, text, cond_index,
              candidates: Optional[Sequence[int]] = None, on_step=None, residual: bool = False):
    """Truncated trajectory (Eq. 2 truncated to S' steps).  ``masks(k)`` -> (skip, proxy).

    Returns (z after S' steps, cache, traces).  ``on_step(k, z)`` is called after each step.
    """
    kv = prepare_text(W, shape, text)
    cache = PoolCache(shape.num_blocks)
    z = np.asarray(z0, f64)
    traces = []
    for k in range(steps_draft):
        skip, proxy = masks(k)
        z, tr = draft_step(W, shape, z, schedule[k], schedule[k + 1], kv, cond_index, skip, proxy,
                           cache, candidates, residual=residual)
        traces.append(tr)
        if on_step is not None:
            on_step(k, z)
    return z, cache, traces


def run_refine(W, shape, z, schedule, start: int, text, cond_index,
               candidates: Optional[Sequence[int]] = None, on_step=None):
    """Stage 3 (Eq. 13): steps start .. S-1 with full computation from the given latent."""
    kv = prepare_text(W, shape, text)
    z = np.asarray(z, f64)
    for k in range(start, len(schedule) - 1):
        z = refine_step(W, shape, z, schedule[k], schedule[k + 1], kv, cond_index, candidates)
        if on_step is not None:
            on_step(k, z)
    return z

