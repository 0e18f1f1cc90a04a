"""A candidate pool driven through the C ABI: torch device buffers + the S'-step loop.

Holds the caller-owned state the library expects (latents, text, text K/V scratch, activation cache,
cache metadata) and calls ``flashbon_draft_step`` / ``flashbon_refine_step`` once per step.  No
arithmetic of the method happens here.
"""
from __future__ import annotations

import ctypes
from typing import Callable, List, Optional, Tuple

import numpy as np

from . import flashbon as fb
from . import synth


class DraftPool:
    def __init__(self, wl: synth.Workload, dtype: Optional[str] = None, weights: Optional[np.ndarray] = None,
                 device: str = "cuda", max_n: Optional[int] = None, max_cond: Optional[int] = None,
                 guidance: Optional[float] = None, proxy_mode: int = 0):
        """``guidance``: classifier-free guidance scale; every candidate then also runs with a null prompt
        (an all-zero text appended as prompt n_cond) and the cache holds 2n rows."""
        import torch
        self.torch = torch
        self.wl = wl
        self.shape = wl.shape
        self.dtype = dtype or wl.dtype
        self.device = device
        if weights is None:
            weights, _ = synth.make_weights(wl.shape, wl.seed_w)
        self.guidance = guidance
        self.proxy_mode = proxy_mode            # 1: residual-delta reading of the proxy
        rows = 2 * wl.n if guidance is not None else wl.n
        n_text = wl.n_cond + (1 if guidance is not None else 0)
        cfg = fb.make_config(wl.shape, fb.BF16 if self.dtype == "bf16" else fb.FP32,
                             max(max_n or rows, rows), wl.tokens, wl.text_len, max(max_cond or n_text, n_text))
        self.cfg = cfg
        self.model = fb.flashbon_init_model(cfg, weights)
        L = wl.shape.num_blocks
        self.L = L
        self.latents = torch.empty((wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w),
                                   dtype=torch.float32, device=device)
        text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
        if guidance is not None:
            text = np.concatenate([text, np.zeros((1,) + text.shape[1:], np.float32)])
        self.text = torch.from_numpy(text).to(device)
        self.cond_index = wl.cond_index()
        self.uncond_index = np.full(wl.n, wl.n_cond, np.int32)
        self.text_kv = torch.empty(fb.flashbon_text_kv_bytes(self.model, text.shape[0], wl.text_len),
                                   dtype=torch.uint8, device=device)
        self.cache = torch.empty(fb.flashbon_cache_bytes(self.model, rows, wl.tokens) // 4,
                                 dtype=torch.float32, device=device)
        self.text_kv_valid = ctypes.c_int32(0)
        self.meta = fb.new_meta(L)
        self.trace = fb.new_trace(L)
        self.schedule = wl.schedule()

    def reset(self, z0: Optional[np.ndarray] = None) -> None:
        """Load initial latents (default: the seeded ones) and clear the cache metadata."""
        wl = self.wl
        if z0 is None:
            z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
        self.latents.copy_(self.torch.from_numpy(np.ascontiguousarray(z0, np.float32)))
        ctypes.memset(self.meta, 0, ctypes.sizeof(self.meta))

    def draft_step(self, k: int, skip=None, proxy=None, hidden_dump=None, stream=None, sde=None,
                   preview=None) -> list:
        """Step k of the schedule; ``sde = (a, seed)`` takes the stochastic update with counter k;
        ``preview`` (device [n, C, H, W] fp32) receives the clean-latent estimate z - t v."""
        if skip is None or proxy is None:
            s, p = self.wl.masks(k)
            skip = s if skip is None else skip
            proxy = p if proxy is None else proxy
        fb.flashbon_draft_step(self.model, self.latents, self.schedule[k], self.schedule[k + 1], self.text,
                               self.cond_index, self.text_kv, self.text_kv_valid, skip, proxy, self.cache,
                               self.meta, self.trace, hidden_dump, stream,
                               None if sde is None else (sde[0], sde[1], k), preview, self._cfg(None),
                               self.proxy_mode)
        return fb.trace_list(self.trace)

    def _cfg(self, rows):
        if self.guidance is None:
            return None
        unc = self.uncond_index if rows is None else self.uncond_index[:rows]
        return (self.guidance, unc)

    def refine_step(self, k: int, latents=None, cond_index=None, hidden_dump=None, stream=None,
                    sde=None) -> list:
        """Step k with every knob off; ``sde = (a, seed[, row0])`` takes the stochastic update."""
        lat = self.latents if latents is None else latents
        cond = self.cond_index if cond_index is None else cond_index
        fb.flashbon_refine_step(self.model, lat, self.schedule[k], self.schedule[k + 1], self.text, cond,
                                self.text_kv, self.text_kv_valid, self.trace, hidden_dump, stream,
                                None if sde is None else (sde[0], sde[1], k, sde[2] if len(sde) > 2 else 0),
                                None, self._cfg(int(lat.shape[0])))
        return fb.trace_list(self.trace)

    def draft(self, steps: Optional[int] = None, on_step: Optional[Callable] = None) -> List[list]:
        traces = []
        for k in range(self.wl.steps_draft if steps is None else steps):
            traces.append(self.draft_step(k))
            if on_step is not None:
                on_step(k, self)
        return traces

    def select(self, scores, judge, rho1: float = 0.5, rho2: float = 0.5, kappa: float = 1.5) -> int:
        """Stage 2 (Sec. 4.2, Eq. 9-12): multi-stage Elo selection over the drafts, run by the library
        on the host; ``scores`` are the verifier's pointwise scores, ``judge(a, b) -> (winner,
        confidence)`` its pairwise calls.  Keeps (winner, ratings, pairwise calls) in
        ``last_selection``."""
        self.last_selection = fb.flashbon_select(scores, judge, rho1, rho2, kappa)
        return self.last_selection[0]

    def refine(self, j: int, out=None, stream=None, sde=None):
        """Stage 3 (Eq. 13): copy draft j's latent device-to-device (the pool stays intact for its
        next use) and run the remaining steps S' .. S-1 with full computation.  ``sde = (a, seed)``
        keeps the stochastic update with candidate j's own normals.  Returns the latent."""
        src = self.latents[j:j + 1]
        z = src.clone() if out is None else out.copy_(src)
        cond = self.cond_index[j:j + 1]
        for k in range(self.wl.steps_draft, self.wl.steps_total):
            self.refine_step(k, latents=z, cond_index=cond, stream=stream,
                             sde=None if sde is None else (sde[0], sde[1], j))
        return z

    def close(self) -> None:
        if self.model:
            fb.flashbon_free(self.model)
            self.model = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

