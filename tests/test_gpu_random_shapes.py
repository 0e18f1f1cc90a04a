"""Seeded random configurations through the draft step against the oracle (GPU).

Shapes the named workloads do not reach: token counts that are not multiples of 4, 64 or 128 (latents of
4..20 x 4..20, patch 2), prompts of 3..70 tokens (ragged key tiles in cross-attention), 1..4 candidates over
1..3 prompts, 2 or 3 blocks, head dim 16 (the VALU attention path) and 128 (the MFMA path), random skip and
proxy masks (Sec. 4.1 (1)-(3)), both readings of the proxy, fp32 and bf16.  Per step: the trace equals the
oracle dispatcher's bit for bit, and latents and velocity are within the bounds of test_gpu_step.py.
"""
import dataclasses

import numpy as np
import pytest

from oracle import dit as odit
from paper_2607_04461_amd import synth
from tests._util import TOL_V, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = {"fp32": (1e-5, TOL_V["fp32"]), "bf16": (2e-2, TOL_V["bf16"])}
SMALL = synth.ModelShape(num_blocks=3, hidden=64, heads=4, mlp_hidden=192, freq_dim=64, text_dim=32)   # dh 16
WIDE = dataclasses.replace(synth.MID, num_blocks=2)                                                      # dh 128
STEPS = 5


def _config(seed):
    rng = np.random.default_rng(seed)
    shape = (SMALL, WIDE)[seed % 2]
    n = int(rng.integers(1, 5))
    n_cond = int(rng.integers(1, min(n, 3) + 1))
    lh, lw = 2 * int(rng.integers(2, 11)), 2 * int(rng.integers(2, 11))
    wl = synth.Workload(f"random{seed}", shape, n=n, latent_h=lh, latent_w=lw, text_len=int(rng.integers(3, 71)),
                        n_cond=n_cond, steps_total=8, steps_draft=STEPS, dtype="fp32", seed_w=1000 + seed)
    L = shape.num_blocks
    masks = [(np.zeros(L, np.uint8), np.zeros(L, np.uint8))]
    for _ in range(1, STEPS):
        masks.append(((rng.random(L) < 0.3).astype(np.uint8), (rng.random(L) < 0.5).astype(np.uint8)))
    return wl, masks, int(rng.integers(0, 2))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("seed", range(6))
def test_random_configuration_matches_oracle(seed, dtype):
    from paper_2607_04461_amd.pool import DraftPool
    wl, masks, proxy_mode = _config(seed)
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    print(f"seed {seed} {dtype}: D={wl.shape.hidden} L={wl.shape.num_blocks} n={wl.n} n_cond={wl.n_cond} "
          f"T={wl.tokens} ({wl.latent_h}x{wl.latent_w}) text_len={wl.text_len} proxy_mode={proxy_mode}", flush=True)
    pool = DraftPool(wl, dtype=dtype, weights=flat, proxy_mode=proxy_mode)
    pool.reset(z0)
    z_ref = z0.astype(np.float64)
    tol_z, tol_v = TOL[dtype]
    for k, (skip, proxy) in enumerate(masks):
        z_prev_gpu = pool.latents.cpu().numpy().astype(np.float64)
        z_next, tr_ref = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip, proxy,
                                         cache, residual=proxy_mode == 1)
        tr = pool.draft_step(k, skip=skip, proxy=proxy)
        torch.cuda.synchronize()
        got = pool.latents.cpu().numpy().astype(np.float64)
        assert tr == [tuple(e) for e in tr_ref], f"trace step {k}"
        dt = float(sched[k + 1]) - float(sched[k])
        ez = rel_l2(got, z_next)
        ev = rel_l2((got - z_prev_gpu) / dt, (z_next - z_ref) / dt)
        print(f"  step {k} skip {skip.tolist()} proxy {proxy.tolist()}: z {ez:.2e} v {ev:.2e}", flush=True)
        assert ez <= tol_z and ev <= tol_v, (k, ez, ev)
        z_ref = z_next
    pool.close()
