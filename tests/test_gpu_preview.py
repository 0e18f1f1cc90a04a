"""The draft preview (clean-latent estimate z - t v, Sec. 4.2 Stage 1 with App. A.1) written by the
step's head epilogue, against the oracle, on the Euler and the stochastic paths."""
import copy

import numpy as np
import pytest

from oracle import dit as odit
from paper_2607_04461_amd import synth
from tests._util import rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
@pytest.mark.parametrize("sde", [None, (0.3, 17)])
def test_preview_matches_oracle(dtype, tol, sde):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    pool = DraftPool(wl, dtype=dtype, weights=flat)
    pool.reset(z0)
    prev = torch.zeros_like(pool.latents)
    z_ref = z0.astype(np.float64)
    for k in range(4):
        skip, proxy = wl.masks(k)
        tc, tn = float(sched[k]), float(sched[k + 1])
        # the velocity of this step, from an Euler step of the oracle on a copy of the cache
        c2 = copy.deepcopy(cache)
        z_e, _ = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip, proxy, c2)
        v = (z_e - z_ref) / (tn - tc)
        expect = odit.clean_estimate(z_ref, v, tc)
        z_ref, _ = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip, proxy,
                                   cache, sde_args=None if sde is None else (sde[0], sde[1], k))
        pool.draft_step(k, sde=sde, preview=prev)
        torch.cuda.synchronize()
        err = rel_l2(prev.cpu().numpy().astype(np.float64), expect)
        print(f"{dtype} sde={sde} step {k}: preview rel-L2 {err:.2e}", flush=True)
        assert err <= tol
    pool.close()


def test_preview_may_not_alias_latents():
    from paper_2607_04461_amd import flashbon as fb
    from paper_2607_04461_amd.pool import DraftPool
    pool = DraftPool(synth.WORKLOADS["tiny"])
    pool.reset()
    with pytest.raises(ValueError):             # the binding rejects it before the library sees it
        pool.draft_step(0, preview=pool.latents)
    pool.close()
