"""qk RMSNorm + 3-D RoPE (reading R26) through the library: whole drafts with the knobs on the rope
workloads (head_dim 16 and 128, ragged token count 130, two prompts) against the oracle, and one
full-quality step of a 1.3B-shaped model with the flag."""
import numpy as np
import pytest

from oracle import dit as odit
from paper_2607_04461_amd import synth
from tests._util import TOL_V, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
@pytest.mark.parametrize("name", ["tiny_rope", "mid_rope"])
def test_rope_draft_matches_oracle(name, dtype, tol):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    pool = DraftPool(wl, dtype=dtype, weights=flat)
    pool.reset(z0)
    z_ref = z0.astype(np.float64)
    for k in range(wl.steps_draft):
        skip, proxy = wl.masks(k)
        z_prev = z_ref
        z_ref, tr_ref = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip,
                                        proxy, cache)
        tr = pool.draft_step(k)
        torch.cuda.synchronize()
        got = pool.latents.cpu().numpy().astype(np.float64)
        assert tr == [tuple(e) for e in tr_ref]
        dt = float(sched[k + 1]) - float(sched[k])
        ez, ev = rel_l2(got, z_ref), rel_l2((got - z_prev) / dt, (z_ref - z_prev) / dt)
        print(f"{name} {dtype} step {k}: z {ez:.2e} v {ev:.2e}", flush=True)
        assert ez <= tol and ev <= TOL_V[dtype]
    pool.close()


def test_rope_changes_the_step():
    """The flag is not a no-op: the same weights without the gains/rotation give another velocity."""
    from paper_2607_04461_amd.pool import DraftPool
    outs = []
    for name in ("mid", "mid_rope"):
        wl = synth.WORKLOADS[name]
        pool = DraftPool(wl, dtype="fp32")
        pool.reset()
        pool.draft_step(0)
        torch.cuda.synchronize()
        outs.append(pool.latents.double().cpu().numpy())
        pool.close()
    assert rel_l2(outs[0], outs[1]) > 1e-6


def test_rope_full_size_one_step():
    """One full-quality step of the 1.3B-shaped model (N = 1, 1560 tokens in a 30 x 52 grid, 512 text
    tokens) with qk RMSNorm + 3-D RoPE, bf16, every output against the oracle."""
    import dataclasses
    import time
    from paper_2607_04461_amd.pool import DraftPool
    base = synth.WORKLOADS["wan1.3b_step"]
    wl = dataclasses.replace(base, shape=dataclasses.replace(base.shape, qk_norm_rope=True))
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    pool = DraftPool(wl, dtype="bf16", weights=flat)
    pool.reset(z0)
    pool.refine_step(0)
    torch.cuda.synchronize()
    got = pool.latents.cpu().numpy().astype(np.float64)
    pool.close()
    t0 = time.time()
    kv = odit.prepare_text(W, wl.shape, text)
    ref = odit.refine_step(W, wl.shape, z0, sched[0], sched[1], kv, wl.cond_index())
    dt = float(sched[1]) - float(sched[0])
    ez, ev = rel_l2(got, ref), rel_l2((got - z0) / dt, (ref - z0) / dt)
    print(f"oracle {time.time() - t0:.1f}s; wan1.3b rope step: z {ez:.2e} v {ev:.2e}", flush=True)
    assert ez <= 2e-2 and ev <= TOL_V["bf16"]
