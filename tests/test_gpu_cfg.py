"""Classifier-free guidance through the library (2n token rows, v = v_u + s (v_c - v_u)) against the
oracle, on the Euler and stochastic paths, in drafting (with the knobs and the 2n-row cache) and in
refinement; and at full size the end points s = 1 (conditional run) and s = 0 (unconditional run)."""
import numpy as np
import pytest

from oracle import dit as odit
from paper_2607_04461_amd import synth
from tests._util import TOL_V, rel_l2, step_velocity

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


def _setup(wl):
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    text_u = np.concatenate([text, np.zeros((1,) + text.shape[1:], np.float32)])   # null prompt = n_cond
    return flat, W, z0, text_u


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
@pytest.mark.parametrize("name,sde", [("tiny", None), ("mid", None), ("mid", (0.3, 5))])
def test_guided_draft_matches_oracle(name, sde, dtype, tol):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, W, z0, text_u = _setup(wl)
    scale = 4.5
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text_u)
    cache = odit.PoolCache(wl.shape.num_blocks)
    unc = np.full(wl.n, wl.n_cond, np.int32)
    pool = DraftPool(wl, dtype=dtype, weights=flat, guidance=scale)
    pool.reset(z0)
    z_ref = z0.astype(np.float64)
    for k in range(wl.steps_draft):
        skip, proxy = wl.masks(k)
        z_prev_ref, z_prev = z_ref, pool.latents.cpu().numpy().astype(np.float64)
        z_ref, tr_ref = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip,
                                        proxy, cache, sde_args=None if sde is None else (sde[0], sde[1], k),
                                        cfg=(scale, unc))
        tr = pool.draft_step(k, sde=sde)
        torch.cuda.synchronize()
        assert tr == [tuple(e) for e in tr_ref], f"trace step {k}"
        got = pool.latents.cpu().numpy().astype(np.float64)
        noise = None if sde is None else (sde[0], sde[1], k, 0)
        ez = rel_l2(got, z_ref)
        ev = rel_l2(step_velocity(got, z_prev, sched[k], sched[k + 1], noise),
                    step_velocity(z_ref, z_prev_ref, sched[k], sched[k + 1], noise))
        print(f"{name} {dtype} cfg {scale} sde={sde} step {k}: z {ez:.2e} v {ev:.2e}", flush=True)
        assert ez <= tol and ev <= TOL_V[dtype], (k, ez, ev)
    # refinement of candidate 1 with guidance, step by step from the GPU's own draft latent
    lat = pool.latents[1:2].clone()
    ref = lat.cpu().numpy().astype(np.float64)
    for k in range(wl.steps_draft, wl.steps_total):
        prev, prev_ref = lat.cpu().numpy().astype(np.float64), ref
        pool.refine_step(k, latents=lat, cond_index=wl.cond_index()[1:2])
        ref = odit.refine_step(W, wl.shape, ref, sched[k], sched[k + 1], kv, wl.cond_index()[1:2],
                               cfg=(scale, unc[:1]))
        torch.cuda.synchronize()
        got = lat.cpu().numpy().astype(np.float64)
        err = rel_l2(got, ref)
        ev = rel_l2(step_velocity(got, prev, sched[k], sched[k + 1]),
                    step_velocity(ref, prev_ref, sched[k], sched[k + 1]))
        print(f"{name} {dtype} guided refine step {k}: z {err:.2e} v {ev:.2e}", flush=True)
        assert err <= tol and ev <= TOL_V[dtype], (k, err, ev)
    pool.close()


def test_guidance_end_points_full_size():
    """1.3B-shaped pool of 16 (bf16), first draft step: s = 1 reproduces the unguided conditional step
    and s = 0 the unguided step with the null prompt, up to the rounding of v_u + s (v_c - v_u)."""
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["wan1.3b_pool16"]
    flat, _, z0, _ = _setup(wl)
    outs = {}
    for label, scale in (("s1", 1.0), ("s0", 0.0)):
        pool = DraftPool(wl, dtype="bf16", weights=flat, guidance=scale)
        pool.reset(z0)
        pool.draft_step(0)
        torch.cuda.synchronize()
        outs[label] = pool.latents.double().cpu().numpy()
        if label == "s1":
            # the same pool object, unguided: the conditional rows alone
            pool.guidance = None
            pool.reset(z0)
            pool.draft_step(0)
            torch.cuda.synchronize()
            outs["cond"] = pool.latents.double().cpu().numpy()
            pool.cond_index = np.full(wl.n, wl.n_cond, np.int32)
            pool.reset(z0)
            pool.draft_step(0)
            torch.cuda.synchronize()
            outs["uncond"] = pool.latents.double().cpu().numpy()
        pool.close()
    e1 = rel_l2(outs["s1"] - z0, outs["cond"] - z0)
    e0 = rel_l2(outs["s0"] - z0, outs["uncond"] - z0)
    print(f"s=1 vs conditional: {e1:.2e}; s=0 vs unconditional: {e0:.2e}", flush=True)
    assert e1 <= 1e-5 and e0 <= 1e-5
    assert rel_l2(outs["cond"] - z0, outs["uncond"] - z0) > 1e-3
