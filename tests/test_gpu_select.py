"""Selection + hand-off on the GPU (Sec. 4.2 Stages 2-3): Elo selection over the drafted pool, then a
device-to-device copy of the winner's latent and full-computation refinement, against the oracle's
trajectory for that candidate (tolerances of the Euler steps: relative L2 fp32 1e-5, bf16 2e-2)."""
import dataclasses

import numpy as np
import pytest

from oracle import dit as odit
from oracle import select as osel
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


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
def test_select_then_refine_matches_oracle(dtype, tol):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    wl = dataclasses.replace(wl, steps_draft=4)           # S' = 4 of S = 8
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    pool = DraftPool(wl, dtype=dtype, weights=flat)
    pool.reset(z0)
    pool.draft()
    drafts = pool.latents.clone()
    v_lib, v_ref = synth.SyntheticVerifier(wl.n, 11), synth.SyntheticVerifier(wl.n, 11)
    j = pool.select(v_lib.scores, v_lib.judge)
    j_ref, _, _ = osel.select(v_ref.scores, v_ref.judge)
    assert j == j_ref
    out = pool.refine(j)
    torch.cuda.synchronize()
    assert torch.equal(pool.latents, drafts)                     # the pool is left intact
    z_draft, _, _ = odit.run_draft(W, wl.shape, z0, sched, wl.steps_draft, wl.masks, text, wl.cond_index(),
                                   candidates=[j])
    ref = odit.run_refine(W, wl.shape, z_draft[j:j + 1], sched, wl.steps_draft, text,
                          wl.cond_index()[j:j + 1])
    err = rel_l2(out.cpu().numpy().astype(np.float64), ref)
    print(f"select+refine {dtype}: winner {j}, rel-L2 {err:.2e}", flush=True)
    assert err <= tol
    # the stochastic variant keeps candidate j's own normals (counter row j) through refinement
    a, seed = 0.3, 99
    out_s = pool.refine(j, sde=(a, seed))
    torch.cuda.synchronize()
    kv = odit.prepare_text(W, wl.shape, text)
    ref_s = z_draft[j:j + 1]
    for k in range(wl.steps_draft, wl.steps_total):
        ref_s = odit.refine_step(W, wl.shape, ref_s, sched[k], sched[k + 1], kv, wl.cond_index()[j:j + 1],
                                 sde_args=(a, seed, k, j))
    err_s = rel_l2(out_s.cpu().numpy().astype(np.float64), ref_s)
    print(f"select+refine {dtype} stochastic: rel-L2 {err_s:.2e}", flush=True)
    assert err_s <= tol
    # per refinement step, from the same input on both sides (the GPU's draft of the winner): latent and
    # velocity (Euler), latent and drift with the known noise removed (stochastic, counter row j)
    for sde in (None, (a, seed)):
        lat = drafts[j:j + 1].clone()
        ref = lat.cpu().numpy().astype(np.float64)
        for k in range(wl.steps_draft, wl.steps_total):
            prev, prev_ref = lat.cpu().numpy().astype(np.float64), ref
            pool.refine_step(k, latents=lat, cond_index=wl.cond_index()[j:j + 1],
                             sde=None if sde is None else (sde[0], sde[1], j))
            ref = odit.refine_step(W, wl.shape, ref, sched[k], sched[k + 1], kv, wl.cond_index()[j:j + 1],
                                   sde_args=None if sde is None else (sde[0], sde[1], k, j))
            torch.cuda.synchronize()
            got = lat.cpu().numpy().astype(np.float64)
            noise = None if sde is None else (sde[0], sde[1], k, j)
            ez = rel_l2(got, ref)
            ev = rel_l2(step_velocity(got, prev, sched[k], sched[k + 1], noise),
                        step_velocity(ref, prev_ref, sched[k], sched[k + 1], noise))
            print(f"refine {dtype} sde={sde} step {k}: z {ez:.2e} v {ev:.2e}", flush=True)
            assert ez <= tol and ev <= TOL_V[dtype], (k, ez, ev)
    pool.close()
