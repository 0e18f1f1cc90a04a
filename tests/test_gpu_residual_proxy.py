"""The residual-delta reading of the activation proxy through the library (cache of block deltas formed
in the down-projection epilogue, proxies added to their input, every proxy live) against the oracle."""
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


@pytest.mark.parametrize("dtype,tol,tile", [("fp32", 1e-5, None), ("bf16", 2e-2, None), ("bf16", 2e-2, "256x256"),
                                            ("bf16", 2e-2, "w8:bm:224"), ("bf16", 2e-2, "deep:160:256:2")])
@pytest.mark.parametrize("name", ["tiny", "mid"])
def test_residual_proxy_trajectory_matches_oracle(name, dtype, tol, tile, monkeypatch):
    """tile: a forced linear-layer tiling (the 8-wave kernels of 256, 224 and 160 rows), so that the
    block-delta cache write of the down-projection's residual epilogue runs on each of them."""
    if tile is not None:
        monkeypatch.setenv("FLASHBON_LINEAR_TILE", tile)
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    pool = DraftPool(wl, dtype=dtype, weights=flat, proxy_mode=1)
    pool.reset(z0)
    z_ref = z0.astype(np.float64)
    live_proxies = 0
    for k in range(wl.steps_draft):
        skip, proxy = wl.masks(k)
        z_prev_ref, z_prev = z_ref, pool.latents.cpu().numpy().astype(np.float64)
        z_ref, tr_ref = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(), skip,
                                        proxy, cache, residual=True)
        tr = pool.draft_step(k)
        torch.cuda.synchronize()
        assert tr == [tuple(e) for e in tr_ref], f"trace step {k}"
        live_proxies += sum(1 for e in tr if e[0] == 2)
        got = pool.latents.cpu().numpy().astype(np.float64)
        ez = rel_l2(got, z_ref)
        ev = rel_l2(step_velocity(got, z_prev, sched[k], sched[k + 1]),
                    step_velocity(z_ref, z_prev_ref, sched[k], sched[k + 1]))
        print(f"{name} {dtype} residual proxy step {k}: z {ez:.2e} v {ev:.2e}", flush=True)
        assert ez <= tol and ev <= TOL_V[dtype], (k, ez, ev)
    assert live_proxies > 0
    pool.close()


def test_residual_and_output_readings_differ_but_share_computed_steps():
    """Steps without proxies are the same computation under both readings (bit for bit); a step with
    proxies differs."""
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    flat, _ = synth.make_weights(wl.shape, wl.seed_w)
    outs = {}
    for mode in (0, 1):
        pool = DraftPool(wl, dtype="fp32", weights=flat, proxy_mode=mode)
        pool.reset()
        steps = []
        for k in range(wl.steps_draft):
            pool.draft_step(k)
            torch.cuda.synchronize()
            steps.append(pool.latents.clone())
        outs[mode] = steps
        pool.close()
    first_proxy = next(k for k in range(wl.steps_draft) if wl.masks(k)[1].any())
    for k in range(first_proxy):
        assert torch.equal(outs[0][k], outs[1][k])
    assert not torch.equal(outs[0][-1], outs[1][-1])
