"""Full-size parity: the draft step at the workloads' real shapes and launch configurations, on
candidates the oracle can follow one by one (candidates are independent, so a subset is a valid
check of the whole pool's launch).  Tolerances as in test_gpu_step.py (bf16 mode: latents 2e-2,
velocity 5e-2, rel-L2 per step); traces bit-exact."""
import time

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


def _run(name, candidates, steps):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, W = synth.make_weights(wl.shape, wl.seed_w, threads=16)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    sched = wl.schedule()
    pool = DraftPool(wl, dtype="bf16", weights=flat)
    pool.reset(z0)
    gpu_z, gpu_tr = [], []
    for k in range(steps):
        gpu_tr.append(pool.draft_step(k))
        torch.cuda.synchronize()
        gpu_z.append(pool.latents.cpu().numpy()[candidates].astype(np.float64))
    pool.close()
    del pool, flat
    t0 = time.time()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    z = z0.astype(np.float64)
    for k in range(steps):
        skip, proxy = wl.masks(k)
        z_prev = z
        z, tr = odit.draft_step(W, wl.shape, z, sched[k], sched[k + 1], kv, wl.cond_index(), skip, proxy,
                                cache, candidates=candidates)
        assert gpu_tr[k] == [tuple(e) for e in tr], f"trace step {k}"
        dt = float(sched[k + 1]) - float(sched[k])
        prev = z0[candidates].astype(np.float64) if k == 0 else gpu_z[k - 1]
        ez = rel_l2(gpu_z[k], z[candidates])
        ev = rel_l2((gpu_z[k] - prev) / dt, (z[candidates] - z_prev[candidates]) / dt)
        print(f"{name} step {k} candidates {candidates}: z {ez:.2e} v {ev:.2e} "
              f"(oracle {time.time() - t0:.0f}s)", flush=True)
        assert ez <= 2e-2 and ev <= 5e-2


def test_pool16_last_candidate_compute_and_proxy_steps():
    """The benchmark pool (N=16, 1560 tokens): step 0 computes 20 blocks, step 1 is all proxies."""
    _run("wan1.3b_pool16", [15], 2)


def test_pool64_four_prompts():
    """N=64 at 1024 tokens, candidates split over 4 prompts; one candidate of prompt 1 and 3."""
    _run("wan1.3b_pool64", [16, 63], 2)


def test_14b_shaped_layers():
    """D=5120, 40 heads, MLP 13824, 4096 tokens, N=4: step 0 computed, step 1 skip + proxy."""
    _run("wan14b_2block", [3], 2)
