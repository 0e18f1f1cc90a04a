"""The configuration search on the GPU (App. C): Sim(phi) measured through the library against the
oracle's drafts, previews and full-compute outputs; a short dual-annealing run on the GPU."""
import numpy as np
import pytest

from oracle import dispatch as odisp
from oracle import dit as odit
from oracle import phi as ophi
from paper_2607_04461_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


def _oracle_sim(W, wl, z0, text, phi):
    sched = wl.schedule()
    S = len(sched) - 1
    base = odit.run_refine(W, wl.shape, z0, sched, 0, text, wl.cond_index())
    zs = {}
    masks = lambda k: odisp.masks_from_phi(phi, wl.shape.num_blocks, k)
    z, _, _ = odit.run_draft(W, wl.shape, z0, sched, phi[0], masks, text, wl.cond_index(),
                             on_step=lambda k, zz: zs.__setitem__(k, zz.copy()))
    t_s = float(sched[phi[0]])
    if t_s > 0:
        prev = zs[phi[0] - 2] if phi[0] >= 2 else z0.astype(np.float64)
        v = (z - prev) / (t_s - float(sched[phi[0] - 1]))
        z = z - t_s * v
    return ophi.similarity([ophi.latent_distance(z[i], base[i]) for i in range(z.shape[0])])


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
def test_similarity_matches_oracle(dtype, tol):
    from paper_2607_04461_amd.phi_search import GpuEvaluator, Phi
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    pool = DraftPool(wl, dtype=dtype, weights=flat)
    pool.reset(z0)
    ev = GpuEvaluator(pool)
    for phi in (Phi(8, 0, 1, 1, 1), Phi(6, 2, 2, 3, 2), Phi(4, 1, 3, 3, 3), Phi(1, 0, 1, 2, 1)):
        speedup, sim = ev(phi)
        ref = _oracle_sim(W, wl, z0, text, phi.astuple())
        print(f"{dtype} {phi.astuple()}: speedup {speedup:.2f} sim {sim:.6f} oracle {ref:.6f}", flush=True)
        assert speedup > 0 and abs(sim - ref) <= tol
    pool.close()


def test_short_search_on_gpu():
    from paper_2607_04461_amd.phi_search import GpuEvaluator, search
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    pool = DraftPool(wl, dtype="bf16")
    pool.reset()
    ev = GpuEvaluator(pool)
    evals, star, best = search(ev, len(pool.schedule) - 1, wl.shape.num_blocks, lam=0.2, maxiter=12, seed=1,
                               f_max=4, min_sim=0.6)
    assert len(evals) >= 5
    print(f"{len(evals)} configurations; best J {evals[best].phi}; phi* "
          f"{None if star is None else (evals[star].phi, evals[star].speedup, evals[star].sim)}", flush=True)
    if star is not None:
        assert evals[star].sim >= 0.6
    pool.close()
