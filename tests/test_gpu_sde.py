"""GPU parity of the stochastic update (App. A.1, Eq. 20) against the oracle, through the C ABI.

* Philox4x32-10 words: bit-exact (integer work).
* Normals: the library forms them in double and rounds to fp32, the oracle keeps fp64: |diff| <= 1e-6.
* Unpatchify + update (fp32 arithmetic on fp32 inputs): |diff| <= 1e-5 (1 + |z|), elementwise.
* Whole steps: the tolerances of the Euler steps (relative L2 of the latents: fp32 1e-5, bf16 2e-2);
  a = 0 with any seed is the Euler step bit for bit.
"""
import numpy as np
import pytest

from oracle import dit as odit
from oracle import sde as osde
from paper_2607_04461_amd import synth
from tests._util import TOL_V, rel_l2, step_velocity

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SEED = 0x0123_4567_89AB_CDEF


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


def _fb():
    from paper_2607_04461_amd import flashbon
    return flashbon


@pytest.mark.parametrize("count,cand,step,seed", [
    (1, 0, 0, 0), (1001, 5, 7, SEED), (16 * 60 * 104, 15, 9, 2 ** 64 - 1), (16 * 128 * 128, 3, 49, 77)])
def test_normals_match_oracle(count, cand, step, seed):
    fb = _fb()
    quads = (count + 3) // 4
    words = torch.zeros(quads * 4, dtype=torch.int32, device="cuda")
    normals = torch.zeros(count, dtype=torch.float32, device="cuda")
    fb.flashbon_op_normals(count, cand, step, seed, words, normals)
    torch.cuda.synchronize()
    ctr = np.zeros((quads, 4), np.uint64)
    ctr[:, 0] = np.arange(quads)
    ctr[:, 1], ctr[:, 2] = cand, step
    ref_w = osde.philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32)).reshape(-1)
    got_w = words.cpu().numpy().view(np.uint32).astype(np.uint64)
    np.testing.assert_array_equal(got_w, ref_w)
    ref_z = osde.latent_normals((count,), cand, step, seed)
    got_z = normals.cpu().numpy().astype(np.float64)
    assert np.max(np.abs(got_z - ref_z)) <= 1e-6


def _ref_unpatch_sde(v_tok, z, C, H, W, p, t_cur, t_next, a, seed, step, row0=0):
    n = z.shape[0]
    T = (H // p) * (W // p)
    out = np.empty_like(z, dtype=np.float64)
    for b in range(n):
        v = odit.unpatchify(v_tok[b * T:(b + 1) * T].astype(np.float64), C, H, W, p)
        eps = osde.latent_normals((C, H, W), row0 + b, step, seed)
        out[b] = osde.sde_update(z[b], v, t_cur, t_next, a, eps)
    return out


@pytest.mark.parametrize("n,C,H,W,p,t_cur,t_next,a,row0", [
    (2, 16, 8, 8, 2, 0.75, 0.5, 0.3, 0),            # tiny latent
    (3, 1, 9, 15, 3, 0.6, 0.5, 0.7, 0),             # count 135 per candidate: ragged last counter
    (1, 3, 2, 2, 1, 1.0, 0.98, 0.3, 0),             # t = 1: sigma from 1 - t_next
    (2, 16, 60, 104, 2, 0.02, 0.0, 0.3, 0),         # 1.3B-shaped latent, last step (t_next = 0)
    (16, 16, 60, 104, 2, 0.8, 0.78, 0.3, 0),        # the 1.3B-shaped pool of 16
    (3, 16, 60, 104, 2, 0.5, 0.48, 0.3, 13),        # rows 13..15 of a pool, drawn on their own
])
def test_unpatch_sde_matches_oracle(n, C, H, W, p, t_cur, t_next, a, row0):
    fb = _fb()
    rng = np.random.default_rng(n * 1000 + C)
    T, P = (H // p) * (W // p), C * p * p
    v = rng.standard_normal((n * T, P)).astype(np.float32)
    z = rng.standard_normal((n, C, H, W)).astype(np.float32)
    zd = torch.from_numpy(z).cuda()
    fb.flashbon_op_unpatch_sde(n, C, H, W, p, torch.from_numpy(v).cuda(), zd, t_cur, t_next, a, SEED, 11, row0)
    torch.cuda.synchronize()
    got = zd.cpu().numpy().astype(np.float64)
    ref = _ref_unpatch_sde(v, z, C, H, W, p, float(np.float32(t_cur)), float(np.float32(t_next)), a, SEED, 11,
                           row0)
    err = np.max(np.abs(got - ref) / (1.0 + np.abs(ref)))
    print(f"unpatch_sde n{n} C{C} {H}x{W} p{p}: {err:.2e}", flush=True)
    assert err <= 1e-5


def test_unpatch_sde_rejects_bad_arguments():
    fb = _fb()
    v = torch.zeros(16, 4, device="cuda")
    z = torch.zeros(1, 1, 8, 8, device="cuda")
    for t_cur, t_next, a in ((0.5, 0.4, -0.1), (0.0, -0.1, 0.3), (1.0, 1.0, 0.3), (1.5, 1.0, 0.3),
                             (0.5, 0.4, float("nan"))):
        with pytest.raises(fb.FlashbonError):
            fb.flashbon_op_unpatch_sde(1, 1, 8, 8, 2, v, z, t_cur, t_next, a, 1, 0)
    assert torch.count_nonzero(z) == 0


def _inputs(wl):
    flat, W = synth.make_weights(wl.shape, wl.seed_w)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    return flat, W, z0, text


@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 2e-2)])
@pytest.mark.parametrize("name", ["tiny", "mid"])
def test_stochastic_draft_trajectory_matches_oracle(name, dtype, tol):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, W, z0, text = _inputs(wl)
    sched = wl.schedule()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    pool = DraftPool(wl, dtype=dtype, weights=flat)
    pool.reset(z0)
    z_ref = z0.astype(np.float64)
    a, seed = 0.3, 4242
    for k in range(wl.steps_draft):
        skip, proxy = wl.masks(k)
        z_prev_ref, z_prev = z_ref, pool.latents.cpu().numpy().astype(np.float64)
        z_ref, tr_ref = odit.draft_step(W, wl.shape, z_ref, sched[k], sched[k + 1], kv, wl.cond_index(),
                                        skip, proxy, cache, sde_args=(a, seed, k))
        tr = pool.draft_step(k, sde=(a, seed))
        torch.cuda.synchronize()
        got = pool.latents.cpu().numpy().astype(np.float64)
        assert tr == [tuple(e) for e in tr_ref], f"trace step {k}"
        ez = rel_l2(got, z_ref)
        # drift v + sigma^2 / (2 t) (z + (1 - t) v): the known noise term removed on both sides
        ev = rel_l2(step_velocity(got, z_prev, sched[k], sched[k + 1], (a, seed, k, 0)),
                    step_velocity(z_ref, z_prev_ref, sched[k], sched[k + 1], (a, seed, k, 0)))
        print(f"{name} {dtype} sde step {k}: z {ez:.2e} drift {ev:.2e}", flush=True)
        assert ez <= tol and ev <= TOL_V[dtype], (k, ez, ev)
    pool.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_a_zero_is_euler_bit_exact(dtype):
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS["mid"]
    flat, _, z0, _ = _inputs(wl)
    outs = []
    for sde in (None, (0.0, 99)):
        pool = DraftPool(wl, dtype=dtype, weights=flat)
        pool.reset(z0)
        for k in range(3):
            pool.draft_step(k, sde=sde)
        pool.refine_step(3, sde=sde)
        torch.cuda.synchronize()
        outs.append(pool.latents.clone())
        pool.close()
    assert torch.equal(outs[0], outs[1])


def test_full_size_stochastic_step_adds_the_right_noise():
    """1.3B-shaped pool of 16, first step (t = 1, sigma from 1 - t_next), bf16.  The stochastic step
    minus the Euler step from the same latents equals dt k (z + (1 - t) v) + g eps with v recovered
    from the Euler step and eps from the normals entry point -- for every candidate row."""
    from paper_2607_04461_amd.pool import DraftPool
    fb = _fb()
    wl = synth.WORKLOADS["wan1.3b_pool16"]
    flat, _, z0, _ = _inputs(wl)
    sched = wl.schedule()
    pool = DraftPool(wl, dtype="bf16", weights=flat)
    a, seed, k = 0.3, 31337, 0
    pool.reset(z0)
    pool.draft_step(k)
    z_euler = pool.latents.clone()
    pool.reset(z0)
    pool.draft_step(k, sde=(a, seed))
    z_sde = pool.latents.clone()
    torch.cuda.synchronize()
    pool.close()
    tc, tn = float(sched[k]), float(sched[k + 1])
    dt = tn - tc
    sigma = osde.sigma(tc, tn, a)
    kk, g = sigma * sigma / (2 * tc), sigma * np.sqrt(abs(dt))
    z = torch.from_numpy(z0).double().cuda()
    v = (z_euler.double() - z) / dt
    per = wl.shape.latent_channels * wl.latent_h * wl.latent_w
    eps = torch.empty(per, dtype=torch.float32, device="cuda")
    worst = 0.0
    for b in range(wl.n):
        fb.flashbon_op_normals(per, b, k, seed, None, eps)
        expect = z[b] + dt * (v[b] + kk * (z[b] + (1 - tc) * v[b])) + g * eps.double().view(z[b].shape)
        err = float(((z_sde[b].double() - expect).abs() / (1 + expect.abs())).max())
        worst = max(worst, err)
    print(f"pool16 step 0 stochastic: worst {worst:.2e}", flush=True)
    assert worst <= 1e-4
