"""Pins of the stochastic-update oracle (App. A.1, Eq. 20) and of its counter-based normals.

Everything here is fixed by something other than the oracle itself:
  * Philox4x32-10 words: the published known-answer vectors of the generator's authors
    (Random123 distribution, kat_vectors, philox4x32 with 10 rounds);
  * Box-Muller: closed-form special words and a Kolmogorov-Smirnov test against scipy's normal CDF;
  * Eq. 20: a = 0 is the Euler update bit for bit; the score identity of App. A.1 for a Gaussian data
    law in closed form; and the marginal of the sampled process at t = 0 for that law, which the
    conversion of App. A.1 is built to preserve (a dropped factor, a flipped sign or a wrong 1 - t in
    the drift all move the final standard deviation by more than 15%).
"""
import numpy as np
import pytest
from scipy import stats

from oracle import sde


@pytest.mark.parametrize("ctr,key,expect", [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
])
def test_philox_known_answers(ctr, key, expect):
    got = sde.philox4x32_10(np.array(ctr, dtype=np.uint64), key)
    assert tuple(int(w) for w in got) == expect


def test_box_muller_special_words():
    # x0 = 2^32 - 1 -> u1 = 1 -> radius 0; x0 = 0 -> u1 = 2^-32 -> radius sqrt(64 ln 2)
    z = sde.box_muller(np.array([[0xFFFFFFFF, 123, 0, 0], [0, 0x40000000, 0, 0xC0000000]], np.uint64))
    assert np.all(z[0, :2] == 0.0)
    r = np.sqrt(64.0 * np.log(2.0))
    np.testing.assert_allclose(z[0, 2:], [r, 0.0], atol=1e-15)          # u2 = 0: cos 1, sin 0
    np.testing.assert_allclose(z[1, :2], [0.0, r], atol=1e-12)          # u2 = 1/4
    np.testing.assert_allclose(z[1, 2:], [0.0, -r], atol=1e-12)         # u2 = 3/4


def test_latent_normals_are_standard_normal_and_distinct():
    shape = (4, 50, 51)                                                  # count not a multiple of 4
    z = sde.latent_normals(shape, candidate=3, step=5, seed=0x1234_5678_9ABC)
    assert z.shape == shape
    ks = stats.kstest(z.reshape(-1), "norm")
    assert ks.pvalue > 1e-3
    assert abs(z.mean()) < 0.05 and abs(z.std() - 1.0) < 0.05
    # every counter field and both key words change the draw
    for other in (sde.latent_normals(shape, 4, 5, 0x1234_5678_9ABC),
                  sde.latent_normals(shape, 3, 6, 0x1234_5678_9ABC),
                  sde.latent_normals(shape, 3, 5, 0x1234_5678_9ABD),
                  sde.latent_normals(shape, 3, 5, 0x1235_5678_9ABC)):
        assert abs(np.corrcoef(z.reshape(-1), other.reshape(-1))[0, 1]) < 0.05
    # element e uses normal e % 4 of counter (e // 4, candidate, step, 0)
    w = sde.philox4x32_10(np.array([7, 3, 5, 0], np.uint64), (0x5678_9ABC, 0x1234))
    np.testing.assert_array_equal(z.reshape(-1)[28:32], sde.box_muller(w))


def test_sigma_schedule():
    assert sde.sigma(0.5, 0.4, 0.3) == pytest.approx(0.3)
    assert sde.sigma(0.8, 0.7, 0.3) == pytest.approx(0.6)
    assert sde.sigma(1.0, 0.9, 0.3) == pytest.approx(0.3 * np.sqrt(10.0))  # t = 1: 1 - t_next
    assert sde.sigma(0.3, 0.2, 0.0) == 0.0


def test_a_zero_is_euler_bit_exact():
    rng = np.random.default_rng(1)
    x, v, eps = rng.standard_normal((3, 16, 8, 8))
    for tc, tn in ((1.0, 0.95), (0.6, 0.5), (0.05, 0.0)):
        np.testing.assert_array_equal(sde.sde_update(x, v, tc, tn, 0.0, eps), x + (tn - tc) * v)


MU, SD = 1.5, 0.5                       # data law N(MU, SD^2); noise at t = 1 is N(0, 1)


def _gauss_velocity(x, t):
    """Exact rectified-flow velocity E[x1 - x0 | x_t = x] for x_t = (1 - t) x0 + t x1."""
    m, var = (1 - t) * MU, (1 - t) ** 2 * SD ** 2 + t * t
    return t * (x - m) / var - (MU + (1 - t) * SD ** 2 * (x - m) / var)


def test_score_identity_gaussian():
    for t in (0.1, 0.37, 0.9):
        x = np.linspace(-3, 3, 13)
        m, var = (1 - t) * MU, (1 - t) ** 2 * SD ** 2 + t * t
        np.testing.assert_allclose(-(x + (1 - t) * _gauss_velocity(x, t)) / t, -(x - m) / var, atol=1e-13)


@pytest.mark.parametrize("a", [0.0, 0.3, 0.7])
def test_sde_preserves_marginal_gaussian(a):
    rng = np.random.default_rng(2)
    x = rng.standard_normal(100_000)
    ts = np.linspace(1.0, 0.0, 201)
    for k in range(200):
        x = sde.sde_update(x, _gauss_velocity(x, ts[k]), ts[k], ts[k + 1], a, rng.standard_normal(x.shape))
    assert abs(x.mean() - MU) < 0.01
    assert abs(x.std() / SD - 1.0) < 0.02


def test_step_level_sde_option():
    """draft_step / refine_step with (a = 0, any seed) are the Euler steps bit for bit; with a > 0 the
    two candidates draw different normals and the result differs from Euler by a term whose noise
    part scales as sigma sqrt(|dt|)."""
    from oracle import dit as od_dit
    from tests.test_oracle_pins import _tiny_setup

    wl, W, z, text = _tiny_setup()
    kv = od_dit.prepare_text(W, wl.shape, text)
    L = wl.shape.num_blocks
    zeros = np.zeros(L, np.uint8)
    base, _ = od_dit.draft_step(W, wl.shape, z, 0.75, 0.5, kv, wl.cond_index(), zeros, zeros,
                                od_dit.PoolCache(L))
    a0, _ = od_dit.draft_step(W, wl.shape, z, 0.75, 0.5, kv, wl.cond_index(), zeros, zeros,
                              od_dit.PoolCache(L), sde_args=(0.0, 99, 3))
    np.testing.assert_array_equal(a0, base)
    np.testing.assert_array_equal(
        od_dit.refine_step(W, wl.shape, z, 0.75, 0.5, kv, wl.cond_index(), sde_args=(0.0, 99, 3)), base)
    noisy = od_dit.refine_step(W, wl.shape, z, 0.75, 0.5, kv, wl.cond_index(), sde_args=(0.3, 99, 3))
    v = (base - z) / (0.5 - 0.75)
    sg = 0.3 * np.sqrt(0.75 / 0.25)
    for n in range(z.shape[0]):
        eps = sde.latent_normals(z.shape[1:], n, 3, 99)
        drift = v[n] + sg * sg / 1.5 * (z[n] + 0.25 * v[n])
        np.testing.assert_allclose(noisy[n], z[n] + drift * (-0.25) + sg * 0.5 * eps, rtol=1e-12, atol=1e-12)
    assert not np.allclose(noisy[0] - base[0], noisy[1] - base[1])


def test_clean_estimate_recovers_a_point_mass():
    """For data concentrated at x0 the exact rectified-flow velocity at x_t = (1 - t) x0 + t x1 is
    x1 - x0 = (x_t - x0) / t, and the preview z - t v returns x0 exactly."""
    from oracle import dit as od_dit
    rng = np.random.default_rng(9)
    x0, x1 = rng.standard_normal((2, 4, 6, 6))
    for t in (1.0, 0.73, 0.2):
        xt = (1 - t) * x0 + t * x1
        np.testing.assert_allclose(od_dit.clean_estimate(xt, (xt - x0) / t, t), x0, atol=1e-12)
