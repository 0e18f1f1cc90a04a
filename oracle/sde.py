"""Oracle of the stochastic flow update (App. A.1, Eq. 20) and its counter-based normal draws.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Eq. 20, with the rectified-flow score of App. A.1 (t = 1 noise, t = 0 data, velocity v):
    x_{t+dt} = x_t + [v + sigma_t^2 / (2 t) (x_t + (1 - t) v)] dt + sigma_t sqrt(|dt|) eps,
    sigma_t = a sqrt(t / (1 - t)),  eps ~ N(0, I).
Readings (the paper is silent): dt = t_next - t_cur < 0 when denoising, so the noise scale uses
sqrt(|dt|); at t = 1 the factor t / (1 - t) is infinite, so 1 - t is replaced by 1 - t_next there.
a = 0 gives exactly the deterministic Euler update.

Normals: eps for latent element e (flat index in [C, H, W]) of candidate n at step s comes from the
Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw, SC'11) with key = seed (two 32-bit
words) and counter = (e // 4, n, s, 0), mapped through the Box-Muller transform: for the output words
(x0, x1, x2, x3), u1 = (x0 + 1) 2^-32, u2 = x1 2^-32 give r = sqrt(-2 ln u1), normals
r cos(2 pi u2), r sin(2 pi u2); (x2, x3) likewise; element e takes normal e % 4.
"""
from __future__ import annotations

import numpy as np

_M0, _M1 = 0xD2511F53, 0xCD9E8D57          # Philox4x32 multipliers
_W0, _W1 = 0x9E3779B9, 0xBB67AE85          # Weyl key increments
_MASK = 0xFFFFFFFF


def _mulhilo(a, b):
    p = a.astype(np.uint64) * np.uint64(b)
    return (p >> np.uint64(32)).astype(np.uint64), (p & np.uint64(_MASK)).astype(np.uint64)


def philox4x32_10(counter, key):
    """counter: uint array [..., 4], key: (k0, k1).  Returns uint64 array [..., 4] of 32-bit words."""
    c = np.asarray(counter, dtype=np.uint64) & np.uint64(_MASK)
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.uint64(key[0] & _MASK)
    k1 = np.uint64(key[1] & _MASK)
    for _ in range(10):
        hi0, lo0 = _mulhilo(c0, _M0)
        hi1, lo1 = _mulhilo(c2, _M1)
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0) & np.uint64(_MASK), lo1, (hi0 ^ c3 ^ k1) & np.uint64(_MASK), lo0
        k0 = (k0 + np.uint64(_W0)) & np.uint64(_MASK)
        k1 = (k1 + np.uint64(_W1)) & np.uint64(_MASK)
    return np.stack([c0, c1, c2, c3], axis=-1)


def box_muller(words):
    """[..., 4] uint words -> [..., 4] standard normals (fp64)."""
    w = np.asarray(words, dtype=np.float64)
    out = np.empty(w.shape, np.float64)
    for a, b in ((0, 1), (2, 3)):
        u1 = (w[..., a] + 1.0) * 2.0 ** -32
        u2 = w[..., b] * 2.0 ** -32
        r = np.sqrt(-2.0 * np.log(u1))
        out[..., a] = r * np.cos(2.0 * np.pi * u2)
        out[..., b] = r * np.sin(2.0 * np.pi * u2)
    return out


def latent_normals(shape_chw, candidate: int, step: int, seed: int) -> np.ndarray:
    """eps for one candidate's latent [C, H, W] at one step."""
    count = int(np.prod(shape_chw))
    quads = (count + 3) // 4
    ctr = np.zeros((quads, 4), np.uint64)
    ctr[:, 0] = np.arange(quads, dtype=np.uint64)
    ctr[:, 1] = candidate
    ctr[:, 2] = step
    key = (seed & _MASK, (seed >> 32) & _MASK)
    z = box_muller(philox4x32_10(ctr, key)).reshape(-1)[:count]
    return z.reshape(shape_chw)


def sigma(t: float, t_next: float, a: float) -> float:
    """sigma_t = a sqrt(t / (1 - t)); at t = 1 the denominator is taken as 1 - t_next."""
    t = float(t)
    one_minus = 1.0 - t if t < 1.0 else 1.0 - float(t_next)
    return a * np.sqrt(t / one_minus)


def sde_update(x, v, t_cur: float, t_next: float, a: float, eps) -> np.ndarray:
    """Eq. 20 for one candidate (fp64)."""
    x = np.asarray(x, np.float64)
    v = np.asarray(v, np.float64)
    dt = float(t_next) - float(t_cur)
    s = sigma(t_cur, t_next, a)
    drift = v + (s * s) / (2.0 * float(t_cur)) * (x + (1.0 - float(t_cur)) * v)
    return x + drift * dt + s * np.sqrt(abs(dt)) * np.asarray(eps, np.float64)
