"""Pins of the oracle's conditioning paths (no GPU): the timestep -> modulation chain, the text
projection -> per-block cross-attention K/V, and the routing of each candidate to its prompt.

The paper does not describe the network (it only says the denoiser is a U-Net or a DiT, Sec. 3), so
these paths follow our Wan-shaped reading of the block of Eq. 7.  Each test below sets the weights to
permutations, scaled identities or constants so that the path's output has a closed form written by
index, and names the plausible mistake it catches.  SiLU, LayerNorm, attention and the timestep
features themselves are pinned to their textbook definitions in test_oracle_pins.py.
"""
import numpy as np
import pytest

from oracle import dit as od_dit
from paper_2607_04461_amd import synth

S = synth.TINY            # D = 64, freq_dim = 64, text_dim = 32, 4 heads


def _weights():
    _, W = synth.make_weights(S, 4321)
    return {k: v.astype(np.float64).copy() for k, v in W.items()}


def _perm_matrix(perm, scale=1.0):
    """P with P[i, perm[i]] = scale, so (x P^T)[i] = scale * x[perm[i]]."""
    n = len(perm)
    P = np.zeros((n, n))
    P[np.arange(n), perm] = scale
    return P


def _silu(x):
    return x / (1.0 + np.exp(-x))


def _non_involution(n, seed):
    """A permutation that is not its own inverse, so a transposed weight gives a different result."""
    rng = np.random.default_rng(seed)
    while True:
        p = rng.permutation(n)
        if not np.array_equal(p[p], np.arange(n)):
            return p


def test_modulation_chain_closed_form():
    """Timestep path (our reading of the conditioning): e = W_t2 SiLU(W_t1 f + b_t1) + b_t2,
    m = W_m SiLU(e) + b_m split into six D-vectors per block (plus the block's table), and the head's
    (shift, scale) = W_hm SiLU(e) + b_hm.

    With W_t1 = P_a (a permutation), W_t2 = 2 P_b, W_m = six scaled identities c_j I and
    W_hm = [3 I; -0.5 I] every output is a closed form by index.  Caught: a SiLU dropped or moved
    (e.g. after W_t2 instead of before it), a transposed W_t1 / W_t2, the six slots permuted, the
    head taking e instead of SiLU(e), a dropped bias or table."""
    D, fd = S.hidden, S.freq_dim
    W = _weights()
    pa, pb = _non_involution(fd, 1), _non_involution(D, 2)
    W["t_w1"][:] = _perm_matrix(pa)
    W["t_w2"][:] = _perm_matrix(pb, 2.0)
    c = np.array([0.5, -1.0, 1.5, 2.0, -0.25, 3.0])
    W["mod_w"][:] = np.concatenate([cj * np.eye(D) for cj in c])
    W["head_mod_w"][:] = np.concatenate([3.0 * np.eye(D), -0.5 * np.eye(D)])
    for l in range(S.num_blocks):
        W[f"blk{l}.mod"][:] = np.random.default_rng(30 + l).standard_normal((6, D))
    t = 0.37
    f = od_dit.timestep_features(t, fd)
    pre = f[pa] + W["t_b1"]                       # (W_t1 f)[i] = f[pa[i]]
    e = 2.0 * _silu(pre)[pb] + W["t_b2"]          # (W_t2 x)[i] = 2 x[pb[i]]
    s = _silu(e)
    m = np.stack([c[j] * s + W["mod_b"][j * D:(j + 1) * D] for j in range(6)])
    bm, hm = od_dit.modulations(W, S.num_blocks, fd, t)
    for l in range(S.num_blocks):
        np.testing.assert_allclose(bm[l], m + W[f"blk{l}.mod"], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(hm[0], 3.0 * s + W["head_mod_b"][:D], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(hm[1], -0.5 * s + W["head_mod_b"][D:], rtol=1e-13, atol=1e-13)
    # the reading's SiLUs matter at these values: without them the result moves far beyond rounding
    assert np.abs(_silu(pre) - pre).max() > 0.1 and np.abs(s - e).max() > 0.1


def test_text_kv_closed_form():
    """Text path (our reading): ctx = text W_txt^T + b_txt; per block K = ctx W_kc^T + b_kc and
    V = ctx W_vc^T + b_vc.

    With W_txt a (scaled) selection of text columns and W_kc, W_vc two different permutations (V's
    scaled by 2), K and V are closed forms by index.  Caught: W_kc and W_vc swapped, b_txt dropped, a
    transposed weight, K and V biases swapped, the same block's K/V used for every block."""
    D, Dt = S.hidden, S.text_dim
    W = _weights()
    rho = _non_involution(Dt, 3)
    W["txt_w"][:] = 0.0
    W["txt_w"][np.arange(Dt), rho] = 1.0                          # ctx[:, i] = text[:, rho[i]], i < Dt
    W["txt_w"][Dt + np.arange(D - Dt), np.arange(D - Dt)] = 0.5   # ctx[:, Dt + j] = 0.5 text[:, j]
    alphas, betas = [], []
    for l in range(S.num_blocks):
        a, b = _non_involution(D, 10 + l), _non_involution(D, 20 + l)
        W[f"blk{l}.wkc"][:] = _perm_matrix(a)
        W[f"blk{l}.wvc"][:] = _perm_matrix(b, 2.0)
        alphas.append(a)
        betas.append(b)
    text = np.random.default_rng(5).standard_normal((7, Dt))
    ctx = np.concatenate([text[:, rho], 0.5 * text[:, :D - Dt]], axis=1) + W["txt_b"]
    kv = od_dit.text_kv(W, S.num_blocks, text)
    assert len(kv) == S.num_blocks
    for l in range(S.num_blocks):
        k, v = kv[l]
        np.testing.assert_allclose(k, ctx[:, alphas[l]] + W[f"blk{l}.bkc"], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(v, 2.0 * ctx[:, betas[l]] + W[f"blk{l}.bvc"], rtol=1e-13, atol=1e-13)


def _gates_off(W):
    """Zero the shared modulation and both gates (table rows 2 and 5): the self-attention and MLP
    branches then add nothing, and a block adds exactly its cross-attention branch."""
    W["mod_w"][:] = 0.0
    W["mod_b"][:] = 0.0
    for l in range(S.num_blocks):
        W[f"blk{l}.mod"][2] = 0.0
        W[f"blk{l}.mod"][5] = 0.0


def test_one_token_prompt_cross_attention_adds_its_value_row():
    """Softmax over a single key is 1 whatever the scores, so with a one-token prompt cross-attention
    returns that token's value row, and a block whose self-attention and MLP gates are zero adds
    (ctx W_vc^T + b_vc) W_oc^T + b_oc to every token, ctx = x W_txt^T + b_txt (Eq. 7 under our block
    reading).  Caught: K used as the value, b_txt or b_vc dropped, the output projection or its bias
    skipped, the cross-attention branch gated."""
    W = _weights()
    _gates_off(W)
    x = np.random.default_rng(6).standard_normal((1, S.text_dim))
    kv = od_dit.text_kv(W, S.num_blocks, x)
    h = np.random.default_rng(7).standard_normal((16, S.hidden))
    bm, _ = od_dit.modulations(W, S.num_blocks, S.freq_dim, 0.5)
    ctx = x @ W["txt_w"].T + W["txt_b"]
    for l in range(S.num_blocks):
        vrow = ctx @ W[f"blk{l}.wvc"].T + W[f"blk{l}.bvc"]
        want = vrow @ W[f"blk{l}.woc"].T + W[f"blk{l}.boc"]
        out = od_dit.block_forward(W, l, h, bm[l], kv[l], S.heads, S.ln_eps)
        np.testing.assert_allclose(out - h, np.tile(want, (16, 1)), rtol=1e-10, atol=1e-13)
        # the same through K in place of V would differ
        krow = ctx @ W[f"blk{l}.wkc"].T + W[f"blk{l}.bkc"]
        assert np.abs((krow - vrow) @ W[f"blk{l}.woc"].T).max() > 1e-3


def test_cond_index_routes_each_candidate_to_its_prompt():
    """Candidates of one pool may carry different prompts (Eq. 8: each draft is x's sample; our
    workloads split a pool over several prompts).  Two prompts whose tokens are all equal give
    constant value rows V_c, so cross-attention returns V_c for every query; with the other branches
    gated off, block l of candidate n adds V_{cond[n]} W_oc^T + b_oc.  Caught: cond_index ignored (every
    candidate on prompt 0), or indexed by the wrong candidate."""
    W = _weights()
    _gates_off(W)
    rng = np.random.default_rng(8)
    u = rng.standard_normal((2, S.text_dim))
    text = np.stack([np.tile(u[0], (5, 1)), np.tile(u[1], (5, 1))])        # [n_cond=2, 5, Dt]
    kv = od_dit.prepare_text(W, S, text)
    z = synth.make_latents(3, 16, 8, 8).astype(np.float64)
    cond = np.array([1, 0, 1], np.int32)
    zeros = np.zeros(S.num_blocks, np.uint8)
    hidden = {}
    od_dit.draft_step(W, S, z, 0.8, 0.6, kv, cond, zeros, zeros, od_dit.PoolCache(S.num_blocks),
                      hidden=hidden)
    want = []
    for c in range(2):
        ctx = u[c] @ W["txt_w"].T + W["txt_b"]
        want.append([(ctx @ W[f"blk{l}.wvc"].T + W[f"blk{l}.bvc"]) @ W[f"blk{l}.woc"].T + W[f"blk{l}.boc"]
                     for l in range(S.num_blocks)])
    for n in range(3):
        for l in range(S.num_blocks):
            delta = hidden[n][l + 1] - hidden[n][l]
            np.testing.assert_allclose(delta, np.tile(want[cond[n]][l], (16, 1)), rtol=1e-10, atol=1e-13)
    assert np.abs(want[0][0] - want[1][0]).max() > 1e-3


@pytest.mark.parametrize("t", [1.0, 0.5, 0.02])
def test_modulation_depends_on_t_only_through_the_features(t):
    """The conditioning is a function of t_k alone (shared by every candidate): two evaluations at the
    same t agree bit for bit, and the block tables enter additively (Eq. 7's B_l(h, x, t))."""
    W = _weights()
    a = od_dit.modulations(W, S.num_blocks, S.freq_dim, t)
    b = od_dit.modulations(W, S.num_blocks, S.freq_dim, t)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    np.testing.assert_allclose(a[0][1] - a[0][0], W["blk1.mod"] - W["blk0.mod"], rtol=0, atol=1e-15)
