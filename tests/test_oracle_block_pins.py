"""Pins of the oracle's block (Eq. 7 under our Wan-shaped reading) beyond the conditioning paths: the
self-attention branch and the cross-attention query path, each isolated by switching the other
branches off and reduced to a closed form through a degenerate attention (no GPU).

* Keys that are the same for every token make every score of a query equal, so softmax is uniform and
  attention returns the mean of the value rows (whatever the queries are).
* With two keys, softmax is a logistic function of the score difference: the output is
  w v1 + (1 - w) v2, w = 1 / (1 + exp(-(q . (k1 - k2)) / sqrt(dh))).

Each test names the plausible mistakes it catches; LayerNorm, the linear orientation and attention
itself are pinned to their textbook definitions in test_oracle_pins.py.
"""
import numpy as np

from oracle import dit as od_dit
from paper_2607_04461_amd import synth

S = synth.TINY            # D = 64, 4 heads of 16, text_dim = 32
T = 16


def _weights(seed=99):
    _, W = synth.make_weights(S, seed)
    return {k: v.astype(np.float64).copy() for k, v in W.items()}


def _tables(rng):
    """Distinct modulation tables per slot (shift1, scale1, gate1, shift2, scale2, gate2)."""
    return rng.standard_normal((6, S.hidden)) * np.array([0.3, 0.2, 0.5, 0.3, 0.2, 0.5])[:, None]


def test_self_attention_branch_with_constant_keys():
    """Constant keys (W_k = 0, b_k != 0): attention returns the mean value row to every query, so the
    block adds g1 (mean_j v_j W_o^T + b_o) with v_j = a_j W_v^T + b_v, a_j = LN(h_j)(1 + scale1) + shift1,
    to every token (MLP gate and cross-attention output switched off).  Caught: queries and keys
    swapped (the keys would then vary by token), values taken from W_k or W_q, b_o or b_v dropped,
    scale1 / shift1 / gate1 taken from another slot, the gate applied outside the projection's bias."""
    rng = np.random.default_rng(1)
    W = _weights()
    mod = _tables(rng)
    mod[5] = 0.0                                     # MLP branch off
    W["blk0.woc"][:] = 0.0
    W["blk0.boc"][:] = 0.0                           # cross-attention branch off
    W["blk0.wk"][:] = 0.0
    W["blk0.bk"][:] = rng.standard_normal(S.hidden)
    h = rng.standard_normal((T, S.hidden))
    kv = od_dit.text_kv(W, 1, rng.standard_normal((5, S.text_dim)))[0]
    out = od_dit.block_forward(W, 0, h, mod, kv, S.heads, S.ln_eps)
    a = od_dit.layer_norm(h, S.ln_eps) * (1.0 + mod[1]) + mod[0]
    v = a @ W["blk0.wv"].T + W["blk0.bv"]
    want = mod[2] * (v.mean(axis=0) @ W["blk0.wo"].T + W["blk0.bo"])
    np.testing.assert_allclose(out - h, np.tile(want, (T, 1)), rtol=1e-9, atol=1e-12)
    # the pin has teeth: the queries vary by token, so swapped roles would not give uniform attention
    q = a @ W["blk0.wq"].T + W["blk0.bq"]
    assert np.abs(q - q.mean(axis=0)).max() > 0.1


def test_self_attention_two_token_logistic_form():
    """Two tokens: each query's output is w v1 + (1 - w) v2 per head, w the logistic function of
    q . (k1 - k2) / sqrt(dh).  With shift1 = 0 and scale1 = 0, a_j = LN(h_j).  Caught: queries and keys
    swapped (the score matrix transposed), the 1/sqrt(dh) scale dropped or taken over D, heads mixed."""
    rng = np.random.default_rng(2)
    W = _weights(7)
    for nm in ("wq", "wk"):
        W[f"blk0.{nm}"][:] *= 20.0                   # scores of order one, so the weights are far from 1/2
    mod = _tables(rng)
    mod[0] = 0.0
    mod[1] = 0.0
    mod[5] = 0.0
    W["blk0.woc"][:] = 0.0
    W["blk0.boc"][:] = 0.0
    h = rng.standard_normal((2, S.hidden))
    kv = od_dit.text_kv(W, 1, rng.standard_normal((3, S.text_dim)))[0]
    out = od_dit.block_forward(W, 0, h, mod, kv, S.heads, S.ln_eps)
    a = od_dit.layer_norm(h, S.ln_eps)
    q = a @ W["blk0.wq"].T + W["blk0.bq"]
    k = a @ W["blk0.wk"].T + W["blk0.bk"]
    v = a @ W["blk0.wv"].T + W["blk0.bv"]
    dh = S.hidden // S.heads
    o = np.empty_like(q)
    for hd in range(S.heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        w = 1.0 / (1.0 + np.exp(-(q[:, sl] @ (k[0, sl] - k[1, sl])) / np.sqrt(dh)))
        o[:, sl] = w[:, None] * v[0, sl] + (1.0 - w[:, None]) * v[1, sl]
    want = mod[2] * (o @ W["blk0.wo"].T + W["blk0.bo"])
    np.testing.assert_allclose(out - h, want, rtol=1e-9, atol=1e-12)
    # the score matrices are not symmetric, so their transposes would give other weights
    asym = max(abs(float(q[0, sl] @ k[1, sl] - q[1, sl] @ k[0, sl]))
               for sl in (slice(hd * dh, (hd + 1) * dh) for hd in range(S.heads)))
    assert asym > 0.1


def test_cross_attention_query_path_two_text_tokens():
    """Cross-attention over a two-token prompt: the query is c W_qc^T + b_qc with the plain (unmodulated)
    LayerNorm c = LN(h) of the stream after the self-attention branch, and the output is the logistic
    mix of the two value rows.  Self-attention and MLP gates off (so that stream is h itself).  Caught:
    a modulated LayerNorm (scale1/shift1 or scale2/shift2) in the cross query, b_qc dropped, W_qc
    transposed, the cross-attention output taken from the self-attention weights."""
    rng = np.random.default_rng(3)
    W = _weights(11)
    W["blk0.wqc"][:] *= 20.0
    W["blk0.wkc"][:] *= 20.0
    mod = _tables(rng)
    mod[2] = 0.0
    mod[5] = 0.0
    h = rng.standard_normal((T, S.hidden))
    text = rng.standard_normal((2, S.text_dim))
    kc, vc = od_dit.text_kv(W, 1, text)[0]
    out = od_dit.block_forward(W, 0, h, mod, (kc, vc), S.heads, S.ln_eps)
    qc = od_dit.layer_norm(h, S.ln_eps) @ W["blk0.wqc"].T + W["blk0.bqc"]
    dh = S.hidden // S.heads
    o = np.empty_like(qc)
    for hd in range(S.heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        w = 1.0 / (1.0 + np.exp(-(qc[:, sl] @ (kc[0, sl] - kc[1, sl])) / np.sqrt(dh)))
        o[:, sl] = w[:, None] * vc[0, sl] + (1.0 - w[:, None]) * vc[1, sl]
    want = o @ W["blk0.woc"].T + W["blk0.boc"]
    np.testing.assert_allclose(out - h, want, rtol=1e-9, atol=1e-12)
    # the weights do vary across queries (the query path matters in this case)
    w0 = 1.0 / (1.0 + np.exp(-(qc[:, :dh] @ (kc[0, :dh] - kc[1, :dh])) / np.sqrt(dh)))
    assert w0.max() - w0.min() > 0.2


def test_branches_add_in_order_on_the_residual_stream():
    """The three branches compose sequentially: the cross-attention query sees the stream after the
    self-attention update, and the MLP's adaLN sees the stream after both.  With every branch on, the
    block equals applying the three single-branch blocks one after another (each with the other two
    switched off).  Caught: the cross or MLP branch reading the block input instead of the running
    stream, two branches' updates applied from the same input."""
    rng = np.random.default_rng(4)
    W = _weights(13)
    mod = _tables(rng)
    h = rng.standard_normal((T, S.hidden))
    text = rng.standard_normal((5, S.text_dim))
    kv = od_dit.text_kv(W, 1, text)[0]
    full = od_dit.block_forward(W, 0, h, mod, kv, S.heads, S.ln_eps)

    def only(branch, x):
        W2 = dict(W)
        m2 = mod.copy()
        if branch != "self":
            m2[2] = 0.0
        if branch != "mlp":
            m2[5] = 0.0
        if branch != "cross":
            W2["blk0.woc"] = np.zeros_like(W["blk0.woc"])
            W2["blk0.boc"] = np.zeros_like(W["blk0.boc"])
        return od_dit.block_forward(W2, 0, x, m2, kv, S.heads, S.ln_eps)

    seq = only("mlp", only("cross", only("self", h)))
    np.testing.assert_allclose(full, seq, rtol=1e-10, atol=1e-12)
    assert np.abs(full - only("self", h)).max() > 1e-3
