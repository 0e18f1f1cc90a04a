"""Kernel-level parity on the GPU: each HIP kernel of the draft step against the CPU oracle's op on
identical seeded inputs, at small ragged shapes (every element) and at the real model shapes
(sampled rows / all elements where cheap).

Tolerances (relative L2 over the compared elements):
  * fp32 operands, fp32 result: 2e-6 (fp32 rounding over K <= 8960 accumulations);
  * bf16 operands (exactly representable, drawn via round_to_bf16), fp32 result: 2e-6;
  * bf16 result: 6e-3 (one bf16 rounding of the output, 2^-9 relative, is the dominant term);
  * attention with bf16 operands: 1e-2 (bf16 rounding of the probabilities before P.V plus output).
"""
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


def fb():
    from paper_2607_04461_amd import flashbon
    return flashbon


def _dev(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to("cuda").to(torch.bfloat16 if dtype == "bf16" else torch.float32)


def _operand(shape, seed, dtype, scale=1.0):
    a = synth.random_matrix(shape, seed, scale)
    return synth.round_to_bf16(a) if dtype == "bf16" else a


LINEAR_SMALL = [(200, 136, 72), (1, 4, 8), (130, 64, 64), (257, 260, 264)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("M,N,K", LINEAR_SMALL)
@pytest.mark.parametrize("epi", ["store", "gelu", "store_f32", "residual"])
def test_linear_small(dtype, M, N, K, epi):
    F = fb()
    dt = F.BF16 if dtype == "bf16" else F.FP32
    A = _operand((M, K), 1, dtype)
    W = _operand((N, K), 2, dtype, 0.05)
    bias = synth.random_matrix((N,), 3)
    gate = synth.random_matrix((N,), 4)
    h0 = synth.random_matrix((M, N), 5)
    ref = odit.linear(A.astype(np.float64), W, bias)
    dA, dW, db, dg = _dev(A, dtype), _dev(W, dtype), _dev(bias, "fp32"), _dev(gate, "fp32")
    if epi in ("store", "gelu"):
        out = torch.empty((M, N), device="cuda", dtype=dA.dtype)
        code = F.EPI_STORE if epi == "store" else F.EPI_GELU
        F.flashbon_op_linear(dt, M, N, K, dA, dW, db, code, out)
        if epi == "gelu":
            ref = odit.gelu_tanh(ref)
        tol = 6e-3 if dtype == "bf16" else 2e-6
    elif epi == "store_f32":
        out = torch.empty((M, N), device="cuda", dtype=torch.float32)
        F.flashbon_op_linear(dt, M, N, K, dA, dW, db, F.EPI_STORE_F32, out)
        tol = 2e-6
    else:
        out = _dev(h0, "fp32")
        cache = torch.zeros((M, N), device="cuda", dtype=torch.float32)
        F.flashbon_op_linear(dt, M, N, K, dA, dW, db, F.EPI_RESIDUAL, out, dg, cache)
        ref = h0 + gate * ref
        torch.cuda.synchronize()
        assert torch.equal(cache, out)
        tol = 2e-6
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert rel_l2(got, ref) <= tol


@pytest.mark.parametrize("tile", ["256x256", "128x128", "split:256", "bm:224", "bm:192", "bm:160", "mix:7:3:1",
                                  "mix:8:3:1", "mix:6:4:2", "w8", "w8:bm:160", "w8:mix:7:3:1", "w8:mix:8:3:1",
                                  "deep:128:128:2", "deep:128:128:3", "deep:160:128:3", "deep:128:256:2",
                                  "deep:128:256:3", "deep:160:256:2", "deep:160:256:3"])
@pytest.mark.parametrize("M,N,K", [(200, 136, 72), (517, 300, 640), (256, 256, 64), (1, 4, 8), (300, 520, 192),
                                   (520, 776, 1024), (300, 520, 128), (1, 8, 128), (33, 264, 128)])
@pytest.mark.parametrize("epi", ["gelu", "residual"])
def test_linear_each_tile_kernel(tile, M, N, K, epi, monkeypatch):
    """Every MFMA tiling (forced: "256x256" is the 8-wave kernel with LDS-writing loads when K % 64 == 0
    and K >= 128, else the 8-wave kernel; "split:256" puts rows 0..255 on 256x256 tiles and the rest
    on 128x128 tiles, when M > 256 and K % 64 == 0; "bm:<rows>" the 4-wave kernel with tiles of one
    height; "mix:w:blocks:tall" the 4-wave kernel with row blocks of two heights, 32 w and 32 (w - 1)
    rows, spread over the blocks; "w8", "w8:bm:<rows>", "w8:mix:..." the 8-wave kernel with LDS-writing
    loads on the same row blocks; "deep:<rows>:<cols>:<stages>" the 8-wave tile with a deeper LDS ring,
    whose K loop is shorter than its ring for the smaller K; plans the
    shape cannot take fall back to 256x256) on ragged M, N
    and K tails, against the oracle.
    The residual case also writes the cache copy."""
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", tile)
    F = fb()
    A = _operand((M, K), 71, "bf16")
    W = _operand((N, K), 72, "bf16", 0.05)
    bias = synth.random_matrix((N,), 73)
    ref = odit.linear(A.astype(np.float64), W, bias)
    if epi == "gelu":
        out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        F.flashbon_op_linear(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"), F.EPI_GELU, out)
        ref, tol = odit.gelu_tanh(ref), 6e-3
    else:
        h0 = synth.random_matrix((M, N), 74)
        gate = synth.random_matrix((N,), 75)
        out = _dev(h0, "fp32")
        cache = torch.full((M, N), 7.0, device="cuda", dtype=torch.float32)
        F.flashbon_op_linear(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"),
                             F.EPI_RESIDUAL, out, _dev(gate, "fp32"), cache)
        ref, tol = h0 + gate * ref, 2e-6
        torch.cuda.synchronize()
        assert torch.equal(cache, out)
    torch.cuda.synchronize()
    assert rel_l2(out.float().cpu().numpy(), ref) <= tol


@pytest.mark.parametrize("epi", ["store", "store_bf16", "gelu", "residual"])
def test_linear_tile_plans_bit_identical(epi, monkeypatch):
    """Every tiling accumulates K in the same order, so an output element does not depend on the tile
    that computed it: all plans give bit-identical results (this is what keeps a candidate's draft
    independent of its position in the pool).  The bf16 store and GELU epilogues of the 256-column
    8-wave tiles and every residual epilogue of the 8-wave tiles pass through LDS; the 4-wave kernels'
    do not, so the comparison also pins the staged epilogues to the direct ones."""
    F = fb()
    M, N, K = 1100, 776, 512
    A = _dev(_operand((M, K), 81, "bf16"), "bf16")
    W = _dev(_operand((N, K), 82, "bf16", 0.05), "bf16")
    bias = _dev(synth.random_matrix((N,), 83), "fp32")
    gate = _dev(synth.random_matrix((N,), 84), "fp32")
    h0 = _dev(synth.random_matrix((M, N), 85), "fp32")
    outs = []
    for tile in ["256x256", "128x128", "split:512", "bm:224", "bm:192", "bm:160", "mix:7:6:1", "mix:8:5:1",
                 "mix:6:7:3", "w8", "w8:bm:224", "w8:bm:192", "w8:bm:160", "w8:mix:7:6:1", "w8:mix:6:7:3",
                 "deep:128:128:2", "deep:128:128:3", "deep:160:128:2", "deep:160:128:3", "deep:128:256:2",
                 "deep:128:256:3", "deep:160:256:2", "deep:160:256:3"]:
        monkeypatch.setenv("FLASHBON_LINEAR_TILE", tile)
        if epi == "store":
            out = torch.empty((M, N), device="cuda", dtype=torch.float32)
            F.flashbon_op_linear(F.BF16, M, N, K, A, W, bias, F.EPI_STORE_F32, out)
        elif epi in ("store_bf16", "gelu"):
            out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
            F.flashbon_op_linear(F.BF16, M, N, K, A, W, bias, F.EPI_STORE if epi == "store_bf16" else F.EPI_GELU, out)
        else:
            out = h0.clone()
            F.flashbon_op_linear(F.BF16, M, N, K, A, W, bias, F.EPI_RESIDUAL, out, gate)
        torch.cuda.synchronize()
        outs.append(out)
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


@pytest.mark.parametrize("tile", [None, "256x256", "128x128", "split:256", "bm:192", "mix:7:3:1", "w8"])
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_linear_residual_separate_source(tile, dtype, monkeypatch):
    """out = residual_in + gate (A W^T + bias) with the residual rows read from another buffer (the
    draft step's self-attention output projection reads the stream from the previous block's cache
    slot): matches the oracle, leaves residual_in untouched, and equals the in-place update bit for bit
    (every tiling; ragged M, N and K)."""
    if tile is None:
        monkeypatch.delenv("FLASHBON_LINEAR_TILE", raising=False)
    else:
        monkeypatch.setenv("FLASHBON_LINEAR_TILE", tile)
    F = fb()
    M, N, K = 517, 300, 640
    A = _operand((M, K), 91, dtype)
    W = _operand((N, K), 92, dtype, 0.05)
    bias = synth.random_matrix((N,), 93)
    gate = synth.random_matrix((N,), 94)
    h0 = synth.random_matrix((M, N), 95)
    dt = F.BF16 if dtype == "bf16" else F.FP32
    res = _dev(h0, "fp32")
    out = torch.full((M, N), 3.0, device="cuda", dtype=torch.float32)
    Ad, Wd, bd, gd = _dev(A, dtype), _dev(W, dtype), _dev(bias, "fp32"), _dev(gate, "fp32")
    F.flashbon_op_linear_residual(dt, M, N, K, Ad, Wd, bd, gd, res, out)
    inplace = _dev(h0, "fp32")
    F.flashbon_op_linear(dt, M, N, K, Ad, Wd, bd, F.EPI_RESIDUAL, inplace, gd)
    torch.cuda.synchronize()
    assert torch.equal(res, _dev(h0, "fp32"))
    assert torch.equal(out, inplace)
    ref = h0 + gate * odit.linear(A.astype(np.float64), W, bias)
    assert rel_l2(out.cpu().numpy(), ref) <= 2e-6


def test_linear_tile_orders_bit_identical(monkeypatch):
    """The 4-wave kernel's tile order (groups of 1..8 row blocks sweeping the column tiles, groups that
    do not divide the row blocks, two tile heights) moves tiles between XCDs and rounds only: outputs
    are bit-identical to the default order and match the oracle."""
    F = fb()
    M, N, K = 1100, 1800, 256
    A_h = _operand((M, K), 86, "bf16")
    W_h = _operand((N, K), 87, "bf16", 0.05)
    bias_h = synth.random_matrix((N,), 88)
    A, W, bias = _dev(A_h, "bf16"), _dev(W_h, "bf16"), _dev(bias_h, "fp32")
    ref = odit.linear(A_h.astype(np.float64), W_h, bias_h)
    for tile in ["bm:160", "mix:7:6:1", "w8", "w8:mix:7:6:1"]:
        monkeypatch.setenv("FLASHBON_LINEAR_TILE", tile)
        outs = []
        for group in [None, 1, 2, 3, 5, 8, 16]:
            if group is None:
                monkeypatch.delenv("FLASHBON_LINEAR_GROUP", raising=False)
            else:
                monkeypatch.setenv("FLASHBON_LINEAR_GROUP", str(group))
            out = torch.empty((M, N), device="cuda", dtype=torch.float32)
            F.flashbon_op_linear(F.BF16, M, N, K, A, W, bias, F.EPI_STORE_F32, out)
            torch.cuda.synchronize()
            outs.append(out)
        assert rel_l2(outs[0].cpu().numpy(), ref) <= 2e-6
        for o in outs[1:]:
            assert torch.equal(o, outs[0])


@pytest.mark.parametrize("M,N,K", [(24960, 4608, 1536), (24960, 8960, 1536), (24960, 1536, 8960),
                                   (24960, 64, 1536), (16384, 15360, 5120)])
def test_linear_full_shapes_bf16_sampled_rows(M, N, K):
    F = fb()
    A = _operand((M, K), 11, "bf16")
    W = _operand((N, K), 12, "bf16", 0.02)
    bias = synth.random_matrix((N,), 13)
    out = torch.empty((M, N), device="cuda", dtype=torch.float32)
    F.flashbon_op_linear(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"),
                         F.EPI_STORE_F32, out)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.random.default_rng(14).integers(0, M, 48), [0, 127, 128, M - 1]]))
    got = out[torch.from_numpy(rows).cuda()].cpu().numpy()
    ref = odit.linear(A[rows].astype(np.float64), W, bias)
    assert rel_l2(got, ref) <= 2e-6


def _attn_ref(q, k, v, heads):
    return odit.multi_head_attention(q.astype(np.float64), k.astype(np.float64), v.astype(np.float64), heads)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("heads,dh,tq,tk", [(2, 128, 130, 130), (4, 16, 16, 8), (3, 64, 70, 200),
                                            (1, 128, 1, 1), (2, 128, 67, 40)])
def test_attention_small(dtype, heads, dh, tq, tk):
    F = fb()
    dt = F.BF16 if dtype == "bf16" else F.FP32
    B = 3
    D = heads * dh
    q = _operand((B, tq, D), 21, dtype)
    k = _operand((B, tk, D), 22, dtype)
    v = _operand((B, tk, D), 23, dtype)
    out = torch.empty((B, tq, D), device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)
    F.flashbon_op_attention(dt, B, heads, dh, tq, tk, _dev(q, dtype), tq * D, D, _dev(k, dtype), _dev(v, dtype),
                            tk * D, D, None, 0, out, tq * D, D)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    ref = np.stack([_attn_ref(q[b], k[b], v[b], heads) for b in range(B)])
    assert rel_l2(got, ref) <= (1e-2 if dtype == "bf16" else 2e-6)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_cross_attention_kv_index(dtype):
    F = fb()
    dt = F.BF16 if dtype == "bf16" else F.FP32
    B, NC, heads, dh, tq, tk = 5, 3, 2, 128, 33, 40
    D = heads * dh
    q = _operand((B, tq, D), 31, dtype)
    kv = _operand((NC, tk, 2 * D), 32, dtype)       # per prompt rows [K | V]
    idx = np.array([2, 0, 1, 1, 2], np.int32)
    dkv = _dev(kv, dtype)
    out = torch.empty((B, tq, D), device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)
    F.flashbon_op_attention(dt, B, heads, dh, tq, tk, _dev(q, dtype), tq * D, D, dkv, dkv[..., D:],
                            tk * 2 * D, 2 * D, torch.from_numpy(idx).cuda(), NC, out, tq * D, D)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    ref = np.stack([_attn_ref(q[b], kv[idx[b], :, :D], kv[idx[b], :, D:], heads) for b in range(B)])
    assert rel_l2(got, ref) <= (1e-2 if dtype == "bf16" else 2e-6)


@pytest.mark.parametrize("tq,tk", [(1, 1), (130, 64), (129, 128), (200, 65), (67, 192), (100, 256),
                                   (33, 255), (64, 257), (160, 321), (128, 384)])
def test_attention_mfma_kernel_tile_edges(tq, tk):
    """The head_dim-128 bf16 kernel over key counts that give one key, 1 to 6 64-key tiles (odd and even
    counts: the step loop runs in pairs and peels the last one or two), full tiles only, a one-key
    ragged tail and a one-key-short one, with query blocks that end mid-wave or leave whole waves idle;
    one of the batches reads its keys through the kv index."""
    F = fb()
    B, NC, heads, dh = 3, 2, 2, 128
    D = heads * dh
    q = _operand((B, tq, D), 51, "bf16")
    kv = _operand((NC, tk, 2 * D), 52, "bf16")
    idx = np.array([1, 0, 1], np.int32)
    dkv = _dev(kv, "bf16")
    out = torch.empty((B, tq, D), device="cuda", dtype=torch.bfloat16)
    F.flashbon_op_attention(F.BF16, B, heads, dh, tq, tk, _dev(q, "bf16"), tq * D, D, dkv, dkv[..., D:],
                            tk * 2 * D, 2 * D, torch.from_numpy(idx).cuda(), NC, out, tq * D, D)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    ref = np.stack([_attn_ref(q[b], kv[idx[b], :, :D], kv[idx[b], :, D:], heads) for b in range(B)])
    assert rel_l2(got, ref) <= 1e-2


@pytest.mark.parametrize("lazy", ["1", "0"])
@pytest.mark.parametrize("order", ["rising", "falling"])
def test_attention_lazy_rescale_moving_maximum(lazy, order, monkeypatch):
    """Keys scaled so that the logits grow (or shrink) by far more than the lazy-rescale margin from
    one 64-key tile to the next: with "rising" the running maximum has to move on every tile, with
    "falling" only on the first.  Both settings of FLASHBON_ATTN_LAZY match the fp64 softmax."""
    monkeypatch.setenv("FLASHBON_ATTN_LAZY", lazy)
    F = fb()
    heads, dh, tq, tk = 2, 128, 130, 321
    D = heads * dh
    q = _operand((1, tq, D), 61, "bf16")
    ramp = np.linspace(0.5, 12.0, tk) if order == "rising" else np.linspace(12.0, 0.5, tk)
    k = synth.round_to_bf16(_operand((tk, D), 62, "bf16") * ramp[:, None].astype(np.float32))
    v = _operand((tk, D), 63, "bf16")
    out = torch.empty((1, tq, D), device="cuda", dtype=torch.bfloat16)
    F.flashbon_op_attention(F.BF16, 1, heads, dh, tq, tk, _dev(q, "bf16"), tq * D, D, _dev(k, "bf16"),
                            _dev(v, "bf16"), tk * D, D, None, 0, out, tq * D, D)
    torch.cuda.synchronize()
    got = out[0].float().cpu().numpy()
    assert np.isfinite(got).all()
    assert rel_l2(got, _attn_ref(q[0], k, v, heads)) <= 1e-2


@pytest.mark.parametrize("B,heads,T,tk", [(16, 12, 1560, 1560), (16, 12, 1560, 512), (4, 40, 4096, 4096)])
def test_attention_full_shapes_bf16_sampled_queries(B, heads, T, tk):
    F = fb()
    dh = 128
    D = heads * dh
    q = _operand((B, T, D), 41, "bf16")
    k = _operand((B, tk, D), 42, "bf16")
    v = _operand((B, tk, D), 43, "bf16")
    out = torch.empty((B, T, D), device="cuda", dtype=torch.bfloat16)
    F.flashbon_op_attention(F.BF16, B, heads, dh, T, tk, _dev(q, "bf16"), T * D, D, _dev(k, "bf16"),
                            _dev(v, "bf16"), tk * D, D, None, 0, out, T * D, D)
    torch.cuda.synchronize()
    rng = np.random.default_rng(44)
    for b in (0, B - 1):
        rows = np.unique(np.concatenate([rng.integers(0, T, 24), [0, T - 1]]))
        got = out[b][torch.from_numpy(rows).cuda()].float().cpu().numpy()
        ref = _attn_ref(q[b][rows], k[b], v[b], heads)
        assert rel_l2(got, ref) <= 1e-2


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("M,D,mod", [(37, 64, True), (24960, 1536, True), (300, 5120, False), (5, 256, False),
                                     (23, 1000, True), (9, 68, True), (1, 4096, True), (2, 8, False),
                                     (4097, 1536, False), (4099, 1536, True)])
def test_ln_mod(dtype, M, D, mod):
    F = fb()
    dt = F.BF16 if dtype == "bf16" else F.FP32
    x = synth.random_matrix((M, D), 51) * 3 + 1
    sh = synth.random_matrix((D,), 52) if mod else None
    sc = synth.random_matrix((D,), 53) if mod else None
    out = torch.empty((M, D), device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)
    F.flashbon_op_ln_mod(dt, M, D, 1e-6, _dev(x, "fp32"), None if sh is None else _dev(sh, "fp32"),
                         None if sc is None else _dev(sc, "fp32"), out)
    torch.cuda.synchronize()
    ref = odit.layer_norm(x.astype(np.float64), 1e-6)
    if mod:
        ref = ref * (1 + sc) + sh
    assert rel_l2(out.float().cpu().numpy(), ref) <= (6e-3 if dtype == "bf16" else 2e-6)


@pytest.mark.parametrize("count", [38_338_560, 1001])
@pytest.mark.parametrize("order", [0, 1, 2])
def test_proxy_kernel(count, order):
    F = fb()
    h = synth.random_cache_entries((count,), 61)
    taus, t = (0.62, 0.7, 0.78), 0.5
    d = [_dev(h[i], "fp32") for i in range(3)]
    out = torch.empty(count, device="cuda", dtype=torch.float32)
    F.flashbon_op_proxy(count, d[0], d[1], d[2], order, taus[0], taus[1], t, out)
    torch.cuda.synchronize()
    entries = [(h[i], np.float32(taus[i])) for i in range(3)]
    ref = odit.taylor_proxy(entries, np.float32(t), order)
    assert rel_l2(out.cpu().numpy(), ref) <= 2e-6


def test_proxy_kernel_constant_is_exact():
    F = fb()
    c = torch.full((4099,), 0.3712, device="cuda", dtype=torch.float32)
    out = torch.empty_like(c)
    F.flashbon_op_proxy(4099, c, c, c, 2, 0.25, 0.5, 0.125, out)
    torch.cuda.synchronize()
    assert torch.equal(out, c)


@pytest.mark.parametrize("M,N,K,epi,split", [(24960, 1536, 8960, "residual", 21760), (24960, 8960, 1536, "gelu", 24320)])
def test_linear_tail_rows_split(M, N, K, epi, split):
    """On 256 CUs these shapes leave the last round of 256x256 tiles mostly idle, so rows from `split`
    on run in the 128x128 kernel (a second launch on moved pointers).  Rows on both sides of the
    split and the last row, against the oracle; the RESIDUAL cache copy must follow the output."""
    F = fb()
    A = _operand((M, K), 81, "bf16")
    W = _operand((N, K), 82, "bf16", 0.02)
    bias = synth.random_matrix((N,), 83)
    rows = np.array([0, 255, split - 256, split - 1, split, split + 1, split + 127, split + 128, M - 2, M - 1])
    ref = odit.linear(A[rows].astype(np.float64), W, bias)
    idx = torch.from_numpy(rows).cuda()
    if epi == "gelu":
        out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        F.flashbon_op_linear(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"), F.EPI_GELU, out)
        torch.cuda.synchronize()
        assert rel_l2(out[idx].float().cpu().numpy(), odit.gelu_tanh(ref)) <= 6e-3
    else:
        h0 = torch.from_numpy(synth.random_matrix((M, N), 84)).cuda()
        gate = synth.random_matrix((N,), 85)
        out = h0.clone()
        cache = torch.zeros((M, N), device="cuda", dtype=torch.float32)
        F.flashbon_op_linear(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"),
                             F.EPI_RESIDUAL, out, _dev(gate, "fp32"), cache)
        torch.cuda.synchronize()
        assert torch.equal(cache, out)
        expect = h0[idx].cpu().numpy().astype(np.float64) + gate * ref
        assert rel_l2(out[idx].cpu().numpy(), expect) <= 2e-6


@pytest.mark.parametrize("M,N,K,epi", [
    (200, 136, 2048, "store"), (200, 136, 2048, "gelu"), (200, 136, 2048, "store_f32"), (200, 136, 2048, "residual"),
    (1560, 1536, 8960, "residual"),      # one candidate's MLP down-projection (refinement)
    (512, 1536, 4096, "store"),          # the text projection of one 512-token prompt
])
def test_linear_splitk_with_workspace(M, N, K, epi):
    """The split-K plan of the linear layers (K ranges of partial sums in a workspace, added in order
    before the epilogue) against the fp64 reference, at a ragged small shape and at the refinement's
    shapes; the plan must actually split there, and a workspace too small falls back to one range."""
    F = fb()
    A = _operand((M, K), 11, "bf16")
    W = _operand((N, K), 12, "bf16", 0.02)
    bias = synth.random_matrix((N,), 13, 0.02)
    gate = synth.random_matrix((N,), 14)
    h0 = synth.random_matrix((M, N), 15)
    dA, dW, db, dg = _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"), _dev(gate, "fp32")
    ws = torch.empty(48 << 18, device="cuda", dtype=torch.float32)          # 48 MiB
    code = {"store": F.EPI_STORE, "gelu": F.EPI_GELU, "store_f32": F.EPI_STORE_F32, "residual": F.EPI_RESIDUAL}[epi]
    rows = np.arange(M) if M <= 256 else np.random.default_rng(16).choice(M, 48, replace=False)
    ref = odit.linear(A[rows].astype(np.float64), W, bias)
    if epi == "gelu":
        ref = odit.gelu_tanh(ref)
    outs = []
    for w in (ws, ws[:1024]):
        if epi in ("store", "gelu"):
            out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
            sp = F.flashbon_op_linear_ws(F.BF16, M, N, K, dA, dW, db, code, out, w)
            tol, expect = 6e-3, ref
        elif epi == "store_f32":
            out = torch.empty((M, N), device="cuda", dtype=torch.float32)
            sp = F.flashbon_op_linear_ws(F.BF16, M, N, K, dA, dW, db, code, out, w)
            tol, expect = 2e-6, ref
        else:
            out = _dev(h0, "fp32")
            sp = F.flashbon_op_linear_ws(F.BF16, M, N, K, dA, dW, db, code, out, w, gate=dg)
            tol, expect = 2e-6, h0[rows] + gate * ref
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()[rows].astype(np.float64)
        err = rel_l2(got, expect)
        print(f"linear_ws {M}x{N}x{K} {epi}: {sp} K ranges, rel-L2 {err:.2e}", flush=True)
        assert err <= tol
        outs.append((sp, got))
    assert outs[0][0] > 1, "the plan should split this shape"
    assert outs[1][0] == 1, "a workspace too small for the plan runs one range"


@pytest.mark.parametrize("plan", ["224:256:2:2", "128:128:3:2", "128:128:2:3", "160:128:3:3", "128:256:3:2",
                                  "160:256:3:2", "160:256:2:3"])
@pytest.mark.parametrize("epi", ["gelu", "residual"])
def test_linear_splitk_forced_plans(plan, epi, monkeypatch):
    """Every split-K tile (FLASHBON_SPLITK = rows:cols:stages:ranges) on ragged M and N, against the fp64
    reference: the K ranges of each tile's partial sums, written to the workspace and added in range
    order, must cover K exactly once for every tile shape and ring depth."""
    monkeypatch.setenv("FLASHBON_SPLITK", plan)
    F = fb()
    M, N, K = 300, 520, 3072
    A = _operand((M, K), 21, "bf16")
    W = _operand((N, K), 22, "bf16", 0.02)
    bias = synth.random_matrix((N,), 23, 0.02)
    gate = synth.random_matrix((N,), 24)
    h0 = synth.random_matrix((M, N), 25)
    ws = torch.empty(48 << 18, device="cuda", dtype=torch.float32)
    ref = odit.linear(A.astype(np.float64), W, bias)
    if epi == "gelu":
        out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        sp = F.flashbon_op_linear_ws(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"),
                                     F.EPI_GELU, out, ws)
        expect, tol = odit.gelu_tanh(ref), 6e-3
    else:
        out = _dev(h0, "fp32")
        sp = F.flashbon_op_linear_ws(F.BF16, M, N, K, _dev(A, "bf16"), _dev(W, "bf16"), _dev(bias, "fp32"),
                                     F.EPI_RESIDUAL, out, ws, gate=_dev(gate, "fp32"))
        expect, tol = h0 + gate * ref, 2e-6
    torch.cuda.synchronize()
    assert sp == int(plan.split(":")[3])
    assert rel_l2(out.float().cpu().numpy(), expect) <= tol
