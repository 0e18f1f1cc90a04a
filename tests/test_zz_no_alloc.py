"""The allocation-free refinement step (flashbon_refine_step_noalloc) against flashbon_refine_step,
through the C ABI: the two share every kernel and its order, so each call must give the same latents
bit for bit.  Two calls in a row, the second with a smaller input (fewer candidates, fewer tokens), so
the second call's buffers are carved anew from a scratch array that still holds the first call's
contents.  Also: sizes beyond the array's limit are rejected before any device work."""
import ctypes

import numpy as np
import pytest

from paper_2607_04461_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04461_amd import flashbon
    flashbon.load()


def _model(shape, dtype, max_n, max_tokens, text_len, n_cond):
    from paper_2607_04461_amd import flashbon as fb
    flat, _ = synth.make_weights(shape, 1234, threads=16)
    cfg = fb.make_config(shape, fb.BF16 if dtype == "bf16" else fb.FP32, max_n, max_tokens, text_len, n_cond)
    return fb.flashbon_init_model(cfg, flat)


def _case(model, shape, n, lh, lw, text, cond, k, sched, sde=None):
    """(latents after flashbon_refine_step, after flashbon_refine_step_noalloc) from the same input; the
    text K/V is prepared by each call itself (text_kv_valid = 0)."""
    from paper_2607_04461_amd import flashbon as fb
    z0 = torch.from_numpy(synth.make_latents(n, shape.latent_channels, lh, lw, first_seed=700 + n)).cuda()
    outs = []
    for fn in (fb.flashbon_refine_step, fb.flashbon_refine_step_noalloc):
        z = z0.clone()
        kv = torch.full((fb.flashbon_text_kv_bytes(model, text.shape[0], text.shape[1]),), 0x7F, dtype=torch.uint8,
                        device="cuda")
        valid = ctypes.c_int32(0)
        tr = fb.new_trace(shape.num_blocks)
        fn(model, z, sched[k], sched[k + 1], text, cond, kv, valid, tr, sde=sde)
        assert valid.value == 1
        assert all(e.action == fb.COMPUTE for e in tr)
        # a second step reusing the text K/V the call made (text_kv_valid = 1)
        fn(model, z, sched[k + 1], sched[k + 2], text, cond, kv, valid, tr, sde=sde)
        torch.cuda.synchronize()
        outs.append(z.cpu().numpy())
    return outs


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_noalloc_refine_equals_refine_mid(dtype):
    from paper_2607_04461_amd import flashbon as fb
    wl = synth.WORKLOADS["mid"]
    s = wl.shape
    model = _model(s, dtype, wl.n, wl.tokens, wl.text_len, wl.n_cond)
    text = torch.from_numpy(synth.make_text(wl.n_cond, wl.text_len, s.text_dim)).cuda()
    sched = wl.schedule()
    try:
        # first call: the pool's 3 candidates at 130 tokens, two prompts
        a, b = _case(model, s, 3, wl.latent_h, wl.latent_w, text, np.array([0, 1, 1], np.int32), 1, sched)
        assert np.array_equal(a, b)
        # second call, smaller: one candidate at 5 x 13 = 65 tokens, with the stochastic update
        a, b = _case(model, s, 1, 10, 26, text, np.array([1], np.int32), 3, sched, sde=(0.3, 17, 3, 2))
        assert np.array_equal(a, b)
        assert np.isfinite(a).all()
    finally:
        fb.flashbon_free(model)


def test_noalloc_refine_equals_refine_1p3b_shape():
    """One candidate of the 1.3B-shaped model at 1560 tokens (the refinement of the benchmark's
    winner), then at 416 tokens; bf16."""
    from paper_2607_04461_amd import flashbon as fb
    s = synth.WAN_1_3B
    model = _model(s, "bf16", 1, 1560, 512, 1)
    text = torch.from_numpy(synth.make_text(1, 512, s.text_dim)).cuda()
    sched = np.linspace(1.0, 0.0, 51).astype(np.float32)
    cond = np.zeros(1, np.int32)
    try:
        a, b = _case(model, s, 1, 60, 104, text, cond, 10, sched)
        assert np.array_equal(a, b)
        a, b = _case(model, s, 1, 32, 52, text, cond, 12, sched)
        assert np.array_equal(a, b)
    finally:
        fb.flashbon_free(model)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    """A call whose buffers exceed the array (the mid model at 9 x 6500 token rows would need far more
    than 128 MiB) fails with FLASHBON_ESHAPE and leaves the latents and the text K/V flag untouched."""
    from paper_2607_04461_amd import flashbon as fb
    s = synth.MID
    model = _model(s, "fp32", 9, 6500, 40, 1)
    try:
        text = torch.from_numpy(synth.make_text(1, 40, s.text_dim)).cuda()
        z = torch.ones((9, 16, 100, 260), device="cuda")
        kv = torch.zeros(fb.flashbon_text_kv_bytes(model, 1, 40), dtype=torch.uint8, device="cuda")
        valid = ctypes.c_int32(0)
        with pytest.raises(fb.FlashbonError) as e:
            fb.flashbon_refine_step_noalloc(model, z, 0.5, 0.4, text, np.zeros(9, np.int32), kv, valid)
        assert e.value.status == fb.ESHAPE
        assert "scratch" in str(e.value)
        torch.cuda.synchronize()
        assert valid.value == 0 and bool((z == 1).all())
    finally:
        fb.flashbon_free(model)
