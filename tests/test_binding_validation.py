"""Host-side checks of the Python binding (no GPU): every tensor a step hands to the library is checked
for dtype, layout, device and size before its address crosses the C ABI, which cannot see them.

The sizes are those the library's kernels address (include/flashbon.h): latents [n, C, H, W] fp32,
text [n_cond, text_len, text_dim] fp32, text K/V [L][n_cond][text_len][2 D] act elements, the
activation cache fp32 [L][3][rows][T][D] with rows = 2n under guidance, hidden_dump fp32
[L + 1][rows][T][D], preview the latents' shape and disjoint from them.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_04461_amd import flashbon as fb
from paper_2607_04461_amd import synth

S = synth.TINY           # L = 2, D = 64, C = 16, text_dim = 32
N, H, W, LT, NC = 2, 8, 8, 8, 1
T = (H // 2) * (W // 2)


def _cfg(dtype=fb.BF16):
    return fb.make_config(S, dtype, 2 * N, T, LT, 2)


def _bufs(cfg, guided=False):
    rows = 2 * N if guided else N
    return dict(
        latents=torch.zeros((N, 16, H, W), dtype=torch.float32),
        text=torch.zeros((NC, LT, 32), dtype=torch.float32),
        text_kv=torch.zeros(fb.text_kv_nbytes(cfg, NC, LT), dtype=torch.uint8),
        cache=torch.zeros(fb.cache_nbytes(cfg, rows, T) // 4, dtype=torch.float32),
        meta=fb.new_meta(S.num_blocks),
        trace=fb.new_trace(S.num_blocks),
    )


def _call(cfg, b, draft=True, guided=False, **kw):
    args = dict(b)
    args.update(kw)
    lat, text, kv = args.pop("latents"), args.pop("text"), args.pop("text_kv")
    fb.validate_step(cfg, lat, text, kv, draft=draft, guided=guided, require_device=False, **args)


def test_sizes_match_the_header_formulas():
    cfg = _cfg()
    assert fb.text_kv_nbytes(cfg, 3, 5) == 2 * 3 * 5 * 2 * 64 * 2
    assert fb.text_kv_nbytes(_cfg(fb.FP32), 3, 5) == 2 * 3 * 5 * 2 * 64 * 4
    assert fb.cache_nbytes(cfg, 4, 16) == 2 * 3 * 4 * 16 * 64 * 4


def test_valid_buffers_pass():
    cfg = _cfg()
    _call(cfg, _bufs(cfg))
    _call(cfg, _bufs(cfg, guided=True), guided=True)
    b = _bufs(cfg)
    _call(cfg, b, draft=False, cache=None, meta=None)
    _call(cfg, b, hidden_dump=torch.zeros(3 * N * T * 64), preview=torch.zeros((N, 16, H, W)))


@pytest.mark.parametrize("case", [
    "latents_bf16", "latents_strided", "latents_channels", "latents_numpy", "text_width", "text_fp64",
    "text_2d", "text_kv_small", "cache_small", "cache_for_n_under_guidance", "cache_missing",
    "cache_bf16", "meta_short", "trace_short", "hidden_small", "preview_shape", "preview_alias",
    "preview_overlap",
])
def test_bad_buffer_rejected(case):
    cfg = _cfg()
    guided = case == "cache_for_n_under_guidance"
    b = _bufs(cfg)
    kw = {}
    if case == "latents_bf16":
        b["latents"] = b["latents"].to(torch.bfloat16)
    elif case == "latents_strided":
        b["latents"] = torch.zeros((N, 16, W, H)).transpose(2, 3)
    elif case == "latents_channels":
        b["latents"] = torch.zeros((N, 8, H, W))
    elif case == "latents_numpy":
        b["latents"] = np.zeros((N, 16, H, W), np.float32)
    elif case == "text_width":
        b["text"] = torch.zeros((NC, LT, 48))
    elif case == "text_fp64":
        b["text"] = torch.zeros((NC, LT, 32), dtype=torch.float64)
    elif case == "text_2d":
        b["text"] = torch.zeros((LT, 32))
    elif case == "text_kv_small":
        b["text_kv"] = b["text_kv"][:-1]
    elif case == "cache_small":
        b["cache"] = b["cache"][:-1]
    elif case == "cache_missing":
        b["cache"] = None
    elif case == "cache_bf16":
        b["cache"] = torch.zeros(b["cache"].numel() * 2, dtype=torch.bfloat16)
    elif case == "meta_short":
        b["meta"] = fb.new_meta(1)
    elif case == "trace_short":
        b["trace"] = fb.new_trace(3)
    elif case == "hidden_small":
        kw["hidden_dump"] = torch.zeros(3 * N * T * 64 - 1)
    elif case == "preview_shape":
        kw["preview"] = torch.zeros((N, 16, H, W + 2))
    elif case == "preview_alias":
        kw["preview"] = b["latents"]
    elif case == "preview_overlap":
        big = torch.zeros(2 * N * 16 * H * W)
        b["latents"] = big[: N * 16 * H * W].view(N, 16, H, W)
        kw["preview"] = big[16 * H * W: 16 * H * W + N * 16 * H * W].view(N, 16, H, W)
    with pytest.raises(ValueError):
        _call(cfg, b, guided=guided, **kw)


def test_cpu_tensors_rejected_for_the_device():
    cfg = _cfg()
    b = _bufs(cfg)
    with pytest.raises(ValueError, match="current device"):
        fb.validate_step(cfg, b["latents"], b["text"], b["text_kv"], draft=True, cache=b["cache"],
                         meta=b["meta"])


def test_unknown_handle_rejected_before_the_library():
    with pytest.raises(ValueError, match="live model handle"):
        fb.model_config(123456)
    with pytest.raises(ValueError, match="live model handle"):
        fb.flashbon_refine_step(123456, torch.zeros((1, 16, 8, 8)), 1.0, 0.9, torch.zeros((1, 8, 32)), [0],
                                torch.zeros(8), ctypes.c_int32(0))


def test_step_args_marshal_every_field():
    cfg = _cfg()
    b = _bufs(cfg)
    valid = ctypes.c_int32(0)
    a = fb.step_args(b["latents"], 0.75, 0.5, b["text"], [0, 0], b["text_kv"], valid,
                     np.array([0, 1]), np.array([1, 0]), b["cache"], b["meta"], b["trace"],
                     sde=(0.3, 7, 2, 1), cfg=(4.5, [0, 0]), proxy_mode=1, stream=0)
    assert (a.n, a.latent_h, a.latent_w, a.n_cond, a.text_len) == (N, H, W, NC, LT)
    assert a.latents == b["latents"].data_ptr() and a.cache == b["cache"].data_ptr()
    assert [a.skip[i] for i in range(2)] == [0, 1] and [a.proxy[i] for i in range(2)] == [1, 0]
    assert (a.cfg, a.cfg_scale, a.proxy_mode) == (1, 4.5, 1)
    assert (round(a.sde_a, 6), a.sde_seed, a.sde_step, a.sde_row0) == (0.3, 7, 2, 1)
    assert a.t_cur == 0.75 and a.t_next == 0.5
