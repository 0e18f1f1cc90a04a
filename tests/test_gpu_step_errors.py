"""Error paths of the step calls, through the C ABI with raw arguments (the binding's own checks are
bypassed).  include/flashbon.h promises that a validation error returns before any device write and
before any change to host state: each case asserts the status and that meta, trace, text_kv_valid
and the latents are byte-identical afterwards.  Every case is rejected on the host, so no kernel runs
with a bad argument.
"""
import ctypes

import numpy as np
import pytest

from paper_2607_04461_amd import synth

pytestmark = pytest.mark.gpu

CASES = [
    # (name, status name, draft only)
    ("n_zero", "ESHAPE", False), ("n_above_max", "ESHAPE", False), ("latent_h_not_patch_multiple", "ESHAPE", False),
    ("tokens_above_max", "ESHAPE", False), ("latents_null", "EINVAL", False), ("text_null", "EINVAL", False),
    ("text_kv_null", "EINVAL", False), ("text_kv_valid_null", "EINVAL", False), ("cond_index_null", "EINVAL", False),
    ("cond_index_out_of_range", "EINVAL", False), ("cond_index_negative", "EINVAL", False),
    ("text_len_above_max", "ESHAPE", False), ("n_cond_above_max", "ESHAPE", False),
    ("t_cur_nan", "EINVAL", False), ("preview_aliases_latents", "EINVAL", False),
    ("proxy_mode_2", "EINVAL", False), ("guidance_without_uncond", "EINVAL", False),
    ("guidance_rows_above_max", "ESHAPE", False), ("sde_at_t_zero", "EINVAL", False),
    ("sde_negative_step", "EINVAL", False),
    ("meta_null", "EINVAL", True), ("cache_null", "EINVAL", True), ("meta_count_4", "ESTATE", True),
    ("meta_head_3", "ESTATE", True), ("cached_tau_coincide", "ESTATE", True),
]


@pytest.fixture(scope="module")
def pool():
    from paper_2607_04461_amd.pool import DraftPool
    p = DraftPool(synth.WORKLOADS["mid"], dtype="bf16")
    p.reset()
    yield p
    p.close()


def _snapshot(pool, a, meta, trace, valid):
    import torch
    torch.cuda.synchronize()
    return (ctypes.string_at(ctypes.addressof(meta), ctypes.sizeof(meta)),
            ctypes.string_at(ctypes.addressof(trace), ctypes.sizeof(trace)), valid.value,
            pool.latents.clone())


# every case through both entry points, except the draft-only ones (refinement ignores meta and cache)
PARAMS = [(kind, name, status) for kind in ("draft", "refine") for name, status, draft_only in CASES
          if kind == "draft" or not draft_only]


@pytest.mark.parametrize("kind,name,status", PARAMS, ids=[f"{k}-{n}" for k, n, _ in PARAMS])
def test_rejected_before_any_side_effect(pool, kind, name, status):
    import torch
    from paper_2607_04461_amd import flashbon as fb
    wl, L = pool.wl, pool.L
    meta = fb.new_meta(L)
    for l in range(L):                       # a valid ring: one computed entry at t = 1
        meta[l].count, meta[l].head, meta[l].t[0] = 1, 1, 1.0
    trace = fb.new_trace(L)
    ctypes.memset(trace, 0x5A, ctypes.sizeof(trace))
    valid = ctypes.c_int32(0)
    ones = np.ones(L, np.uint8)
    zeros = np.zeros(L, np.uint8)
    a = fb.step_args(pool.latents, 0.875, 0.75, pool.text, pool.cond_index, pool.text_kv, valid,
                     zeros, ones, pool.cache, meta, trace, stream=torch.cuda.current_stream().cuda_stream)
    keep = []
    if name == "n_zero":
        a.n = 0
    elif name == "n_above_max":
        a.n = pool.cfg.max_n + 1
    elif name == "latent_h_not_patch_multiple":
        a.latent_h = wl.latent_h + 1
    elif name == "tokens_above_max":
        a.latent_h = 2 * wl.latent_h
    elif name == "latents_null":
        a.latents = None
    elif name == "text_null":
        a.text = None
    elif name == "text_kv_null":
        a.text_kv = None
    elif name == "text_kv_valid_null":
        a.text_kv_valid = ctypes.POINTER(ctypes.c_int32)()
    elif name == "cond_index_null":
        a.cond_index = ctypes.POINTER(ctypes.c_int32)()
    elif name in ("cond_index_out_of_range", "cond_index_negative"):
        bad = np.array([0, wl.n_cond if name == "cond_index_out_of_range" else -1, 0], np.int32)
        keep.append(bad)
        a.cond_index = bad.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    elif name == "text_len_above_max":
        a.text_len = pool.cfg.max_text_len + 1
    elif name == "n_cond_above_max":
        a.n_cond = pool.cfg.max_cond + 1
    elif name == "t_cur_nan":
        a.t_cur = float("nan")
    elif name == "preview_aliases_latents":
        a.preview = a.latents
    elif name == "proxy_mode_2":
        a.proxy_mode = 2
    elif name == "guidance_without_uncond":
        a.n = 1                              # 2n rows within max_n, so the missing uncond_index is the error
        a.cfg, a.cfg_scale = 1, 5.0
    elif name == "guidance_rows_above_max":
        unc = np.zeros(wl.n, np.int32)
        keep.append(unc)
        a.cfg, a.cfg_scale = 1, 5.0
        a.uncond_index = unc.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    elif name == "sde_at_t_zero":
        a.sde_a, a.t_cur, a.t_next = 0.5, 0.0, -0.125
    elif name == "sde_negative_step":
        a.sde_a, a.sde_step = 0.5, -1
    elif name == "meta_null":
        a.meta = ctypes.POINTER(fb.CacheMeta)()
    elif name == "cache_null":
        a.cache = None
    elif name == "meta_count_4":
        meta[1].count = 4
    elif name == "meta_head_3":
        meta[2].head = 3
    elif name == "cached_tau_coincide":
        # block 2 is the last proxy (live) with two entries at the same t: Eq. 3 would divide by zero
        meta[2].count, meta[2].head, meta[2].t[0], meta[2].t[1] = 2, 2, 0.9, 0.9
    before = _snapshot(pool, a, meta, trace, valid)
    fn = fb.load().flashbon_draft_step if kind == "draft" else fb.load().flashbon_refine_step
    st = fn(pool.model, ctypes.byref(a))
    msg = fb.load().flashbon_last_error().decode()
    print(f"{kind} {name}: status {st} ({msg})", flush=True)
    assert st == getattr(fb, status), msg
    after = _snapshot(pool, a, meta, trace, valid)
    assert after[0] == before[0], "meta changed"
    assert after[1] == before[1], "trace changed"
    assert after[2] == before[2], "text_kv_valid changed"
    assert torch.equal(after[3], before[3]), "latents changed"


def test_valid_call_after_errors_still_steps(pool):
    """The model is usable after rejected calls: a draft step from reset state plans and runs."""
    import torch
    pool.reset()
    tr = pool.draft_step(0)
    torch.cuda.synchronize()
    assert [e[0] for e in tr] == [0] * pool.L
    assert torch.isfinite(pool.latents).all()


def test_preview_alias_rejected_by_the_binding(pool):
    pool.reset()
    with pytest.raises(ValueError):
        pool.draft_step(0, preview=pool.latents)


def test_init_out_of_memory_returns_enomem():
    """A workspace far beyond the device's memory (max_n x max_tokens = 2^30 rows of the tiny model,
    several hundred GB) fails its allocation: FLASHBON_ENOMEM, no handle, and the library still works."""
    from paper_2607_04461_amd import flashbon as fb
    cfg = fb.make_config(synth.TINY, fb.BF16, 1 << 14, 1 << 16, 8, 1)
    w, _ = synth.make_weights(synth.TINY)
    with pytest.raises(fb.FlashbonError) as e:
        fb.flashbon_init_model(cfg, w)
    assert e.value.status == fb.ENOMEM
    ok = fb.make_config(synth.TINY, fb.BF16, 2, 16, 8, 1)
    h = fb.flashbon_init_model(ok, w)
    fb.flashbon_free(h)
