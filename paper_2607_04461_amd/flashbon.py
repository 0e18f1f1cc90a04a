"""Python binding of ``libflashbon.so`` (include/flashbon.h, include/flashbon_ops.h).

Argument marshalling only: every step of the draft path runs in the library's HIP kernels.  Device
buffers are anything with ``data_ptr()`` (torch CUDA tensors); ``stream=None`` means torch's current
stream on the current device.  The library must have been built (``__graft_entry__.build()``); a
missing library raises, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflashbon.so")
_lib: Optional[ctypes.CDLL] = None

OK, EINVAL, ESHAPE, ENOMEM, EHIP, ESTATE = 0, -1, -2, -3, -4, -5
FP32, BF16 = 0, 1
COMPUTE, SKIP, PROXY = 0, 1, 2
EPI_STORE, EPI_GELU, EPI_STORE_F32, EPI_RESIDUAL = 0, 1, 2, 3
SITES = ["qkv", "attn_self", "out", "cross_q", "attn_cross", "out_cross", "mlp_up", "mlp_down", "norm",
         "proxy", "embed", "head", "time", "text"]


class FlashbonError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where} failed with status {status}: {msg}")
        self.status = status


class ModelConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("num_blocks", "hidden", "heads", "mlp_hidden",
                                               "latent_channels", "patch", "freq_dim", "text_dim",
                                               "dtype")] + \
               [("ln_eps", ctypes.c_float)] + \
               [(n, ctypes.c_int32) for n in ("max_n", "max_tokens", "max_text_len", "max_cond", "qk_norm_rope")]


class CacheMeta(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int32), ("head", ctypes.c_int32), ("t", ctypes.c_float * 3)]


class TraceEntry(ctypes.Structure):
    _fields_ = [("action", ctypes.c_int8), ("order", ctypes.c_int8), ("slot", ctypes.c_int8),
                ("live", ctypes.c_int8)]


class StepArgs(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int32), ("latent_h", ctypes.c_int32), ("latent_w", ctypes.c_int32),
        ("latents", ctypes.c_void_p), ("t_cur", ctypes.c_float), ("t_next", ctypes.c_float),
        ("text", ctypes.c_void_p), ("n_cond", ctypes.c_int32), ("text_len", ctypes.c_int32),
        ("cond_index", ctypes.POINTER(ctypes.c_int32)), ("text_kv", ctypes.c_void_p),
        ("text_kv_valid", ctypes.POINTER(ctypes.c_int32)),
        ("skip", ctypes.POINTER(ctypes.c_uint8)), ("proxy", ctypes.POINTER(ctypes.c_uint8)),
        ("cache", ctypes.c_void_p), ("meta", ctypes.POINTER(CacheMeta)),
        ("trace", ctypes.POINTER(TraceEntry)), ("hidden_dump", ctypes.c_void_p),
        ("stream", ctypes.c_void_p),
        ("sde_a", ctypes.c_float), ("sde_step", ctypes.c_int32), ("sde_seed", ctypes.c_uint64),
        ("sde_row0", ctypes.c_int32), ("preview", ctypes.c_void_p),
        ("cfg", ctypes.c_int32), ("cfg_scale", ctypes.c_float), ("uncond_index", ctypes.POINTER(ctypes.c_int32)),
        ("proxy_mode", ctypes.c_int32),
    ]


EXPORTS = [
    "flashbon_weight_count", "flashbon_init_model", "flashbon_text_kv_bytes", "flashbon_cache_bytes",
    "flashbon_draft_step", "flashbon_refine_step", "flashbon_free", "flashbon_plan_step",
    "flashbon_last_error", "flashbon_set_timing", "flashbon_read_timing", "flashbon_op_linear", "flashbon_op_linear_residual", "flashbon_op_linear_plan", "flashbon_op_attention", "flashbon_op_ln_mod",
    "flashbon_op_proxy", "flashbon_op_normals", "flashbon_op_unpatch_sde", "flashbon_select",
    "flashbon_refine_step_noalloc", "flashbon_op_linear_ws",
]
NOALLOC_SCRATCH_BYTES = 128 << 20

JUDGE_FN = ctypes.CFUNCTYPE(ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                            ctypes.POINTER(ctypes.c_int32))


def lib_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load the built library (raises FileNotFoundError if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise FileNotFoundError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    L.flashbon_weight_count.argtypes = [ctypes.POINTER(ModelConfig)]
    L.flashbon_weight_count.restype = sz
    L.flashbon_init_model.argtypes = [ctypes.POINTER(ModelConfig), vp, sz, ctypes.POINTER(vp)]
    L.flashbon_init_model.restype = i32
    L.flashbon_text_kv_bytes.argtypes = [vp, i32, i32]
    L.flashbon_text_kv_bytes.restype = sz
    L.flashbon_cache_bytes.argtypes = [vp, i32, i32]
    L.flashbon_cache_bytes.restype = sz
    L.flashbon_draft_step.argtypes = [vp, ctypes.POINTER(StepArgs)]
    L.flashbon_draft_step.restype = i32
    L.flashbon_refine_step.argtypes = [vp, ctypes.POINTER(StepArgs)]
    L.flashbon_refine_step.restype = i32
    L.flashbon_refine_step_noalloc.argtypes = [vp, ctypes.POINTER(StepArgs)]
    L.flashbon_refine_step_noalloc.restype = i32
    L.flashbon_free.argtypes = [vp]
    L.flashbon_free.restype = None
    L.flashbon_plan_step.argtypes = [i32, ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_uint8),
                                     ctypes.POINTER(CacheMeta), f32, ctypes.POINTER(TraceEntry), i32]
    L.flashbon_plan_step.restype = i32
    L.flashbon_set_timing.argtypes = [vp, ctypes.c_uint32]
    L.flashbon_set_timing.restype = i32
    L.flashbon_read_timing.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    L.flashbon_read_timing.restype = i32
    L.flashbon_last_error.argtypes = []
    L.flashbon_last_error.restype = ctypes.c_char_p
    L.flashbon_op_linear.argtypes = [i32, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp]
    L.flashbon_op_linear.restype = i32
    L.flashbon_op_linear_ws.argtypes = [i32, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp, sz,
                                        ctypes.POINTER(ctypes.c_int32), vp]
    L.flashbon_op_linear_ws.restype = i32
    L.flashbon_op_linear_residual.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    L.flashbon_op_linear_residual.restype = i32
    L.flashbon_op_linear_plan.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int32), ctypes.c_char_p, i32]
    L.flashbon_op_linear_plan.restype = i32
    L.flashbon_op_attention.argtypes = [i32, i32, i32, i32, i32, i32, vp, i64, i64, vp, vp, i64, i64,
                                        vp, i32, vp, i64, i64, vp]
    L.flashbon_op_attention.restype = i32
    L.flashbon_op_ln_mod.argtypes = [i32, i32, i32, f32, vp, vp, vp, vp, vp]
    L.flashbon_op_ln_mod.restype = i32
    L.flashbon_op_proxy.argtypes = [i64, vp, vp, vp, i32, f32, f32, f32, vp, vp]
    L.flashbon_op_proxy.restype = i32
    L.flashbon_op_normals.argtypes = [i64, i32, i32, ctypes.c_uint64, vp, vp, vp]
    L.flashbon_op_normals.restype = i32
    L.flashbon_op_unpatch_sde.argtypes = [i32, i32, i32, i32, i32, vp, vp, f32, f32, f32, ctypes.c_uint64,
                                          i32, i32, vp]
    L.flashbon_op_unpatch_sde.restype = i32
    L.flashbon_select.argtypes = [i32, ctypes.POINTER(ctypes.c_int32), ctypes.c_double, ctypes.c_double,
                                  ctypes.c_double, JUDGE_FN, vp, ctypes.POINTER(ctypes.c_int32),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]
    L.flashbon_select.restype = i32
    _lib = L
    return L


def _check(status: int, where: str) -> None:
    if status != OK:
        raise FlashbonError(status, where, load().flashbon_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return int(stream)
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def _u8(mask: Optional[Sequence[int]], n: int):
    if mask is None:
        return None, None
    a = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    if a.shape != (n,):
        raise ValueError(f"mask must have shape ({n},)")
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))


def make_config(shape, dtype: int, max_n: int, max_tokens: int, max_text_len: int, max_cond: int) -> ModelConfig:
    return ModelConfig(shape.num_blocks, shape.hidden, shape.heads, shape.mlp_hidden,
                       shape.latent_channels, shape.patch, shape.freq_dim, shape.text_dim, dtype,
                       shape.ln_eps, max_n, max_tokens, max_text_len, max_cond,
                       1 if getattr(shape, "qk_norm_rope", False) else 0)


def flashbon_weight_count(cfg: ModelConfig) -> int:
    return int(load().flashbon_weight_count(ctypes.byref(cfg)))


# Shape of every live model handle, so that the step wrappers can check the caller's tensors before
# their addresses cross the C ABI (which cannot see sizes, dtypes or devices).
_MODELS: Dict[int, ModelConfig] = {}


def flashbon_init_model(cfg: ModelConfig, host_weights: np.ndarray) -> int:
    w = np.ascontiguousarray(host_weights, dtype=np.float32)
    h = ctypes.c_void_p()
    _check(load().flashbon_init_model(ctypes.byref(cfg), w.ctypes.data, w.size, ctypes.byref(h)),
           "flashbon_init_model")
    kept = ModelConfig()
    ctypes.pointer(kept)[0] = cfg
    _MODELS[int(h.value)] = kept
    return int(h.value)


def flashbon_free(model: Optional[int]) -> None:
    if model:
        _MODELS.pop(int(model), None)
        load().flashbon_free(model)


def model_config(model: int) -> ModelConfig:
    """The configuration a live handle was created with (ValueError for an unknown handle)."""
    try:
        return _MODELS[int(model)]
    except (KeyError, TypeError):
        raise ValueError("not a live model handle from flashbon_init_model") from None


def text_kv_nbytes(cfg: ModelConfig, n_cond: int, text_len: int) -> int:
    """flashbon_text_kv_bytes for a configuration: [L][n_cond][text_len][2 D] act elements."""
    return cfg.num_blocks * n_cond * text_len * 2 * cfg.hidden * (2 if cfg.dtype == BF16 else 4)


def cache_nbytes(cfg: ModelConfig, rows: int, tokens: int) -> int:
    """flashbon_cache_bytes for a configuration: fp32 [L][3][rows][tokens][D]."""
    return cfg.num_blocks * 3 * rows * tokens * cfg.hidden * 4


def _nbytes(t) -> int:
    return int(t.numel()) * int(t.element_size())


def _check_tensor(name: str, t, *, dtype=None, ndim=None, require_device: bool = True) -> None:
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if require_device:
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the current device (a GPU), got {t.device}")
        if t.device.index != torch.cuda.current_device():
            raise ValueError(f"{name} must be on the current device (cuda:{torch.cuda.current_device()}), "
                             f"got {t.device}")


def validate_step(cfg: ModelConfig, latents, text, text_kv, *, draft: bool, guided: bool = False,
                  cache=None, hidden_dump=None, preview=None, meta=None, trace=None,
                  require_device: bool = True) -> None:
    """Raise ValueError unless every buffer a step would hand to the library has the dtype, layout,
    device and size the step's kernels read and write (include/flashbon.h, flashbon_step_args).
    ``require_device=False`` skips only the device check (host-only tests of the other checks)."""
    import torch
    f32 = torch.float32
    _check_tensor("latents", latents, dtype=f32, ndim=4, require_device=require_device)
    n, C, H, W = (int(x) for x in latents.shape)
    if C != cfg.latent_channels:
        raise ValueError(f"latents have {C} channels, the model {cfg.latent_channels}")
    _check_tensor("text", text, dtype=f32, ndim=3, require_device=require_device)
    n_cond, text_len, text_dim = (int(x) for x in text.shape)
    if text_dim != cfg.text_dim:
        raise ValueError(f"text tokens are {text_dim} wide, the model takes {cfg.text_dim}")
    _check_tensor("text_kv", text_kv, require_device=require_device)
    need = text_kv_nbytes(cfg, n_cond, text_len)
    if _nbytes(text_kv) < need:
        raise ValueError(f"text_kv holds {_nbytes(text_kv)} bytes, needs {need}")
    rows = 2 * n if guided else n
    p = max(cfg.patch, 1)
    tokens = (H // p) * (W // p)
    if draft:
        if cache is None:
            raise ValueError("a draft step needs the activation cache")
        _check_tensor("cache", cache, dtype=f32, require_device=require_device)
        need = cache_nbytes(cfg, rows, tokens)
        if _nbytes(cache) < need:
            raise ValueError(f"cache holds {_nbytes(cache)} bytes, needs {need} for {rows} rows x {tokens} tokens")
        if meta is None or len(meta) != cfg.num_blocks:
            raise ValueError(f"meta must hold {cfg.num_blocks} entries")
    if trace is not None and len(trace) != cfg.num_blocks:
        raise ValueError(f"trace must hold {cfg.num_blocks} entries")
    if hidden_dump is not None:
        _check_tensor("hidden_dump", hidden_dump, dtype=f32, require_device=require_device)
        need = (cfg.num_blocks + 1) * rows * tokens * cfg.hidden
        if int(hidden_dump.numel()) < need:
            raise ValueError(f"hidden_dump holds {int(hidden_dump.numel())} floats, needs {need}")
    if preview is not None:
        _check_tensor("preview", preview, dtype=f32, ndim=4, require_device=require_device)
        if tuple(preview.shape) != tuple(latents.shape):
            raise ValueError(f"preview must have the latents' shape {tuple(latents.shape)}")
        a0, a1 = latents.data_ptr(), latents.data_ptr() + _nbytes(latents)
        b0, b1 = preview.data_ptr(), preview.data_ptr() + _nbytes(preview)
        if a0 < b1 and b0 < a1:
            raise ValueError("preview must not overlap latents")


def flashbon_text_kv_bytes(model: int, n_cond: int, text_len: int) -> int:
    return int(load().flashbon_text_kv_bytes(model, n_cond, text_len))


def flashbon_cache_bytes(model: int, n: int, tokens: int) -> int:
    return int(load().flashbon_cache_bytes(model, n, tokens))


def new_meta(num_blocks: int):
    return (CacheMeta * num_blocks)()


def new_trace(num_blocks: int):
    return (TraceEntry * num_blocks)()


def trace_list(trace) -> list:
    return [(e.action, e.order, e.slot, e.live) for e in trace]


def _step(fn, where, model, latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid,
          skip=None, proxy=None, cache=None, meta=None, trace=None, hidden_dump=None, stream=None,
          num_blocks=None, sde=None, preview=None, cfg=None, proxy_mode=0, draft=True):
    validate_step(model_config(model), latents, text, text_kv, draft=draft, guided=cfg is not None,
                  cache=cache, hidden_dump=hidden_dump, preview=preview, meta=meta, trace=trace)
    a = step_args(latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid, skip, proxy, cache,
                  meta, trace, hidden_dump, stream, num_blocks, sde, preview, cfg, proxy_mode)
    _check(fn(model, ctypes.byref(a)), where)


def step_args(latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid, skip=None, proxy=None,
              cache=None, meta=None, trace=None, hidden_dump=None, stream=None, num_blocks=None, sde=None,
              preview=None, cfg=None, proxy_mode=0) -> StepArgs:
    """flashbon_step_args for the given buffers, without any check (the library validates the rest;
    tests of the library's own validation build arguments with this).  The host arrays it points to
    are kept alive on the returned structure."""
    n, C, H, W = (int(x) for x in latents.shape)
    n_cond, text_len = int(text.shape[0]), int(text.shape[1])
    cond = np.ascontiguousarray(np.asarray(cond_index, dtype=np.int32))
    if cond.shape != (n,):
        raise ValueError(f"cond_index must have shape ({n},)")
    L = num_blocks if num_blocks is not None else (len(meta) if meta is not None else None)
    sk, skp = _u8(skip, L) if skip is not None else (None, None)
    px, pxp = _u8(proxy, L) if proxy is not None else (None, None)
    a = StepArgs()
    a.n, a.latent_h, a.latent_w = n, H, W
    a.latents = _ptr(latents)
    a.t_cur, a.t_next = float(t_cur), float(t_next)
    a.text = _ptr(text)
    a.n_cond, a.text_len = n_cond, text_len
    a.cond_index = cond.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    a.text_kv = _ptr(text_kv)
    a.text_kv_valid = ctypes.pointer(text_kv_valid)
    a.skip, a.proxy = skp, pxp
    a.cache = _ptr(cache)
    a.meta = meta
    a.trace = trace
    a.hidden_dump = _ptr(hidden_dump)
    a.preview = _ptr(preview)
    a.proxy_mode = int(proxy_mode)
    if cfg is not None:
        unc = np.ascontiguousarray(np.asarray(cfg[1], dtype=np.int32))
        if unc.shape != (n,):
            raise ValueError(f"uncond_index must have shape ({n},)")
        a.cfg, a.cfg_scale = 1, float(cfg[0])
        a.uncond_index = unc.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    a.stream = _stream(stream)
    if sde is not None:
        a.sde_a, a.sde_seed, a.sde_step = float(sde[0]), int(sde[1]), int(sde[2])
        a.sde_row0 = int(sde[3]) if len(sde) > 3 else 0
    a._keep = (cond, sk, px, unc if cfg is not None else None, text_kv_valid)
    return a


def flashbon_draft_step(model, latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid,
                        skip, proxy, cache, meta, trace=None, hidden_dump=None, stream=None, sde=None,
                        preview=None, cfg=None, proxy_mode=0):
    """One draft step; ``text_kv_valid`` is a ctypes.c_int32, ``meta``/``trace`` ctypes arrays;
    ``sde = (a, seed, step[, row0])`` selects the stochastic update (None or a = 0: Euler);
    ``preview`` (device [n, C, H, W] fp32) receives z - t_cur v; ``cfg = (scale, uncond_index)``
    turns on classifier-free guidance (the cache then holds 2n rows); ``proxy_mode`` 1 takes the
    residual-delta reading of the proxy."""
    _step(load().flashbon_draft_step, "flashbon_draft_step", model, latents, t_cur, t_next, text,
          cond_index, text_kv, text_kv_valid, skip, proxy, cache, meta, trace, hidden_dump, stream,
          num_blocks=len(meta), sde=sde, preview=preview, cfg=cfg, proxy_mode=proxy_mode)


def flashbon_refine_step(model, latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid,
                         trace=None, hidden_dump=None, stream=None, sde=None, preview=None, cfg=None):
    _step(load().flashbon_refine_step, "flashbon_refine_step", model, latents, t_cur, t_next, text,
          cond_index, text_kv, text_kv_valid, None, None, None, None, trace, hidden_dump, stream, sde=sde,
          preview=preview, cfg=cfg, draft=False)


def flashbon_refine_step_noalloc(model, latents, t_cur, t_next, text, cond_index, text_kv, text_kv_valid,
                                 trace=None, hidden_dump=None, stream=None, sde=None, preview=None, cfg=None):
    """flashbon_refine_step with its working buffers in the library's static per-GPU scratch array
    (allocates nothing; overlapping calls on one GPU race)."""
    _step(load().flashbon_refine_step_noalloc, "flashbon_refine_step_noalloc", model, latents, t_cur, t_next,
          text, cond_index, text_kv, text_kv_valid, None, None, None, None, trace, hidden_dump, stream, sde=sde,
          preview=preview, cfg=cfg, draft=False)


def flashbon_select(scores, judge, rho1=0.5, rho2=0.5, kappa=1.5):
    """Multi-stage Elo selection; ``judge(a, b) -> (winner, confidence)`` is the verifier.
    Returns (winner, ratings [m] float64, pairwise calls)."""
    sc = np.ascontiguousarray(np.asarray(scores, dtype=np.int32))
    m = int(sc.size)
    failure = []

    def _cb(_ctx, a, b, conf):
        try:
            w, c = judge(int(a), int(b))
            conf[0] = int(c)
            return int(w)
        except BaseException as e:  # the exception cannot cross the C frame; report it afterwards
            failure.append(e)
            return -1

    cb = JUDGE_FN(_cb)
    winner, calls = ctypes.c_int32(), ctypes.c_int32()
    ratings = np.zeros(m, np.float64)
    st = load().flashbon_select(m, sc.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), rho1, rho2, kappa, cb,
                                None, ctypes.byref(winner),
                                ratings.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.byref(calls))
    if failure:
        raise failure[0]
    _check(st, "flashbon_select")
    return int(winner.value), ratings, int(calls.value)


def flashbon_plan_step(skip, proxy, meta, t_cur: float, trace=None, proxy_mode: int = 0):
    L = len(meta)
    sk, skp = _u8(skip, L)
    px, pxp = _u8(proxy, L)
    if trace is None:
        trace = new_trace(L)
    _check(load().flashbon_plan_step(L, skp, pxp, meta, float(t_cur), trace, int(proxy_mode)),
           "flashbon_plan_step")
    return trace


def flashbon_set_timing(model: int, sites) -> None:
    """Time the named launch sites (see SITES) on later steps; empty = off."""
    mask = 0
    for name in sites:
        mask |= 1 << SITES.index(name)
    _check(load().flashbon_set_timing(model, mask), "flashbon_set_timing")


def flashbon_read_timing(model: int, site: str):
    """(total device ms, launches) of one site since the last read."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(load().flashbon_read_timing(model, SITES.index(site), ctypes.byref(ms), ctypes.byref(n)),
           "flashbon_read_timing")
    return ms.value, n.value


# --------------------------------------------------------------------------- kernel-level entry points

def flashbon_op_linear(dtype, M, N, K, A, W, bias, epilogue, out, gate=None, cache_out=None, stream=None):
    _check(load().flashbon_op_linear(dtype, M, N, K, _ptr(A), _ptr(W), _ptr(bias), epilogue, _ptr(out),
                                     _ptr(gate), _ptr(cache_out), _stream(stream)), "flashbon_op_linear")


def flashbon_op_linear_ws(dtype, M, N, K, A, W, bias, epilogue, out, workspace, gate=None, cache_out=None,
                          stream=None) -> int:
    """flashbon_op_linear with a split-K workspace (a device tensor); returns the number of K ranges."""
    sp = ctypes.c_int32()
    nbytes = 0 if workspace is None else int(workspace.numel()) * int(workspace.element_size())
    _check(load().flashbon_op_linear_ws(dtype, M, N, K, _ptr(A), _ptr(W), _ptr(bias), epilogue, _ptr(out),
                                        _ptr(gate), _ptr(cache_out), _ptr(workspace), nbytes, ctypes.byref(sp),
                                        _stream(stream)), "flashbon_op_linear_ws")
    return sp.value


def flashbon_op_linear_residual(dtype, M, N, K, A, W, bias, gate, residual_in, out, stream=None):
    _check(load().flashbon_op_linear_residual(dtype, M, N, K, _ptr(A), _ptr(W), _ptr(bias), _ptr(gate),
                                              _ptr(residual_in), _ptr(out), _stream(stream)),
           "flashbon_op_linear_residual")


def flashbon_op_linear_plan(dtype, M, N, K, epilogue):
    """(number of kernel launches, description) of the tile plan flashbon_op_linear takes."""
    n = ctypes.c_int32()
    buf = ctypes.create_string_buffer(256)
    _check(load().flashbon_op_linear_plan(dtype, M, N, K, epilogue, ctypes.byref(n), buf, len(buf)),
           "flashbon_op_linear_plan")
    return n.value, buf.value.decode()


def flashbon_op_attention(dtype, batch, heads, head_dim, tq, tk, q, q_bs, q_rs, k, v, kv_bs, kv_rs,
                          kv_index, n_kv, out, o_bs, o_rs, stream=None):
    _check(load().flashbon_op_attention(dtype, batch, heads, head_dim, tq, tk, _ptr(q), q_bs, q_rs, _ptr(k),
                                        _ptr(v), kv_bs, kv_rs, _ptr(kv_index), n_kv, _ptr(out), o_bs, o_rs,
                                        _stream(stream)), "flashbon_op_attention")


def flashbon_op_ln_mod(dtype, M, D, eps, x, shift, scale, out, stream=None):
    _check(load().flashbon_op_ln_mod(dtype, M, D, eps, _ptr(x), _ptr(shift), _ptr(scale), _ptr(out),
                                     _stream(stream)), "flashbon_op_ln_mod")


def flashbon_op_proxy(count, h1, h2, h3, order, tau1, tau2, t_cur, out, stream=None):
    _check(load().flashbon_op_proxy(count, _ptr(h1), _ptr(h2), _ptr(h3), order, tau1, tau2, t_cur, _ptr(out),
                                    _stream(stream)), "flashbon_op_proxy")


def flashbon_op_normals(count, candidate, step, seed, words=None, normals=None, stream=None):
    _check(load().flashbon_op_normals(count, candidate, step, seed, _ptr(words), _ptr(normals),
                                      _stream(stream)), "flashbon_op_normals")


def flashbon_op_unpatch_sde(n, C, H, W, p, v, z, t_cur, t_next, a, seed, step, row0=0, stream=None):
    _check(load().flashbon_op_unpatch_sde(n, C, H, W, p, _ptr(v), _ptr(z), t_cur, t_next, a, seed, step, row0,
                                          _stream(stream)), "flashbon_op_unpatch_sde")
