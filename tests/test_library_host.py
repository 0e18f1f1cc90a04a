"""Host-only checks of the C-ABI library (no GPU): it loads, exports every declared symbol, its
dispatcher is bit-exact with the oracle's, and its validation rejects bad configurations."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import dispatch as od
from paper_2607_04461_amd import flashbon as fb
from paper_2607_04461_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("flashbon.h", "flashbon_ops.h"):
        txt = open(os.path.join(ROOT, "include", h)).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)          # drop comments
        names |= set(re.findall(r"(?:flashbon_status|size_t|void|const char)\s*\*?\s*(flashbon_[a-z_0-9]+)\s*\(", txt))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    lib = fb.load()
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(fb.EXPORTS)


def test_headers_are_plain_c_and_the_handle_is_typed(tmp_path):
    """The two headers compile as C99 on their own, and the model handle is the opaque flashbon_model type
    (a wrong handle type is a compile error, not a silent void* conversion)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    src.write_text('#include "flashbon_ops.h"\n'
                   "flashbon_status step(flashbon_model *m, const flashbon_step_args *a) {\n"
                   "  return flashbon_draft_step(m, a);\n}\n")
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), "-c", str(src),
                        "-o", str(tmp_path / "use.o")], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    bad = tmp_path / "bad.c"
    bad.write_text('#include "flashbon.h"\nflashbon_status f(const flashbon_model_config *c, const flashbon_step_args *a) {\n'
                   "  return flashbon_draft_step(c, a);\n}\n")
    r = subprocess.run([cc, "-std=c99", "-Werror", "-I", os.path.join(ROOT, "include"), "-c", str(bad),
                        "-o", str(tmp_path / "bad.o")], capture_output=True, text=True)
    assert r.returncode != 0


@pytest.mark.parametrize("name", ["tiny", "mid", "wan1.3b_pool16", "wan14b_pool4", "wan1.3b_pool64"])
def test_plan_step_matches_oracle_on_workloads(name):
    wl = synth.WORKLOADS[name]
    L = wl.shape.num_blocks
    meta_c = fb.new_meta(L)
    meta_o = od.empty_meta(L)
    sched = wl.schedule()
    for k in range(wl.steps_draft):
        skip, proxy = wl.masks(k)
        tr_c = fb.trace_list(fb.flashbon_plan_step(skip, proxy, meta_c, sched[k]))
        tr_o, meta_o = od.plan_step(skip, proxy, meta_o, sched[k])
        assert tr_c == [tuple(e) for e in tr_o], f"step {k}"
        for l in range(L):
            assert (meta_c[l].count, meta_c[l].head) == (meta_o[l]["count"], meta_o[l]["head"])
            assert list(meta_c[l].t) == meta_o[l]["t"]


@pytest.mark.parametrize("mode", [0, 1])
def test_plan_step_random_masks_bit_exact(mode):
    rng = np.random.default_rng(42)
    for trial in range(200):
        L = int(rng.integers(1, 12))
        meta_c = fb.new_meta(L)
        meta_o = od.empty_meta(L)
        t = 1.0
        for k in range(int(rng.integers(1, 9))):
            skip = (rng.random(L) < rng.random()).astype(np.uint8)
            proxy = (rng.random(L) < rng.random()).astype(np.uint8)
            tr_c = fb.trace_list(fb.flashbon_plan_step(skip, proxy, meta_c, t, proxy_mode=mode))
            tr_o, meta_o = od.plan_step(skip, proxy, meta_o, t, residual=bool(mode))
            assert tr_c == [tuple(e) for e in tr_o]
            t -= float(rng.random()) * 0.1


def test_plan_step_rejects_unknown_proxy_mode():
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_plan_step(np.zeros(3), np.zeros(3), fb.new_meta(3), 0.5, proxy_mode=2)


def test_plan_step_rejects_bad_meta():
    meta = fb.new_meta(3)
    meta[1].count = 4
    with pytest.raises(fb.FlashbonError) as e:
        fb.flashbon_plan_step(np.zeros(3), np.zeros(3), meta, 0.5)
    assert e.value.status == fb.ESTATE
    meta[1].count = 2
    meta[1].head = 3
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_plan_step(np.zeros(3), np.zeros(3), meta, 0.5)


@pytest.mark.parametrize("shape", [synth.TINY, synth.MID, synth.WAN_1_3B, synth.WAN_14B,
                                   synth.WORKLOADS["mid_rope"].shape,
                                   synth.dataclasses.replace(synth.WAN_1_3B, qk_norm_rope=True)])
def test_weight_count_matches_packing(shape):
    cfg = fb.make_config(shape, fb.BF16, 1, 16, 8, 1)
    assert fb.flashbon_weight_count(cfg) == synth.weight_count(shape)


def test_weight_count_of_published_shapes():
    # the blocks of the 1.3B-shaped model hold 1.39e9 parameters, of the 14B-shaped one 14.05e9;
    # the shared timestep / text / patch / head layers add a little on top
    for shape, blocks in ((synth.WAN_1_3B, 1.39e9), (synth.WAN_14B, 14.05e9)):
        D, F = shape.hidden, shape.mlp_hidden
        assert abs(shape.num_blocks * (8 * D * D + 2 * D * F) - blocks) < 0.01e9
        assert blocks < synth.weight_count(shape) < 1.03 * blocks


@pytest.mark.parametrize("field,value", [("hidden", 60), ("heads", 5), ("mlp_hidden", 12), ("dtype", 7),
                                         ("mlp_hidden", 65544), ("text_dim", 65544), ("hidden", 6152),
                                         ("max_n", 0), ("ln_eps", 0.0), ("freq_dim", 6), ("num_blocks", 0),
                                         ("qk_norm_rope", 2)])
def test_invalid_config_rejected(field, value):
    cfg = fb.make_config(synth.TINY, fb.FP32, 2, 16, 8, 1)
    setattr(cfg, field, value)
    assert fb.flashbon_weight_count(cfg) == 0


def test_init_rejects_wrong_weight_count_without_device():
    cfg = fb.make_config(synth.TINY, fb.FP32, 2, 16, 8, 1)
    w = np.zeros(10, np.float32)
    with pytest.raises(fb.FlashbonError) as e:
        fb.flashbon_init_model(cfg, w)
    assert e.value.status == fb.ESHAPE


def test_round_to_bf16_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e38], np.float32)
    y = synth.round_to_bf16(x)
    assert list(y[:3]) == [1.0, 1.0, 1.0 + 2 ** -6]   # ties to even, then round up past the tie
    assert y[3] == -2.5


@pytest.mark.parametrize("t_cur,t_next,a", [(0.5, 0.4, -0.1), (0.0, -0.1, 0.3), (1.0, 1.0, 0.3),
                                            (1.5, 1.0, 0.3), (0.5, 0.4, float("nan")),
                                            (0.5, 0.4, float("inf"))])
def test_unpatch_sde_rejects_bad_noise_arguments_before_device_work(t_cur, t_next, a):
    """Host validation of the stochastic update (App. A.1, Eq. 20): no kernel is launched, so the
    (never dereferenced) placeholder pointers are safe without a device."""
    lib = fb.load()
    st = lib.flashbon_op_unpatch_sde(1, 1, 8, 8, 2, 0x1000, 0x2000, t_cur, t_next, a, 1, 0, 0, None)
    assert st == fb.EINVAL
    assert b"t_cur" in lib.flashbon_last_error()


@pytest.mark.parametrize("args", [(0, 1, 8, 8, 2), (1, 1, 7, 8, 2), (1, 0, 8, 8, 2), (1, 1, 8, 8, 0)])
def test_unpatch_sde_rejects_bad_shapes(args):
    lib = fb.load()
    st = lib.flashbon_op_unpatch_sde(*args, 0x1000, 0x2000, 0.5, 0.4, 0.3, 1, 0, 0, None)
    assert st == fb.ESHAPE


def test_unpatch_sde_rejects_negative_counters():
    lib = fb.load()
    assert lib.flashbon_op_unpatch_sde(1, 1, 8, 8, 2, 0x1000, 0x2000, 0.5, 0.4, 0.3, 1, -1, 0, None) == fb.EINVAL
    assert lib.flashbon_op_unpatch_sde(1, 1, 8, 8, 2, 0x1000, 0x2000, 0.5, 0.4, 0.3, 1, 0, -3, None) == fb.EINVAL


def test_normals_rejects_bad_arguments():
    lib = fb.load()
    assert lib.flashbon_op_normals(0, 0, 0, 1, 0x1000, None, None) == fb.ESHAPE
    assert lib.flashbon_op_normals(8, -1, 0, 1, 0x1000, None, None) == fb.EINVAL
    assert lib.flashbon_op_normals(8, 0, 0, 1, None, None, None) == fb.EINVAL


@pytest.mark.parametrize("params", [(0.5, 0.5, 1.5), (0.25, 0.5, 1.0), (1.0, 1.0, 0.0), (0.3, 0.7, 2.5),
                                    (1.0, 1.0, 3.0)])
def test_select_matches_oracle_bit_exact(params):
    """Host Elo selection (Sec. 4.2 Stage 2, Eq. 9-12) against the oracle: same matches in the same
    order (the synthetic verifier's outcomes depend on the pair and its meeting count only), same
    winner, bit-identical ratings and call count."""
    from oracle import select as osel
    for seed in range(6):
        for m in (1, 2, 3, 5, 16, 33, 64, 100):
            v_ref, v_lib = synth.SyntheticVerifier(m, seed), synth.SyntheticVerifier(m, seed)
            w_ref, r_ref, st = osel.select(v_ref.scores, v_ref.judge, *params)
            w, r, calls = fb.flashbon_select(v_lib.scores, v_lib.judge, *params)
            assert (w, calls) == (w_ref, len(st["matches"])), (seed, m)
            np.testing.assert_array_equal(r, np.array(r_ref))
            assert v_lib.meetings == v_ref.meetings


def test_select_rejects_bad_arguments():
    judge = lambda a, b: (a, 0)
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([5, 11], judge)                        # score outside 1..10
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([5, 6], judge, rho1=0.0)
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([5, 6], judge, kappa=float("nan"))
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([], judge)
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([5, 6, 7, 8], lambda a, b: (99, 0))   # winner not a or b
    with pytest.raises(fb.FlashbonError):
        fb.flashbon_select([5, 6, 7, 8], lambda a, b: (a, 3))    # unknown confidence

    def broken(a, b):
        raise KeyError("verifier down")
    with pytest.raises(KeyError):
        fb.flashbon_select([5, 6, 7, 8], broken)


@pytest.mark.parametrize("shape,kernels,desc", [
    ((24960, 4608, 1536, 0), 1, "k_linear_dma8 (8 waves): 99 row blocks x 18, 87 of 256 rows and 12 of 224"),
    ((24960, 8960, 1536, 1), 1, "k_linear_dma8 (8 waves): 102 row blocks x 35, 66 of 256 rows and 36 of 224"),
    ((24960, 1536, 1536, 3), 1, "k_linear_dma8 (8 waves): 128 row blocks x 6, 12 of 224 rows and 116 of 192"),
    ((24960, 1536, 8960, 3), 1, "k_linear_dma8 (8 waves): 128 row blocks x 6, 12 of 224 rows and 116 of 192"),
    ((16384, 15360, 5120, 0), 1, "k_linear_dma8 (8 waves): 256x256 tiles, 64 row blocks x 60"),
    ((200, 136, 72, 0), 1, "k_linear_mfma: 256x256 tiles, 8 waves"),
    ((1560, 4608, 1536, 0), 1, "k_linear_deep (8 waves): 128x256 tiles, 3 LDS stages"),
    ((1560, 8960, 1536, 1), 1, "k_linear_dma8 (8 waves): 224x256 tiles, 7 row blocks x 35"),
    ((1560, 1536, 1536, 3), 1, "k_linear_deep (8 waves): 128x128 tiles, 3 LDS stages"),
    ((1560, 1536, 8960, 3), 1, "k_linear_deep (8 waves): 128x128 tiles, 3 LDS stages"),
    ((3120, 1536, 1536, 3), 1, "k_linear_deep (8 waves): 160x128 tiles, 3 LDS stages"),
])
def test_linear_plan_of_model_shapes(shape, kernels, desc, monkeypatch):
    """The tile plan is a host decision (no device needed; 256 CUs assumed without one).  At the
    1.3B-shaped pool's M = 16 x 1560 rows: QKV and MLP up on row blocks of 256 and 224 rows of the
    8-wave kernel that fill 7 and 14 rounds, the N = 1536 projections on 128 row blocks of 224 and 192
    rows that fill three rounds exactly;
    K % 64 != 0 takes the generic 8-wave kernel with register-staged loads.  One candidate's projections
    (M = 1560) and two candidates' N = 1536 projections fit one round of the deep-ring tile, on the tile
    that gives the most workgroups within it; MLP up at M = 1560 does not (7 x 35 tiles of 224 rows)."""
    monkeypatch.delenv("FLASHBON_LINEAR_TILE", raising=False)
    assert fb.flashbon_op_linear_plan(fb.BF16, *shape) == (kernels, desc)
    # the row blocks named cover M with no block starting past it
    m = re.search(r"(\d+) row blocks x \d+, (\d+) of (\d+) rows and (\d+) of (\d+)", desc)
    if m:
        mb, tall, hi, short, lo = map(int, m.groups())
        assert tall + short == mb and hi == lo + 32
        total = tall * hi + short * lo
        assert shape[0] <= total < shape[0] + lo


def test_linear_plan_follows_override_and_rejects_bad_arguments(monkeypatch):
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", "split:24320")
    n, d = fb.flashbon_op_linear_plan(fb.BF16, 24960, 8960, 1536, 1)
    assert n == 2 and "rows 0..24319" in d and "remaining 640 rows" in d
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", "mix:7:128:12")
    assert fb.flashbon_op_linear_plan(fb.BF16, 24960, 1536, 1536, 3)[1] == \
        "k_linear_dma: 128 row blocks x 6, 12 of 224 rows and 116 of 192"
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", "w8:mix:7:128:12")
    assert fb.flashbon_op_linear_plan(fb.BF16, 24960, 1536, 1536, 3)[1] == \
        "k_linear_dma8 (8 waves): 128 row blocks x 6, 12 of 224 rows and 116 of 192"
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", "w8:bm:192")
    assert fb.flashbon_op_linear_plan(fb.BF16, 24960, 1536, 1536, 3)[1] == \
        "k_linear_dma8 (8 waves): 192x256 tiles, 130 row blocks x 6"
    monkeypatch.setenv("FLASHBON_LINEAR_TILE", "mix:7:100:0")    # does not cover M: ignored
    assert "256x256" in fb.flashbon_op_linear_plan(fb.BF16, 24960, 1536, 1536, 3)[1]
    monkeypatch.delenv("FLASHBON_LINEAR_TILE")
    assert fb.flashbon_op_linear_plan(fb.FP32, 100, 64, 64, 0)[1].startswith("k_linear_valu")
    lib = fb.load()
    n = ctypes.c_int32()
    buf = ctypes.create_string_buffer(8)
    for args in [(fb.BF16, 0, 64, 64, 0), (fb.BF16, 64, 62, 64, 0), (fb.BF16, 64, 64, 12, 0), (7, 64, 64, 64, 0),
                 (fb.BF16, 64, 64, 64, 4)]:
        assert lib.flashbon_op_linear_plan(*args, ctypes.byref(n), buf, len(buf)) != 0
    assert lib.flashbon_op_linear_plan(fb.BF16, 64, 64, 64, 0, None, buf, len(buf)) != 0
    assert lib.flashbon_op_linear_plan(fb.BF16, 64, 64, 64, 0, ctypes.byref(n), buf, len(buf)) == 0
    assert len(buf.value) == 7    # truncated to desc_len - 1 characters


@pytest.mark.parametrize("args,status", [
    ((7, 64, 64, 64), fb.EINVAL),          # bad dtype
    ((fb.BF16, 0, 64, 64), fb.ESHAPE),     # M < 1
    ((fb.BF16, 64, 6, 64), fb.ESHAPE),     # N % 4 != 0
    ((fb.BF16, 64, 64, 12), fb.ESHAPE),    # K % 8 != 0
])
def test_linear_ws_rejects_bad_arguments_before_device_work(args, status):
    """flashbon_op_linear_ws validates on the host and returns before any launch (no device needed)."""
    sp = ctypes.c_int32(-7)
    st = fb.load().flashbon_op_linear_ws(*args, None, None, None, fb.EPI_STORE, None, None, None, None, 0,
                                         ctypes.byref(sp), None)
    assert st == status
    assert sp.value == -7                  # nothing reported for a rejected call


def test_linear_ws_requires_operands():
    sp = ctypes.c_int32(-7)
    st = fb.load().flashbon_op_linear_ws(fb.BF16, 64, 64, 64, None, None, None, fb.EPI_STORE, None, None, None,
                                         None, 0, ctypes.byref(sp), None)
    assert st == fb.EINVAL and sp.value == -7
