"""Seeded synthetic inputs for the batched draft step: model shapes, workloads, weights, latents, text.

This module holds shapes, seeds and random-number draws only; none of the method's arithmetic lives
here.  Both the CPU oracle (through the tests) and the HIP library (through the binding) take their
inputs from it, so neither side ever produces the other's inputs.

Recipe (all values float32):
  * every weight matrix, bias and per-block modulation table ~ N(0, 0.02^2), one generator per tensor,
    ``default_rng([seed_w, tensor_index])`` in the fixed tensor order of :func:`weight_specs`;
  * candidate j's initial latent z_T^(j) ~ N(0, I) from ``default_rng(10_000 + j)`` -- distinct seeds
    per candidate, as in the paper's Stage 1 (Sec. 4.2, Eq. 8);
  * text conditioning c ~ N(0, 1), shape [text_len, text_dim], from ``default_rng(20_000 + c)``;
  * timestep schedule ``linspace(1, 0, S + 1)`` (rectified flow, t = 1 is noise; App. A.1).
The shapes are those of Wan2.1-1.3B / 14B-sized DiTs and of the workloads the paper evaluates
(Sec. 5, App. A.2); the paper's prompts and benchmarks are replaced by these random tensors.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Tuple

import numpy as np

WEIGHT_STD = 0.02
NORM_GAINS = ("nq", "nk", "nqc", "nkc")


@dataclasses.dataclass(frozen=True)
class ModelShape:
    num_blocks: int
    hidden: int
    heads: int
    mlp_hidden: int
    freq_dim: int
    text_dim: int
    latent_channels: int = 16
    patch: int = 2
    ln_eps: float = 1e-6
    qk_norm_rope: bool = False      # RMSNorm on q/k (self and cross) + 3-D RoPE on self-attention

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def patch_dim(self) -> int:
        return self.latent_channels * self.patch * self.patch


@dataclasses.dataclass(frozen=True)
class Workload:
    """One workload: a model shape, a candidate pool, a schedule and the per-step knob masks."""
    name: str
    shape: ModelShape
    n: int                      # candidates in the pool
    latent_h: int
    latent_w: int
    text_len: int
    n_cond: int
    steps_total: int            # S, length of the full schedule
    steps_draft: int            # S', truncated draft length
    dtype: str                  # "fp32" or "bf16" compute mode
    seed_w: int = 1234

    @property
    def tokens(self) -> int:
        return (self.latent_h // self.shape.patch) * (self.latent_w // self.shape.patch)

    def cond_index(self) -> np.ndarray:
        # candidates split into n_cond equal groups, group c conditioned on prompt c
        return (np.arange(self.n) * self.n_cond // self.n).astype(np.int32)

    def schedule(self) -> np.ndarray:
        return np.linspace(1.0, 0.0, self.steps_total + 1).astype(np.float32)

    def masks(self, k: int) -> Tuple[np.ndarray, np.ndarray]:
        return step_masks(self.name, self.shape.num_blocks, k)


TINY = ModelShape(num_blocks=2, hidden=64, heads=4, mlp_hidden=256, freq_dim=64, text_dim=32)
WAN_1_3B = ModelShape(num_blocks=30, hidden=1536, heads=12, mlp_hidden=8960, freq_dim=256, text_dim=4096)
WAN_14B = ModelShape(num_blocks=40, hidden=5120, heads=40, mlp_hidden=13824, freq_dim=256, text_dim=4096)
# Mid-size shape used by parity tests: head_dim 128 like the real models, several tiles, ragged tails.
MID = ModelShape(num_blocks=3, hidden=256, heads=2, mlp_hidden=704, freq_dim=64, text_dim=96)

WORKLOADS: Dict[str, Workload] = {
    # tiny fp32 pool: 2 blocks, 16 tokens, 4-step schedule
    "tiny": Workload("tiny", TINY, n=2, latent_h=8, latent_w=8, text_len=8, n_cond=1,
                     steps_total=4, steps_draft=4, dtype="fp32"),
    # one full-quality 1.3B-shaped step, N=1
    "wan1.3b_step": Workload("wan1.3b_step", WAN_1_3B, n=1, latent_h=60, latent_w=104, text_len=512,
                             n_cond=1, steps_total=50, steps_draft=1, dtype="bf16"),
    # 1.3B-shaped draft pool: N=16, 10 of 50 steps, every 3rd block skipped, proxies on odd steps
    "wan1.3b_pool16": Workload("wan1.3b_pool16", WAN_1_3B, n=16, latent_h=60, latent_w=104,
                               text_len=512, n_cond=1, steps_total=50, steps_draft=10, dtype="bf16"),
    # 14B-shaped draft pool: N=4 at 4096 tokens, 8 of 50 steps, blocks 24..35 skipped
    "wan14b_pool4": Workload("wan14b_pool4", WAN_14B, n=4, latent_h=128, latent_w=128, text_len=512,
                             n_cond=1, steps_total=50, steps_draft=8, dtype="bf16"),
    # 1.3B-shaped large pool: N=64 at 1024 tokens, 4 prompts x 16, 12 of 50 steps, varying masks
    "wan1.3b_pool64": Workload("wan1.3b_pool64", WAN_1_3B, n=64, latent_h=64, latent_w=64,
                               text_len=512, n_cond=4, steps_total=50, steps_draft=12, dtype="bf16"),
    # 14B-shaped layers (D=5120, 40 heads, MLP 13824, 4096 tokens, N=4) in a 2-block model, so the
    # oracle can follow a full step at these shapes in seconds
    "wan14b_2block": Workload("wan14b_2block", dataclasses.replace(WAN_14B, num_blocks=2), n=4,
                              latent_h=128, latent_w=128, text_len=512, n_cond=1, steps_total=50,
                              steps_draft=2, dtype="bf16"),
    # mid-size parity pool (head_dim 128, ragged token count 130, 2 prompts)
    "mid": Workload("mid", MID, n=3, latent_h=10, latent_w=52, text_len=40, n_cond=2,
                    steps_total=8, steps_draft=8, dtype="fp32"),
    # the same two pools with qk RMSNorm + 3-D RoPE
    "tiny_rope": Workload("tiny_rope", dataclasses.replace(TINY, qk_norm_rope=True), n=2, latent_h=8, latent_w=8,
                          text_len=8, n_cond=1, steps_total=4, steps_draft=4, dtype="fp32"),
    "mid_rope": Workload("mid_rope", dataclasses.replace(MID, qk_norm_rope=True), n=3, latent_h=10, latent_w=52,
                         text_len=40, n_cond=2, steps_total=8, steps_draft=8, dtype="fp32"),
}


def step_masks(name: str, num_blocks: int, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Per-step (skip, proxy) uint8 masks over 0-based blocks for the named workload, step k (0-based)."""
    skip = np.zeros(num_blocks, np.uint8)
    proxy = np.zeros(num_blocks, np.uint8)
    if name in ("tiny", "tiny_rope"):
        # skip block 1 on steps 2-3, proxies on step 3
        if k in (2, 3):
            skip[1] = 1
        if k == 3:
            proxy[:] = 1
    elif name == "wan1.3b_pool16":
        skip[2::3] = 1
        if k % 2 == 1:
            proxy[:] = 1
    elif name == "wan14b_pool4":
        skip[24:36] = 1
        if k % 2 == 1:
            proxy[:] = 1
    elif name == "wan1.3b_pool64":
        n_k = 6 + (9 * k) // 11
        perm = np.random.default_rng(1000 + k).permutation(num_blocks)
        skip[perm[:n_k]] = 1
        if k % 2 == 1:
            proxy[:] = 1
    elif name == "wan14b_2block":
        if k == 1:
            skip[1] = 1
            proxy[0] = 1
    elif name in ("mid", "mid_rope"):
        # exercises the empty-cache fallback, warm-up orders 0/1/2, dead and live proxies,
        # skip-over-proxy and proxies over unequally spaced cached steps
        if k >= 2:
            skip[1] = 1
        if k in (1, 3, 5, 7):
            proxy[:] = 1
        if k == 4:
            proxy[0] = proxy[1] = 1
        if k == 0:
            proxy[2] = 1
    return skip, proxy


def weight_specs(s: ModelShape) -> List[Tuple[str, Tuple[int, ...]]]:
    """Named weight tensors in packing order; matrices are [out, in] row-major."""
    D, F, P, Dt, fd = s.hidden, s.mlp_hidden, s.patch_dim, s.text_dim, s.freq_dim
    specs: List[Tuple[str, Tuple[int, ...]]] = [
        ("t_w1", (D, fd)), ("t_b1", (D,)), ("t_w2", (D, D)), ("t_b2", (D,)),
        ("mod_w", (6 * D, D)), ("mod_b", (6 * D,)),
        ("head_mod_w", (2 * D, D)), ("head_mod_b", (2 * D,)),
        ("pe_w", (D, P)), ("pe_b", (D,)),
        ("txt_w", (D, Dt)), ("txt_b", (D,)),
    ]
    for l in range(s.num_blocks):
        b = f"blk{l}."
        specs += [
            (b + "mod", (6, D)),
            (b + "wq", (D, D)), (b + "wk", (D, D)), (b + "wv", (D, D)),
            (b + "bq", (D,)), (b + "bk", (D,)), (b + "bv", (D,)),
            (b + "wo", (D, D)), (b + "bo", (D,)),
            (b + "wqc", (D, D)), (b + "bqc", (D,)),
            (b + "wkc", (D, D)), (b + "wvc", (D, D)), (b + "bkc", (D,)), (b + "bvc", (D,)),
            (b + "woc", (D, D)), (b + "boc", (D,)),
            (b + "w1", (F, D)), (b + "b1", (F,)),
            (b + "w2", (D, F)), (b + "b2", (D,)),
        ]
        if s.qk_norm_rope:
            specs += [(b + "nq", (D,)), (b + "nk", (D,)), (b + "nqc", (D,)), (b + "nkc", (D,))]
    specs += [("head_w", (P, D)), ("head_b", (P,))]
    return specs


def weight_count(s: ModelShape) -> int:
    return int(sum(int(np.prod(sh)) for _, sh in weight_specs(s)))


def make_weights(s: ModelShape, seed_w: int = 1234, threads: int = 8,
                 out: Optional[np.ndarray] = None) -> Tuple[np.ndarray, Dict[str, np.ndarray]]:
    """Draw every weight ~ N(0, 0.02^2) as float32 (RMSNorm gains ~ 1 + N(0, 0.02^2)).

    Returns (flat, views): ``flat`` is one contiguous float32 array in packing order, ``views`` maps
    each tensor name to a reshaped view into it.
    """
    specs = weight_specs(s)
    sizes = [int(np.prod(sh)) for _, sh in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    total = int(offs[-1])
    flat = np.empty(total, np.float32) if out is None else out
    assert flat.shape == (total,) and flat.dtype == np.float32

    def fill(i: int) -> None:
        rng = np.random.default_rng([seed_w, i])
        seg = flat[offs[i]:offs[i + 1]]
        rng.standard_normal(out=seg, dtype=np.float32)
        seg *= np.float32(WEIGHT_STD)
        if specs[i][0].rsplit(".", 1)[-1] in NORM_GAINS:
            seg += np.float32(1.0)

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(fill, range(len(specs))))
    views = {name: flat[offs[i]:offs[i + 1]].reshape(sh) for i, (name, sh) in enumerate(specs)}
    return flat, views


def make_latents(n: int, channels: int, h: int, w: int, first_seed: int = 10_000) -> np.ndarray:
    """Candidate j's latent z_T^(j) ~ N(0, I) from its own seed (10_000 + j): [n, C, H, W] float32."""
    z = np.empty((n, channels, h, w), np.float32)
    for j in range(n):
        z[j] = np.random.default_rng(first_seed + j).standard_normal((channels, h, w), dtype=np.float32)
    return z


def make_text(n_cond: int, text_len: int, text_dim: int, first_seed: int = 20_000) -> np.ndarray:
    """Text-conditioning tokens ~ N(0, 1): [n_cond, text_len, text_dim] float32."""
    x = np.empty((n_cond, text_len, text_dim), np.float32)
    for c in range(n_cond):
        x[c] = np.random.default_rng(first_seed + c).standard_normal((text_len, text_dim), dtype=np.float32)
    return x


def random_cache_entries(shape: Tuple[int, ...], seed: int) -> np.ndarray:
    """Three ~N(0,1) cached activations stacked on axis 0 (for proxy-kernel tests)."""
    return np.random.default_rng(seed).standard_normal((3,) + tuple(shape), dtype=np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32.

    Used to draw test operands that are exactly representable in bf16, so that a bf16 kernel and
    an fp64 reference see identical input values."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def random_matrix(shape: Tuple[int, ...], seed: int, scale: float = 1.0) -> np.ndarray:
    """~N(0, scale^2) float32 tensor."""
    a = np.random.default_rng(seed).standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        a *= np.float32(scale)
    return a


class SyntheticVerifier:
    """Seeded stand-in for the paper's VLM verifier (Sec. 4.2 Stage 2), which is not part of this
    library: every candidate has a hidden quality q_j ~ N(0, 1) (``default_rng(seed)``).

    * pointwise score: integer 1..10, round(5.5 + 1.5 q_j + 0.75 n_j) clipped, n_j ~ N(0, 1) -- coarse
      and tie-prone, like the integer scores the paper describes;
    * pairwise judgement of (a, b): a wins with probability 1 / (1 + exp(-(q_a - q_b) / 0.5)), the
      uniform draw coming from ``default_rng([seed, min(a, b), max(a, b), m])`` for the m-th meeting
      of that pair, so an outcome depends only on the pair and how often it has met; confidence 0
      (high) if |q_a - q_b| > 1, 1 (medium) if > 0.3, else 2 (low).
    """

    def __init__(self, m: int, seed: int):
        rng = np.random.default_rng(seed)
        self.seed = seed
        self.quality = rng.standard_normal(m)
        noise = rng.standard_normal(m)
        self.scores = np.clip(np.rint(5.5 + 1.5 * self.quality + 0.75 * noise), 1, 10).astype(np.int32)
        self.meetings: Dict[Tuple[int, int], int] = {}
        self.calls = 0

    def judge(self, a: int, b: int) -> Tuple[int, int]:
        lo, hi = (a, b) if a < b else (b, a)
        m = self.meetings.get((lo, hi), 0)
        self.meetings[(lo, hi)] = m + 1
        self.calls += 1
        u = np.random.default_rng([self.seed, lo, hi, m]).random()
        d = float(self.quality[a] - self.quality[b])
        p_a = 1.0 / (1.0 + np.exp(-d / 0.5))
        conf = 0 if abs(d) > 1.0 else (1 if abs(d) > 0.3 else 2)
        return (a if u < p_a else b), conf
