import numpy as np


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# Velocity tolerances of the step tests (relative L2 of v = (z_next - z) / dt per step).  The latent
# check alone is weak: |dt v| / |z| is about 0.04 per step on these workloads, so a latent bound of 2e-2
# would let a velocity off by half pass.  bf16 mode: every GEMM and attention takes bf16 operands (one
# rounding, 2^-9 relative, per operand).  Measured: <= 8.3e-3 on the 1.3B-shaped pools and the
# mid/tiny workloads; 1.8e-2 at the 14B layer shapes, whose attention logits spread about 3.4x wider
# (std 0.02^2 D = 2.0 against 0.6 at D = 1536), so the same rounding of q and k moves the softmax more;
# 2.1e-2 with qk RMSNorm + RoPE on the mid workload.  The bound sits just above the widest of these.
TOL_V = {"fp32": 1e-4, "bf16": 3e-2}


def step_velocity(z_next, z_prev, t_cur, t_next, noise=None):
    """The step's velocity (z_next - z_prev) / dt, per candidate row [n, C, H, W].

    With ``noise = (a, seed, step, row0)`` (the stochastic update of Eq. 20), the known noise term
    sigma sqrt(|dt|) eps of each row -- eps drawn by the oracle's counter-based generator for counter
    row row0 + b -- is removed first, leaving the drift v + sigma^2 / (2 t) (z + (1 - t) v)."""
    z_next = np.asarray(z_next, np.float64)
    z_prev = np.asarray(z_prev, np.float64)
    dt = float(np.float32(t_next)) - float(np.float32(t_cur))
    if noise is None:
        return (z_next - z_prev) / dt
    from oracle import sde as osde
    a, seed, step, row0 = noise
    g = osde.sigma(float(np.float32(t_cur)), float(np.float32(t_next)), a) * np.sqrt(abs(dt))
    out = np.empty_like(z_next)
    for b in range(z_next.shape[0]):
        eps = osde.latent_normals(z_next.shape[1:], row0 + b, step, seed)
        out[b] = (z_next[b] - g * eps - z_prev[b]) / dt
    return out
