"""Oracle dispatch: which action each block takes at one step, and the activation-cache bookkeeping.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package; the product path never does.

Pure integer/host logic, written from the paper's knob definitions:
  * Layer skipping (Sec. 4.1 (3), Eq. 6): a skipped block propagates its input unchanged.
  * Activation proxies (Sec. 4.1 (2), Eq. 3-5): the block output is forecast from up to three cached
    outputs of the same block at earlier (larger) timesteps.
  * Configuration phi = (S', n_skip, l_start, l_end, f_full) (Sec. 4.1, "Configuration Space").

Readings where the paper is silent (each is listed with its reason in the design notes):
  * skip wins over proxy on the same (step, block);
  * only fully computed blocks write the cache; the proxy uses the most recent computed entries of
    that block, with their own timesteps; with c entries the Taylor order is min(c, 3) - 1; a proxy
    requested with an empty cache falls back to full computation;
  * the cache per block is a 3-slot ring: meta = {count, head, t[3]}; a COMPUTE writes slot ``head``,
    records its timestep there, advances head modulo 3 and saturates count at 3.  Most recent entry
    is slot (head + 2) % 3, then (head + 1) % 3, then head;
  * a proxied block's output is "live" only if something reads it before another proxy overwrites
    the residual stream: the next non-skipped block is a full computation, or there is none (the
    output head reads it).
"""
from __future__ import annotations

import copy
from typing import Dict, List, Tuple

import numpy as np

COMPUTE, SKIP, PROXY = 0, 1, 2


def empty_meta(num_blocks: int) -> List[Dict]:
    return [{"count": 0, "head": 0, "t": [0.0, 0.0, 0.0]} for _ in range(num_blocks)]


def recent_slots(meta_l: Dict) -> List[int]:
    """Slots of the cached entries of one block, most recent first."""
    h = meta_l["head"]
    return [(h + 2) % 3, (h + 1) % 3, h][: min(meta_l["count"], 3)]


def plan_step(skip: np.ndarray, proxy: np.ndarray, meta: List[Dict], t_cur: float, residual: bool = False
              ) -> Tuple[List[Tuple[int, int, int, int]], List[Dict]]:
    """Return (trace, new_meta) for one step.

    trace[l] = (action, order, slot, live):
      COMPUTE: order -1, slot written, live 1
      SKIP:    order -1, slot -1,      live 0
      PROXY:   order 0..2, slot of the most recent entry, live 0/1
    ``t_cur`` is stored as float32, the precision the cache metadata holds.
    ``residual``: proxies forecast the block's residual delta and add it to their input, so every
    proxy's output is read (live 1).
    """
    L = len(meta)
    actions = []
    for l in range(L):
        if skip[l]:
            actions.append(SKIP)
        elif proxy[l] and meta[l]["count"] >= 1:
            actions.append(PROXY)
        else:
            actions.append(COMPUTE)
    new_meta = copy.deepcopy(meta)
    trace = []
    for l in range(L):
        a = actions[l]
        if a == SKIP:
            trace.append((SKIP, -1, -1, 0))
        elif a == PROXY:
            order = min(meta[l]["count"], 3) - 1
            nxt = [actions[j] for j in range(l + 1, L) if actions[j] != SKIP]
            live = 1 if (residual or not nxt or nxt[0] == COMPUTE) else 0
            trace.append((PROXY, order, recent_slots(meta[l])[0], live))
        else:
            m = new_meta[l]
            slot = m["head"]
            m["t"][slot] = float(np.float32(t_cur))
            m["head"] = (slot + 1) % 3
            m["count"] = min(m["count"] + 1, 3)
            trace.append((COMPUTE, -1, slot, 1))
    return trace, new_meta


def masks_from_phi(phi: Tuple[int, int, int, int, int], num_blocks: int, k: int
                   ) -> Tuple[np.ndarray, np.ndarray]:
    """(skip, proxy) masks at 0-based step k for phi = (S', n_skip, l_start, l_end, f_full).

    Readings: layer skipping is active from step n_skip on; full computation happens on steps with
    k mod f_full == 0 and every other step proxies every block; l_start..l_end are 1-based inclusive.
    Steps k >= S' are not part of the draft.
    """
    s_draft, n_skip, l_start, l_end, f_full = phi
    if not (0 <= k < s_draft):
        raise ValueError("step outside the draft")
    skip = np.zeros(num_blocks, np.uint8)
    proxy = np.zeros(num_blocks, np.uint8)
    if k >= n_skip:
        for l in range(l_start, l_end + 1):
            skip[l - 1] = 1
    if f_full > 1 and k % f_full != 0:
        proxy[:] = 1
    return skip, proxy
