"""Plain reference for the router's threshold control (Sec. 3).

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module.

Probe feedback: when a window's probe error (Eq. 3) exceeds its tolerance the
router lowers the window's threshold, so more tokens get the higher residual
rank; when the error stays below tolerance for several probe intervals in a
row it raises the threshold and residual storage shrinks.  The paper gives no
constants.  Reading used here: thresholds are logits theta = logit(tau) (as the
router compares them); every threshold of the window moves by the same step
(down by step_down on an error above tol, up by step_up after `patience`
consecutive intervals at or below tol), clamped to [theta_min, theta_max]; the
window's error is the largest Eq. 3 error over its probed layers, heads and
sequences; an error that is not a number counts as above tolerance; the
interval counter resets on every move.

Budget: tau_m is chosen to satisfy the memory budget.  Reading used here, for
the two-level form of Eq. 2 (rho_min, rho_max): with E residual entries
allowed for the window and head, and N tokens, the n = floor((E - N rho_min) /
(rho_max - rho_min)) tokens of largest router score z (ties to the lower token
index; clamped to [0, N]) get rho_max and the rest rho_min.

Probe schedule: the probe runs every p decode steps on a small subset of heads
and recent query positions.  Reading used here: decode step s (0-based, counted
from the first decode step after prefill) probes when s mod p == 0; the k-th
probe (k = s / p) takes the n KV heads (k n + i) mod Hkv, i = 0..n-1, so the
subset rotates and every head is probed in every ceil(Hkv / n) consecutive
probes; it evaluates min(P, s + 1) recent positions (the decode steps so far,
the current one included).
"""
from __future__ import annotations

import math

import numpy as np


def controller_update(theta, below, err, tol, step_down, step_up, patience, theta_min, theta_max):
    """One probe interval: theta [M][n_thr] and below [M] updated in place."""
    theta = np.asarray(theta)
    for m in range(theta.shape[0]):
        e = float(err[m])
        if math.isnan(e) or e > tol:
            theta[m] = np.clip(theta[m] - np.float32(step_down), theta_min, theta_max)
            below[m] = 0
        else:
            below[m] += 1
            if below[m] >= patience:
                theta[m] = np.clip(theta[m] + np.float32(step_up), theta_min, theta_max)
                below[m] = 0
    return theta, below


def budget_select(z: np.ndarray, entries: int, rho_min: int, rho_max: int) -> np.ndarray:
    """Two-level codes (0 = rho_min, 1 = rho_max) for router scores z [N] under a
    budget of `entries` residual entries: the largest-z tokens first, ties to
    the lower index."""
    N = len(z)
    n = (entries - N * rho_min) // (rho_max - rho_min) if rho_max > rho_min else 0
    n = max(0, min(N, n))
    order = sorted(range(N), key=lambda t: (-float(z[t]), t))
    codes = np.zeros(N, dtype=np.uint8)
    codes[order[:n]] = 1
    return codes


def route_budget(phi, u, entries, levels, t0: int, t1: int, codes, off):
    """Two-level routing of tokens [t0, t1) under a budget per (window, head):
    entries [M][Hkv] residual entries allowed over the range.  Writes
    codes[m][h][t] (0 or 1) and continues off[m][h][t+1] from off[m][h][t0]
    (0 when t0 == 0).  Router scores as the router computes them (Eq. 2)."""
    from .router import router_score
    lev = np.asarray(levels, dtype=np.int64)
    M, Hk = codes.shape[0], codes.shape[1]
    if t0 == 0:
        off[:, :, 0] = 0
    for m in range(M):
        z = router_score(phi[m, :, t0:t1], u[m])
        for h in range(Hk):
            k = budget_select(z[h], int(entries[m][h]), int(lev[0]), int(lev[1]))
            codes[m, h, t0:t1] = k
            off[m, h, t0 + 1:t1 + 1] = int(off[m, h, t0]) + np.cumsum(lev[k.astype(np.int64)])
    return codes, off


def probe_schedule(step: int, period: int, n_heads: int, n_kv_heads: int, n_pos: int):
    """(probed KV heads, positions) at decode step `step`; ([], 0) when the
    step does not probe."""
    if step % period != 0:
        return [], 0
    k = step // period
    return [(k * n_heads + i) % n_kv_heads for i in range(n_heads)], min(n_pos, step + 1)
