"""Plain reference for the token-conditional depth router (Eq. 2) and the
residual-offset table it implies.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module.

Eq. 2 (Sec. 3) routes token t of window m, head h to residual rank
    rho = rho_min + (rho_max - rho_min) * 1[ sigma(u^T phi_{m,h,t}) > tau_m ],
with u a router vector shared by the layers of window m and tau_m the
window's adaptive threshold.  The paper then states that three (or more) rank
levels are used in practice rather than a binary decision.  Reading used here:
with ascending thresholds tau_{m,0} < tau_{m,1} < ..., the level index is the
number of thresholds the gate exceeds, k = #{j : sigma(u^T phi) > tau_{m,j}},
and rho = levels[k]; with two levels this is exactly Eq. 2.  Because sigma is
strictly increasing, sigma(z) > tau  <=>  z > logit(tau), so the thresholds are
passed as logits theta = logit(tau) in float32 and compared with strict ">".

Precision (the paper fixes none): the score z = u^T phi is evaluated in
float32, left to right, each product and each sum rounded to float32 on its
own: z = ((u0*phi0 + u1*phi1) + u2*phi2) + u3*phi3.

The offsets are the exclusive running sum of the routed ranks per (window,
head) over the packed tokens of all sequences: token t's residual entries
occupy [off[t], off[t+1]).
"""
from __future__ import annotations

import numpy as np


def router_score(phi: np.ndarray, u: np.ndarray) -> np.ndarray:
    """phi [..., 4] float32, u [4] float32 -> z [...] float32."""
    phi = np.asarray(phi, dtype=np.float32)
    u = np.asarray(u, dtype=np.float32)
    z = np.float32(u[0]) * phi[..., 0]
    z = z + np.float32(u[1]) * phi[..., 1]
    z = z + np.float32(u[2]) * phi[..., 2]
    z = z + np.float32(u[3]) * phi[..., 3]
    return z.astype(np.float32)


def level_index(z: np.ndarray, theta: np.ndarray) -> np.ndarray:
    """k = number of thresholds exceeded (strictly)."""
    z = np.asarray(z, dtype=np.float32)
    k = np.zeros(z.shape, dtype=np.int64)
    for th in np.asarray(theta, dtype=np.float32):
        k += (z > th)
    return k


def route(phi: np.ndarray, u: np.ndarray, theta: np.ndarray, levels):
    """phi [M][Hkv][T][4], u [M][4], theta [M][n_levels-1] (float32).
    Returns rank_code uint8 [M][Hkv][T] and res_off uint32 [M][Hkv][T+1]."""
    M, Hk, T, _ = phi.shape
    lev = np.asarray(levels, dtype=np.int64)
    codes = np.empty((M, Hk, T), dtype=np.uint8)
    off = np.zeros((M, Hk, T + 1), dtype=np.uint32)
    for m in range(M):
        z = router_score(phi[m], u[m])                        # [Hk, T]
        k = level_index(z, theta[m])
        codes[m] = k
        run = np.cumsum(lev[k], axis=1)
        if T and run[:, -1].max() > np.iinfo(np.uint32).max:
            raise OverflowError("residual offsets exceed 32 bits")
        off[m, :, 1:] = run
    return codes, off


def theta_from_tau(tau) -> np.ndarray:
    """Thresholds on the gate sigma(z) -> thresholds on z (float64 logit,
    rounded to float32)."""
    tau = np.asarray(tau, dtype=np.float64)
    return np.log(tau / (1.0 - tau)).astype(np.float32)


def route_range(phi: np.ndarray, u: np.ndarray, theta: np.ndarray, levels, t0: int, t1: int,
                codes: np.ndarray, off: np.ndarray):
    """Route packed tokens [t0, t1) in place, continuing an existing table:
    codes[m][h][t] for those tokens and off[m][h][t+1] = off[m][h][t] + rho,
    starting from the off[m][h][t0] already there (0 when t0 == 0).  The
    append of a decode token is the range [T-1, T)."""
    M, Hk = codes.shape[0], codes.shape[1]
    lev = np.asarray(levels, dtype=np.int64)
    if t0 == 0:
        off[:, :, 0] = 0
    for m in range(M):
        z = router_score(phi[m, :, t0:t1], u[m])
        k = level_index(z, theta[m])
        codes[m, :, t0:t1] = k
        run = off[m, :, t0:t0 + 1].astype(np.int64) + np.cumsum(lev[k], axis=1)
        if run.size and run.max() > np.iinfo(np.uint32).max:
            raise OverflowError("residual offsets exceed 32 bits")
        off[m, :, t0 + 1:t1 + 1] = run
    return codes, off
