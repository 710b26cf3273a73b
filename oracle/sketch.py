"""Plain reference for the online basis initialization (Sec. 3).

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module.

In Sec. 3 the shared bases of a depth window start out, once the prompt has
been prefilled, as a low-rank random projection of that window's keys and of
its values (each head on its own, keys apart from values).  Reading used here: for sequence b, window m,
KV head h and Z, stack the window's prefill vectors of that head (every layer
of the window, every token) as the rows of X ((w T_b) x d); with a random
sketch matrix Omega (r_b x (w T_b), an input, shared by the heads and by K and
V), the sketch is Y = Omega X (r_b x d) and the basis is the orthonormalized
rows of Y (Gram-Schmidt in order, each row's component along the earlier ones
removed, then normalized), rounded to fp16.  A row whose remaining norm falls
below 1e-9 of the largest sketch row norm (a rank-deficient sketch) becomes
zero.  Arithmetic here is float64 on the fp16 inputs.
"""
from __future__ import annotations

import numpy as np


def sketch(x_rows: np.ndarray, omega: np.ndarray) -> np.ndarray:
    """Y = Omega X: x_rows [(w T_b), d], omega [r_b, (w T_b)] -> [r_b, d] float64."""
    return np.asarray(omega, np.float64) @ np.asarray(x_rows, np.float64)


def orthonormal_rows(Y: np.ndarray) -> np.ndarray:
    """Modified Gram-Schmidt over the rows of Y, in order (float64)."""
    Y = np.array(Y, dtype=np.float64)
    Q = np.zeros_like(Y)
    floor = 1e-9 * (np.linalg.norm(Y, axis=1).max() if Y.size else 0.0)
    for i in range(Y.shape[0]):
        v = Y[i].copy()
        for j in range(i):
            v -= (v @ Q[j]) * Q[j]
        n = np.linalg.norm(v)
        Q[i] = v / n if n > floor and n > 0 else 0.0
    return Q


def sketch_basis(x: np.ndarray, omega: np.ndarray, h: int, z: int) -> np.ndarray:
    """fp16 basis [r_b, d] of head h, Z = z from the window's prefill
    x [w][2][T_b][Hkv][d] (fp16) and omega [(w T_b)][r_b] (fp16, row l T_b + t)."""
    w, _, Tb, _, d = x.shape
    rows = np.asarray(x[:, z, :, h, :], np.float64).reshape(w * Tb, d)
    Y = sketch(rows, np.asarray(omega, np.float64).T)
    return orthonormal_rows(Y).astype(np.float16)
