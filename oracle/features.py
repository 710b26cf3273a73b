"""Plain reference for the router's attention features taken from a decode.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module.

Sec. 3 scores each token for the router from online features, among them its
accumulated attention mass and its maximum attention spike.  Reading used
here (the paper gives no formula): for one decode layer l in window m, KV head
h and packed token t of sequence b, with p the softmax probability of t for
query head hq (Eq. 1 keys, the decode's own attention),
    mass_t  = sum over the query heads hq of KV head h of p
    spike_t = max over the same heads of p
and the window's feature table accumulates them over its layers and over
decode steps: phi[m][h][t][0] += mass_t, phi[m][h][t][1] = max(phi, spike_t).
Columns 2 and 3 of phi (delimiter indicator, previous probe error) are not
attention features and are left alone.
"""
from __future__ import annotations

import numpy as np

from . import factorized as F


def attention_features(cache, layer: int, q=None, sm_scale=None):
    """mass, spike [Hkv][T] (float64) of one decode layer."""
    _, probs = F.decode(cache, layer, q, sm_scale, with_probs=True)
    Hk, T = cache.n_kv_heads, int(cache.cu_seqlens[-1])
    mass = np.zeros((Hk, T))
    spike = np.zeros((Hk, T))
    for (b, h), p in probs.items():
        t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
        if t1 > t0:
            mass[h, t0:t1] = p.sum(axis=0)
            spike[h, t0:t1] = p.max(axis=0)
    return mass, spike


def update_features(phi: np.ndarray, window: int, mass: np.ndarray, spike: np.ndarray) -> np.ndarray:
    """Fold one layer's features into phi [M][Hkv][T][4] (in place)."""
    phi[window, :, :, 0] += mass
    phi[window, :, :, 1] = np.maximum(phi[window, :, :, 1], spike)
    return phi
