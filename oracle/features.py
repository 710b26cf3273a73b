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
attention features and are left alone by update_features.

The fourth router feature is the attention-output reconstruction error of
the previous probe interval (Eq. 3).  Eq. 3 gives one error per sequence and
query head, while the router scores tokens.  Reading used here: for window m,
KV head h and sequence b, the feature is the largest Eq. 3 error over the
window's probed layers of the interval and over h's G query heads, and every
token of (b, h) carries it in phi[m][h][t][3]; the first probed layer of an
interval overwrites the column, later ones keep the maximum, and heads not
probed in the interval keep their previous value.
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


def probe_feature(phi: np.ndarray, cu_seqlens, window: int, kv_heads, err: np.ndarray, G: int,
                  fresh: bool) -> np.ndarray:
    """Fold one probed layer's Eq. 3 errors err [B][n*G] (probed KV head
    kv_heads[i], group member g at column i*G + g) into column 3 of window
    `window` of phi [M][Hkv][T][4] (in place)."""
    err = np.asarray(err, dtype=np.float32)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    for i, h in enumerate(kv_heads):
        for b in range(len(cu) - 1):
            e = float(np.max(err[b, i * G:(i + 1) * G]))
            for t in range(int(cu[b]), int(cu[b + 1])):
                if fresh:
                    phi[window, h, t, 3] = e
                else:
                    phi[window, h, t, 3] = max(float(phi[window, h, t, 3]), e)
    return phi
