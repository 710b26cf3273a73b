"""Plain reference for the append/compress step: one dense key or value vector
of a token becomes its Eq. 1 factors (coefficient row, routed residual
channels with int4 codes, gate-folded scale).

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module.

What it computes, following Sec. 3 (the storage half of Eq. 1): the
coefficient row is the projection of the cache vector x (1 x d) onto the
window's current basis B (r_b x d), A = x B^T, kept in half precision; the
residual is what the basis term leaves, r = x - A B; the router's rank rho
decides how many residual channels are kept, and they are stored 4-bit
quantized with one scale per token, the token's gate g folded into it.

Readings where the paper is silent (each listed in the design notes):

* Projection: A = x B^T with the stored fp16 basis rows, the orthogonal
  projection for orthonormal rows (the bases come from an orthonormalising
  sketch and deviate from orthonormal only by fp16 rounding), not a
  least-squares solve against B B^T.
* Kept channels: the rho channels of largest |r|, ties to the lower channel.
* Quantization: symmetric int4 with codes in [-7, 7]: S = max_c |r_c| / 7 over
  all d channels, code = round-half-even(r_c / S); S = 0 gives code 0.
* Gate: the stored scale is fp16(g * S); g defaults to 1; a rank-0 token
  stores scale 0.
* Entry order inside a token: descending |code|, then ascending channel (the
  order the layout validator checks).
* 8-bit blockwise coefficients (Sec. 3 stores A in that form; reading C7):
  per token and block of 16 coefficients [16 s, 16 s + 16), the scale is
  S_s = fp16(max_i |A_i| / 127) from the float32 projection (not the fp16
  one), and code_i = round-half-even(A_i / S_s) clamped to [-127, 127] (0 when
  S_s == 0).  The residual is then taken against the coefficients the decode
  rebuilds, code_i * S_s (exact in float32).

Precision.  The kept channels and the codes are integers decided by floating
point, and the paper fixes no arithmetic for them.  Reading used here: single
precision written out in the plainest order, the one a scalar loop takes.
Every product and every sum is rounded to float32 on its own (no fused
multiply-add).  A sum over the contracted index (the d channels for A, the
r_b basis rows for the basis term of r) runs left to right, starting from its
first product.  A is rounded to fp16 (round-half-even) before the residual,
and r_c = x_c - p_c with p_c the basis term of channel c.  S = |r|_max / 7 and
r_c / S are correctly rounded float32 divisions.  Every fp16 conversion
rounds half to even.
"""
from __future__ import annotations

import numpy as np

from .factorized import window_of


# ------------------------------------------------------------ one vector
def _sum_in_order(terms):
    """A sum of float32 terms (a list, summed along the list) left to right:
    the first term, then each next term added with one rounding."""
    acc = terms[0]
    for t in terms[1:]:
        acc = acc + t
    return acc


def project32(x: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Coefficient rows A = x B^T for vectors x [n, d] against basis rows
    B [r_b, d] (fp16 values): float32 products summed over the d channels left
    to right.  Returns float32 [n, r_b]."""
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    B = np.asarray(B, dtype=np.float16).astype(np.float32)
    terms = [x[:, j:j + 1] * B[None, :, j] for j in range(x.shape[1])]
    return _sum_in_order(terms)


def project(x: np.ndarray, B: np.ndarray) -> np.ndarray:
    """project32 rounded to fp16 (the fp16 coefficient form).  Returns float16 [n, r_b]."""
    return project32(x, B).astype(np.float16)


def quantize_coefficients(a32: np.ndarray):
    """8-bit blockwise form of float32 coefficient rows a32 [n, r_b] (r_b a
    multiple of 16).  Returns (codes int8 [n, r_b], scales float16 [n, r_b/16],
    the rebuilt rows code * scale as float32 [n, r_b])."""
    a = np.asarray(a32, dtype=np.float32)
    n, rb = a.shape
    codes = np.zeros((n, rb), dtype=np.int8)
    scales = np.zeros((n, rb // 16), dtype=np.float16)
    for k in range(n):
        for s in range(rb // 16):
            blk = a[k, 16 * s:16 * s + 16]
            S = np.float16(np.float32(np.abs(blk).max()) / np.float32(127.0))
            scales[k, s] = S
            if S == 0:
                continue
            q = np.rint(blk / np.float32(S))
            codes[k, 16 * s:16 * s + 16] = np.clip(q, -127, 127).astype(np.int8)
    rebuilt = codes.astype(np.float32) * np.repeat(scales.astype(np.float32), 16, axis=1)
    return codes, scales, rebuilt


def residual(x: np.ndarray, B: np.ndarray, a: np.ndarray) -> np.ndarray:
    """r = x - A B in float32 for coefficient rows a [n, r_b] (the values the
    decode rebuilds: fp16 rows, or the dequantized 8-bit form): the basis term
    of each channel summed over the basis rows left to right, then subtracted
    from x.  Returns float32 [n, d]."""
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    B = np.asarray(B, dtype=np.float16).astype(np.float32)
    a = np.asarray(a, dtype=np.float32)
    terms = [a[:, i:i + 1] * B[None, i, :] for i in range(B.shape[0])]
    return x - _sum_in_order(terms)


def select_channels(r: np.ndarray, rho: int) -> np.ndarray:
    """The rho channels of largest |r| (ties to the lower channel), in that order."""
    mag = np.abs(np.asarray(r, dtype=np.float32))
    order = sorted(range(mag.size), key=lambda c: (-float(mag[c]), c))
    return np.asarray(order[:rho], dtype=np.int64)


def quant_scale(r: np.ndarray) -> np.float32:
    """Symmetric int4 scale: max |r| over every channel / 7 (float32)."""
    return np.float32(np.abs(np.asarray(r, dtype=np.float32)).max()) / np.float32(7.0)


def quantize(values: np.ndarray, S: np.float32) -> np.ndarray:
    """Codes round-half-even(v / S) clamped to [-7, 7]; S = 0 gives zeros."""
    v = np.asarray(values, dtype=np.float32)
    if S == 0:
        return np.zeros(v.shape, dtype=np.int64)
    q = np.rint(v / np.float32(S))
    return np.clip(q, -7, 7).astype(np.int64)


def entry_order(chans: np.ndarray, codes: np.ndarray):
    """Entries of one token sorted by descending |code|, then ascending channel."""
    idx = sorted(range(len(chans)), key=lambda e: (-abs(int(codes[e])), int(chans[e])))
    return np.asarray(chans, np.int64)[idx], np.asarray(codes, np.int64)[idx]


def fold_gate(S: np.float32, g: float) -> np.float16:
    """Stored scale fp16(g * S), the product rounded to float32 first."""
    return np.float16(np.float32(g) * np.float32(S))


def compress_vectors(x: np.ndarray, B: np.ndarray, rhos, gates=None, coef_format: str = "f16"):
    """Compress n vectors x [n, d] sharing basis B [r_b, d].

    Returns (coef, entries, scale16 [n] float16) where entries[k] = (channels,
    codes) of vector k in storage order, and coef is the float16 rows [n, r_b]
    or, for coef_format "int8", the pair (codes int8 [n, r_b], block scales
    float16 [n, r_b/16])."""
    x = np.asarray(x, dtype=np.float16)
    n = x.shape[0]
    if coef_format == "int8":
        codes8, cscales, rows = quantize_coefficients(project32(x, B))
        a16 = (codes8, cscales)
    else:
        a16 = rows = project(x, B)
    r = residual(x, B, rows)
    entries, scales = [], np.zeros(n, dtype=np.float16)
    for k in range(n):
        rho = int(rhos[k])
        if rho == 0:
            entries.append((np.zeros(0, np.int64), np.zeros(0, np.int64)))
            continue
        S = quant_scale(r[k])
        ch = select_channels(r[k], rho)
        codes = quantize(r[k][ch], S)
        entries.append(entry_order(ch, codes))
        scales[k] = fold_gate(S, 1.0 if gates is None else float(gates[k]))
    return a16, entries, scales


# ------------------------------------------------------- into the layout
def _pack_pairs(codes: np.ndarray) -> np.ndarray:
    u = (np.asarray(codes, dtype=np.int64) & 0xF).astype(np.uint8)
    return (u[0::2] | (u[1::2] << 4)).astype(np.uint8)


def sequence_of(cu_seqlens, t: int) -> int:
    """Sequence b with cu_seqlens[b] <= t < cu_seqlens[b+1] (non-empty ones)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    return int(np.searchsorted(cu, t, side="right") - 1)


def compress(cache, layer: int, x_k: np.ndarray, x_v: np.ndarray, t0: int, t1: int, gate=None):
    """Write the Eq. 1 factors of packed tokens [t0, t1) of `layer` into the
    cache arrays (in place), for every KV head and both Z.

    x_k, x_v: fp16 [t1-t0][Hkv][d] dense keys / values of those tokens.
    gate: None (g = 1) or float32 [2][Hkv][t1-t0].
    The routed ranks and offsets of the tokens (rank_code, res_off of the
    layer's window) must already be in the cache.  Coefficients go to coef_k
    (row-major) and coef_v (16-token blocks, token fastest), fp16 rows or, for
    an int8 cache, codes with their block scales in coef_scale_k / _v
    ([L][Hkv][r_b/16][T]); entries to res_idx / res_val at the token's
    offsets; the folded scale to res_scale."""
    m = window_of(layer, cache.window)
    levels = np.asarray(cache.levels, dtype=np.int64)
    Hk = cache.n_kv_heads
    n = t1 - t0
    if n <= 0:
        return cache
    seq = np.array([sequence_of(cache.cu_seqlens, t) for t in range(t0, t1)])
    for z, X in ((0, x_k), (1, x_v)):
        X = np.asarray(X, dtype=np.float16)
        for h in range(Hk):
            for b in np.unique(seq):
                ks = np.nonzero(seq == b)[0]
                toks = t0 + ks
                B = cache.basis[b, m, h, z]
                rhos = levels[cache.rank_code[m, h, toks]]
                g = None if gate is None else np.asarray(gate, np.float32)[z, h, ks]
                c8 = getattr(cache, "coef_format", "f16") == "int8"
                coef, entries, scales = compress_vectors(X[ks, h], B, rhos, g, "int8" if c8 else "f16")
                for j, t in enumerate(toks):
                    if c8:
                        store_coefficients(cache, layer, z, h, int(t), coef[0][j])
                        (cache.coef_scale_k if z == 0 else cache.coef_scale_v)[layer, h, :, t] = coef[1][j]
                    else:
                        store_coefficients(cache, layer, z, h, int(t), coef[j])
                    cache.res_scale[layer, z, h, t] = scales[j]
                    store_entries(cache, layer, z, h, int(t), *entries[j])
    return cache


def store_coefficients(cache, layer: int, z: int, h: int, t: int, row) -> None:
    """Keys row-major [T][r_b]; values in 16-token blocks, token index fastest."""
    if z == 0:
        cache.coef_k[layer, h, t] = row
    else:
        cache.coef_v[layer, h, t // 16, :, t % 16] = row


def store_entries(cache, layer: int, z: int, h: int, t: int, chans, codes) -> None:
    """Entries of token t at [res_off[t], res_off[t+1]) of the window's table:
    channel bytes, and int4 codes two per byte, low nibble first."""
    m = window_of(layer, cache.window)
    e0 = int(cache.res_off[m, h, t])
    if int(cache.res_off[m, h, t + 1]) - e0 != len(chans):
        raise ValueError("residual offsets disagree with the routed rank")
    cache.res_idx[layer, z, h, e0:e0 + len(chans)] = chans
    if len(chans):
        if e0 % 2 or len(chans) % 2:
            raise ValueError("token entries must fill whole bytes")
        cache.res_val[layer, z, h, e0 // 2:(e0 + len(chans)) // 2] = _pack_pairs(codes)
