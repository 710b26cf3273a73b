"""Plain float64 reference for decode attention over the cross-depth factorized cache.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports or calls this module;
only the tests, the smoke check and the benchmark's CPU-baseline leg may.

What it computes, following the paper's Method section (Sec. 3):

* Eq. 1: the key or value of token t at layer l (window m = the depth window
  holding l) and head h is rebuilt explicitly as
      X_hat = A^Z_{l,h,t} B^Z_{m,h} + g^Z_{l,h,t} R^Z_{l,h,t},   Z in {K, V},
  with A the token's coefficient row, B the window's shared basis (r_b x d),
  and R the token's residual holding the routed number of channels.  The
  storage keeps, per routed channel, its index and a 4-bit two's-complement
  code, and one per-token scale with the gate folded in (g * s), so
  g R = scale * code at each stored channel and 0 elsewhere.
* The decode query then attends to all cached tokens of its sequence with
  plain softmax attention (the fused kernel in Sec. 3 feeds the rebuilt
  fragments straight into the score and value product; this module
  materialises them instead).
* Eq. 3: the probe error e = ||Attn(Q,K,V) - Attn(Q,K_hat,V_hat)||_2 /
  (||Attn(Q,K,V)||_2 + eps), with (K,V) the higher-fidelity reference cache.
  The probe may evaluate several recent query positions; then the norms run
  over those positions and d together, and the query j steps back attends to
  the first T_b - j tokens of its sequence (the prefix its position saw), in
  the current cache.

Readings where the paper is silent (each listed in the design notes):
depth windows are contiguous non-overlapping groups (m = l // w); the routed
rank is shared by the layers of a window and by K and V; query head hq reads
KV head hq // (Hq/Hkv); keys are stored post-positional-encoding, so no
transform is applied; the softmax scale defaults to 1/sqrt(d); an empty
context yields a zero output.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------- encodings
def int4_from_nibble(nib):
    """4-bit two's complement: nibble 0..7 -> 0..7, 8..15 -> -8..-1."""
    nib = np.asarray(nib, dtype=np.int64)
    return np.where(nib >= 8, nib - 16, nib)


def entry_codes(val_bytes: np.ndarray, start: int, count: int) -> np.ndarray:
    """Signed codes of entries [start, start+count) of one packed slab:
    entry e sits in byte e // 2, low nibble when e is even."""
    e = np.arange(start, start + count, dtype=np.int64)
    byte = val_bytes[e // 2].astype(np.int64)
    nib = np.where(e % 2 == 0, byte & 0xF, byte >> 4)
    return int4_from_nibble(nib)


def q_to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def coefficient_rows(cache, layer: int, z: int, h: int, t0: int, t1: int) -> np.ndarray:
    """Coefficient rows A^Z_{l,h,t} of packed tokens [t0, t1) as [t1-t0, r_b] float64.

    Keys are stored row-major [T][r_b]; values in 16-token blocks with the token
    index fastest ([T16/16][r_b][16]): row t of the values is column t % 16 of
    block t // 16.  In the 8-bit blockwise form (Sec. 3 stores coefficients
    8-bit blockwise quantized) the stored entries are int8 codes and
    A_{t,i} = code_{t,i} * scale[i // 16][t], one fp16 scale per token and
    block of 16 coefficients."""
    if z == 0:
        rows = cache.coef_k[layer, h, t0:t1].astype(np.float64)
    else:
        blocks = cache.coef_v[layer, h]                                 # [NB, r_b, 16]
        rows = np.swapaxes(blocks, 1, 2).reshape(-1, blocks.shape[1])   # [NB*16, r_b]
        rows = rows[t0:t1].astype(np.float64)
    if getattr(cache, "coef_format", "f16") == "int8":
        sc = (cache.coef_scale_k if z == 0 else cache.coef_scale_v)[layer, h, :, t0:t1]   # [r_b/16, n]
        rows = rows * np.repeat(sc.astype(np.float64).T, 16, axis=1)
    return rows


def window_of(layer: int, window: int) -> int:
    return layer // window


def kv_head_of(hq: int, n_q_heads: int, n_kv_heads: int) -> int:
    return hq // (n_q_heads // n_kv_heads)


# ------------------------------------------------------------ Eq. 1 rebuild
def reconstruct(cache, layer: int, z: int, h: int, b: int) -> np.ndarray:
    """Explicit Eq. 1 for every token of sequence b: returns [T_b, d] float64."""
    m = window_of(layer, cache.window)
    t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
    A = coefficient_rows(cache, layer, z, h, t0, t1)                # [T_b, r_b]
    Bz = cache.basis[b, m, h, z].astype(np.float64)                 # [r_b, d]
    X = A @ Bz                                                      # shared-basis term
    off = cache.res_off[m, h].astype(np.int64)
    rho = off[t0 + 1:t1 + 1] - off[t0:t1]
    lev = np.asarray(cache.levels, dtype=np.int64)[cache.rank_code[m, h, t0:t1]]
    if not np.array_equal(rho, lev):
        raise ValueError("residual offsets disagree with the routed rank codes")
    e0, e1 = int(off[t0]), int(off[t1])
    tok = np.repeat(np.arange(t1 - t0), rho)                        # token of each entry
    chan = cache.res_idx[layer, z, h, e0:e1].astype(np.int64)
    code = entry_codes(cache.res_val[layer, z, h], e0, e1 - e0)
    if np.any(code == -8):
        raise ValueError("int4 code -8 is not a valid residual code")
    gs = cache.res_scale[layer, z, h, t0:t1].astype(np.float64)     # gate * scale
    R = np.zeros_like(X)
    R[tok, chan] = code                                             # channels distinct per token
    return X + gs[:, None] * R


# -------------------------------------------------------------- attention
def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, sm_scale: float):
    """Softmax attention of query rows q [G, d] over K, V [T, d] (float64).
    Returns (out [G, d], probabilities [G, T])."""
    if K.shape[0] == 0:
        return np.zeros((q.shape[0], V.shape[1])), np.zeros((q.shape[0], 0))
    s = sm_scale * (q @ K.T)
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    p = w / w.sum(axis=1, keepdims=True)
    return p @ V, p


def default_scale(d: int) -> float:
    return 1.0 / np.sqrt(d)


def decode(cache, layer: int, q: np.ndarray | None = None, sm_scale: float | None = None,
           heads=None, with_probs: bool = False):
    """Per-layer decode attention output [B, Hq, d] (float64).

    q defaults to the cache's stored query of that layer.  ``heads`` restricts
    the work to a list of (b, kv_head) pairs (others stay zero)."""
    B, Hq, Hk, d = cache.batch, cache.n_q_heads, cache.n_kv_heads, cache.head_dim
    G = Hq // Hk
    if q is None:
        q = q_to_f64(cache.q_bits[layer], cache.q_dtype)
    scale = default_scale(d) if sm_scale is None or sm_scale <= 0 else sm_scale
    out = np.zeros((B, Hq, d))
    probs = {}
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hk)]
    for b, h in pairs:
        K = reconstruct(cache, layer, 0, h, b)
        V = reconstruct(cache, layer, 1, h, b)
        hq = [x for x in range(Hq) if kv_head_of(x, Hq, Hk) == h]
        o, p = attention(q[b, hq], K, V, scale)
        out[b, hq] = o
        if with_probs:
            probs[(b, h)] = p
    return (out, probs) if with_probs else out


# ------------------------------------------------------------------ Eq. 3
def probe_error(o_ref: np.ndarray, o: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """Eq. 3 per query row: ||o_ref - o||_2 / (||o_ref||_2 + eps)."""
    o_ref = np.asarray(o_ref, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    return np.linalg.norm(o_ref - o, axis=-1) / (np.linalg.norm(o_ref, axis=-1) + eps)


def probe(cache, layer: int, kv_heads, k_ref: np.ndarray, v_ref: np.ndarray,
          q: np.ndarray | None = None, sm_scale: float | None = None, eps: float = 1e-6):
    """Eq. 3 for the probed KV heads: attention over the dense reference cache
    k_ref/v_ref [n_probe, T, d] against attention over the rebuilt cache.
    Returns err [B, n_probe * G] (probed head i, group member g at i*G+g)."""
    B, Hq, Hk, d = cache.batch, cache.n_q_heads, cache.n_kv_heads, cache.head_dim
    G = Hq // Hk
    if q is None:
        q = q_to_f64(cache.q_bits[layer], cache.q_dtype)
    scale = default_scale(d) if sm_scale is None or sm_scale <= 0 else sm_scale
    err = np.zeros((B, len(kv_heads) * G))
    for i, h in enumerate(kv_heads):
        for b in range(B):
            t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
            qq = q[b, h * G:(h + 1) * G]
            o_ref, _ = attention(qq, k_ref[i, t0:t1].astype(np.float64),
                                 v_ref[i, t0:t1].astype(np.float64), scale)
            o, _ = attention(qq, reconstruct(cache, layer, 0, h, b),
                             reconstruct(cache, layer, 1, h, b), scale)
            err[b, i * G:(i + 1) * G] = probe_error(o_ref, o, eps)
    return err


def probe_positions(cache, layer: int, kv_heads, k_ref: np.ndarray, v_ref: np.ndarray, qs: np.ndarray,
                    sm_scale: float | None = None, eps: float = 1e-6):
    """Eq. 3 over several recent query positions.  qs [P][B][Hq][d]: the
    queries of the last P decode positions of every sequence, j = 0 the
    current one.  The query j steps back attends to the tokens its position
    could see, the first T_b - j of the sequence (none when T_b <= j).  Per
    sequence and probed query head, with O_j and O_ref_j the outputs over the
    rebuilt and the reference cache,
        e = sqrt(sum_j ||O_ref_j - O_j||^2) / (sqrt(sum_j ||O_ref_j||^2) + eps),
    the 2-norm taken over the positions and d together.
    Returns err [B, n_probe * G]."""
    B, Hq, Hk, d = cache.batch, cache.n_q_heads, cache.n_kv_heads, cache.head_dim
    G = Hq // Hk
    scale = default_scale(d) if sm_scale is None or sm_scale <= 0 else sm_scale
    qs = np.asarray(qs, dtype=np.float64)
    err = np.zeros((B, len(kv_heads) * G))
    for i, h in enumerate(kv_heads):
        for b in range(B):
            t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
            K = reconstruct(cache, layer, 0, h, b)
            V = reconstruct(cache, layer, 1, h, b)
            d2 = np.zeros(G)
            r2 = np.zeros(G)
            for j in range(qs.shape[0]):
                n = max(t1 - t0 - j, 0)
                qq = qs[j, b, h * G:(h + 1) * G]
                o_ref, _ = attention(qq, k_ref[i, t0:t0 + n].astype(np.float64),
                                     v_ref[i, t0:t0 + n].astype(np.float64), scale)
                o, _ = attention(qq, K[:n], V[:n], scale)
                d2 += ((o_ref - o) ** 2).sum(axis=-1)
                r2 += (o_ref ** 2).sum(axis=-1)
            err[b, i * G:(i + 1) * G] = np.sqrt(d2) / (np.sqrt(r2) + eps)
    return err


# ------------------------------------------------------- residual decoding
def residual_map(cache, layer: int, z: int, h: int, t0: int, t1: int) -> np.ndarray:
    """Dense g*R rows for packed tokens [t0, t1) of slab (layer, z, h): scale*code
    at each routed channel, zero elsewhere ([t1-t0, d] float64)."""
    m = window_of(layer, cache.window)
    d = cache.head_dim
    off = cache.res_off[m, h].astype(np.int64)
    out = np.zeros((t1 - t0, d))
    for t in range(t0, t1):
        e0, e1 = int(off[t]), int(off[t + 1])
        chan = cache.res_idx[layer, z, h, e0:e1].astype(np.int64)
        code = entry_codes(cache.res_val[layer, z, h], e0, e1 - e0)
        out[t - t0, chan] = float(cache.res_scale[layer, z, h, t]) * code
    return out
