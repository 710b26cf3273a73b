"""Pins of the float64 oracle against facts that do not come from the oracle.

Each ``pin_*`` function takes the oracle package (so the mutation test can hand
it a copy with a planted mistake) and returns None on success or a string that
says what disagreed.  The pins are:

* brute force in 40-digit decimal arithmetic with scalar loops on tiny caches;
* closed forms on hand-built caches (one-hot coefficients over permutation
  bases, residual-only caches, a single token, a zero query);
* reductions to library attention (torch CPU float64 scaled_dot_product_attention):
  rank-0 residuals, an identity basis, and a full-rank residual with no basis term;
* invariants: probabilities sum to one, token-permutation invariance, sequence
  independence, the query-head to KV-head grouping;
* Eq. 3 closed forms (e = 0 for an exact reference, e = |1-c|/(|c| + eps/||O||)
  for a value reference scaled by c); over several recent positions, the same
  scaled-reference form with the norm over positions, a last-token change
  seen by the current position only, and the one-position reduction;
* the router score in exact rational arithmetic rounded per operation, Eq. 2 in
  float64 for two levels, infinite thresholds, monotonicity, and offsets by a
  running loop;
* the int4 nibble table in ``tests/golden/int4_nibbles.txt``;
* the append/compress step: signed-permutation bases (exact projection and
  residual), the round-half-even tie table in ``tests/golden/int4_rne_ties.txt``,
  the float32 decision path in exact rational arithmetic, enumeration of the
  kept channels, the 8-bit blockwise encode (exact model, round-half-even
  ties, zero block, half-step bound, rows rebuilt from the cache), float64 error bounds with an orthonormal basis, the rebuilt
  Eq. 1 vectors after writing into the layout, and range routing against a
  running loop;
* the router's attention features: per-sequence masses summing to G, spike
  below mass below G spike, uniform and ln-3 closed forms, the table fold;
  the probe-error feature on a hand-worked case (fresh fold, maximum fold,
  unprobed heads, an empty sequence);
* the probe schedule: a hand-worked rotation table and its period, coverage
  and distinctness invariants;
* threshold control: a hand-worked feedback trace with clamps, the
  budget-driven selection against enumeration of the promoted sets, and
  budget routing of a token range against a running loop (exact scores,
  planted ties, offsets continued from a non-zero start);
* sketch basis: Gram-Schmidt against numpy's QR, the exact row space of a
  rank-r_b prefill, zero rows of a rank-deficient sketch;
* 8-bit blockwise coefficients: a scalar loop over code * block scale, and an
  fp16 twin with power-of-two scales decoding identically.
"""
from __future__ import annotations

import copy
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np

from synth import generate, router_inputs, Workload
from synth.layout import block_values, unblock_values

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ helpers
def small_workload(**kw) -> Workload:
    base = dict(name="pin", batch=2, n_layers=4, window=2, n_kv_heads=2, n_q_heads=4,
                head_dim=16, context=7, basis_rank=4, levels=(0, 2, 4),
                probs=(0.5, 0.3, 0.2), q_dtype="f16", seed=11, ragged=(3, 9))
    base.update(kw)
    return Workload(**base)


def small_cache(**kw):
    return generate(small_workload(**kw), threads=2)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.linalg.norm(b), 1e-300)
    return float(np.linalg.norm(a - b) / den)


def _q64(o, cache, layer):
    return o.q_to_f64(cache.q_bits[layer], cache.q_dtype)


def coef_rows(c, layer, z, h):
    """Logical [T][r_b] coefficient rows (a copy)."""
    if z == 0:
        return c.coef_k[layer, h].copy()
    return unblock_values(c.coef_v[layer, h], c.total_tokens).copy()


def set_coef_rows(c, layer, z, h, rows):
    if z == 0:
        c.coef_k[layer, h] = rows
    else:
        c.coef_v[layer, h] = block_values(np.asarray(rows, dtype=np.float16))


def coef_set(c, layer, z, h, t, i, value):
    if z == 0:
        c.coef_k[layer, h, t, i] = value
    else:
        c.coef_v[layer, h, t // 16, i, t % 16] = value


def coef_get(c, layer, z, h, t, i):
    return c.coef_k[layer, h, t, i] if z == 0 else c.coef_v[layer, h, t // 16, i, t % 16]


def zero_coefs(c, layer=None):
    sl = slice(None) if layer is None else layer
    c.coef_k[sl] = 0
    c.coef_v[sl] = 0


def _pack(codes):
    u = [(int(c) & 0xF) for c in codes]
    if len(u) % 2:
        u.append(0)
    return np.array([u[i] | (u[i + 1] << 4) for i in range(0, len(u), 2)], dtype=np.uint8)


def set_entries(cache, layer, z, h, token, chans, codes):
    """Overwrite the stored entries of one token (its rank must equal len(chans))."""
    m = layer // cache.window
    e0 = int(cache.res_off[m, h, token])
    assert int(cache.res_off[m, h, token + 1]) - e0 == len(chans)
    for j, (c, k) in enumerate(zip(chans, codes)):
        e = e0 + j
        cache.res_idx[layer, z, h, e] = c
        byte = int(cache.res_val[layer, z, h, e // 2])
        nib = int(k) & 0xF
        byte = (byte & 0xF0) | nib if e % 2 == 0 else (byte & 0x0F) | (nib << 4)
        cache.res_val[layer, z, h, e // 2] = byte


# ------------------------------------------------------- 40-digit brute force
def _nibble_value(byte, high):
    n = (byte >> 4) & 0xF if high else byte & 0xF
    return n - 16 if n & 0x8 else n


def brute_force_decode(cache, layer, b, hq, scale):
    """Scalar-loop Eq. 1 + softmax attention in 40-digit decimal arithmetic."""
    getcontext().prec = 40
    d, rb = cache.head_dim, cache.basis_rank
    G = cache.n_q_heads // cache.n_kv_heads
    h = hq // G
    m = layer // cache.window
    t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
    qd = [Decimal(float(v)) for v in _qvals(cache, layer, b, hq)]
    rows = {}
    for z in (0, 1):
        basis = cache.basis[b, m, h, z]
        rows[z] = []
        for t in range(t0, t1):
            x = [Decimal(0)] * d
            for c in range(d):
                acc = Decimal(0)
                for i in range(rb):
                    acc += Decimal(float(coef_get(cache, layer, z, h, t, i))) * Decimal(float(basis[i, c]))
                x[c] = acc
            e = int(cache.res_off[m, h, t])
            while e < int(cache.res_off[m, h, t + 1]):
                byte = int(cache.res_val[layer, z, h, e >> 1])
                code = _nibble_value(byte, e & 1)
                c = int(cache.res_idx[layer, z, h, e])
                x[c] += Decimal(float(cache.res_scale[layer, z, h, t])) * Decimal(code)
                e += 1
            rows[z].append(x)
    if t1 == t0:
        return [0.0] * d
    sc = Decimal(scale)
    s = [sc * sum(qd[c] * k[c] for c in range(d)) for k in rows[0]]
    mx = max(s)
    w = [(v - mx).exp() for v in s]
    tot = sum(w)
    return [float(sum(w[i] * rows[1][i][c] for i in range(len(w))) / tot) for c in range(d)]


def _qvals(cache, layer, b, hq):
    bits = int(0)
    out = []
    for v in cache.q_bits[layer, b, hq]:
        v = int(v)
        if cache.q_dtype == "f16":
            out.append(float(np.array([v], dtype=np.uint16).view(np.float16)[0]))
        else:
            out.append(float(np.array([v << 16], dtype=np.uint32).view(np.float32)[0]))
    return out


def pin_brute_force(o):
    cache = small_cache(head_dim=8, basis_rank=3, context=4, ragged=(0, 4), levels=(0, 2, 4),
                        probs=(0.3, 0.4, 0.3), batch=3, n_q_heads=4, n_kv_heads=2)
    scale = 0.37
    for layer in (1, 2):
        got = o.decode(cache, layer, sm_scale=scale)
        for b in range(cache.batch):
            for hq in range(cache.n_q_heads):
                ref = brute_force_decode(cache, layer, b, hq, scale)
                if np.linalg.norm(ref) == 0:
                    if np.abs(got[b, hq]).max() != 0:
                        return f"empty sequence b={b} should give zeros"
                    continue
                if _rel(got[b, hq], ref) > 1e-13:
                    return f"brute force mismatch layer={layer} b={b} hq={hq}: {_rel(got[b, hq], ref):.3e}"
    return None


# -------------------------------------------------------------- closed forms
def _perm_basis(cache, seed):
    """Replace every basis by one-hot rows e_{pi(i)} (a non-involutive permutation
    per (b, m, h, z)); returns the permutations."""
    rng = np.random.default_rng(seed)
    B, M, Hk = cache.basis.shape[:3]
    rb, d = cache.basis_rank, cache.head_dim
    perms = {}
    for b in range(B):
        for m in range(M):
            for h in range(Hk):
                for z in range(2):
                    p = rng.permutation(d)[:rb]
                    cache.basis[b, m, h, z] = 0
                    cache.basis[b, m, h, z, np.arange(rb), p] = 1
                    perms[(b, m, h, z)] = p
    return perms


def pin_closed_forms(o):
    # (1) zero residual rank, one-hot coefficients, permutation bases: V_hat_t is a
    # basis row; q = 0 gives the plain mean of the selected rows.
    c = small_cache(levels=(0,), probs=(1.0,), head_dim=16, basis_rank=5)
    perms = _perm_basis(c, 3)
    rng = np.random.default_rng(4)
    layer = 3
    m = layer // c.window
    Hq, Hk = c.n_q_heads, c.n_kv_heads
    G = Hq // Hk
    zero_coefs(c, layer)
    sel = rng.integers(0, c.basis_rank, size=(2, Hk, c.total_tokens))
    for z in range(2):
        for h in range(Hk):
            rows = np.zeros((c.total_tokens, c.basis_rank), np.float16)
            rows[np.arange(c.total_tokens), sel[z, h]] = 1
            set_coef_rows(c, layer, z, h, rows)
    q0 = np.zeros((c.batch, Hq, c.head_dim))
    out = o.decode(c, layer, q=q0)
    for b in range(c.batch):
        t0, t1 = int(c.cu_seqlens[b]), int(c.cu_seqlens[b + 1])
        for hq in range(Hq):
            h = hq // G
            exp = np.zeros(c.head_dim)
            for t in range(t0, t1):
                exp[perms[(b, m, h, 1)][sel[1, h, t]]] += 1.0 / (t1 - t0)
            if np.abs(out[b, hq] - exp).max() > 1e-15:
                return f"q=0 mean of one-hot value rows wrong at b={b} hq={hq}"
    # (2) two tokens, keys one-hot along a basis row, query along the same output
    # channel: scores differ by exactly ln 3, so p = (1/4, 3/4).
    c = small_cache(levels=(0,), probs=(1.0,), head_dim=16, basis_rank=5, batch=1,
                    ragged=None, context=2)
    perms = _perm_basis(c, 5)
    layer = 2
    m = layer // c.window
    zero_coefs(c, layer)
    for h in range(Hk):
        coef_set(c, layer, 0, h, 1, 2, 2.0)              # K_hat_1 = 2 e_{pi_K(2)}, K_hat_0 = 0
        coef_set(c, layer, 1, h, 0, 0, 1.0)              # V_hat_0 = e_{pi_V(0)}
        coef_set(c, layer, 1, h, 1, 1, -4.0)             # V_hat_1 = -4 e_{pi_V(1)}
    q = np.zeros((1, Hq, c.head_dim))
    for hq in range(Hq):
        h = hq // G
        q[0, hq, perms[(0, m, h, 0)][2]] = math.log(3.0) / 2.0
    out = o.decode(c, layer, q=q, sm_scale=1.0)
    for hq in range(Hq):
        h = hq // G
        exp = np.zeros(c.head_dim)
        exp[perms[(0, m, h, 1)][0]] += 0.25
        exp[perms[(0, m, h, 1)][1]] += 0.75 * -4.0
        if np.abs(out[0, hq] - exp).max() > 1e-14:
            return f"two-token ln3 closed form wrong at hq={hq}: {out[0, hq]} vs {exp}"
    # (3) single token: output is that token's rebuilt value row, here a basis row
    # plus one residual entry s*k at a chosen channel.
    c = small_cache(levels=(2,), probs=(1.0,), head_dim=16, basis_rank=4, batch=1,
                    ragged=None, context=1)
    perms = _perm_basis(c, 7)
    layer = 1
    m = 0
    zero_coefs(c, layer)
    for h in range(Hk):
        coef_set(c, layer, 1, h, 0, 3, 1.0)
        set_entries(c, layer, 1, h, 0, [5, 11], [-7, 3])
        c.res_scale[layer, 1, h, 0] = np.float16(0.0625)
    out = o.decode(c, layer)
    for hq in range(Hq):
        h = hq // G
        exp = np.zeros(c.head_dim)
        exp[perms[(0, m, h, 1)][3]] += 1.0
        exp[5] += 0.0625 * -7
        exp[11] += 0.0625 * 3
        if np.abs(out[0, hq] - exp).max() > 1e-15:
            return f"single-token output is not V_hat_0 at hq={hq}"
    # (4) residual-only keys: A^K = 0, one K entry per token -> score s*k*q[c].
    c = small_cache(levels=(2,), probs=(1.0,), head_dim=16, basis_rank=4, batch=1,
                    ragged=None, context=2)
    layer = 0
    zero_coefs(c, layer)
    for h in range(Hk):
        set_entries(c, layer, 0, h, 0, [1, 9], [2, 0])      # K_hat_0 = 2 s0 e_1
        set_entries(c, layer, 0, h, 1, [4, 9], [-1, 0])     # K_hat_1 = -s1 e_4
        c.res_scale[layer, 0, h, 0] = np.float16(0.5)
        c.res_scale[layer, 0, h, 1] = np.float16(0.25)
        coef_set(c, layer, 1, h, 0, 0, 1.0)
        coef_set(c, layer, 1, h, 1, 0, 0.0)
        set_entries(c, layer, 1, h, 0, [0, 1], [0, 0])
        set_entries(c, layer, 1, h, 1, [0, 1], [0, 0])
    q = np.zeros((1, Hq, c.head_dim))
    q[0, :, 1] = 3.0
    q[0, :, 4] = 2.0
    out = o.decode(c, layer, q=q, sm_scale=0.5)
    # s0 = 0.5 * (2*0.5*3) = 1.5 ; s1 = 0.5 * (-0.25*2) = -0.25
    p0 = 1.0 / (1.0 + math.exp(-0.25 - 1.5))
    for hq in range(Hq):
        h = hq // G
        vrow = c.basis[0, 0, h, 1, 0].astype(np.float64)
        if np.abs(out[0, hq] - p0 * vrow).max() > 1e-14:
            return f"residual-only key closed form wrong at hq={hq}"
    return None


# ------------------------------------------------ reductions to library attention
def _sdpa(q, K, V, scale):
    import torch
    qt = torch.tensor(q, dtype=torch.float64)[None, None]
    kt = torch.tensor(K, dtype=torch.float64)[None, None]
    vt = torch.tensor(V, dtype=torch.float64)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)[0, 0].numpy()


def pin_reductions(o):
    # R0: rank-0 residuals: K = A^K B^K, V = A^V B^V built here with torch matmul
    import torch
    c = small_cache(levels=(0,), probs=(1.0,), head_dim=32, basis_rank=8, context=40,
                    ragged=(20, 60), n_layers=6, window=3, n_kv_heads=3, n_q_heads=6)
    scale = 0.2
    for layer in (0, 4, 5):
        out = o.decode(c, layer, sm_scale=scale)
        m = layer // 3
        for b in range(c.batch):
            t0, t1 = int(c.cu_seqlens[b]), int(c.cu_seqlens[b + 1])
            for hq in range(c.n_q_heads):
                h = hq // 2
                K = torch.tensor(coef_rows(c, layer, 0, h)[t0:t1].astype(np.float64)) @ \
                    torch.tensor(c.basis[b, m, h, 0].astype(np.float64))
                V = torch.tensor(coef_rows(c, layer, 1, h)[t0:t1].astype(np.float64)) @ \
                    torch.tensor(c.basis[b, m, h, 1].astype(np.float64))
                ref = _sdpa(_q64(o, c, layer)[b, hq][None], K.numpy(), V.numpy(), scale)[0]
                if _rel(out[b, hq], ref) > 1e-12:
                    return f"R0 mismatch layer={layer} b={b} hq={hq}"
    # R1: identity basis (r_b = d): attention over the raw fp16 coefficient rows
    c = small_cache(levels=(0,), probs=(1.0,), head_dim=16, basis_rank=16, context=30,
                    ragged=None, batch=1)
    c.basis[:] = np.eye(16, dtype=np.float16)
    for layer in range(c.n_layers):
        out = o.decode(c, layer)
        for hq in range(c.n_q_heads):
            h = hq // 2
            ref = _sdpa(_q64(o, c, layer)[0, hq][None], coef_rows(c, layer, 0, h).astype(np.float64),
                        coef_rows(c, layer, 1, h).astype(np.float64), 0.25)[0]
            if _rel(out[0, hq], ref) > 1e-12:
                return f"R1 mismatch layer={layer} hq={hq}"
    # R2: full-rank residual (every channel), no basis term: attention over the
    # dequantised dense int4 cache, built here entry by entry.
    c = small_cache(levels=(16,), probs=(1.0,), head_dim=16, basis_rank=4, context=25,
                    ragged=None, batch=1)
    zero_coefs(c)
    for layer in range(c.n_layers):
        out = o.decode(c, layer)
        m = layer // c.window
        for hq in range(c.n_q_heads):
            h = hq // 2
            dense = {0: np.zeros((25, 16)), 1: np.zeros((25, 16))}
            for z in (0, 1):
                for t in range(25):
                    for e in range(int(c.res_off[m, h, t]), int(c.res_off[m, h, t + 1])):
                        byte = int(c.res_val[layer, z, h, e >> 1])
                        dense[z][t, int(c.res_idx[layer, z, h, e])] = \
                            float(c.res_scale[layer, z, h, t]) * _nibble_value(byte, e & 1)
            ref = _sdpa(_q64(o, c, layer)[0, hq][None], dense[0], dense[1], 0.25)[0]
            if _rel(out[0, hq], ref) > 1e-12:
                return f"R2 mismatch layer={layer} hq={hq}"
    return None


# ---------------------------------------------------------------- invariants
def pin_invariants(o):
    c = small_cache(head_dim=16, basis_rank=6, context=50, ragged=(30, 70),
                    levels=(0, 2, 4, 8), probs=(0.4, 0.3, 0.2, 0.1))
    layer = 3
    out, probs = o.decode(c, layer, with_probs=True)
    for key, p in probs.items():
        if p.size and (np.abs(p.sum(axis=1) - 1).max() > 1e-12 or p.min() < 0):
            return f"probabilities of {key} do not sum to one"
    # token permutation within sequence 1 (with metadata and rebuilt offsets)
    c2 = permute_tokens(c, b=1, seed=9)
    out2 = o.decode(c2, layer)
    if np.abs(out2 - out).max() > 1e-13 * max(1.0, np.abs(out).max()):
        return "output changed under token permutation"
    # another sequence's data does not leak
    c3 = copy.deepcopy(c)
    t0, t1 = int(c.cu_seqlens[0]), int(c.cu_seqlens[1])
    for layer in range(c3.n_layers):
        for z in range(2):
            for h in range(c3.n_kv_heads):
                rows = coef_rows(c3, layer, z, h)
                rows[t0:t1] = -rows[t0:t1]
                set_coef_rows(c3, layer, z, h, rows)
    out3 = o.decode(c3, layer)
    if np.abs(out3[1:] - out[1:]).max() != 0:
        return "sequence 0's data changed another sequence's output"
    # query-head grouping: each group member matches a one-head attention
    G = c.n_q_heads // c.n_kv_heads
    for hq in range(c.n_q_heads):
        h = hq // G
        for b in range(c.batch):
            K = o.reconstruct(c, layer, 0, h, b)
            V = o.reconstruct(c, layer, 1, h, b)
            ref = _sdpa(_q64(o, c, layer)[b, hq][None], K, V, 0.25)[0]
            if _rel(out[b, hq], ref) > 1e-12:
                return f"query head {hq} does not read KV head {h}"
    return None


def permute_tokens(cache, b, seed):
    """Copy of ``cache`` with sequence b's tokens permuted, carrying every
    per-token field and residual entry and rebuilding the offsets."""
    c = copy.deepcopy(cache)
    rng = np.random.default_rng(seed)
    t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
    perm = t0 + rng.permutation(t1 - t0)
    M, Hk = cache.rank_code.shape[:2]
    levels = np.asarray(cache.levels)
    for m in range(M):
        for h in range(Hk):
            c.rank_code[m, h, t0:t1] = cache.rank_code[m, h, perm]
            c.res_off[m, h, 1:] = np.cumsum(levels[c.rank_code[m, h]])
    for layer in range(cache.n_layers):
        m = layer // cache.window
        for z in range(2):
            for h in range(Hk):
                rows = coef_rows(cache, layer, z, h)
                rows[t0:t1] = rows[perm]
                set_coef_rows(c, layer, z, h, rows)
                c.res_scale[layer, z, h, t0:t1] = cache.res_scale[layer, z, h, perm]
                # gather entries token by token in the new order
                idx, codes = [], []
                for t in range(cache.total_tokens):
                    src = perm[t - t0] if t0 <= t < t1 else t
                    for e in range(int(cache.res_off[m, h, src]), int(cache.res_off[m, h, src + 1])):
                        idx.append(int(cache.res_idx[layer, z, h, e]))
                        byte = int(cache.res_val[layer, z, h, e >> 1])
                        codes.append(_nibble_value(byte, e & 1))
                c.res_idx[layer, z, h, :len(idx)] = idx
                pk = _pack(codes)
                c.res_val[layer, z, h, :pk.size] = pk
    return c


# ----------------------------------------------------------------- Eq. 3 probe
def pin_probe(o):
    # reference rows exactly representable in fp16: small-integer coefficients
    # over one-hot bases, fp16-exact residuals.
    c = small_cache(head_dim=16, basis_rank=4, context=20, ragged=None, batch=2,
                    levels=(0, 2), probs=(0.5, 0.5))
    _perm_basis(c, 13)
    rng = np.random.default_rng(14)
    c.coef_k[:] = rng.integers(-3, 4, size=c.coef_k.shape).astype(np.float16)
    c.coef_v[:] = rng.integers(-3, 4, size=c.coef_v.shape).astype(np.float16)
    c.res_scale[:] = np.float16(0.5)
    layer = 2
    heads = [1, 0]
    K = np.stack([np.concatenate([o.reconstruct(c, layer, 0, h, b) for b in range(c.batch)]) for h in heads])
    V = np.stack([np.concatenate([o.reconstruct(c, layer, 1, h, b) for b in range(c.batch)]) for h in heads])
    if not np.array_equal(K.astype(np.float16).astype(np.float64), K):
        return "probe test setup: reference not fp16-exact"
    e = o.probe(c, layer, heads, K.astype(np.float16), V.astype(np.float16))
    if np.abs(e).max() != 0:
        return "Eq. 3 error is not zero for an exact reference"
    for cval in (2.0, -0.5):
        eps = 1e-6
        e = o.probe(c, layer, heads, K.astype(np.float16), (cval * V).astype(np.float16), eps=eps)
        out = o.decode(c, layer)
        G = c.n_q_heads // c.n_kv_heads
        for i, h in enumerate(heads):
            for g in range(G):
                n = np.linalg.norm(out[:, h * G + g], axis=-1)
                exp = abs(1 - cval) * n / (abs(cval) * n + eps)
                if np.abs(e[:, i * G + g] - exp).max() > 1e-12:
                    return f"Eq. 3 scaled-reference closed form wrong (c={cval})"
    return None


def _probe_pos_setup(o):
    c = small_cache(head_dim=16, basis_rank=4, batch=4, ragged=(0, 7), context=7, seed=28,
                    levels=(0, 2), probs=(0.5, 0.5))
    _perm_basis(c, 29)
    rng = np.random.default_rng(30)
    c.coef_k[:] = rng.integers(-3, 4, size=c.coef_k.shape).astype(np.float16)
    c.coef_v[:] = rng.integers(-3, 4, size=c.coef_v.shape).astype(np.float16)
    c.res_scale[:] = np.float16(0.5)
    layer, heads = 1, [1, 0]
    K = np.stack([np.concatenate([o.reconstruct(c, layer, 0, h, b) for b in range(c.batch)]) for h in heads])
    V = np.stack([np.concatenate([o.reconstruct(c, layer, 1, h, b) for b in range(c.batch)]) for h in heads])
    P = 3
    qs = rng.standard_normal((P, c.batch, c.n_q_heads, c.head_dim)).astype(np.float16).astype(np.float64)
    return c, layer, heads, K, V, qs


def pin_probe_positions(o):
    """Eq. 3 over several recent positions (norm over the positions and d).
    Lengths 0, 6, 1 and 4 with three positions: the query j steps back sees
    the first T_b - j tokens, none when T_b <= j.  Expected values come from
    torch's attention over prefixes of the rebuilt rows."""
    c, layer, heads, K, V, qs = _probe_pos_setup(o)
    if not np.array_equal(V.astype(np.float16).astype(np.float64), V):
        return "probe positions setup: reference not fp16-exact"
    G = c.n_q_heads // c.n_kv_heads
    P = qs.shape[0]
    scale = 1.0 / np.sqrt(c.head_dim)
    cu = c.cu_seqlens
    # one position is the single-position probe
    e1 = o.probe_positions(c, layer, heads, K.astype(np.float16), V.astype(np.float16), qs[:1])
    e0 = o.probe(c, layer, heads, K.astype(np.float16), V.astype(np.float16), q=qs[0])
    if not np.array_equal(e1, e0):
        return "probe over one position differs from the single-position probe"

    def rows(i, b, j, Vm):
        h = heads[i]
        n = max(int(cu[b + 1] - cu[b]) - j, 0)
        t0 = int(cu[b])
        if n == 0:
            return np.zeros((G, c.head_dim))
        return _sdpa(qs[j, b, h * G:(h + 1) * G], K[i, t0:t0 + n], Vm[i, t0:t0 + n], scale)

    # scaled reference values: every position's reference output is cval times
    # the rebuilt one, e = |1 - c| N / (|c| N + eps) with N^2 summed over positions
    eps = 0.5
    for cval in (2.0, -0.5):
        e = o.probe_positions(c, layer, heads, K.astype(np.float16), (cval * V).astype(np.float16), qs, eps=eps)
        for i in range(len(heads)):
            for b in range(c.batch):
                N = np.sqrt(sum((rows(i, b, j, V) ** 2).sum(axis=-1) for j in range(P)))
                want = abs(1 - cval) * N / (abs(cval) * N + eps)
                if np.abs(e[b, i * G:(i + 1) * G] - want).max() > 1e-12:
                    return f"probe positions scaled-reference closed form wrong (c={cval}, b={b}, head {i})"
    # a change to the last token of every sequence is seen by the current
    # position only
    Vr = V.copy()
    last = cu[1:][cu[1:] > cu[:-1]] - 1
    Vr[:, last, :] += 1.0
    e = o.probe_positions(c, layer, heads, K.astype(np.float16), Vr.astype(np.float16), qs, eps=1e-6)
    for i in range(len(heads)):
        for b in range(c.batch):
            d2 = ((rows(i, b, 0, Vr) - rows(i, b, 0, V)) ** 2).sum(axis=-1)
            r2 = (rows(i, b, 0, Vr) ** 2).sum(axis=-1) + sum((rows(i, b, j, V) ** 2).sum(axis=-1) for j in range(1, P))
            want = np.sqrt(d2) / (np.sqrt(r2) + 1e-6)
            if np.abs(e[b, i * G:(i + 1) * G] - want).max() > 1e-12:
                return f"probe positions last-token case wrong (b={b}, head {i}): {e[b, i * G:(i + 1) * G]} vs {want}"
            if cu[b + 1] == cu[b] and np.any(e[b, i * G:(i + 1) * G] != 0):
                return "probe positions: an empty sequence has a non-zero error"
    if not np.any(e > 0):
        return "probe positions last-token case: no error seen"
    return None


# -------------------------------------------------------------------- router
def fp32_round(x: Fraction) -> Fraction:
    """Round an exact rational to the nearest float32, ties to even."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, -126)
    ulp = Fraction(2) ** (e - 23)
    n = a / ulp
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sign * fl * ulp


def exact_score(u, phi):
    z = fp32_round(Fraction(float(u[0])) * Fraction(float(phi[0])))
    for i in (1, 2, 3):
        z = fp32_round(z + fp32_round(Fraction(float(u[i])) * Fraction(float(phi[i]))))
    return z


def pin_router(o):
    w = small_workload(levels=(0, 4, 8, 16), probs=(0.25, 0.25, 0.25, 0.25))
    phi, u, theta = router_inputs(w, n_windows=2, T=300)
    rng = np.random.default_rng(21)
    # per-operation rounded float32 score, checked in exact rational arithmetic
    for m in range(2):
        z = o.router_score(phi[m], u[m])
        for h in range(phi.shape[1]):
            for t in rng.integers(0, 300, size=60):
                if Fraction(float(z[h, t])) != exact_score(u[m], phi[m, h, t]):
                    return f"router score not the per-op rounded float32 sum at m={m} h={h} t={t}"
    # adversarial magnitudes where fused or reordered sums round differently
    u2 = np.array([1.0, 1e-8, -1.0, 3.0], np.float32)
    ph = rng.standard_normal((500, 4)).astype(np.float32) * np.array([1e4, 1.0, 1e4, 1e-3], np.float32)
    z = o.router_score(ph, u2)
    for t in range(500):
        if Fraction(float(z[t])) != exact_score(u2, ph[t]):
            return "router score order/rounding differs on cancelling inputs"
    codes, off = o.route(phi, u, theta, w.levels)
    lev = np.asarray(w.levels)
    # offsets by a running loop
    for m in range(2):
        for h in range(phi.shape[1]):
            run = 0
            for t in range(300):
                if int(off[m, h, t]) != run:
                    return "offsets are not the exclusive running sum of ranks"
                run += int(lev[codes[m, h, t]])
            if int(off[m, h, 300]) != run:
                return "final offset is not the total rank"
    # Eq. 2 with two levels, in float64 with the logistic gate, away from ties
    tau = np.array([[0.7], [0.9]])
    th = np.stack([o.theta_from_tau(t) for t in tau])
    c2, _ = o.route(phi, u, th, (2, 8))
    for m in range(2):
        s = phi[m].astype(np.float64) @ u[m].astype(np.float64)
        gate = 1 / (1 + np.exp(-s))
        ref = np.where(gate > tau[m, 0], 1, 0)
        far = np.abs(s - np.log(tau[m, 0] / (1 - tau[m, 0]))) > 1e-4
        if not np.array_equal(c2[m][far], ref[far]):
            return "two-level routing disagrees with Eq. 2"
        if not np.any(ref == 1) or not np.any(ref == 0):
            return "router pin setup does not reach both levels"
    # infinite thresholds
    inf = np.full_like(theta, np.inf)
    c_hi, _ = o.route(phi, u, inf, w.levels)
    c_lo, _ = o.route(phi, u, -inf, w.levels)
    if c_hi.max() != 0 or c_lo.min() != len(w.levels) - 1:
        return "infinite thresholds do not pin the extreme levels"
    # exact ties: Eq. 2 uses a strict inequality, so z == theta keeps the lower level
    ut = np.array([1.0, 0.0, 0.0, 0.0], np.float32)
    pt = np.zeros((1, 1, 4, 4), np.float32)
    pt[0, 0, :, 0] = [0.5, 1.5, 1.5000001, 2.5]
    ct, _ = o.route(pt, ut[None], np.array([[0.5, 1.5, 2.5]], np.float32), (0, 2, 4, 6))
    if [int(x) for x in ct[0, 0]] != [0, 1, 2, 2]:
        return f"ties at the threshold must keep the lower level, got {ct[0, 0]}"
    # monotone in each feature with positive weight
    bump = phi.copy()
    bump[..., 0] += 0.5
    c_b, _ = o.route(bump, u, theta, w.levels)
    if np.any(c_b < codes):
        return "raising a positively weighted feature lowered the level"
    return None


# --------------------------------------------------------- nibble + residual map
def pin_nibbles(o):
    table = []
    with open(os.path.join(GOLDEN, "int4_nibbles.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                a, b = line.split()
                table.append((int(a, 16), int(b)))
    got = o.int4_from_nibble(np.array([a for a, _ in table]))
    if [int(x) for x in got] != [b for _, b in table]:
        return "int4 nibble decoding disagrees with the two's-complement table"
    # byte order: entry e lives in byte e//2, low nibble when e is even
    vb = np.array([0x1F, 0x72], dtype=np.uint8)
    if [int(x) for x in o.entry_codes(vb, 0, 4)] != [-1, 1, 2, 7]:
        return "entry -> (byte, nibble) placement wrong"
    return None


def pin_residual_map(o):
    c = small_cache(levels=(2, 4), probs=(0.5, 0.5), head_dim=16, context=3, ragged=None, batch=1)
    layer, z, h = 1, 1, 0
    set_entries(c, layer, z, h, 1, [3, 0] + ([7, 9] if c.res_off[0, h, 2] - c.res_off[0, h, 1] == 4 else []),
                [-7, 5] + ([1, -1] if c.res_off[0, h, 2] - c.res_off[0, h, 1] == 4 else []))
    c.res_scale[layer, z, h, 1] = np.float16(0.125)
    got = o.residual_map(c, layer, z, h, 1, 2)
    exp = np.zeros((1, 16))
    exp[0, 3], exp[0, 0] = -7 * 0.125, 5 * 0.125
    if c.res_off[0, h, 2] - c.res_off[0, h, 1] == 4:
        exp[0, 7], exp[0, 9] = 0.125, -0.125
    if not np.array_equal(got, exp):
        return "residual map of a hand-set token is wrong"
    return None


def pin_query_formats(o):
    """fp16 / bf16 query bits decode as torch's own dtypes do."""
    import torch
    rng = np.random.default_rng(31)
    bits = rng.integers(0, 2**16, size=4096, dtype=np.uint64).astype(np.uint16)
    bits = bits[(bits & 0x7C00) != 0x7C00]                      # finite fp16 patterns
    ref16 = torch.from_numpy(bits.astype(np.int16)).view(torch.float16).double().numpy()
    if not np.array_equal(o.q_to_f64(bits, "f16"), ref16):
        return "fp16 query decoding differs from torch.float16"
    b2 = bits[(bits & 0x7F80) != 0x7F80]                        # finite bf16 patterns
    ref_bf = torch.from_numpy(b2.astype(np.int16)).view(torch.bfloat16).double().numpy()
    if not np.array_equal(o.q_to_f64(b2, "bf16"), ref_bf):
        return "bf16 query decoding differs from torch.bfloat16"
    return None



# ------------------------------------------------------------ append/compress
def fp16_round(x: Fraction) -> Fraction:
    """Round an exact rational to the nearest float16, ties to even."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, -14)
    ulp = Fraction(2) ** (e - 10)
    n = a / ulp
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sign * fl * ulp


def _expected_entries(r, rho, S):
    """Kept channels by the pairwise definition (every kept channel beats every
    dropped one: larger |r|, or equal |r| and lower channel), codes rounded
    half to even in exact arithmetic from the float32 quotient, storage order
    by descending |code| then channel.  r, S exact rationals."""
    d = len(r)
    beats = lambda a, b: abs(r[a]) > abs(r[b]) or (abs(r[a]) == abs(r[b]) and a < b)
    kept = [c for c in range(d) if sum(1 for c2 in range(d) if beats(c2, c)) < rho]
    assert len(kept) == rho
    codes = {}
    for c in kept:
        q = Fraction(0) if S == 0 else fp32_round(r[c] / S)
        codes[c] = max(-7, min(7, round(q)))           # Fraction rounds half to even
    order = sorted(kept, key=lambda c: (-abs(codes[c]), c))
    return [(c, codes[c]) for c in order]


def _f16(vals):
    return np.asarray(vals, dtype=np.float64).astype(np.float16)


def pin_compress_closed_forms(o):
    """Signed-permutation bases make the projection and residual exact:
    A_i = s_i x_{pi(i)}, r = x off the basis channels and 0 on them."""
    C = o.compress
    rng = np.random.default_rng(41)
    d, r_b = 16, 4
    for trial in range(6):
        perm = rng.permutation(d)
        sgn = rng.choice([-1.0, 1.0], size=r_b)
        B = np.zeros((r_b, d))
        for i in range(r_b):
            B[i, perm[i]] = sgn[i]
        B = _f16(B)
        x = _f16(rng.uniform(0.05, 2.0, size=(3, d)) * rng.choice([-1, 1], size=(3, d)))
        x[1, perm[r_b]] = x[1, perm[r_b + 1]]          # an exact |r| tie
        x[2, perm[r_b + 2]] = -x[2, perm[r_b + 3]]
        gates = np.array([1.0, 0.5, 0.3], np.float32)
        for rho in (0, 2, 6, 12, d):
            a16, entries, scales = C.compress_vectors(x, B, [rho] * 3, gates)
            for k in range(3):
                xs = [Fraction(float(v)) for v in x[k]]
                exp_a = [sgn[i] * xs[perm[i]] for i in range(r_b)]
                if [Fraction(float(v)) for v in a16[k]] != exp_a:
                    return f"projection on a signed permutation basis is not A_i = s_i x_pi(i) (trial {trial})"
                on_basis = set(int(perm[i]) for i in range(r_b))
                rr = [Fraction(0) if c in on_basis else xs[c] for c in range(d)]
                S = fp32_round(max(abs(v) for v in rr) / 7)
                want = _expected_entries(rr, rho, S) if rho else []
                got = [(int(c), int(q)) for c, q in zip(*entries[k])]
                if got != want:
                    return f"kept channels / codes / order wrong (trial {trial}, rho {rho}): {got} vs {want}"
                exp_s = Fraction(0) if rho == 0 else fp16_round(fp32_round(Fraction(float(gates[k])) * S))
                if Fraction(float(scales[k])) != exp_s:
                    return f"stored scale is not fp16(g * max|r| / 7) (trial {trial}, rho {rho})"
    return None


def pin_compress_rne_table(o):
    """Codes at and around rounding ties against tests/golden/int4_rne_ties.txt."""
    C = o.compress
    rows = []
    with open(os.path.join(GOLDEN, "int4_rne_ties.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                v, k = line.split()
                rows.append((float(v), int(k)))
    d, r_b = 32, 2
    B = np.zeros((r_b, d))
    B[0, 0] = B[1, 1] = 1.0                           # identity rows: r = x off channels 0, 1
    S = 2.0 ** -6
    x = np.zeros(d)
    x[0], x[1] = 0.75, -1.25
    for j, (v, _) in enumerate(rows):
        x[2 + j] = v * S
    a16, entries, scales = C.compress_vectors(_f16(x[None]), _f16(B), [d])
    got = dict(zip((int(c) for c in entries[0][0]), (int(q) for q in entries[0][1])))
    for j, (v, k) in enumerate(rows):
        if got.get(2 + j) != k:
            return f"r/S = {v} quantized to {got.get(2 + j)}, expected {k}"
    if float(scales[0]) != S:
        return "scale of the tie table is not max|r| / 7"
    return None


def _exact_ordered_sum(terms):
    """Exact-arithmetic model of a float32 sum left to right: the first term,
    then every next term added with one rounding to float32."""
    acc = terms[0] if terms else Fraction(0)
    for t in terms[1:]:
        acc = fp32_round(acc + t)
    return acc


def _exact_project(x, B):
    """A_i = fp16 of the left-to-right float32 sum of the rounded products x_j B_ij."""
    out = []
    for i in range(B.shape[0]):
        terms = [fp32_round(Fraction(float(x[j])) * Fraction(float(B[i, j]))) for j in range(len(x))]
        out.append(fp16_round(_exact_ordered_sum(terms)))
    return out


def _exact_residual(x, B, a):
    out = []
    for c in range(len(x)):
        terms = [fp32_round(a[i] * Fraction(float(B[i, c]))) for i in range(B.shape[0])]
        out.append(fp32_round(Fraction(float(x[c])) - _exact_ordered_sum(terms)))
    return out


def pin_compress_arithmetic(o):
    """The float32 decision path in exact rational arithmetic, each operation
    rounded, on inputs whose magnitudes span many binades (so a reordered or
    fused sum rounds differently), and the kept set by enumeration on a tiny
    case."""
    from itertools import combinations
    C = o.compress
    rng = np.random.default_rng(43)
    d, r_b = 24, 6
    B = _f16(rng.standard_normal((r_b, d)) * 2.0 ** rng.integers(-6, 3, size=(r_b, d)))
    x = _f16(rng.standard_normal((4, d)) * 2.0 ** rng.integers(-8, 6, size=(4, d)))
    a16 = C.project(x, B)
    r = C.residual(x, B, a16)
    for k in range(4):
        ea = _exact_project(x[k], B)
        if [Fraction(float(v)) for v in a16[k]] != ea:
            return f"projection is not the per-op rounded left-to-right float32 sum (vector {k})"
        er = _exact_residual(x[k], B, ea)
        if [Fraction(float(v)) for v in r[k]] != er:
            return f"residual is not x - (left-to-right float32 basis term) (vector {k})"
        for rho in (2, 8):
            S = fp32_round(max(abs(v) for v in er) / 7)
            want = _expected_entries(er, rho, S)
            _, entries, _ = C.compress_vectors(x[k:k + 1], B, [rho])
            if [(int(c), int(q)) for c, q in zip(*entries[0])] != want:
                return f"entries of vector {k} at rho {rho} differ from the exact computation"
    # cancelling pairs: small terms, then +1024 and -1024, then more small
    # terms, so the float32 running sum absorbs a different set of the small
    # terms in any other order (and a float64 or fused sum keeps them all)
    x2 = _f16(rng.uniform(0.01, 0.02, size=(3, d)) * rng.choice([-1, 1], size=(3, d)))
    B2 = _f16(rng.uniform(0.01, 0.02, size=(r_b, d)) * rng.choice([-1, 1], size=(r_b, d)))
    x2[:, d // 3] = 32.0
    x2[:, 2 * d // 3] = 32.0
    B2[:, d // 3] = 32.0
    B2[:, 2 * d // 3] = -32.0
    B2[0, 2 * d // 3] = 32.0              # one row that does not cancel: large A_0
    a2 = C.project(x2, B2)
    r2 = C.residual(x2, B2, a2)
    for k in range(3):
        ea = _exact_project(x2[k], B2)
        if [Fraction(float(v)) for v in a2[k]] != ea:
            return f"projection of cancelling terms is not the left-to-right float32 sum (vector {k})"
        if [Fraction(float(v)) for v in r2[k]] != _exact_residual(x2[k], B2, ea):
            return f"residual of cancelling terms is not the left-to-right float32 sum (vector {k})"
    # enumeration: on 6 channels with repeated magnitudes, the kept set is the
    # lexicographically first subset (by channel) among those with the largest
    # sorted |r| profile
    rr = np.array([0.5, -0.25, 0.5, 0.125, -0.5, 0.25], np.float32)
    for rho in range(0, 7):
        best = None
        for sub in combinations(range(6), rho):
            prof = sorted((abs(float(rr[c])) for c in sub), reverse=True)
            key = ([-v for v in prof], list(sub))
            if best is None or key < best[0]:
                best = (key, sub)
        got = sorted(int(c) for c in C.select_channels(rr, rho))
        if got != list(best[1]):
            return f"top-{rho} channels {got}, enumeration gives {list(best[1])}"
    return None


def _rne_int(q: Fraction) -> int:
    """Round a rational to the nearest integer, ties to even."""
    fl = q.numerator // q.denominator
    rem = q - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return int(fl)


def pin_compress_int8(o):
    """The 8-bit blockwise encode (reading C7): the whole decision path in
    exact rational arithmetic rounded per operation (float32 projection left
    to right, S = fp16(fp32(max|A| / 127)), code = rne(fp32(A / S)) clamped,
    the residual against code * S); round-half-even ties at an exact scale of
    2^-4; a zero block; the half-step bound; and the rows rebuilt from the
    cache after writing."""
    C = o.compress
    rng = np.random.default_rng(59)
    d, r_b = 32, 32
    B = _f16(rng.standard_normal((r_b, d)) * 2.0 ** rng.integers(-4, 2, size=(r_b, d)))
    x = _f16(rng.standard_normal((3, d)) * 2.0 ** rng.integers(-6, 4, size=(3, d)))
    codes, scales, rows = C.quantize_coefficients(C.project32(x, B))
    for k in range(3):
        a32 = []
        for i in range(r_b):
            terms = [fp32_round(Fraction(float(x[k, j])) * Fraction(float(B[i, j]))) for j in range(d)]
            a32.append(_exact_ordered_sum(terms))
        want_rows = []
        for sblk in range(r_b // 16):
            blk = a32[16 * sblk:16 * sblk + 16]
            S = fp16_round(fp32_round(max(abs(v) for v in blk) / 127))
            if Fraction(float(scales[k, sblk])) != S:
                return f"vector {k} block {sblk}: scale {float(scales[k, sblk])} is not fp16(max|A| / 127)"
            for i, v in enumerate(blk):
                q = 0 if S == 0 else max(-127, min(127, _rne_int(fp32_round(v / S))))
                if int(codes[k, 16 * sblk + i]) != q:
                    return f"vector {k} coefficient {16 * sblk + i}: code {int(codes[k, 16 * sblk + i])}, want {q}"
                want_rows.append(q * S)
        if [Fraction(float(v)) for v in rows[k]] != want_rows:
            return f"vector {k}: rebuilt rows are not code * scale"
        er = _exact_residual(x[k], B, want_rows)
        _, entries, _ = C.compress_vectors(x[k:k + 1], B, [8], coef_format="int8")
        Sr = fp32_round(max(abs(v) for v in er) / 7)
        if [(int(c), int(q)) for c, q in zip(*entries[0])] != _expected_entries(er, 8, Sr):
            return f"vector {k}: residual entries are not taken against code * scale"
    # a vector in the span of an orthonormal basis: its residual is the
    # coefficients' quantization error, so only residuals taken against
    # code * scale give these entries
    qb, _ = np.linalg.qr(rng.standard_normal((32, 16)))
    Bo = _f16(qb.T)
    xo = _f16(rng.standard_normal((2, 16)) @ Bo.astype(np.float64))
    _, _, rows_o = C.quantize_coefficients(C.project32(xo, Bo))
    for k in range(2):
        er = _exact_residual(xo[k], Bo, [Fraction(float(v)) for v in rows_o[k]])
        _, entries, _ = C.compress_vectors(xo[k:k + 1], Bo, [6], coef_format="int8")
        Sr = fp32_round(max(abs(v) for v in er) / 7)
        if [(int(c), int(q)) for c, q in zip(*entries[0])] != _expected_entries(er, 6, Sr):
            return f"in-span vector {k}: residual entries are not taken against code * scale"
    # ties: a signed-permutation basis makes A exact; block 0's largest entry is
    # 127 * 2^-4, so S = 2^-4 and the others sit on half steps
    d2, rb2 = 32, 16
    perm = rng.permutation(d2)
    B2 = np.zeros((rb2, d2))
    for i in range(rb2):
        B2[i, perm[i]] = 1.0 if i % 3 else -1.0
    B2 = _f16(B2)
    vals = [127, 2.5, 3.5, -2.5, -0.5, 126.5, 0.5, 1.5, -1.5, 7.25, -127, 64.5, 0, 3, -3.5, 5.5]
    want = [127, 2, 4, -2, 0, 126, 0, 2, -2, 7, -127, 64, 0, 3, -4, 6]
    x2 = np.zeros((1, d2))
    for i in range(rb2):
        x2[0, perm[i]] = (1.0 if i % 3 else -1.0) * vals[i] * 2.0 ** -4
    c2, s2, _ = C.quantize_coefficients(C.project32(_f16(x2), B2))
    if float(s2[0, 0]) != 2.0 ** -4 or [int(v) for v in c2[0]] != want:
        return f"int8 ties: scale {float(s2[0, 0])}, codes {[int(v) for v in c2[0]]}, want 2^-4 and {want}"
    # a zero block stores scale 0 and codes 0
    c3, s3, r3 = C.quantize_coefficients(np.zeros((2, 32), np.float32))
    if np.any(c3 != 0) or np.any(s3 != 0) or np.any(r3 != 0):
        return "a zero block must store scale 0 and codes 0"
    # the half-step bound on a realistic orthonormal basis
    q, _ = np.linalg.qr(rng.standard_normal((128, 48)))
    B4 = _f16(q.T)
    x4 = _f16(rng.standard_normal((20, 128)))
    a4 = x4.astype(np.float64) @ B4.astype(np.float64).T
    c4, s4, r4 = C.quantize_coefficients(C.project32(x4, B4))
    S4 = np.repeat(s4.astype(np.float64), 16, axis=1)
    if np.any(np.abs(r4 - a4) > S4 * 0.5 * (1 + 2.0 ** -9) + 1e-6):
        return "int8 coefficients off by more than half a step"
    # written into an int8 cache, the rows rebuilt from it are code * scale
    c = small_cache(levels=(0, 2, 4), probs=(0.4, 0.3, 0.3), context=20, ragged=(13, 30), basis_rank=32,
                    head_dim=32, coef_format="int8")
    layer, t0, t1 = 1, 3, 17
    Hk = c.n_kv_heads
    xk = _f16(rng.standard_normal((t1 - t0, Hk, 32)))
    xv = _f16(rng.standard_normal((t1 - t0, Hk, 32)))
    c2c = copy.deepcopy(c)
    C.compress(c2c, layer, xk, xv, t0, t1)
    for z, X in ((0, xk), (1, xv)):
        for h in range(Hk):
            b = C.sequence_of(c.cu_seqlens, t0)
            _, _, want_rows = C.quantize_coefficients(C.project32(X[:int(c.cu_seqlens[b + 1]) - t0, h],
                                                                   c.basis[b, 0, h, z]))
            got = o.factorized.coefficient_rows(c2c, layer, z, h, t0, min(t1, int(c.cu_seqlens[b + 1])))
            if not np.array_equal(got, want_rows.astype(np.float64)):
                return f"int8 rows rebuilt from the cache differ (z={z}, h={h})"
    return None


def pin_compress_bounds(o):
    """With a realistic orthonormal basis (d = 128): A matches the float64
    projection to fp16 rounding, every kept channel is reproduced within
    S/2 (+ rounding), every dropped channel is no larger than any kept one, and
    the stored scale is max|r|/7 to fp16 accuracy."""
    C = o.compress
    rng = np.random.default_rng(47)
    d, r_b = 128, 32
    q, _ = np.linalg.qr(rng.standard_normal((d, r_b)))
    B16 = _f16(q.T)
    B = B16.astype(np.float64)
    x16 = _f16(rng.standard_normal((40, d)))
    x = x16.astype(np.float64)
    rhos = rng.choice([0, 4, 8, 16, 32], size=40)
    a16, entries, scales = C.compress_vectors(x16, B16, rhos)
    a_exact = x @ B.T
    tol_a = np.abs(a_exact) * 2.0 ** -11 + 1e-5
    if np.any(np.abs(a16.astype(np.float64) - a_exact) > tol_a):
        return "coefficients are not the projection x B^T"
    r = x - a16.astype(np.float64) @ B
    for k in range(40):
        ch, codes = entries[k]
        if len(ch) != rhos[k] or len(set(int(c) for c in ch)) != len(ch):
            return f"vector {k}: {len(ch)} distinct channels kept, routed rank {rhos[k]}"
        if rhos[k] == 0:
            if float(scales[k]) != 0.0:
                return "a rank-0 vector must store scale 0"
            continue
        S = np.abs(r[k]).max() / 7
        if abs(float(scales[k]) - S) > S * 2.0 ** -10 + 1e-7:
            return f"vector {k}: stored scale {float(scales[k])} vs max|r|/7 = {S}"
        err = np.abs(r[k, ch] - S * codes)
        if np.any(err > S * (0.5 + 1e-3) + 1e-6):
            return f"vector {k}: a kept channel is off by more than half a step"
        dropped = np.setdiff1d(np.arange(d), ch)
        if dropped.size and np.abs(r[k, dropped]).max() > np.abs(r[k, ch]).min() + 1e-6:
            return f"vector {k}: a dropped channel is larger than a kept one"
        mags = np.abs(codes)
        if np.any(np.diff(mags) > 0) or np.any((np.diff(mags) == 0) & (np.diff(ch) < 0)):
            return f"vector {k}: entries not ordered by |code| then channel"
    return None


def pin_compress_into_cache(o):
    """Writing the factors into the layout: the rebuilt Eq. 1 vectors of the
    compressed tokens approximate the dense inputs within the quantization
    bound, tokens outside the range are untouched, gates scale the residual."""
    C = o.compress
    c = small_cache(levels=(0, 2, 4, 16), probs=(0.25, 0.25, 0.25, 0.25), context=20,
                    ragged=(13, 30), basis_rank=4)
    layer, m = 3, 1
    before = {(z, h, b): o.reconstruct(c, layer, z, h, b)
              for z in range(2) for h in range(c.n_kv_heads) for b in range(c.batch)}
    T, Hk, d = c.total_tokens, c.n_kv_heads, c.head_dim
    t0, t1 = int(c.cu_seqlens[0]) + 5, int(c.cu_seqlens[1]) + 4      # spans both sequences
    rng = np.random.default_rng(53)
    xk = _f16(rng.standard_normal((t1 - t0, Hk, d)))
    xv = _f16(rng.standard_normal((t1 - t0, Hk, d)))
    gate = rng.uniform(0.2, 1.0, size=(2, Hk, t1 - t0)).astype(np.float32)
    c2 = copy.deepcopy(c)
    C.compress(c2, layer, xk, xv, t0, t1, gate)
    lev = np.asarray(c.levels)
    for z, X in ((0, xk), (1, xv)):
        for h in range(Hk):
            for b in range(c.batch):
                s0, s1 = int(c.cu_seqlens[b]), int(c.cu_seqlens[b + 1])
                got = o.reconstruct(c2, layer, z, h, b)
                Bm = c.basis[b, m, h, z].astype(np.float64)
                for t in range(s0, s1):
                    if not (t0 <= t < t1):
                        if not np.array_equal(got[t - s0], before[(z, h, b)][t - s0]):
                            return "a token outside the compressed range changed"
                        continue
                    x = X[t - t0, h].astype(np.float64)
                    a = (x @ Bm.T).astype(np.float16).astype(np.float64)
                    rr = x - a @ Bm
                    rho = lev[c.rank_code[m, h, t]]
                    g = float(gate[z, h, t - t0])
                    kept = np.argsort(-np.abs(rr), kind="stable")[:rho]
                    want = a @ Bm
                    want[kept] += g * rr[kept]
                    S = np.abs(rr).max() / 7
                    if np.abs(got[t - s0] - want).max() > g * S * 0.51 + 2e-3:
                        return f"rebuilt vector of token {t} (z={z}, h={h}) is not A B + g R"
    for l in range(c.n_layers):
        if l == layer:
            continue
        for name in ("coef_k", "coef_v", "res_idx", "res_val", "res_scale"):
            if not np.array_equal(getattr(c2, name)[l], getattr(c, name)[l]):
                return f"{name} of another layer changed"
    return None


def pin_route_range(o):
    """Routing a token range continues the offset table: the result equals a
    running loop over all tokens, and the decode-token append [T-1, T) adds
    exactly one rank."""
    w = small_workload(levels=(0, 4, 8, 16), probs=(0.25, 0.25, 0.25, 0.25))
    phi, u, theta = router_inputs(w, n_windows=2, T=200)
    M, Hk, T = phi.shape[0], phi.shape[1], phi.shape[2]
    lev = np.asarray(w.levels)
    codes = np.zeros((M, Hk, T), np.uint8)
    off = np.full((M, Hk, T + 1), 7, np.uint32)
    for a, b in ((0, 37), (37, 120), (120, 199), (199, 200)):
        o.route_range(phi, u, theta, w.levels, a, b, codes, off)
    for m in range(M):
        for h in range(Hk):
            run = 0
            for t in range(T):
                z = exact_score(u[m], phi[m, h, t])
                k = sum(1 for th in theta[m] if z > Fraction(float(th)))
                if int(codes[m, h, t]) != k:
                    return f"range routing code differs at m={m} h={h} t={t}"
                if int(off[m, h, t]) != run:
                    return f"range routing offsets break at m={m} h={h} t={t}"
                run += int(lev[k])
            if int(off[m, h, T]) != run:
                return "range routing final offset wrong"
    return None


def pin_attention_features(o):
    """Mass and spike of the decode's own probabilities: a sequence's masses sum
    to G (each head's probabilities sum to one), spike <= mass <= G spike; a
    zero query spreads 1/T_b over every token; two tokens whose scores differ
    by ln 3 get 1/4 and 3/4 per head; the table folds sums and maxima."""
    OF = o.features
    c = small_cache(levels=(0, 2, 4), probs=(0.4, 0.3, 0.3), context=9, ragged=(0, 9), batch=4)
    G = c.n_q_heads // c.n_kv_heads
    for layer in range(c.n_layers):
        mass, spike = OF.attention_features(c, layer)
        for b in range(c.batch):
            t0, t1 = int(c.cu_seqlens[b]), int(c.cu_seqlens[b + 1])
            for h in range(c.n_kv_heads):
                if t1 > t0 and abs(mass[h, t0:t1].sum() - G) > 1e-9:
                    return f"masses of sequence {b}, head {h} sum to {mass[h, t0:t1].sum()}, not G = {G}"
                if np.any(spike[h, t0:t1] > mass[h, t0:t1] + 1e-15) or \
                        np.any(mass[h, t0:t1] > G * spike[h, t0:t1] + 1e-12):
                    return "spike and mass out of order"
        q0 = np.zeros((c.batch, c.n_q_heads, c.head_dim))
        mass0, spike0 = OF.attention_features(c, layer, q=q0)
        for b in range(c.batch):
            t0, t1 = int(c.cu_seqlens[b]), int(c.cu_seqlens[b + 1])
            if t1 > t0 and (not np.allclose(mass0[:, t0:t1], G / (t1 - t0), rtol=0, atol=1e-12)
                            or not np.allclose(spike0[:, t0:t1], 1.0 / (t1 - t0), rtol=0, atol=1e-12)):
                return "a zero query must give mass G/T_b and spike 1/T_b"
    # two tokens, one-hot coefficients over a permutation basis: scores 0 and ln 3
    c2 = small_cache(levels=(0,), probs=(1.0,), context=2, ragged=None, batch=1, basis_rank=4)
    zero_coefs(c2)
    for z in range(2):
        c2.basis[0, 0, 0, z] = 0
        c2.basis[0, 0, 0, z, 0, 0] = 1.0
    coef_set(c2, 0, 0, 0, 1, 0, 1.0)
    q = np.zeros((1, c2.n_q_heads, c2.head_dim))
    q[0, :, 0] = np.log(3.0) * np.sqrt(c2.head_dim)
    mass2, spike2 = OF.attention_features(c2, 0, q=q)
    G2 = c2.n_q_heads // c2.n_kv_heads
    if not (np.allclose(mass2[0], [G2 / 4, 3 * G2 / 4], atol=1e-12) and np.allclose(spike2[0], [0.25, 0.75], atol=1e-12)):
        return f"ln 3 score gap must give 1/4, 3/4 per head, got mass {mass2[0]}, spike {spike2[0]}"
    phi = np.zeros((1, 1, 2, 4))
    phi[0, 0, :, 1] = [0.5, 0.1]
    phi[0, 0, :, 2:] = 7.0
    OF.update_features(phi, 0, np.array([[0.2, 0.3]]), np.array([[0.4, 0.2]]))
    OF.update_features(phi, 0, np.array([[0.1, 0.1]]), np.array([[0.1, 0.6]]))
    if not np.allclose(phi[0, 0], [[0.3, 0.5, 7, 7], [0.4, 0.6, 7, 7]]):
        return f"feature table must add masses and keep maxima, got {phi[0, 0]}"
    return None


def pin_probe_feature(o):
    """The probe-error feature on a hand-worked case: two sequences (one empty),
    three KV heads of which two are probed in a different order, G = 2; a fresh
    fold writes each probed head's largest group error on every token of the
    sequence, a second fold keeps the maximum, the unprobed head and columns
    0-2 stay as they were."""
    OF = o.features
    cu = [0, 3, 3, 5]                                  # sequence 1 is empty
    phi = np.full((2, 3, 5, 4), 9.0, np.float32)
    phi[1, :, :, 3] = 0.5
    err = np.array([[0.1, 0.3, 0.2, 0.05],             # b = 0: head 2 -> 0.3, head 0 -> 0.2
                    [0.7, 0.7, 0.7, 0.7],              # b = 1 (empty): nothing to write
                    [0.0, 0.25, 0.6, 0.4]], np.float32)  # b = 2: head 2 -> 0.25, head 0 -> 0.6
    OF.probe_feature(phi, cu, 1, [2, 0], err, 2, True)
    want = np.full((3, 5), 0.5, np.float32)
    want[2, 0:3], want[0, 0:3] = 0.3, 0.2
    want[2, 3:5], want[0, 3:5] = 0.25, 0.6
    if not np.array_equal(phi[1, :, :, 3], want):
        return f"fresh probe feature: got {phi[1, :, :, 3]}, want {want}"
    if not (np.all(phi[:, :, :, :3] == 9.0) and np.all(phi[0, :, :, 3] == 9.0)):
        return "probe feature touched other columns or another window"
    err2 = np.array([[0.35, 0.0, 0.1, 0.1], [0, 0, 0, 0], [0.1, 0.2, 0.9, 0.0]], np.float32)
    OF.probe_feature(phi, cu, 1, [2, 0], err2, 2, False)
    want[2, 0:3] = 0.35                               # max(0.3, 0.35)
    want[0, 3:5] = 0.9                                # max(0.6, 0.9); the rest keep the larger earlier value
    if not np.array_equal(phi[1, :, :, 3], want):
        return f"accumulated probe feature must keep the maximum: got {phi[1, :, :, 3]}, want {want}"
    return None


def pin_control(o):
    """Threshold feedback on a hand-worked trace (down on an error above
    tolerance or a NaN, up after `patience` quiet intervals, clamps) and the
    budget selection against enumeration."""
    OC = o.control
    theta = np.array([[0.0, 1.0]], np.float32)
    below = np.array([0])
    want = [([-0.5, 0.5], 0), ([-0.5, 0.5], 1), ([-0.5, 0.5], 2), ([-0.25, 0.75], 0), ([-0.75, 0.25], 0),
            ([-1.25, -0.25], 0)]
    for e, (th, bl) in zip([0.2, 0.05, 0.1, 0.05, 0.3, float("nan")], want):
        OC.controller_update(theta, below, [e], 0.1, 0.5, 0.25, 3, -4.0, 4.0)
        if not (np.allclose(theta[0], th) and below[0] == bl):
            return f"feedback trace: after error {e} got theta {theta[0]}, below {below[0]}; want {th}, {bl}"
    theta = np.array([[-3.8, 3.9]], np.float32)
    below = np.array([2])
    OC.controller_update(theta, below, [0.0], 0.1, 0.5, 0.25, 3, -4.0, 4.0)
    if not (np.allclose(theta[0], [-3.55, 4.0]) and below[0] == 0):
        return f"step up must clamp at theta_max, got {theta[0]}"
    OC.controller_update(theta, below, [1.0], 0.1, 1.0, 0.25, 3, -4.0, 4.0)
    if not np.allclose(theta[0], [-4.0, 3.0]):
        return f"step down must clamp at theta_min, got {theta[0]}"
    from itertools import combinations
    z = np.array([0.5, 0.9, 0.5, -1.0, 0.9, 0.5], np.float32)
    for rmin, rmax in ((0, 8), (2, 8), (4, 16)):
        for E in range(0, 6 * rmax + 3):
            got = OC.budget_select(z, E, rmin, rmax)
            # enumeration: the largest promoted set within the budget whose
            # members all beat every other token (larger z, or equal z and lower index)
            best = ()
            for n in range(len(z) + 1):
                if len(z) * rmin + n * (rmax - rmin) > E:
                    break
                for sub in combinations(range(len(z)), n):
                    rest = [t for t in range(len(z)) if t not in sub]
                    if all(z[a] > z[b] or (z[a] == z[b] and a < b) for a in sub for b in rest):
                        best = sub
            if [int(t) for t in np.nonzero(got)[0]] != sorted(best):
                return f"budget {E} at levels ({rmin}, {rmax}): promoted {np.nonzero(got)[0]}, want {sorted(best)}"
    return None


def pin_probe_schedule(o):
    """The probe schedule on a hand-worked table (Hkv 8, 3 heads, every 4
    steps), and its invariants over many steps: probes only every p steps,
    distinct heads, every head within each ceil(Hkv / n) consecutive probes
    (exactly once per Hkv / n probes when n divides Hkv), positions limited by
    the decode steps so far."""
    OC = o.control
    table = {0: [0, 1, 2], 4: [3, 4, 5], 8: [6, 7, 0], 12: [1, 2, 3], 16: [4, 5, 6]}
    for s in range(20):
        heads, npos = OC.probe_schedule(s, 4, 3, 8, 5)
        if s in table:
            if heads != table[s] or npos != min(5, s + 1):
                return f"probe schedule step {s}: got {heads}, {npos}"
        elif heads or npos:
            return f"probe schedule probes at step {s}"
    for hk, n, p in ((8, 1, 1), (8, 2, 3), (8, 3, 2), (5, 4, 1), (64, 8, 16), (8, 8, 2)):
        probes = []
        for s in range(0, 60 * p):
            heads, npos = OC.probe_schedule(s, p, n, hk, 4)
            if (s % p == 0) != bool(heads):
                return f"probe schedule (Hkv {hk}, n {n}, p {p}) wrong at step {s}"
            if heads:
                if len(heads) != n or len(set(heads)) != n or not all(0 <= h < hk for h in heads):
                    return f"probe schedule heads {heads} invalid"
                if npos != min(4, s + 1):
                    return "probe schedule positions wrong"
                probes.append(heads)
        span = -(-hk // n)
        for k in range(len(probes) - span + 1):
            seen = set(h for hs in probes[k:k + span] for h in hs)
            if len(seen) != hk:
                return f"probe schedule (Hkv {hk}, n {n}): probes {k}..{k + span - 1} miss a head"
            if hk % n == 0 and sum(len(hs) for hs in probes[k:k + span]) != hk:
                return "probe schedule repeats a head within a rotation"
    return None


def pin_route_budget(o):
    """Budget routing of a token range against a running loop written here:
    router scores in exact rational arithmetic rounded per operation, the n
    tokens of largest score promoted (ties to the lower token, n from the
    budget and clamped to [0, N]), codes as level indices 0 / 1, and offsets
    continued from a non-zero off[t0] by the routed levels.  Budgets run from
    infeasible to generous; the promotion boundary falls inside a group of
    exactly tied scores; rho_min is positive in one level pair; codes and
    offsets outside the range stay untouched."""
    OC = o.control
    w = small_workload(levels=(0, 16), probs=(0.5, 0.5))
    M, Hk, T = 2, 2, 120
    phi, u, _ = router_inputs(w, n_windows=M, T=T)
    t0, t1 = 30, 100
    N = t1 - t0
    # a tie group: tokens 50..59 share one feature row, so their scores tie
    # exactly; budgets below put the promotion boundary inside it
    for m in range(M):
        for h in range(Hk):
            phi[m, h, 50:60] = phi[m, h, 41]
    for lo, hi in ((0, 16), (2, 8)):
        lev = (lo, hi)
        for which in range(5):
            entries = np.zeros((M, Hk), np.int64)
            for m in range(M):
                for h in range(Hk):
                    zs = [exact_score(u[m], phi[m, h, t]) for t in range(t0, t1)]
                    order = sorted(range(N), key=lambda k: (-zs[k], k))
                    tie = [k for k in order if zs[k] == zs[50 - t0]]
                    cut = order.index(tie[len(tie) // 2])       # a boundary inside the tie group
                    n_want = (0, cut, N, N // 3, N)[which]
                    extra = (-(N * lo) - 5 if lo else -3, 0, 7, hi - lo - 1, 10 * N * hi)[which]
                    entries[m, h] = N * lo + n_want * (hi - lo) + extra
            codes = np.full((M, Hk, T), 9, np.uint8)
            off = np.full((M, Hk, T + 1), 7, np.uint32)
            off[:, :, t0] = 1234
            OC.route_budget(phi, u, entries, lev, t0, t1, codes, off)
            for m in range(M):
                for h in range(Hk):
                    zs = [exact_score(u[m], phi[m, h, t]) for t in range(t0, t1)]
                    E = int(entries[m, h])
                    n = max(0, min(N, (E - N * lo) // (hi - lo)))
                    order = sorted(range(N), key=lambda k: (-zs[k], k))
                    promoted = set(order[:n])
                    run = 1234
                    for k in range(N):
                        t = t0 + k
                        want = 1 if k in promoted else 0
                        if int(codes[m, h, t]) != want:
                            return (f"levels {lev}, budget {E}: code of token {t} (m={m}, h={h}) is "
                                    f"{int(codes[m, h, t])}, the loop gives {want}")
                        if int(off[m, h, t]) != run:
                            return f"levels {lev}, budget {E}: offset of token {t} is {int(off[m, h, t])}, want {run}"
                        run += lev[want]
                    if int(off[m, h, t1]) != run:
                        return f"levels {lev}, budget {E}: final offset {int(off[m, h, t1])}, want {run}"
                    if np.any(codes[m, h, :t0] != 9) or np.any(codes[m, h, t1:] != 9):
                        return "budget routing wrote codes outside the range"
                    if np.any(off[m, h, :t0] != 7) or np.any(off[m, h, t1 + 1:] != 7):
                        return "budget routing wrote offsets outside the range"
    return None


def pin_sketch(o):
    """Sketch basis: Gram-Schmidt rows against numpy's QR (same signs after
    fixing R's diagonal positive), orthonormality, the exact row space of a
    rank-r_b prefill, and a rank-deficient sketch giving zero rows."""
    S = o.sketch
    rng = np.random.default_rng(61)
    Y = rng.standard_normal((12, 40))
    Q = S.orthonormal_rows(Y)
    qq, rr = np.linalg.qr(Y.T)
    qq = qq * np.sign(np.diag(rr))[None, :]
    if not np.allclose(Q, qq.T, atol=1e-12):
        return "Gram-Schmidt rows differ from the QR factor"
    if not np.allclose(Q @ Q.T, np.eye(12), atol=1e-12):
        return "sketch basis not orthonormal"
    # a prefill of exact rank r_b (exact in fp16: integer mixes of unit
    # channel vectors): the basis spans its row space
    w, Tb, Hk, d, rb = 2, 30, 2, 16, 4
    V = np.zeros((d, rb))
    V[rng.permutation(d)[:rb], np.arange(rb)] = 1.0
    coeff = rng.integers(-3, 4, size=(w, 2, Tb, Hk, rb)).astype(np.float64)
    x = np.einsum("lztha,da->lzthd", coeff, V).astype(np.float16)
    omega = rng.standard_normal((w * Tb, rb)).astype(np.float16)
    for h in range(Hk):
        for z in range(2):
            B = S.sketch_basis(x, omega, h, z).astype(np.float64)
            rows = x[:, z, :, h, :].astype(np.float64).reshape(-1, d)
            resid = rows - (rows @ B.T) @ B
            if np.abs(resid).max() > 4e-3 * np.abs(rows).max():
                return f"basis of a rank-{rb} prefill misses its row space (h={h}, z={z})"
            if not np.allclose(B @ B.T, np.eye(rb), atol=3e-3):
                return "fp16 basis rows far from orthonormal"
    # rank-deficient: a single-direction prefill leaves rows 1.. zero
    x1 = np.zeros((1, 2, 10, 1, d), np.float16)
    x1[0, :, :, 0, 3] = rng.standard_normal((2, 10))
    B1 = S.sketch_basis(x1, rng.standard_normal((10, 3)).astype(np.float16), 0, 0).astype(np.float64)
    if not (abs(abs(B1[0, 3]) - 1) < 1e-3 and np.all(B1[1:] == 0)):
        return f"rank-deficient sketch must give one unit row and zero rows, got {B1[:, 3]}"
    return None


def pin_int8_coefficients(o):
    """The 8-bit blockwise coefficient form: a scalar loop over (token, i) gives
    code * scale of block i // 16; with power-of-two scales the int8 cache and
    the fp16 cache holding the same products decode identically."""
    c = small_cache(coef_format="int8", head_dim=128, basis_rank=48, context=20, ragged=(5, 40))
    F = o.factorized
    for layer in range(c.n_layers):
        for z in range(2):
            for h in range(c.n_kv_heads):
                t0, t1 = 3, c.total_tokens - 2
                rows = F.coefficient_rows(c, layer, z, h, t0, t1)
                sc = c.coef_scale_k if z == 0 else c.coef_scale_v
                for t in (t0, t0 + 1, t1 - 1):
                    for i in (0, 1, 15, 16, 20, 31, 32, 33, 47):
                        code = int(c.coef_k[layer, h, t, i]) if z == 0 else int(c.coef_v[layer, h, t // 16, i, t % 16])
                        want = code * float(sc[layer, h, i // 16, t])
                        if rows[t - t0, i] != want:
                            return f"int8 coefficient (layer {layer}, z {z}, h {h}, t {t}, i {i}) is not code * block scale"
    c.coef_scale_k[:] = np.float16(0.125)
    c.coef_scale_v[:] = np.float16(0.25)
    twin = copy.deepcopy(c)
    twin.coef_format = "f16"
    twin.coef_k = (c.coef_k.astype(np.float64) * 0.125).astype(np.float16)
    twin.coef_v = (c.coef_v.astype(np.float64) * 0.25).astype(np.float16)
    for layer in range(c.n_layers):
        if not np.array_equal(o.decode(c, layer), o.decode(twin, layer)):
            return "int8 cache with power-of-two scales decodes differently from its fp16 twin"
    return None


ALL_PINS = [pin_query_formats, pin_nibbles, pin_residual_map, pin_brute_force, pin_closed_forms,
            pin_reductions, pin_invariants, pin_probe, pin_probe_positions, pin_router, pin_compress_closed_forms,
            pin_compress_rne_table, pin_compress_arithmetic, pin_compress_int8, pin_compress_bounds,
            pin_compress_into_cache, pin_route_range, pin_attention_features, pin_probe_feature, pin_control, pin_probe_schedule, pin_route_budget, pin_sketch,
            pin_int8_coefficients]


def run_all(o):
    """Run every pin; returns the list of failure messages (empty when all hold)."""
    fails = []
    for pin in ALL_PINS:
        try:
            r = pin(o)
        except Exception as exc:                      # a mutant may also crash
            r = f"{pin.__name__} raised {type(exc).__name__}: {exc}"
        if r is not None:
            fails.append(f"{pin.__name__}: {r}")
    return fails
