"""Plant plausible mistakes in the oracle (on the CPU) and check that at least
one pin fails for each.  A pin suite that lets a mutant through is too weak to
trust the oracle with."""
import numpy as np
import pytest

import oracle
import oracle.factorized as F
import oracle.router as R
import oracle.compress as CP
import oracle.features as FE
import oracle.control as CT
import oracle.sketch as SK
import pins

_orig_reconstruct = F.reconstruct
_orig_attention = F.attention
_orig_entry_codes = F.entry_codes


def _reconstruct_variant(kind):
    def rec(cache, layer, z, h, b):
        m = F.window_of(layer, cache.window)
        t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
        zb = 1 - z if kind == "other_basis" else z
        A = F.coefficient_rows(cache, layer, z, h, t0, t1)
        if kind == "coef_shift":
            A = F.coefficient_rows(cache, layer, z, h, t0 + 1, t1 + 1)
            A = np.concatenate([A, np.zeros((t1 - t0 - A.shape[0], A.shape[1]))])
        X = A @ cache.basis[b, m, h, zb].astype(np.float64)
        if kind == "no_residual":
            return X
        off = cache.res_off[m, h].astype(np.int64)
        rho = off[t0 + 1:t1 + 1] - off[t0:t1]
        e0, e1 = int(off[t0]), int(off[t1])
        tok = np.repeat(np.arange(t1 - t0), rho)
        chan = cache.res_idx[layer, z, h, e0:e1].astype(np.int64)
        code = F.entry_codes(cache.res_val[layer, z, h], e0, e1 - e0)
        gs = cache.res_scale[layer, z, h, t0:t1].astype(np.float64)
        Rm = np.zeros_like(X)
        Rm[tok, chan] = code
        if kind == "residual_sign":
            return X - gs[:, None] * Rm
        if kind == "no_gate":
            return X + Rm
        if kind == "residual_layer":       # residual of the window's first layer
            l0 = m * cache.window
            chan = cache.res_idx[l0, z, h, e0:e1].astype(np.int64)
            code = F.entry_codes(cache.res_val[l0, z, h], e0, e1 - e0)
            Rm = np.zeros_like(X)
            Rm[tok, chan] = code
        return X + gs[:, None] * Rm
    return rec


def _attention_variant(kind):
    def att(q, K, V, sm_scale):
        if K.shape[0] == 0:
            return np.zeros((q.shape[0], V.shape[1])), np.zeros((q.shape[0], 0))
        s = (q @ K.T) * (1.0 if kind == "no_scale" else sm_scale)
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        ax = 0 if kind == "wrong_axis" else 1
        p = w / w.sum(axis=ax, keepdims=True)
        return (p @ (K if kind == "keys_as_values" else V)), p
    return att


def _entry_codes_swapped(val_bytes, start, count):
    e = np.arange(start, start + count, dtype=np.int64)
    byte = val_bytes[e // 2].astype(np.int64)
    nib = np.where(e % 2 == 1, byte & 0xF, byte >> 4)
    return F.int4_from_nibble(nib)


def _router_fused(phi, u):
    phi = np.asarray(phi, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    return (phi @ u).astype(np.float32)


def _router_reordered(phi, u):
    phi = np.asarray(phi, dtype=np.float32)
    u = np.asarray(u, dtype=np.float32)
    z = np.float32(u[3]) * phi[..., 3]
    for i in (2, 1, 0):
        z = z + np.float32(u[i]) * phi[..., i]
    return z


def _level_ge(z, theta):
    k = np.zeros(np.shape(z), dtype=np.int64)
    for th in np.asarray(theta, dtype=np.float32):
        k += (np.asarray(z, np.float32) >= th)
    return k


def _route_inclusive(phi, u, theta, levels):
    codes, off = R.__dict__["_orig_route"](phi, u, theta, levels)
    lev = np.asarray(levels)
    off2 = np.zeros_like(off)
    off2[..., :-1] = off[..., 1:]
    off2[..., -1] = off[..., -1]
    return codes, off2


def _project_reversed(x, B):
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    B = np.asarray(B, dtype=np.float16).astype(np.float32)
    d = x.shape[1]
    acc = x[:, d - 1:d] * B[None, :, d - 1]
    for j in range(d - 2, -1, -1):
        acc = acc + x[:, j:j + 1] * B[None, :, j]
    return acc.astype(np.float16)


def _blocked_sum(terms):
    """Four contiguous quarters, each left to right, combined (q0 + q1) + (q2 + q3)."""
    n = len(terms)
    b = [q * n // 4 for q in range(5)]
    part = []
    for q in range(4):
        acc = terms[b[q]]
        for j in range(b[q] + 1, b[q + 1]):
            acc = acc + terms[j]
        part.append(acc)
    return (part[0] + part[1]) + (part[2] + part[3])


def _project_quarters(x, B):
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    B = np.asarray(B, dtype=np.float16).astype(np.float32)
    return _blocked_sum([x[:, j:j + 1] * B[None, :, j] for j in range(x.shape[1])]).astype(np.float16)


def _residual_quarters(x, B, a16):
    xx = np.asarray(x, dtype=np.float16).astype(np.float32)
    BB = np.asarray(B, dtype=np.float16).astype(np.float32)
    a = np.asarray(a16, dtype=np.float16).astype(np.float32)
    return xx - _blocked_sum([a[:, i:i + 1] * BB[None, i, :] for i in range(BB.shape[0])])


def _project_f64(x, B):
    return (np.asarray(x, np.float64) @ np.asarray(B, np.float64).T).astype(np.float16)


def _residual_unrounded_a(x, B, a16):
    xx = np.asarray(x, dtype=np.float16).astype(np.float32)
    BB = np.asarray(B, dtype=np.float16).astype(np.float32)
    a = xx[:, 0:1] * BB[None, :, 0]
    for j in range(1, xx.shape[1]):
        a = a + xx[:, j:j + 1] * BB[None, :, j]
    p = a[:, 0:1] * BB[None, 0, :]
    for i in range(1, BB.shape[0]):
        p = p + a[:, i:i + 1] * BB[None, i, :]
    return xx - p


def _residual_reversed(x, B, a16):
    xx = np.asarray(x, dtype=np.float16).astype(np.float32)
    BB = np.asarray(B, dtype=np.float16).astype(np.float32)
    a = np.asarray(a16, dtype=np.float16).astype(np.float32)
    r = BB.shape[0]
    p = a[:, r - 1:r] * BB[None, r - 1, :]
    for i in range(r - 2, -1, -1):
        p = p + a[:, i:i + 1] * BB[None, i, :]
    return xx - p


def _select_ties_up(r, rho):
    mag = np.abs(np.asarray(r, dtype=np.float32))
    order = sorted(range(mag.size), key=lambda c: (-float(mag[c]), -c))
    return np.asarray(order[:rho], dtype=np.int64)


def _quantize_half_away(values, S):
    v = np.asarray(values, dtype=np.float32)
    if S == 0:
        return np.zeros(v.shape, dtype=np.int64)
    q = v / np.float32(S)
    return np.clip(np.sign(q) * np.floor(np.abs(q) + 0.5), -7, 7).astype(np.int64)


def _store_values_row_major(cache, layer, z, h, t, row):
    if z == 0:
        cache.coef_k[layer, h, t] = row
    else:
        cache.coef_v[layer, h].reshape(-1, cache.coef_v.shape[3])[t] = row


def _store_entries_at_next(cache, layer, z, h, t, chans, codes):
    m = layer // cache.window
    e0 = int(cache.res_off[m, h, t + 1])
    cache.res_idx[layer, z, h, e0:e0 + len(chans)] = chans
    if len(chans):
        cache.res_val[layer, z, h, e0 // 2:(e0 + len(chans)) // 2] = CP._pack_pairs(codes)


def _route_range_from_zero(phi, u, theta, levels, t0, t1, codes, off):
    off[:, :, t0] = 0
    return R.__dict__["_orig_route_range"](phi, u, theta, levels, t0, t1, codes, off)


def _features_variant(kind):
    def feat(cache, layer, q=None, sm_scale=None):
        _, probs = F.decode(cache, layer, q, sm_scale, with_probs=True)
        Hk, T = cache.n_kv_heads, int(cache.cu_seqlens[-1])
        mass, spike = np.zeros((Hk, T)), np.zeros((Hk, T))
        for (b, h), p in probs.items():
            t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
            if t1 > t0:
                if kind == "mean":
                    mass[h, t0:t1] = p.mean(axis=0)
                else:
                    mass[h, t0:t1] = p.sum(axis=0)
                spike[h, t0:t1] = p.sum(axis=0) if kind == "spike_sum" else p.max(axis=0)
        return mass, spike
    return feat


def _update_overwrite(phi, window, mass, spike):
    phi[window, :, :, 0] = mass
    phi[window, :, :, 1] = np.maximum(phi[window, :, :, 1], spike)
    return phi


def _update_spike_last(phi, window, mass, spike):
    phi[window, :, :, 0] += mass
    phi[window, :, :, 1] = spike
    return phi


def _ctl_variant(kind):
    def upd(theta, below, err, tol, step_down, step_up, patience, theta_min, theta_max):
        theta = np.asarray(theta)
        for m in range(theta.shape[0]):
            e = float(err[m])
            above = (e > tol) if kind == "nan_quiet" else (np.isnan(e) or e > tol)
            if above:
                theta[m] = theta[m] - np.float32(step_down)
                if kind != "no_clamp":
                    theta[m] = np.clip(theta[m], theta_min, theta_max)
                below[m] = 0
            else:
                below[m] += 1
                if (below[m] > patience) if kind == "patience_late" else (below[m] >= patience):
                    theta[m] = theta[m] + np.float32(step_up)
                    if kind != "no_clamp":
                        theta[m] = np.clip(theta[m], theta_min, theta_max)
                    below[m] = 0
        return theta, below
    return upd


def _budget_ties_up(z, entries, rho_min, rho_max):
    N = len(z)
    n = max(0, min(N, (entries - N * rho_min) // (rho_max - rho_min)))
    order = sorted(range(N), key=lambda t: (-float(z[t]), -t))
    codes = np.zeros(N, dtype=np.uint8)
    codes[order[:n]] = 1
    return codes


def _budget_ceil(z, entries, rho_min, rho_max):
    N = len(z)
    n = max(0, min(N, -(-(entries - N * rho_min) // (rho_max - rho_min))))
    order = sorted(range(N), key=lambda t: (-float(z[t]), t))
    codes = np.zeros(N, dtype=np.uint8)
    codes[order[:n]] = 1
    return codes


def _budget_offsets_from_zero(phi, u, entries, levels, t0, t1, codes, off):
    off[:, :, t0] = 0
    return CT.__dict__["_orig_route_budget"](phi, u, entries, levels, t0, t1, codes, off)


def _budget_code_as_level(phi, u, entries, levels, t0, t1, codes, off):
    CT.__dict__["_orig_route_budget"](phi, u, entries, levels, t0, t1, codes, off)
    codes[:, :, t0:t1] = np.asarray(levels, np.uint8)[codes[:, :, t0:t1]]
    return codes, off


def _pf_mean(phi, cu, window, kv_heads, err, G, fresh):
    err = np.asarray(err, np.float32)
    e2 = np.repeat(err.reshape(err.shape[0], -1, G).mean(axis=2), G, axis=1)
    return FE.__dict__["_orig_probe_feature"](phi, cu, window, kv_heads, e2, G, fresh)


def _pf_overwrite(phi, cu, window, kv_heads, err, G, fresh):
    return FE.__dict__["_orig_probe_feature"](phi, cu, window, kv_heads, err, G, True)


def _pf_all_heads(phi, cu, window, kv_heads, err, G, fresh):
    FE.__dict__["_orig_probe_feature"](phi, cu, window, kv_heads, err, G, fresh)
    h0 = kv_heads[0]
    for h in range(phi.shape[1]):
        phi[window, h, :, 3] = phi[window, h0, :, 3]
    return phi


def _q8_variant(kind):
    def q8(a32):
        a = np.asarray(a32, dtype=np.float32)
        n, rb = a.shape
        bw = 8 if kind == "block8" else 16
        codes = np.zeros((n, rb), dtype=np.int8)
        scales = np.zeros((n, rb // 16), dtype=np.float16)
        rows = np.zeros((n, rb), dtype=np.float32)
        for k in range(n):
            for s in range(rb // bw):
                blk = a[k, bw * s:bw * s + bw]
                S = np.float16(np.float32(np.abs(blk).max()) / np.float32(128.0 if kind == "div128" else 127.0))
                if bw == 16:
                    scales[k, s] = S
                if S == 0:
                    continue
                q = blk / np.float32(S)
                q = np.sign(q) * np.floor(np.abs(q) + 0.5) if kind == "half_away" else np.rint(q)
                codes[k, bw * s:bw * s + bw] = np.clip(q, -127, 127).astype(np.int8)
                rows[k, bw * s:bw * s + bw] = codes[k, bw * s:bw * s + bw].astype(np.float32) * np.float32(S)
        return codes, scales, rows
    return q8


def _cv_residual_fp16(x, B, rhos, gates=None, coef_format="f16"):
    if coef_format != "int8":
        return CP.__dict__["_orig_compress_vectors"](x, B, rhos, gates, coef_format)
    x = np.asarray(x, dtype=np.float16)
    codes8, cscales, _ = CP.quantize_coefficients(CP.project32(x, B))
    r = CP.residual(x, B, CP.project(x, B))
    entries, scales = [], np.zeros(x.shape[0], dtype=np.float16)
    for k in range(x.shape[0]):
        rho = int(rhos[k])
        if rho == 0:
            entries.append((np.zeros(0, np.int64), np.zeros(0, np.int64)))
            continue
        S = CP.quant_scale(r[k])
        ch = CP.select_channels(r[k], rho)
        entries.append(CP.entry_order(ch, CP.quantize(r[k][ch], S)))
        scales[k] = CP.fold_gate(S, 1.0 if gates is None else float(gates[k]))
    return (codes8, cscales), entries, scales


def _gs_no_normalize(Y):
    Y = np.array(Y, dtype=np.float64)
    Q = np.zeros_like(Y)
    for i in range(Y.shape[0]):
        v = Y[i].copy()
        for j in range(i):
            v -= (v @ Q[j]) * Q[j]
        Q[i] = v / max(np.abs(v).max(), 1e-300)
    return Q


def _sketch_transposed(x_rows, omega):
    return (np.asarray(x_rows, np.float64).T @ np.asarray(omega, np.float64).T).T[:, :np.asarray(x_rows).shape[1]] \
        if False else np.asarray(omega, np.float64)[:, ::-1] @ np.asarray(x_rows, np.float64)


def _coef_rows_variant(kind):
    orig = F.__dict__.setdefault("_orig_coefficient_rows", F.coefficient_rows)
    def rows(cache, layer, z, h, t0, t1):
        if getattr(cache, "coef_format", "f16") != "int8":
            return orig(cache, layer, z, h, t0, t1)
        if z == 0:
            r = cache.coef_k[layer, h, t0:t1].astype(np.float64)
        else:
            blocks = cache.coef_v[layer, h]
            r = np.swapaxes(blocks, 1, 2).reshape(-1, blocks.shape[1])[t0:t1].astype(np.float64)
        sc = (cache.coef_scale_k if z == 0 else cache.coef_scale_v)[layer, h].astype(np.float64)   # [NB, T]
        nb = sc.shape[0]
        if kind == "block_mod":
            idx = np.arange(r.shape[1]) % nb
            return r * sc[idx][:, t0:t1].T
        if kind == "next_token":
            return r * np.repeat(sc[:, t0 + 1:t1 + 1].T if t1 < sc.shape[1] else
                                 np.concatenate([sc[:, t0 + 1:t1], sc[:, t1 - 1:t1]], axis=1).T, 16, axis=1)
        return r
    return rows



def _pp_variant(kind):
    def pp(cache, layer, kv_heads, k_ref, v_ref, qs, sm_scale=None, eps=1e-6):
        G = cache.n_q_heads // cache.n_kv_heads
        scale = F.default_scale(cache.head_dim) if not sm_scale or sm_scale <= 0 else sm_scale
        qs = np.asarray(qs, np.float64)
        P = qs.shape[0]
        err = np.zeros((cache.batch, len(kv_heads) * G))
        for i, h in enumerate(kv_heads):
            for b in range(cache.batch):
                t0, t1 = int(cache.cu_seqlens[b]), int(cache.cu_seqlens[b + 1])
                K, V = F.reconstruct(cache, layer, 0, h, b), F.reconstruct(cache, layer, 1, h, b)
                d2, r2, per = np.zeros(G), np.zeros(G), []
                for j in range(P):
                    n = max(t1 - t0 - j, 0)
                    lo, hi = (j, t1 - t0) if kind == "front" else (0, n)
                    if kind == "plus_one" and j > 0:
                        hi = min(n + 1, t1 - t0)
                    lo = min(lo, hi)
                    qq = qs[P - 1 - j if kind == "reverse" else j, b, h * G:(h + 1) * G]
                    o_ref, _ = F.attention(qq, np.asarray(k_ref[i, t0 + lo:t0 + hi], np.float64),
                                           np.asarray(v_ref[i, t0 + lo:t0 + hi], np.float64), scale)
                    o, _ = F.attention(qq, K[lo:hi], V[lo:hi], scale)
                    dd, rr = ((o_ref - o) ** 2).sum(-1), (o_ref ** 2).sum(-1)
                    if kind == "first_only" and j > 0:
                        dd = rr = 0 * dd
                    d2, r2 = d2 + dd, r2 + rr
                    per.append(np.sqrt(dd) / (np.sqrt(rr) + eps))
                err[b, i * G:(i + 1) * G] = (np.mean(per, axis=0) if kind == "mean"
                                             else np.sqrt(d2) / (np.sqrt(r2) + eps))
        return err
    return pp

MUTANTS = {
    "residual dropped": [(F, "reconstruct", _reconstruct_variant("no_residual"))],
    "residual sign flipped": [(F, "reconstruct", _reconstruct_variant("residual_sign"))],
    "gate scale dropped": [(F, "reconstruct", _reconstruct_variant("no_gate"))],
    "K/V basis swapped": [(F, "reconstruct", _reconstruct_variant("other_basis"))],
    "coefficient rows shifted by one token": [(F, "reconstruct", _reconstruct_variant("coef_shift"))],
    "residual read from the window's first layer": [(F, "reconstruct", _reconstruct_variant("residual_layer"))],
    "window index l % w": [(F, "window_of", lambda layer, w: layer % w)],
    "interleaved GQA grouping": [(F, "kv_head_of", lambda hq, nq, nk: hq % nk)],
    "softmax scale dropped": [(F, "attention", _attention_variant("no_scale"))],
    "softmax over tokens of the wrong axis": [(F, "attention", _attention_variant("wrong_axis"))],
    "keys used as values": [(F, "attention", _attention_variant("keys_as_values"))],
    "unsigned int4": [(F, "int4_from_nibble", lambda nib: np.asarray(nib, dtype=np.int64))],
    "nibble order swapped": [(F, "entry_codes", _entry_codes_swapped)],
    "default scale 1/d": [(F, "default_scale", lambda d: 1.0 / d)],
    "probe denominator uses the compressed output": [
        (F, "probe_error", lambda o_ref, o, eps=1e-6: np.linalg.norm(np.asarray(o_ref) - o, axis=-1)
         / (np.linalg.norm(o, axis=-1) + eps))],
    "probe eps dropped": [
        (F, "probe_error", lambda o_ref, o, eps=1e-6: np.linalg.norm(np.asarray(o_ref) - o, axis=-1)
         / np.maximum(np.linalg.norm(o_ref, axis=-1), 1e-300))],
    "probe positions average the per-position errors": [(F, "probe_positions", _pp_variant("mean"))],
    "probe positions trimmed from the front": [(F, "probe_positions", _pp_variant("front"))],
    "probe positions see one token too many": [(F, "probe_positions", _pp_variant("plus_one"))],
    "probe positions pair the queries in reverse": [(F, "probe_positions", _pp_variant("reverse"))],
    "probe positions keep only the current one": [(F, "probe_positions", _pp_variant("first_only"))],
    "probe schedule rotates by one head": [(CT, "probe_schedule", lambda s, p, n, hk, P: (
        ([((s // p) + i) % hk for i in range(n)], min(P, s + 1)) if s % p == 0 else ([], 0)))],
    "probe schedule probes one step late": [(CT, "probe_schedule", lambda s, p, n, hk, P: (
        ([(((s - 1) // p) * n + i) % hk for i in range(n)], min(P, s)) if s % p == 1 % p else ([], 0)))],
    "probe schedule ignores the step count for positions": [(CT, "probe_schedule", lambda s, p, n, hk, P: (
        ([((s // p) * n + i) % hk for i in range(n)], P) if s % p == 0 else ([], 0)))],
    "router score in float64": [(R, "router_score", _router_fused)],
    "router score summed in reverse": [(R, "router_score", _router_reordered)],
    "router ties go up": [(R, "level_index", _level_ge)],
    "inclusive offsets": [(R, "route", _route_inclusive)],
    "value blocks read row-major": [(F, "coefficient_rows", lambda cache, layer, z, h, t0, t1:
        cache.coef_k[layer, h, t0:t1].astype(np.float64) if z == 0 else
        cache.coef_v[layer, h].reshape(-1, cache.coef_v.shape[3])[t0:t1].astype(np.float64))],
    "projection summed right to left": [(CP, "project", _project_reversed)],
    "projection in float64": [(CP, "project", _project_f64)],
    "projection summed in four blocked quarters": [(CP, "project", _project_quarters)],
    "basis term summed in four blocked quarters": [(CP, "residual", _residual_quarters)],
    "residual from the unrounded coefficients": [(CP, "residual", _residual_unrounded_a)],
    "residual basis term summed right to left": [(CP, "residual", _residual_reversed)],
    "residual sign flipped in compress": [(CP, "residual", lambda x, B, a16:
        -_residual_reversed.__globals__["CP"].__dict__["_orig_residual"](x, B, a16))],
    "kept-channel ties go to the higher channel": [(CP, "select_channels", _select_ties_up)],
    "int4 scale max|r| / 8": [(CP, "quant_scale", lambda r: np.float32(np.abs(np.asarray(r, np.float32)).max())
                                / np.float32(8.0))],
    "codes round half away from zero": [(CP, "quantize", _quantize_half_away)],
    "entries stored in channel order": [(CP, "entry_order", lambda ch, k: (np.asarray(ch)[np.argsort(ch)],
                                                                        np.asarray(k)[np.argsort(ch)]))],
    "gate not folded into the scale": [(CP, "fold_gate", lambda S, g: np.float16(S))],
    "int8 block scale max|A| / 128": [(CP, "quantize_coefficients", _q8_variant("div128"))],
    "int8 codes round half away from zero": [(CP, "quantize_coefficients", _q8_variant("half_away"))],
    "int8 blocks of 8 coefficients": [(CP, "quantize_coefficients", _q8_variant("block8"))],
    "int8 residual against the fp16 projection": [(CP, "compress_vectors", _cv_residual_fp16)],
    "value coefficients written row-major": [(CP, "store_coefficients", _store_values_row_major)],
    "entries written at the next token's offset": [(CP, "store_entries", _store_entries_at_next)],
    "range routing restarts the offsets at zero": [(R, "route_range", _route_range_from_zero)],
    "attention mass averaged over heads": [(FE, "attention_features", _features_variant("mean"))],
    "attention spike summed over heads": [(FE, "attention_features", _features_variant("spike_sum"))],
    "feature mass overwritten instead of accumulated": [(FE, "update_features", _update_overwrite)],
    "feature spike keeps the last value": [(FE, "update_features", _update_spike_last)],
    "probe feature averages the group's errors": [(FE, "probe_feature", _pf_mean)],
    "probe feature overwrites when folding": [(FE, "probe_feature", _pf_overwrite)],
    "probe feature written to every head": [(FE, "probe_feature", _pf_all_heads)],
    "threshold steps not clamped": [(CT, "controller_update", _ctl_variant("no_clamp"))],
    "NaN probe error counted as quiet": [(CT, "controller_update", _ctl_variant("nan_quiet"))],
    "step up one interval late": [(CT, "controller_update", _ctl_variant("patience_late"))],
    "budget ties go to the higher token": [(CT, "budget_select", _budget_ties_up)],
    "budget count rounded up": [(CT, "budget_select", _budget_ceil)],
    "budget routing restarts the offsets at zero": [(CT, "route_budget", _budget_offsets_from_zero)],
    "budget routing writes the level as the code": [(CT, "route_budget", _budget_code_as_level)],
    "Gram-Schmidt rows scaled by max instead of norm": [(SK, "orthonormal_rows", _gs_no_normalize)],
    "sketch with the token order reversed": [(SK, "sketch", _sketch_transposed)],
    "int8 block scale indexed by i mod blocks": [(F, "coefficient_rows", _coef_rows_variant("block_mod"))],
    "int8 block scale of the next token": [(F, "coefficient_rows", _coef_rows_variant("next_token"))],
    "int8 block scale ignored": [(F, "coefficient_rows", _coef_rows_variant("none"))],
    "bf16 query read as fp16": [(F, "q_to_f64", lambda bits, dtype: np.asarray(bits, np.uint16)
                                 .view(np.float16).astype(np.float64))],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    R.__dict__.setdefault("_orig_route", R.route)
    R.__dict__.setdefault("_orig_route_range", R.route_range)
    CP.__dict__.setdefault("_orig_residual", CP.residual)
    CT.__dict__.setdefault("_orig_route_budget", CT.route_budget)
    FE.__dict__.setdefault("_orig_probe_feature", FE.probe_feature)
    CP.__dict__.setdefault("_orig_compress_vectors", CP.compress_vectors)
    for mod, attr, fn in MUTANTS[name]:
        monkeypatch.setattr(mod, attr, fn)
        if hasattr(oracle, attr):
            monkeypatch.setattr(oracle, attr, fn)
    fails = pins.run_all(oracle)
    assert fails, f"no pin caught the mutant '{name}'"


def test_unmutated_oracle_passes_every_pin():
    assert pins.run_all(oracle) == []
