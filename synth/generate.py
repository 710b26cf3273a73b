"""Seeded synthetic factorized KV caches in the library's storage layout.

Every random draw comes from a PCG64DXSM stream keyed by
(workload seed, tensor id, indices), so any slab (one sequence, layer,
K-or-V, head) regenerates on its own and equals the same slab of a full
generation.  The draws follow the workload's stated distributions:

* shared bases: r_b x d N(0,1) rows, orthonormalised in float64, rounded to fp16;
* per-token basis coefficients: N(0,1) rounded to fp16; or, for the 8-bit
  blockwise form, int8 codes Binomial(254, 1/2) - 127 (mean 0, sd about 8)
  with one fp16 scale per 16-coefficient block drawn U(0.11, 0.14);
* routed residual rank: categorical over the level table (salient spans, when
  the workload has them, force one level for every window and head);
* residual entries: the routed number of distinct channels drawn uniformly,
  int4 codes uniform on [-7, 7], stored largest |code| first, then by channel;
* per-token residual scale (gate folded in, gate = 1): U(0.01, 0.1) in fp16;
  or, in the "wide" scale mode, scales spanning fp16's range: within every
  run of `scale_period` tokens of a sequence the binary exponent ramps up
  from the subnormals (2^-24) to 2^15 for values and to 2^1 for keys, times
  U(1, 2), with 4% of the scales zero and the last token of every run at the
  ramp's top (so that the largest scale of a chunk comes late);
* int8 block scales in the "wide" coefficient-scale mode: 2^U(-12, 7) for
  values and 2^U(-5, -2) for keys (several binades within one token);
* queries: N(0,1)/sqrt(d) rounded to the workload's query dtype.

Packing variable-length residual entries needs the running position of each
token's first entry; that is storage layout, computed here with a cumulative
sum of the drawn ranks.  Nothing in this module evaluates the method itself
(reconstruction, routing scores, attention or probe error).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

from .layout import BLOCK, padded_tokens
from .workloads import Workload

# tensor ids used to key the random streams
_BASIS, _COEF, _RANK, _RES_CH, _RES_CODE, _RES_SCALE, _Q, _SPANS = 1, 2, 3, 4, 5, 6, 7, 8
_PHI, _ROUTER_U, _PROBE = 10, 11, 12
_COEF8, _COEF8_SCALE = 13, 14

RES_TAIL_PAD = 512      # spare entries after the longest slab
RES_ALIGN = 256         # res_stride is a multiple of this


def rng_for(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64DXSM(np.random.SeedSequence(list(key))))


def _residual_scales(w: Workload, g: np.random.Generator, z: int, n: int) -> np.ndarray:
    """fp16 residual scales of one sequence's n tokens of a (layer, Z, head) slab."""
    if getattr(w, "scale_mode", "uniform") != "wide":
        return g.uniform(0.01, 0.1, size=n).astype(np.float16)
    P = max(int(w.scale_period), 2)
    top = 15.0 if z == 1 else 1.0
    pos = np.arange(n) % P
    e = np.floor(-24.0 + (top + 24.0) * pos / (P - 1))
    s = np.exp2(e) * g.uniform(1.0, 2.0, size=n)
    s[pos == P - 1] = np.exp2(top) * 1.99
    s[g.random(n) < 0.04] = 0.0
    return np.minimum(s, 65504.0).astype(np.float16)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def f16_bits(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


@dataclass
class CompressedCache:
    """Host copy of one factorized cache, laid out as the C ABI expects.

    Shapes (M windows, L layers held, T packed tokens over all sequences):
      basis     fp16  [B][M][Hkv][2][r_b][d]   Z=0 keys, Z=1 values
      coef_k    fp16  [L][Hkv][T][r_b]           key coefficient rows A^K
      coef_v    fp16  [L][Hkv][T16/16][r_b][16]  value coefficients A^V in 16-token
                                                 blocks, token fastest (T16 = T rounded
                                                 up to 16, zero padded)
      rank_code uint8 [M][Hkv][T]
      res_off   uint32[M][Hkv][T+1]
      res_idx   uint8 [L][2][Hkv][res_stride]
      res_val   uint8 [L][2][Hkv][res_stride/2]  two int4 codes per byte, low nibble first
      res_scale fp16  [L][2][Hkv][T]
      q_bits    uint16[L][B][Hq][d]              fp16 or bf16 bit patterns
    With coef_format "int8" (the 8-bit blockwise form), coef_k / coef_v hold
    int8 codes in the same shapes and coef_scale_k / coef_scale_v fp16
    [L][Hkv][r_b/16][T] the scale of each 16-coefficient block.
    """
    workload: Workload
    layer0: int                 # absolute index of the first layer held
    n_layers: int               # layers held (a whole number of windows)
    seqlens: list
    cu_seqlens: np.ndarray      # int32 [B+1]
    levels: tuple
    res_stride: int
    basis: np.ndarray
    coef_k: np.ndarray
    coef_v: np.ndarray
    rank_code: np.ndarray
    res_off: np.ndarray
    res_idx: np.ndarray
    res_val: np.ndarray
    res_scale: np.ndarray
    q_bits: np.ndarray
    q_dtype: str
    coef_format: str = "f16"
    coef_scale_k: np.ndarray | None = None
    coef_scale_v: np.ndarray | None = None

    @property
    def batch(self): return len(self.seqlens)
    @property
    def window(self): return self.workload.window
    @property
    def n_kv_heads(self): return self.workload.n_kv_heads
    @property
    def n_q_heads(self): return self.workload.n_q_heads
    @property
    def head_dim(self): return self.workload.head_dim
    @property
    def basis_rank(self): return self.workload.basis_rank
    @property
    def total_tokens(self): return int(self.cu_seqlens[-1])
    @property
    def n_windows(self): return self.n_layers // self.window

    def nbytes_layer(self) -> int:
        """Compressed bytes one per-layer decode reads (bases, coefficients,
        offsets, residual scales/indices/values) plus q in and fp32 out."""
        Hk, T, rb, d = self.n_kv_heads, self.total_tokens, self.basis_rank, self.head_dim
        B, Hq = self.batch, self.n_q_heads
        basis = B * Hk * 2 * rb * d * 2
        coef = 2 * Hk * T * rb * 2 if self.coef_format == "f16" else 2 * Hk * T * (rb + 2 * (rb // 16))
        off = Hk * (T + 1) * 4
        ent = 0
        for h in range(Hk):      # average over windows of the entries per slab
            ent += sum(int(self.res_off[m, h, -1]) for m in range(self.n_windows)) / self.n_windows
        resid = 2 * (ent * 1 + ent / 2) + 2 * Hk * T * 2
        qo = B * Hq * d * (2 + 4)
        return int(basis + coef + off + resid + qo)


def _window_codes(w: Workload, b: int, m: int, h: int, T: int) -> np.ndarray:
    rng = rng_for(w.seed, _RANK, b, m, h)
    codes = rng.choice(len(w.levels), size=T, p=np.asarray(w.probs, dtype=np.float64))
    codes = codes.astype(np.uint8)
    if w.salient_frac > 0:
        span = w.salient_span
        n_slots = T // span
        n_spans = min(n_slots, int(round(w.salient_frac * T / span)))
        srng = rng_for(w.seed, _SPANS, b)          # shared by every (window, head)
        slots = srng.choice(n_slots, size=n_spans, replace=False)
        for s in slots:
            codes[s * span:(s + 1) * span] = w.salient_level
    return codes


def _orthonormal_rows(rng: np.random.Generator, r: int, d: int) -> np.ndarray:
    x = rng.standard_normal((r, d))
    q, rr = np.linalg.qr(x.T)                    # columns of q: orthonormal
    q = q * np.sign(np.diag(rr))[None, :]        # fixed sign convention
    return q.T                                   # r x d, orthonormal rows


def _slab_entries(w: Workload, b: int, l: int, z: int, h: int, ranks: np.ndarray):
    """Residual channels and codes for one (sequence, layer, Z, head) slab,
    in token order, each token's entries largest |code| first then by channel."""
    d = w.head_dim
    T = ranks.shape[0]
    n_e = int(ranks.sum())
    chans = np.empty(n_e, dtype=np.uint8)
    codes = np.empty(n_e, dtype=np.int8)
    starts = np.zeros(T, dtype=np.int64)
    np.cumsum(ranks[:-1], out=starts[1:])
    rng_c = rng_for(w.seed, _RES_CH, b, l, z, h)
    rng_k = rng_for(w.seed, _RES_CODE, b, l, z, h)
    for r in sorted(set(int(x) for x in np.unique(ranks)) - {0}):
        toks = np.nonzero(ranks == r)[0]
        keys = rng_c.random((toks.size, d))
        ch = np.argpartition(keys, r - 1, axis=1)[:, :r] if r < d else np.argsort(keys, axis=1)
        k = rng_k.integers(-7, 8, size=(toks.size, r))
        order = np.argsort((7 - np.abs(k)) * 256 + ch, axis=1, kind="stable")
        ch = np.take_along_axis(ch, order, axis=1)
        k = np.take_along_axis(k, order, axis=1)
        pos = starts[toks][:, None] + np.arange(r)[None, :]
        chans[pos] = ch
        codes[pos] = k
    return chans, codes


def _pack_nibbles(codes: np.ndarray) -> np.ndarray:
    n = codes.size
    u = (codes.astype(np.int16) & 0xF).astype(np.uint8)
    if n % 2:
        u = np.concatenate([u, np.zeros(1, np.uint8)])
    return (u[0::2] | (u[1::2] << 4)).astype(np.uint8)


def generate(w: Workload, layers: tuple | None = None, threads: int | None = None,
             with_q: bool = True) -> CompressedCache:
    """Build the cache of workload ``w``.

    ``layers`` = (start, stop) restricts the cache to whole depth windows
    [start, stop); every draw keeps its absolute layer/window key, so the slice
    equals the same layers of a full generation.
    """
    L0, L1 = (0, w.n_layers) if layers is None else layers
    assert L0 % w.window == 0 and L1 % w.window == 0 and 0 <= L0 < L1 <= w.n_layers
    nL, nM = L1 - L0, (L1 - L0) // w.window
    m0 = L0 // w.window
    B, Hk, Hq, d, rb = w.batch, w.n_kv_heads, w.n_q_heads, w.head_dim, w.basis_rank
    seqlens = w.seqlens()
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(seqlens)
    T = int(cu[-1])
    levels = np.asarray(w.levels, dtype=np.int64)
    threads = threads or min(16, os.cpu_count() or 1)
    pool = ThreadPoolExecutor(threads)

    # routed ranks, shared by the layers of a window and by K and V
    rank_code = np.empty((nM, Hk, T), dtype=np.uint8)
    def _codes(job):
        m, h = job
        for b in range(B):
            rank_code[m, h, cu[b]:cu[b + 1]] = _window_codes(w, b, m0 + m, h, seqlens[b])
    list(pool.map(_codes, [(m, h) for m in range(nM) for h in range(Hk)]))
    res_off = np.zeros((nM, Hk, T + 1), dtype=np.uint32)
    totals = np.zeros((nM, Hk), dtype=np.int64)
    for m in range(nM):
        for h in range(Hk):
            c = np.cumsum(levels[rank_code[m, h]])
            totals[m, h] = c[-1] if T else 0
            assert totals[m, h] < 2**32
            res_off[m, h, 1:] = c
    res_stride = int(-(-(int(totals.max()) + RES_TAIL_PAD) // RES_ALIGN) * RES_ALIGN)

    basis = np.empty((B, nM, Hk, 2, rb, d), dtype=np.float16)
    def _basis(job):
        b, m, h, z = job
        basis[b, m, h, z] = _orthonormal_rows(rng_for(w.seed, _BASIS, b, m0 + m, h, z), rb, d).astype(np.float16)
    list(pool.map(_basis, [(b, m, h, z) for b in range(B) for m in range(nM)
                           for h in range(Hk) for z in range(2)]))

    c8 = getattr(w, "coef_format", "f16") == "int8"
    cdt = np.int8 if c8 else np.float16
    coef_k = np.empty((nL, Hk, T, rb), dtype=cdt)
    coef_v = np.zeros((nL, Hk, padded_tokens(T) // BLOCK, rb, BLOCK), dtype=cdt)
    cs_k = np.empty((nL, Hk, rb // 16, T), dtype=np.float16) if c8 else None
    cs_v = np.empty((nL, Hk, rb // 16, T), dtype=np.float16) if c8 else None
    res_scale = np.empty((nL, 2, Hk, T), dtype=np.float16)
    res_idx = np.zeros((nL, 2, Hk, res_stride), dtype=np.uint8)
    res_val = np.zeros((nL, 2, Hk, res_stride // 2), dtype=np.uint8)

    def _slab(job):
        li, z, h = job
        l = L0 + li
        m = li // w.window
        for b in range(B):
            t0, t1 = int(cu[b]), int(cu[b + 1])
            n = t1 - t0
            if n == 0:
                continue
            if c8:
                rows = (rng_for(w.seed, _COEF8, b, l, z, h).binomial(254, 0.5, size=(n, rb)) - 127).astype(np.int8)
                gs = rng_for(w.seed, _COEF8_SCALE, b, l, z, h)
                if getattr(w, "coef_scale_mode", "narrow") == "wide":
                    lo, hi = (-12.0, 7.0) if z == 1 else (-5.0, -2.0)
                    sc = np.exp2(gs.uniform(lo, hi, size=(rb // 16, n)))
                else:
                    sc = gs.uniform(0.11, 0.14, size=(rb // 16, n))
                (cs_k if z == 0 else cs_v)[li, h, :, t0:t1] = sc.astype(np.float16)
            else:
                g = rng_for(w.seed, _COEF, b, l, z, h)
                rows = g.standard_normal((n, rb), dtype=np.float32).astype(np.float16)
            if z == 0:
                coef_k[li, h, t0:t1] = rows
            else:   # scatter into the token-fastest blocks
                tt = np.arange(t0, t1)
                coef_v[li, h, tt // BLOCK, :, tt % BLOCK] = rows
            res_scale[li, z, h, t0:t1] = _residual_scales(w, rng_for(w.seed, _RES_SCALE, b, l, z, h), z, n)
        # entries of every sequence, packed in token order
        all_ch, all_k = [], []
        for b in range(B):
            t0, t1 = int(cu[b]), int(cu[b + 1])
            ranks = levels[rank_code[m, h, t0:t1]]
            ch, k = _slab_entries(w, b, l, z, h, ranks)
            all_ch.append(ch)
            all_k.append(k)
        ch = np.concatenate(all_ch) if all_ch else np.zeros(0, np.uint8)
        k = np.concatenate(all_k) if all_k else np.zeros(0, np.int8)
        assert ch.size == totals[m, h]
        res_idx[li, z, h, :ch.size] = ch
        packed = _pack_nibbles(k)
        res_val[li, z, h, :packed.size] = packed
    list(pool.map(_slab, [(li, z, h) for li in range(nL) for z in range(2) for h in range(Hk)]))

    q_bits = np.empty((nL, B, Hq, d), dtype=np.uint16)
    if with_q:
        for li in range(nL):
            x = rng_for(w.seed, _Q, L0 + li).standard_normal((B, Hq, d)) / np.sqrt(d)
            q_bits[li] = f16_bits(x) if w.q_dtype == "f16" else f32_to_bf16_bits(x.astype(np.float32))
    pool.shutdown()
    return CompressedCache(
        workload=w, layer0=L0, n_layers=nL, seqlens=list(seqlens), cu_seqlens=cu,
        levels=tuple(int(x) for x in w.levels), res_stride=res_stride, basis=basis,
        coef_k=coef_k, coef_v=coef_v, rank_code=rank_code, res_off=res_off, res_idx=res_idx,
        res_val=res_val, res_scale=res_scale, q_bits=q_bits, q_dtype=w.q_dtype,
        coef_format="int8" if c8 else "f16", coef_scale_k=cs_k, coef_scale_v=cs_v)


def router_inputs(w: Workload, n_windows: int, T: int, window0: int = 0):
    """Router features phi [M][Hkv][T][4] (float32), router weights u [M][4] and
    ascending thresholds theta [M][n_levels-1] (float32), seeded.

    Features: attention mass and spike (non-negative, heavy tailed), a 0/1
    delimiter flag and the previous probe error; thresholds are spread so every
    level is reached."""
    Hk = w.n_kv_heads
    n_lev = len(w.levels)
    phi = np.empty((n_windows, Hk, T, 4), dtype=np.float32)
    u = np.empty((n_windows, 4), dtype=np.float32)
    theta = np.empty((n_windows, max(n_lev - 1, 0)), dtype=np.float32)
    for m in range(n_windows):
        g = rng_for(w.seed, _ROUTER_U, window0 + m)
        u[m] = g.uniform(0.25, 1.5, size=4).astype(np.float32)
        theta[m] = np.sort(g.uniform(0.5, 4.0, size=n_lev - 1)).astype(np.float32)
        for h in range(Hk):
            r = rng_for(w.seed, _PHI, window0 + m, h)
            phi[m, h, :, 0] = r.exponential(1.0, size=T)
            phi[m, h, :, 1] = r.exponential(0.5, size=T)
            phi[m, h, :, 2] = (r.random(T) < 0.05)
            phi[m, h, :, 3] = r.uniform(0.0, 0.2, size=T)
    return phi, u, theta
