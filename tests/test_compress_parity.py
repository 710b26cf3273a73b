"""Append/compress (Sec. 3, the storage half of Eq. 1) and range routing on
the GPU through the C ABI, against the oracle bit for bit.

Every array the call writes (coefficient rows in both layouts, residual
channel bytes, packed int4 codes, gate-folded scales) must equal the oracle's
exactly, and nothing outside the compressed tokens may change.  Cases: the
decode-token append [T-1, T) and a multi-token tail append (routed with
dwkv_route_range, then compressed), a whole-layer prefill, a range across
sequences with empty ones and per-token gates, full-rank residuals, basis
ranks 16..128, inputs exactly in the basis span (zero residual, scale 0) and
exact |r| ties; then the decode over the appended cache matches the float64
decode of the oracle's cache, and the layout validator accepts it.  The
64K-token workload shape compresses a whole layer in the benchmark's launch
configuration and is checked on sampled tokens."""
import copy

import numpy as np
import pytest

import oracle
import oracle.compress as OC
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate, router_inputs

pytestmark = pytest.mark.gpu


class _Fixed:
    """Workload wrapper with explicit per-sequence lengths."""
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        if k.startswith("_"):              # copying makes the object before its fields
            raise AttributeError(k)
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


WRITTEN = ("coef_k", "coef_v", "res_idx", "res_val", "res_scale")


WRITTEN_I8 = ("coef_k", "coef_v", "coef_scale_k", "coef_scale_v", "res_idx", "res_val", "res_scale")


def _host_arrays(dc):
    keys, values = dc.coef_host()       # back from the ABI's tiled layouts
    if dc.coef_format == "int8":
        extra = {"coef_k": keys.view(np.int8), "coef_v": values.view(np.int8),
                 "coef_scale_k": dc.coef_scale_k.cpu().numpy().view(np.float16),
                 "coef_scale_v": dc.coef_scale_v.cpu().numpy().view(np.float16)}
    else:
        extra = {"coef_k": keys.view(np.float16), "coef_v": values.view(np.float16)}
    return {
        **extra,
        "res_idx": dc.res_idx.cpu().numpy(),
        "res_val": dc.res_val.cpu().numpy(),
        "res_scale": dc.res_scale.cpu().numpy().view(np.float16),
        "rank_code": dc.rank_code.cpu().numpy(),
        "res_off": dc.res_off.cpu().numpy().view(np.uint32),
    }


def _assert_same(got, host, names, label):
    for name in names:
        want = getattr(host, name)
        g = got[name].reshape(want.shape)
        if not np.array_equal(g.view(np.uint8), np.ascontiguousarray(want).view(np.uint8)):
            diff = np.argwhere(g.view(np.uint8).reshape(-1) != np.ascontiguousarray(want).view(np.uint8).reshape(-1))
            raise AssertionError(f"{label}: {name} differs from the oracle at byte(s) {diff[:5].ravel()}")


def _inputs(host, layer, t0, t1, kind, rng):
    """Dense fp16 keys / values [t1-t0, Hkv, d] of the tokens."""
    Hk, d = host.n_kv_heads, host.head_dim
    n = t1 - t0
    if kind == "normal":
        return [rng.standard_normal((n, Hk, d)).astype(np.float16) for _ in range(2)]
    if kind == "near-cache":             # the cache's own rebuilt vectors plus a small deviation
        out = []
        for z in range(2):
            x = np.zeros((n, Hk, d))
            for h in range(Hk):
                for b in range(host.batch):
                    s0, s1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
                    a, e = max(s0, t0), min(s1, t1)
                    if e > a:
                        X = oracle.reconstruct(host, layer, z, h, b)
                        x[a - t0:e - t0, h] = X[a - s0:e - s0]
            out.append((x + 0.05 * rng.standard_normal(x.shape)).astype(np.float16))
        return out
    raise ValueError(kind)


def _perm_basis(host, rng):
    """Signed-permutation basis rows (exactly orthonormal in fp16)."""
    rb, d = host.basis_rank, host.head_dim
    for idx in np.ndindex(*host.basis.shape[:4]):
        perm = rng.permutation(d)[:rb]
        B = np.zeros((rb, d), np.float16)
        B[np.arange(rb), perm] = rng.choice([-1.0, 1.0], size=rb)
        host.basis[idx] = B


def _room_for_routing(host, routing, t0, t1):
    """Widen res_stride when the new routing of [t0, t1) needs more entries than
    the synthetic cache reserved (padding only; entries keep their positions)."""
    phi, u, theta = routing
    codes, off = host.rank_code.copy(), host.res_off.copy()
    oracle.route_range(phi, u, theta, host.levels, t0, t1, codes, off)
    need = int(off[..., -1].max()) + 512
    if need > host.res_stride:
        new = -(-need // 256) * 256
        pad = new - host.res_stride
        host.res_idx = np.pad(host.res_idx, [(0, 0)] * 3 + [(0, pad)])
        host.res_val = np.pad(host.res_val, [(0, 0)] * 3 + [(0, pad // 2)])
        host.res_stride = new


def _run_case(host, dc, layers, t0, t1, xs, gates, routing=None, label=""):
    """Optionally route [t0, t1), then compress it in every listed layer on both
    sides and compare every array.  Returns the oracle's updated cache."""
    torch = torch_gpu()
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ref = copy.deepcopy(host)
    if routing is not None:
        phi, u, theta = routing
        announce(f"route_range {label} [{t0},{t1})")
        dc.route_range(dev(phi), dev(u), dev(theta), t0, t1)
        oracle.route_range(phi, u, theta, ref.levels, t0, t1, ref.rank_code, ref.res_off)
        _assert_same(_host_arrays(dc), ref, ("rank_code", "res_off"), label + " routing")
    for layer, (xk, xv), gate in zip(layers, xs, gates):
        announce(f"compress {label} layer={layer} [{t0},{t1})")
        dc.compress(layer, dev(xk), dev(xv), t0, t1, gate=None if gate is None else dev(gate))
        torch.cuda.synchronize()
        OC.compress(ref, layer, xk, xv, t0, t1, gate)
    written = WRITTEN_I8 if getattr(host, "coef_format", "f16") == "int8" else WRITTEN
    _assert_same(_host_arrays(dc), ref, written + ("rank_code", "res_off"), label)
    announce(f"validate {label}")
    ok, bad = dc.validate()
    assert ok, f"{label}: the validator rejects the compressed cache at {bad}"
    return ref


CASES = [
    # name, r_b, levels, probs, lengths, layer, range, gate, x, route
    ("rb32-decode-token-append", 32, (0, 8, 16), (0.2, 0.4, 0.4), [4096], 1, "last", False, "near-cache", True),
    ("rb48-tail-append-100", 48, (0, 4, 8, 16), (0.25, 0.25, 0.25, 0.25), [700, 1500], 3, "tail100", True,
     "normal", True),
    ("rb48-across-seqs-gated", 48, (0, 4, 8, 16), (0.25, 0.25, 0.25, 0.25), [0, 129, 700, 0, 300], 2,
     (100, 1100), True, "normal", False),
    ("rb64-full-rank", 64, (0, 2, 128), (0.3, 0.3, 0.4), [257, 70], 0, "all", True, "normal", True),
    ("rb128-prefill", 128, (0, 16, 32), (0.4, 0.3, 0.3), [1000], 1, "all", False, "near-cache", True),
    ("rb16-one-level", 16, (8,), (1.0,), [63, 65], 0, "all", False, "normal", False),
    ("rb80-rank-zero-only", 80, (0,), (1.0,), [333], 1, (5, 300), True, "normal", False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_compress_bit_exact(case):
    """A routed case re-routes [t0, t1) in every window and compresses it in
    every layer (the append of a real decode step); an unrouted one
    recompresses existing tokens of one layer under their stored routing."""
    torch = torch_gpu()
    name, rb, levels, probs, lengths, layer, rng_spec, use_gate, xkind, route = case
    w = _Fixed(Workload(name=name, batch=len(lengths), n_layers=4, window=2, n_kv_heads=2, n_q_heads=8,
                        head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                        q_dtype="bf16", seed=300 + len(name)), lengths)
    host = generate(w, threads=4)
    T = host.total_tokens
    t0, t1 = {"last": (T - 1, T), "tail100": (T - 100, T), "all": (0, T)}.get(rng_spec, rng_spec)
    rng = np.random.default_rng(7 + len(name))
    routing = None
    layers = [layer]
    if route:                            # routing covers every window: compress every layer
        routing = router_inputs(w, host.n_windows, T)
        _room_for_routing(host, routing, t0, t1)
        layers = list(range(host.n_layers))
    xs = [_inputs(host, l, t0, t1, xkind, rng) for l in layers]
    gates = [rng.uniform(0.0, 1.0, size=(2, host.n_kv_heads, t1 - t0)).astype(np.float32) if use_gate else None
             for _ in layers]
    dc = device_cache(host)
    ref = _run_case(host, dc, layers, t0, t1, xs, gates, routing, name)
    # the decode over the appended cache against the float64 decode of the oracle's cache
    pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
    for l in layers:
        announce(f"decode after compress {name} layer={l}")
        out = dc.decode(l).cpu().numpy()
        torch.cuda.synchronize()
        compare(out, oracle.decode(ref, l), pairs, host.n_q_heads // host.n_kv_heads, f"{name} decode l={l}")


I8_CASES = [
    # name, r_b, levels, probs, lengths, layer, range, gate, x, route, decode afterwards
    ("i8-rb48-decode-token-append", 48, (0, 4, 8, 16), (0.25, 0.25, 0.25, 0.25), [2048], 1, "last", False,
     "near-cache", True, True),
    ("i8-rb32-across-seqs-gated", 32, (0, 8, 16), (0.3, 0.4, 0.3), [0, 129, 700, 0, 300], 2, (100, 1100), True,
     "normal", False, True),
    ("i8-rb64-prefill", 64, (0, 4, 8, 16), (0.4, 0.3, 0.2, 0.1), [1000], 3, "all", False, "near-cache", True,
     True),
    ("i8-rb16-tail", 16, (0, 2), (0.5, 0.5), [63, 65], 0, "tail100", False, "normal", True, True),
    ("i8-rb128-compress-only", 128, (0, 16, 32), (0.4, 0.3, 0.3), [500], 1, "all", True, "normal", False, False),
]


@pytest.mark.parametrize("case", I8_CASES, ids=[c[0] for c in I8_CASES])
def test_compress_int8_bit_exact(case):
    """dwkv_compress writing the 8-bit blockwise coefficient form (reading C7):
    codes, block scales, residual channels, codes and scales equal the
    oracle's byte for byte; then the int8 decode over the written cache matches
    the float64 decode of the oracle's cache (r_b above 64 is encoded only: the
    int8 decode serves r_b up to 64)."""
    torch = torch_gpu()
    name, rb, levels, probs, lengths, layer, rng_spec, use_gate, xkind, route, decode = case
    w = _Fixed(Workload(name=name, batch=len(lengths), n_layers=4, window=2, n_kv_heads=2, n_q_heads=8,
                        head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                        q_dtype="bf16", seed=500 + len(name), coef_format="int8"), lengths)
    host = generate(w, threads=4)
    T = host.total_tokens
    t0, t1 = {"last": (T - 1, T), "tail100": (T - 100, T), "all": (0, T)}.get(rng_spec, rng_spec)
    rng = np.random.default_rng(9 + len(name))
    routing = None
    layers = [layer]
    if route:
        routing = router_inputs(w, host.n_windows, T)
        _room_for_routing(host, routing, t0, t1)
        layers = list(range(host.n_layers))
    xs = [_inputs(host, l, t0, t1, xkind, rng) for l in layers]
    gates = [rng.uniform(0.0, 1.0, size=(2, host.n_kv_heads, t1 - t0)).astype(np.float32) if use_gate else None
             for _ in layers]
    dc = device_cache(host)
    ref = _run_case(host, dc, layers, t0, t1, xs, gates, routing, name)
    if decode:
        pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
        for l in layers:
            announce(f"int8 decode after compress {name} layer={l}")
            out = dc.decode(l).cpu().numpy()
            torch.cuda.synchronize()
            compare(out, oracle.decode(ref, l), pairs, host.n_q_heads // host.n_kv_heads, f"{name} decode l={l}")


def test_compress_zero_residual_and_ties():
    """Signed-permutation bases: inputs on the basis channels leave r = 0 exactly
    (scale 0, codes 0, channels 0..rho-1 by the tie rule); inputs with repeated
    magnitudes off the basis produce exact |r| ties."""
    torch_gpu()
    w = _Fixed(Workload(name="perm", batch=2, n_layers=2, window=2, n_kv_heads=2, n_q_heads=4, head_dim=128,
                        context=200, basis_rank=32, levels=(4, 16, 128), probs=(0.3, 0.3, 0.4), q_dtype="f16",
                        seed=77), [200, 90])
    host = generate(w, threads=4)
    rng = np.random.default_rng(5)
    _perm_basis(host, rng)
    T, Hk, d = host.total_tokens, host.n_kv_heads, host.head_dim
    xs = []
    for z in range(2):
        x = np.zeros((T, Hk, d), np.float16)
        for t in range(T):
            b = 0 if t < 200 else 1
            for h in range(Hk):
                B = host.basis[b, 0, h, z].astype(np.float32)
                on = np.nonzero(np.abs(B).sum(axis=0))[0]
                if t % 2 == 0:            # in the span: zero residual
                    x[t, h, on] = rng.standard_normal(on.size)
                else:                     # few distinct magnitudes: many exact ties
                    x[t, h] = rng.choice([-0.5, 0.5, 0.25, -1.0, 1.0], size=d)
        xs.append(x)
    dc = device_cache(host)
    ref = _run_case(host, dc, [1], 0, T, [(xs[0], xs[1])], [None], None, "perm-basis")
    m = 0
    for t in range(0, T, 2):
        assert float(ref.res_scale[1, 0, 0, t]) == 0.0
    lev = np.asarray(host.levels)
    t = 0
    rho = int(lev[host.rank_code[m, 0, t]])
    e0 = int(host.res_off[m, 0, t])
    assert list(ref.res_idx[1, 0, 0, e0:e0 + rho]) == list(range(rho)), "zero residual must keep channels 0.."


def test_compress_full_size_sampled():
    """The 64K-token shape (r_b 48, 8 KV heads): a whole-layer compress in one
    launch, sampled tokens against the oracle bit for bit, then the validator."""
    torch = torch_gpu()
    host = generate(LLAMA8B_64K, layers=(0, 4), with_q=False)
    T, Hk, d = host.total_tokens, host.n_kv_heads, host.head_dim
    rng = np.random.default_rng(64)
    layer, m = 2, 0
    xk = rng.standard_normal((T, Hk, d)).astype(np.float16)
    xv = rng.standard_normal((T, Hk, d)).astype(np.float16)
    dc = device_cache(host)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    announce(f"compress 64k layer={layer} T={T}")
    dc.compress(layer, dev(xk), dev(xv), 0, T)
    torch.cuda.synchronize()
    got = _host_arrays(dc)
    coef_k = got["coef_k"].reshape(host.coef_k.shape)
    coef_v = got["coef_v"].reshape(host.coef_v.shape)
    res_idx = got["res_idx"].reshape(host.res_idx.shape)
    res_val = got["res_val"].reshape(host.res_val.shape)
    res_scale = got["res_scale"].reshape(host.res_scale.shape)
    lev = np.asarray(host.levels)
    toks = np.concatenate([[0, 1, 15, 16, T - 2, T - 1], rng.choice(T, size=120, replace=False)])
    for z, X in ((0, xk), (1, xv)):
        for h in range(Hk):
            B = host.basis[0, m, h, z]
            rhos = lev[host.rank_code[m, h, toks]]
            a16, entries, scales = OC.compress_vectors(X[toks, h], B, rhos)
            for j, t in enumerate(toks):
                row = coef_k[layer, h, t] if z == 0 else coef_v[layer, h, t // 16, :, t % 16]
                assert np.array_equal(row.view(np.uint16), a16[j].view(np.uint16)), f"coef z={z} h={h} t={t}"
                assert res_scale[layer, z, h, t].view(np.uint16) == scales[j].view(np.uint16), f"scale t={t}"
                e0 = int(host.res_off[m, h, t])
                ch, codes = entries[j]
                assert list(res_idx[layer, z, h, e0:e0 + len(ch)]) == list(ch), f"channels z={z} h={h} t={t}"
                got_codes = oracle.entry_codes(res_val[layer, z, h], e0, len(ch))
                assert list(got_codes) == list(codes), f"codes z={z} h={h} t={t}"
    for name, arr in (("coef_k", coef_k), ("res_idx", res_idx), ("res_scale", res_scale)):
        other = [l for l in range(host.n_layers) if l != layer]
        assert np.array_equal(arr[other], getattr(host, name)[other]), f"{name} of another layer changed"
    announce("validate 64k")
    ok, bad = dc.validate()
    assert ok, f"validator rejects the compressed 64K layer at {bad}"
