"""The comparison paths on the GPU through the C ABI: the rebuilt cache written
out (dwkv_materialize, Eq. 1 with one fp16 rounding) against the oracle's
explicit Eq. 1 rebuild; decode attention over a dense fp16 cache
(dwkv_dense_decode) against softmax attention in float64 on the same fp16
data; and the unfused path (materialize, then dense decode) against the
oracle's factorized decode."""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate
from synth.layout import unblock_values

pytestmark = pytest.mark.gpu


class _Fixed:
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        if k.startswith("_"):
            raise AttributeError(k)
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


CASES = [
    # name, r_b, G, levels, probs, lengths
    ("rb16-g1-tails", 16, 1, (0, 2), (0.6, 0.4), [1, 63, 65, 300]),
    ("rb48-g4-empty-seqs", 48, 4, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [0, 129, 700, 0, 37]),
    ("rb64-g8-rank32", 64, 8, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [1000, 517]),
    ("rb128-g2-full-rank", 128, 2, (0, 128), (0.5, 0.5), [257, 70]),
    ("rb80-g16-no-residual", 80, 16, (0,), (1.0,), [333]),
]


def _small(case):
    name, rb, G, levels, probs, lengths = case
    w = _Fixed(Workload(name=name, batch=len(lengths), n_layers=2, window=2, n_kv_heads=2, n_q_heads=2 * G,
                        head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                        q_dtype="bf16", seed=500 + len(name)), lengths)
    return generate(w, threads=4)


def _abs_terms(host, layer, z, h, b):
    """Per-element sum of the magnitudes of the Eq. 1 terms (float64 [T_b, d]):
    the scale of the float32 accumulation error."""
    m = layer // host.window
    t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
    A = oracle.factorized.coefficient_rows(host, layer, z, h, t0, t1)
    B = host.basis[b, m, h, z].astype(np.float64)
    R = oracle.residual_map(host, layer, z, h, t0, t1)
    return np.abs(A) @ np.abs(B) + np.abs(R)


def _check_materialized(host, dc, layer, label):
    announce(f"materialize {label} layer={layer}")
    k_dev, v_dev = dc.materialize(layer)
    k = k_dev.cpu().numpy().astype(np.float64)
    v_blocks = v_dev.cpu().numpy()
    T = host.total_tokens
    T16 = -(-T // 16) * 16
    assert np.all(v_blocks.reshape(host.n_kv_heads, T16 // 16, host.head_dim, 16)
                  .swapaxes(-1, -2).reshape(host.n_kv_heads, T16, host.head_dim)[:, T:] == 0), "value padding not zero"
    vv = unblock_values(v_blocks, T).astype(np.float64)
    worst = 0.0
    for z, X in ((0, k), (1, vv)):
        for h in range(host.n_kv_heads):
            for b in range(host.batch):
                t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
                if t1 == t0:
                    continue
                ref = oracle.reconstruct(host, layer, z, h, b)
                got = X[h, t0:t1]
                # one fp16 rounding of the float32 sum: half an fp16 ulp of the
                # value, plus the float32 accumulation error, plus fp16's
                # smallest step
                tol = np.abs(ref) * 2.0 ** -11 + _abs_terms(host, layer, z, h, b) * 2.0 ** -21 + 2.0 ** -24
                excess = np.abs(got - ref) / tol
                worst = max(worst, float(excess.max()))
                assert np.all(excess <= 1.0), (f"{label}: z={z} h={h} b={b}: materialized value off by "
                                               f"{excess.max():.2f} x its bound")
    print(f"[parity] {label} materialize: worst error {worst:.3f} of the bound", flush=True)
    return k_dev, v_dev


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_materialize_and_unfused(case):
    torch = torch_gpu()
    host = _small(case)
    dc = device_cache(host)
    G = host.n_q_heads // host.n_kv_heads
    pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
    for layer in range(host.n_layers):
        k, v = _check_materialized(host, dc, layer, case[0])
        # dense decode over the materialized cache: against float64 attention
        # on the same fp16 keys / values ...
        announce(f"dense decode {case[0]} layer={layer}")
        q = dc.q[layer]
        out = dc.dense_decode(k, v, q).cpu().numpy()
        torch.cuda.synchronize()
        qf = oracle.q_to_f64(host.q_bits[layer], host.q_dtype)
        kk = k.cpu().numpy().astype(np.float64)
        vv = unblock_values(v.cpu().numpy(), host.total_tokens).astype(np.float64)
        ref = np.zeros_like(out, dtype=np.float64)
        for b, h in pairs:
            t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
            o, _ = oracle.attention(qf[b, h * G:(h + 1) * G], kk[h, t0:t1], vv[h, t0:t1],
                                    oracle.default_scale(host.head_dim))
            ref[b, h * G:(h + 1) * G] = o
        compare(out, ref, pairs, G, f"{case[0]} dense l={layer}")
        # ... and the unfused path against the oracle's factorized decode
        compare(out, oracle.decode(host, layer), pairs, G, f"{case[0]} unfused vs factorized l={layer}",
                regression=None)
        for b in range(host.batch):
            if host.cu_seqlens[b + 1] == host.cu_seqlens[b]:
                assert np.all(out[b] == 0), "empty sequence must give zeros"


def test_dense_decode_random_cache():
    """A dense fp16 cache that is not a rebuilt one (N(0,1) keys and values)."""
    torch = torch_gpu()
    host = _small(CASES[1])
    dc = device_cache(host)
    rng = np.random.default_rng(9)
    Hk, T, d = host.n_kv_heads, host.total_tokens, host.head_dim
    T16 = -(-T // 16) * 16
    kk = rng.standard_normal((Hk, T, d)).astype(np.float16)
    vrows = np.zeros((Hk, T16, d), np.float16)
    vrows[:, :T] = rng.standard_normal((Hk, T, d)).astype(np.float16)
    vb = np.ascontiguousarray(vrows.reshape(Hk, T16 // 16, 16, d).swapaxes(-1, -2))
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    q = dc.q[0]
    announce("dense decode random cache")
    out = dc.dense_decode(dev(kk), dev(vb), q).cpu().numpy()
    torch.cuda.synchronize()
    G = host.n_q_heads // Hk
    qf = oracle.q_to_f64(host.q_bits[0], host.q_dtype)
    pairs = [(b, h) for b in range(host.batch) for h in range(Hk)]
    ref = np.zeros(out.shape)
    for b, h in pairs:
        t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
        ref[b, h * G:(h + 1) * G], _ = oracle.attention(qf[b, h * G:(h + 1) * G], kk[h, t0:t1].astype(np.float64),
                                                        vrows[h, t0:t1].astype(np.float64), 1.0 / np.sqrt(d))
    compare(out, ref, pairs, G, "dense random")


def test_unfused_full_size_sampled():
    """The 64K-token shape: materialize one layer, dense decode over it, sampled
    (KV head) outputs against the oracle's factorized decode."""
    torch = torch_gpu()
    host = generate(LLAMA8B_64K, layers=(28, 32))
    dc = device_cache(host)
    layer = 1
    announce("materialize 64k")
    k, v = dc.materialize(layer)
    announce("dense decode 64k")
    out = dc.dense_decode(k, v, dc.q[layer]).cpu().numpy()
    torch.cuda.synchronize()
    pairs = [(0, 0), (0, 5)]
    G = host.n_q_heads // host.n_kv_heads
    ref = oracle.decode(host, layer, heads=pairs)
    compare(out, ref, pairs, G, "unfused 64k", regression=None)
