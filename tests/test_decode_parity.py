"""GPU decode (through the C ABI) against the float64 oracle, element by element.

Small shapes cover every compiled basis rank and group size, ragged lengths
with partial tiles, empty sequences, several split sizes, many-entry tiles
(more than one staged entry chunk) and the no-residual path; the workload
shapes run at their full per-layer size on one depth window, in the launch
configuration the benchmark uses, on sampled (sequence, KV head) outputs."""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import (BATCH16, LLAMA70B_128K, LLAMA8B_32K, LLAMA8B_64K, TINY, Workload, generate)

pytestmark = pytest.mark.gpu


class _Fixed:
    """Workload wrapper with explicit per-sequence lengths."""
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


SMALL = [
    # name, r_b, G, levels, probs, lengths, split, q dtype
    ("rb16-g1-tails", 16, 1, (0, 2), (0.6, 0.4), [1, 63, 65, 300], 64, "bf16"),
    ("rb32-g4-tiny-shape", 32, 4, (0, 8, 16), (0.8, 0.15, 0.05), [4096], 0, "f16"),
    ("rb48-g2-empty-seq", 48, 2, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [0, 129, 700], 128, "bf16"),
    ("rb64-g8-five-levels", 64, 8, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [1000, 2048], 0, "bf16"),
    ("rb80-g16-short-tiles", 80, 16, (0, 8), (0.5, 0.5), [333], 64, "f16"),
    ("rb96-g1-no-residual", 96, 1, (0,), (1.0,), [500, 37], 128, "bf16"),
    ("rb112-g2", 112, 2, (0, 2, 6), (0.3, 0.3, 0.4), [777], 256, "bf16"),
    ("rb128-g4-full-rank-residual", 128, 4, (0, 128), (0.5, 0.5), [257, 70], 128, "bf16"),
    ("rb32-g16-many-entries", 32, 16, (32, 64), (0.5, 0.5), [200, 4097], 0, "bf16"),
    # token-lane kernel: ~900 entries per 64-token tile (past the preloaded batches)
    ("rb64-g4-entry-heavy", 64, 4, (0, 16), (0.1, 0.9), [1500, 64], 256, "bf16"),
    # token-lane kernel, more sequences than the kernel-argument work table holds
    ("rb32-g4-20-seqs", 32, 4, (0, 8), (0.7, 0.3), [37 + 23 * i for i in range(20)], 64, "bf16"),
    # token-lane merge over more chunks than one load round covers (79 and 47 partials)
    ("rb48-g4-many-chunks", 48, 4, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [5000, 37], 64, "bf16"),
    ("rb64-g2-many-chunks", 64, 2, (0, 8, 16), (0.8, 0.15, 0.05), [3000], 64, "f16"),
    # token-lane kernel, groups of 8 heads (ranks to 32): ragged tails, empty
    # sequences, every basis rank, rank-32-heavy tiles (past the preloaded
    # value-entry batches and up to the 2048-entry map), and many chunks
    ("rb32-g8-tails", 32, 8, (0, 2, 4, 8, 16, 32), (0.4, 0.2, 0.15, 0.1, 0.1, 0.05), [1, 63, 65, 300, 0], 64, "f16"),
    ("rb16-g8", 16, 8, (0, 8), (0.5, 0.5), [777], 128, "bf16"),
    ("rb48-g8-five-levels", 48, 8, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [2000, 33], 0, "bf16"),
    ("rb64-g8-rank32-heavy", 64, 8, (0, 32), (0.1, 0.9), [1500, 64], 256, "bf16"),
    ("rb64-g8-many-chunks", 64, 8, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [5000, 37], 64, "bf16"),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_shapes_all_outputs(case):
    torch = torch_gpu()
    name, rb, G, levels, probs, lengths, split, qd = case
    base = Workload(name=name, batch=len(lengths), n_layers=2, window=2, n_kv_heads=2,
                    n_q_heads=2 * G, head_dim=128, context=max(lengths), basis_rank=rb,
                    levels=levels, probs=probs, q_dtype=qd, seed=100 + len(name))
    w = _Fixed(base, lengths)
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=split)
    pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
    for layer in range(host.n_layers):
        announce(f"decode {name} layer={layer} split={dc.split_tokens}")
        out = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        ref = oracle.decode(host, layer)
        compare(out, ref, pairs, G, f"{name} layer {layer}")
        for b, L in enumerate(lengths):
            if L == 0:
                assert np.all(out[b] == 0), "empty sequence must give zeros"


def test_tiny_workload_all_layers():
    torch_gpu()
    host = generate(TINY, threads=4)
    dc = device_cache(host)
    pairs = [(0, h) for h in range(host.n_kv_heads)]
    for layer in range(host.n_layers):
        announce(f"decode tiny layer={layer}")
        compare(dc.decode(layer).cpu().numpy(), oracle.decode(host, layer), pairs, host.n_q_heads // host.n_kv_heads,
                f"tiny layer {layer}")


def _needles(host, layer, n_needles, seed, scale_q=1.0):
    """Plant tokens whose key coefficients point along the query's basis
    projection, so a handful of tokens own most of the softmax mass (exercises
    running-max updates late in a split and across splits)."""
    rng = np.random.default_rng(seed)
    m = layer // host.window
    G = host.n_q_heads // host.n_kv_heads
    q = oracle.q_to_f64(host.q_bits[layer], host.q_dtype) * scale_q
    for b in range(host.batch):
        t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
        if t1 - t0 < 2:
            continue
        for h in range(host.n_kv_heads):
            qt = host.basis[b, m, h, 0].astype(np.float64) @ q[b, h * G]
            dirn = qt / np.linalg.norm(qt)
            lam = (np.log(t1 - t0) + 3.0) / (np.linalg.norm(qt) / np.sqrt(host.head_dim))
            for t in rng.choice(np.arange(t0, t1), size=min(n_needles, t1 - t0), replace=False):
                host.coef_k[layer, h, t] = (lam * dirn).astype(np.float16)


@pytest.mark.parametrize("G", [4, 8])
def test_needles_and_peaked_queries(G):
    torch = torch_gpu()
    w = _Fixed(Workload(name="needles", batch=2, n_layers=2, window=2, n_kv_heads=2, n_q_heads=2 * G,
                        head_dim=128, context=9000, basis_rank=48, levels=(0, 4, 8, 16),
                        probs=(0.75, 0.12, 0.08, 0.05), q_dtype="bf16", seed=77), [9000, 5000])
    host = generate(w, threads=4)
    _needles(host, 0, 4, seed=5)
    dc = device_cache(host, split_tokens=512)
    pairs = [(b, h) for b in range(2) for h in range(2)]
    announce(f"decode needles G={G} layer 0")
    out = dc.decode(0).cpu().numpy()
    ref, probs = oracle.decode(host, 0, with_probs=True)
    top = max(p.max() for p in probs.values())
    assert top > 0.1, f"needle setup did not concentrate the softmax (max p {top:.3f})"
    compare(out, ref, pairs, G, f"needles G={G}")
    # peaked: query scaled by 32 (bf16 scaling by a power of two is exact)
    q = dc.q[1].float() * 32
    q = q.to(torch.bfloat16)
    announce(f"decode peaked G={G} layer 1")
    out = dc.decode(1, q=q).cpu().numpy()
    ref = oracle.decode(host, 1, q=oracle.q_to_f64(host.q_bits[1], "bf16") * 32)
    compare(out, ref, pairs, G, f"peaked q x32 G={G}")


def test_softmax_scale_argument():
    torch_gpu()
    host = generate(TINY, threads=4)
    dc = device_cache(host)
    announce("decode tiny sm_scale=0.37")
    out = dc.decode(1, sm_scale=0.37).cpu().numpy()
    compare(out, oracle.decode(host, 1, sm_scale=0.37), [(0, 0), (0, 1)], 4, "sm_scale 0.37")


FULL = [
    # workload, window start layer, sampled (b, kv head) pairs
    (LLAMA8B_32K, 6, [(0, 0), (0, 5)]),
    (LLAMA8B_64K, 4, [(0, 1), (0, 7)]),
    (BATCH16, 2, [(0, 0), (7, 3), (15, 6)]),
    (LLAMA70B_128K, 8, [(0, 2), (1, 7)]),
]


@pytest.mark.parametrize("wl,layer0,pairs", FULL, ids=[f[0].name for f in FULL])
def test_workload_full_size_sampled(wl, layer0, pairs):
    torch_gpu()
    announce(f"generate {wl.name} layers [{layer0}, {layer0 + wl.window})")
    host = generate(wl, layers=(layer0, layer0 + wl.window))
    dc = device_cache(host)
    G = wl.group
    for li in (0, wl.window - 1):
        announce(f"decode {wl.name} layer={layer0 + li} split={dc.split_tokens}")
        out = dc.decode(li).cpu().numpy()
        ref = oracle.decode(host, li, heads=pairs)
        compare(out, ref, pairs, G, f"{wl.name} layer {layer0 + li}")


def test_determinism_and_split_invariance():
    torch_gpu()
    host = generate(LLAMA8B_64K.with_(context=20000), layers=(0, 4))
    dc = device_cache(host)
    announce("determinism: two runs, auto split")
    a = dc.decode(2).cpu().numpy()
    b = dc.decode(2).cpu().numpy()
    assert np.array_equal(a, b), "two runs with the same plan differ"
    outs = {}
    for split in (256, 1024, 4096, 20480):
        dc.set_split(split)
        announce(f"split {split}")
        outs[split] = dc.decode(2).cpu().numpy()
    ref = oracle.decode(host, 2, heads=[(0, 0), (0, 3)])
    for split, o in outs.items():
        compare(o, ref, [(0, 0), (0, 3)], 4, f"split {split}")


def test_two_phase_calls_equal_decode():
    """dwkv_decode_partials + dwkv_decode_merge give dwkv_decode's output bit for bit."""
    torch_gpu()
    host = generate(BATCH16.with_(n_layers=2), layers=(0, 2))
    dc = device_cache(host)
    announce("two-phase decode batch16 layer 1")
    full = dc.decode(1).cpu().numpy()
    dc.decode_partials(1)
    two = dc.decode_merge(1).cpu().numpy()
    assert np.array_equal(full, two)
