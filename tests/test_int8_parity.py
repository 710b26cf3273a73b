"""Decode over the 8-bit blockwise coefficient form (dwkv_decode with int8
codes and per-block fp16 scales) on the GPU against the float64 oracle, which
rebuilds A = code * scale explicitly: every token-lane basis rank and group
size, ragged lengths with partial tiles, empty sequences, several splits, the
no-residual path, and the 64K-token shape on sampled heads.  The call that
rebuilds fp16 rows (materialize) refuses the format; compress writes it
(tests/test_compress_parity.py)."""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate

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
    # name, r_b, G, levels, probs, lengths, split
    ("i8-rb16-g1-tails", 16, 1, (0, 2), (0.6, 0.4), [1, 63, 65, 300], 64),
    ("i8-rb32-g4", 32, 4, (0, 8, 16), (0.8, 0.15, 0.05), [4096], 0),
    ("i8-rb48-g2-empty-seq", 48, 2, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [0, 129, 700], 128),
    ("i8-rb64-g4-entry-heavy", 64, 4, (0, 16), (0.1, 0.9), [1500, 64], 256),
    ("i8-rb48-g4-no-residual", 48, 4, (0,), (1.0,), [2000, 37], 0),
    ("i8-rb48-g4-many-chunks", 48, 4, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [5000, 37], 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_int8_small_shapes(case):
    torch = torch_gpu()
    name, rb, G, levels, probs, lengths, split = case
    w = _Fixed(Workload(name=name, batch=len(lengths), n_layers=2, window=2, n_kv_heads=2, n_q_heads=2 * G,
                        head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                        q_dtype="bf16", seed=900 + len(name), coef_format="int8"), lengths)
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=split)
    pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
    for layer in range(host.n_layers):
        announce(f"int8 decode {name} layer={layer}")
        out = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        compare(out, oracle.decode(host, layer), pairs, G, f"{name} layer {layer}")
        for b, L in enumerate(lengths):
            if L == 0:
                assert np.all(out[b] == 0)


def test_int8_refused_where_unsupported():
    torch = torch_gpu()
    from paper_2607_06523_amd import DwkvError
    w = Workload(name="i8-refuse", batch=1, n_layers=2, window=2, n_kv_heads=2, n_q_heads=16, head_dim=128,
                 context=300, basis_rank=32, levels=(0, 8), probs=(0.5, 0.5), q_dtype="bf16", seed=3,
                 coef_format="int8")
    host = generate(w, threads=4)
    dc = device_cache(host)                    # int8 is built for groups of up to 4 heads
    with pytest.raises(DwkvError) as e:
        dc.decode(0)
    assert e.value.status == 3
    w4 = w.with_(n_q_heads=8)
    dc4 = device_cache(generate(w4, threads=4))
    with pytest.raises(DwkvError) as e:        # the rebuild writes fp16 rows
        dc4.materialize(0)
    assert e.value.status == 3


def test_int8_full_size_sampled():
    torch = torch_gpu()
    host = generate(LLAMA8B_64K.with_(coef_format="int8"), layers=(28, 32))
    dc = device_cache(host)
    G = host.n_q_heads // host.n_kv_heads
    for layer in (0, 3):
        announce(f"int8 decode 64k layer={layer}")
        out = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        pairs = [(0, 2), (0, 7)]
        compare(out, oracle.decode(host, layer, heads=pairs), pairs, G, f"int8 64k layer {layer}")


@pytest.mark.parametrize("G,rb", [(4, 48), (1, 16), (2, 64)])
def test_int8_with_probe(G, rb):
    """Eq. 3 on an int8 cache (the current position): the int8 token-lane pass
    and the dense reference pass in one launch, Eq. 3 in the wide merge,
    against the oracle; a probe over several positions is refused (its earlier
    positions run the general kernel, which reads fp16 coefficients)."""
    torch = torch_gpu()
    from paper_2607_06523_amd import DwkvError, ProbeRef
    from synth.layout import block_values
    w = _Fixed(Workload(name=f"i8-probe-g{G}-rb{rb}", batch=3, n_layers=2, window=2, n_kv_heads=4, n_q_heads=4 * G,
                        head_dim=128, context=1500, basis_rank=rb, levels=(0, 4, 8, 16), probs=(0.7, 0.1, 0.1, 0.1),
                        q_dtype="bf16", seed=77 + G, coef_format="int8"), [1500, 0, 700])
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=256)
    heads, layer = [2, 0], 1
    rng = np.random.default_rng(3)
    K = np.stack([np.concatenate([oracle.reconstruct(host, layer, 0, h, b) for b in range(host.batch)])
                  for h in heads])
    V = np.stack([np.concatenate([oracle.reconstruct(host, layer, 1, h, b) for b in range(host.batch)])
                  for h in heads])
    K = (K + rng.normal(0, 0.05, K.shape)).astype(np.float16)
    V = (V + rng.normal(0, 0.05, V.shape)).astype(np.float16)
    pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                  torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda(), 1e-6)
    announce(f"int8 decode with a probe, G {G}, r_b {rb}")
    out, err, _ = dc.decode(layer, probe=pr)
    err = err.cpu().numpy()
    e_ref = oracle.probe(host, layer, heads, K, V)
    assert np.abs(err - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max(), (err, e_ref)
    assert np.all(err[1] == 0)
    compare(out.cpu().numpy(), oracle.decode(host, layer), [(b, h) for b in range(3) for h in range(4)], G,
            "int8 with probe")
    q_prev = torch.zeros((1, host.batch, host.n_q_heads, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(DwkvError) as e:
        dc.decode(layer, probe=ProbeRef(heads, pr.k_ref, pr.v_ref, 1e-6, q_prev=q_prev))
    assert e.value.status == 3
