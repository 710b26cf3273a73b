"""Seeded random shapes on the GPU (through the C ABI) against the float64
oracle: group size, basis rank, ranks, ragged lengths (with empty
sequences), chunk size, query dtype, coefficient format and an Eq. 3 probe
over one or two positions drawn together, so that combinations the
hand-picked cases do not list also run.  Every draw is a fixed function of
its index."""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import Workload, generate

N_DRAWS = 40


class _Fixed:
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        if k.startswith("_"):
            raise AttributeError(k)
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


def _draw(i):
    rng = np.random.default_rng(1000 + i)
    G = int(rng.choice([1, 2, 4, 8, 16]))
    rb = int(rng.choice([16, 32, 48, 64, 96, 128] if G < 16 else [16, 32, 64]))
    Hk = int(rng.choice([1, 2, 4]))
    token_lane = rb <= 64 and G <= 8
    top = 16 if G <= 4 else 32
    pool = [2, 4, 8, 16, 32, 64] if not token_lane else [2, 4, 8, 16, 32][: 4 if top == 16 else 5]
    n_lev = int(rng.integers(1, 4))
    levels = tuple(sorted({0, *[int(v) for v in rng.choice(pool, n_lev)]}))
    probs = tuple(float(p) for p in rng.dirichlet(np.ones(len(levels)) * 2))
    B = int(rng.integers(1, 6))
    lengths = [int(v) if rng.random() > 0.15 else 0 for v in rng.integers(1, 2500, B)]
    if max(lengths) == 0:
        lengths[0] = 1 + int(rng.integers(0, 600))
    split = int(rng.choice([0, 64, 128, 256, 512]))
    qd = str(rng.choice(["f16", "bf16"]))
    n_pos = int(rng.choice([1, 1, 2]))
    c8 = token_lane and G <= 4 and n_pos == 1 and rng.random() < 0.6
    n_probe = int(rng.integers(0, Hk + 1))
    return dict(G=G, rb=rb, Hk=Hk, levels=levels, probs=probs, lengths=lengths, split=split, qd=qd,
                n_pos=n_pos, c8=c8, n_probe=n_probe, seed=int(rng.integers(1, 1 << 30)))


def test_draws_cover_both_kernels_and_formats():
    """The draws include the token-lane and general kernels, int8 and fp16
    coefficients, probes over one and two positions, and empty sequences."""
    ds = [_draw(i) for i in range(N_DRAWS)]
    assert any(d["rb"] <= 64 and d["G"] <= 8 for d in ds) and any(d["rb"] > 64 or d["G"] == 16 for d in ds)
    assert any(d["c8"] for d in ds) and any(d["n_probe"] and d["n_pos"] == 2 for d in ds)
    assert any(0 in d["lengths"] for d in ds)


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_DRAWS))
def test_random_shape(i):
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    d = _draw(i)
    G, Hk = d["G"], d["Hk"]
    w = _Fixed(Workload(name=f"random-{i}", batch=len(d["lengths"]), n_layers=2, window=2, n_kv_heads=Hk,
                        n_q_heads=Hk * G, head_dim=128, context=max(d["lengths"]), basis_rank=d["rb"],
                        levels=d["levels"], probs=d["probs"], q_dtype=d["qd"], seed=d["seed"],
                        coef_format="int8" if d["c8"] else "f16"), d["lengths"])
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=d["split"])
    layer = 1
    announce(f"random shape {i}: {d}")
    pairs = [(b, h) for b in range(host.batch) for h in range(Hk)]
    if not d["n_probe"]:
        compare(dc.decode(layer).cpu().numpy(), oracle.decode(host, layer), pairs, G, f"random {i}")
        return
    rng = np.random.default_rng(d["seed"])
    heads = [int(h) for h in rng.permutation(Hk)[: d["n_probe"]]]
    K = np.stack([np.concatenate([oracle.reconstruct(host, layer, 0, h, b) for b in range(host.batch)])
                  for h in heads])
    V = np.stack([np.concatenate([oracle.reconstruct(host, layer, 1, h, b) for b in range(host.batch)])
                  for h in heads])
    K = (K + rng.normal(0, 0.05, K.shape)).astype(np.float16)
    V = (V + rng.normal(0, 0.05, V.shape)).astype(np.float16)
    qdt = torch.float16 if d["qd"] == "f16" else torch.bfloat16
    q_prev = None
    qs = oracle.q_to_f64(host.q_bits[layer], d["qd"])[None]
    if d["n_pos"] > 1:
        q_prev = torch.from_numpy(rng.standard_normal((d["n_pos"] - 1, host.batch, host.n_q_heads, 128))
                                  .astype(np.float32)).to(qdt)
        qs = np.concatenate([qs, q_prev.float().numpy().astype(np.float64)])
        q_prev = q_prev.cuda()
    pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                  torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda(), 1e-6,
                  q_prev=q_prev)
    out, err, _ = dc.decode(layer, probe=pr)
    compare(out.cpu().numpy(), oracle.decode(host, layer), pairs, G, f"random {i} with probe")
    e_ref = oracle.probe_positions(host, layer, heads, K, V, qs) if d["n_pos"] > 1 else \
        oracle.probe(host, layer, heads, K, V)
    err = err.cpu().numpy()
    assert np.abs(err - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max(), (err, e_ref)
