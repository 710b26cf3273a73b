"""Randomized-sketch basis initialization (dwkv_sketch_basis) on the GPU
against the oracle: every basis row within one fp16 step of the oracle's
(float64 sketch and Gram-Schmidt on both sides), other sequences' and windows'
bases untouched, rank-deficient sketches giving zero rows, and the 64K-token
prefill of the benchmark shape on two sampled heads."""
import numpy as np
import pytest

import oracle.sketch as OS
from gpu_util import announce, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate

pytestmark = pytest.mark.gpu


def _ulp16(v):
    a = np.abs(v.astype(np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -14)))
    return 2.0 ** (e - 10)


def _compare(got, ref, label):
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    d = np.abs(g - r)
    bad = d > _ulp16(r) * 1.0001
    assert not np.any(bad), f"{label}: {int(bad.sum())} basis entries more than one fp16 step off (max {d.max():.3e})"
    print(f"[parity] {label}: {int((d > 0).sum())} of {d.size} entries one step off", flush=True)


@pytest.mark.parametrize("rb,n_tok,kind", [(16, 3000, "normal"), (48, 5000, "lowrank"), (128, 700, "normal"),
                                           (32, 7, "short")])
def test_sketch_small(rb, n_tok, kind):
    torch = torch_gpu()
    w = Workload(name=f"sk{rb}", batch=2, n_layers=4, window=2, n_kv_heads=2, n_q_heads=4, head_dim=128,
                 context=max(n_tok, 64), basis_rank=rb, levels=(0, 8), probs=(0.5, 0.5), q_dtype="bf16", seed=rb)
    host = generate(w, threads=4)
    dc = device_cache(host)
    rng = np.random.default_rng(rb + n_tok)
    Hk, d = host.n_kv_heads, host.head_dim
    if kind == "lowrank":                       # rank 8 plus small noise
        V = np.linalg.qr(rng.standard_normal((d, 8)))[0]
        x = (rng.standard_normal((2, 2, n_tok, Hk, 8)) @ V.T + 0.01 * rng.standard_normal((2, 2, n_tok, Hk, d)))
    else:
        x = rng.standard_normal((2, 2, n_tok, Hk, d))
    x = x.astype(np.float16)
    omega = rng.standard_normal((2 * n_tok, rb)).astype(np.float16)
    before = dc.basis.cpu().numpy().view(np.float16).reshape(host.basis.shape).copy()
    seq, window = 1, 1
    announce(f"sketch rb={rb} n={n_tok} {kind}")
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    dc.sketch_basis(window, seq, dev(x), dev(omega))
    torch.cuda.synchronize()
    after = dc.basis.cpu().numpy().view(np.float16).reshape(host.basis.shape)
    for h in range(Hk):
        for z in range(2):
            ref = OS.sketch_basis(x, omega, h, z)
            _compare(after[seq, window, h, z], ref, f"rb {rb} {kind} h={h} z={z}")
            if kind == "short":                # 14 sketch rows of rank <= 14 < r_b: the rest are zero
                assert np.all(after[seq, window, h, z, 2 * n_tok:] == 0)
    mask = np.ones(after.shape[:2], bool)
    mask[seq, window] = False
    assert np.array_equal(after[mask], before[mask]), "another sequence's or window's basis changed"


def test_sketch_full_size_sampled():
    torch = torch_gpu()
    host = generate(LLAMA8B_64K, layers=(0, 4), with_q=False)
    dc = device_cache(host)
    T, Hk, d, w, rb = host.total_tokens, host.n_kv_heads, host.head_dim, host.window, host.basis_rank
    g = torch.Generator(device="cuda").manual_seed(11)
    x = torch.randn((w, 2, T, Hk, d), generator=g, device="cuda", dtype=torch.float16)
    omega = torch.randn((w * T, rb), generator=g, device="cuda", dtype=torch.float16)
    announce("sketch 64k")
    dc.sketch_basis(0, 0, x, omega)
    torch.cuda.synchronize()
    after = dc.basis.cpu().numpy().view(np.float16).reshape(host.basis.shape)
    om = omega.cpu().numpy()
    for h in (0, 7):
        xh = x[:, :, :, h:h + 1].cpu().numpy()
        for z in range(2):
            _compare(after[0, 0, h, z], OS.sketch_basis(xh, om, 0, z), f"64k h={h} z={z}")
