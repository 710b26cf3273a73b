"""The router's attention features from the decode (dwkv_decode_features)
against the oracle: per-token attention mass and spike of every layer, folded
into the window's feature table, over ragged sequences with empty ones, every
token-lane group size and a run of layers; the decode output stays bit-equal
to dwkv_decode's; the 64K-token shape on the benchmark's launch."""
import numpy as np
import pytest

import oracle
import oracle.features as OF
from gpu_util import announce, device_cache, torch_gpu
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
    ("rb32-g4-ragged", 32, 4, (0, 8, 16), (0.8, 0.15, 0.05), [0, 700, 129, 0, 2100], 256),
    ("rb48-g2-one-seq", 48, 2, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [3000], 0),
    ("rb16-g1-short", 16, 1, (0, 2), (0.6, 0.4), [1, 63, 65], 64),
    ("rb64-g4-no-residual", 64, 4, (0,), (1.0,), [1500, 37], 128),
    ("rb64-g8-ranks-to-32", 64, 8, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [0, 900, 2100], 256),
    # 8-bit blockwise coefficients
    ("i8-rb48-g4-ragged", 48, 4, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [0, 700, 129, 2100], 256),
    ("i8-rb64-g2-one-seq", 64, 2, (0, 8, 16), (0.7, 0.2, 0.1), [1800], 0),
]


def _check(phi_gpu, phi_ref, label):
    d0 = np.abs(phi_gpu[..., 0] - phi_ref[..., 0])
    d1 = np.abs(phi_gpu[..., 1] - phi_ref[..., 1])
    tol0 = 2e-4 * np.abs(phi_ref[..., 0]) + 1e-9
    tol1 = 2e-4 * np.abs(phi_ref[..., 1]) + 1e-9
    print(f"[parity] {label}: mass max rel {float((d0 / (np.abs(phi_ref[..., 0]) + 1e-30)).max()):.2e}, "
          f"spike max rel {float((d1 / (np.abs(phi_ref[..., 1]) + 1e-30)).max()):.2e}", flush=True)
    assert np.all(d0 <= tol0), f"{label}: attention mass off by {float((d0 / tol0).max()):.2f} x tolerance"
    assert np.all(d1 <= tol1), f"{label}: attention spike off by {float((d1 / tol1).max()):.2f} x tolerance"
    assert np.array_equal(phi_gpu[..., 2:], phi_ref[..., 2:]), f"{label}: columns 2, 3 changed"


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_features_small(case):
    torch = torch_gpu()
    name, rb, G, levels, probs, lengths, split = case
    w = _Fixed(Workload(name=name, batch=len(lengths), n_layers=4, window=2, n_kv_heads=2, n_q_heads=2 * G,
                        head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                        q_dtype="bf16", seed=700 + len(name),
                        coef_format="int8" if name.startswith("i8") else "f16"), lengths)
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=split)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    rng = np.random.default_rng(3)
    phi0 = rng.uniform(0.0, 0.5, size=(M, Hk, T, 4)).astype(np.float32)
    phi = torch.from_numpy(phi0.copy()).cuda()
    ref = phi0.astype(np.float64)
    for layer in range(host.n_layers):
        announce(f"decode_features {name} layer={layer}")
        out = dc.decode_features(layer, phi).cpu().numpy()
        base = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        assert np.array_equal(out.view(np.uint32), base.view(np.uint32)), "decode output differs from dwkv_decode"
        mass, spike = OF.attention_features(host, layer)
        OF.update_features(ref, layer // host.window, mass, spike)
        _check(phi.cpu().numpy().astype(np.float64), ref, f"{name} after layer {layer}")


def test_features_full_size_sampled():
    """The 64K shape: one layer's features on two sampled KV heads."""
    torch = torch_gpu()
    host = generate(LLAMA8B_64K, layers=(0, 4))
    dc = device_cache(host)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    phi = torch.zeros((M, Hk, T, 4), dtype=torch.float32, device="cuda")
    layer = 2
    announce("decode_features 64k")
    dc.decode_features(layer, phi)
    torch.cuda.synchronize()
    got = phi.cpu().numpy().astype(np.float64)
    _, probs = oracle.decode(host, layer, heads=[(0, 1), (0, 6)], with_probs=True)
    for (b, h), p in probs.items():
        ref = np.zeros((1, 1, T, 4))
        ref[0, 0, :, 0] = p.sum(axis=0)
        ref[0, 0, :, 1] = p.max(axis=0)
        _check(got[0:1, h:h + 1], ref, f"64k head {h}")


def test_probe_feature_matches_oracle():
    """The probe-error feature (column 3 of phi) from the Eq. 3 errors of two
    probed layers of one window: a fresh fold then a maximum fold, on the GPU
    through dwkv_probe_feature, against the oracle's fold of the same errors,
    bit for bit (a maximum and a copy, no arithmetic)."""
    torch = torch_gpu()
    import oracle.features as OFE
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    w = _Fixed(Workload(name="probe-feature", batch=3, n_layers=4, window=2, n_kv_heads=4, n_q_heads=16,
                        head_dim=128, context=900, basis_rank=32, levels=(0, 8, 16), probs=(0.8, 0.15, 0.05),
                        q_dtype="bf16", seed=91), [500, 0, 900])
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=256)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    rng = np.random.default_rng(4)
    phi0 = rng.uniform(0.0, 0.5, size=(M, Hk, T, 4)).astype(np.float32)
    phi = torch.from_numpy(phi0.copy()).cuda()
    ref = phi0.copy()
    heads = [3, 1]
    for k, layer in enumerate((2, 3)):              # window 1, fresh then folded
        K = rng.standard_normal((len(heads), T, 128)).astype(np.float16)
        V = rng.standard_normal((len(heads), T, 128)).astype(np.float16)
        pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                      torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda())
        announce(f"probe feature layer {layer}")
        _, err, _ = dc.decode(layer, probe=pr)
        dc.probe_feature(layer, heads, err, phi, fresh=(k == 0))
        torch.cuda.synchronize()
        OFE.probe_feature(ref, host.cu_seqlens, layer // host.window, heads, err.cpu().numpy(), 4, k == 0)
    got = phi.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), "probe feature differs from the oracle"
    assert np.array_equal(got[:, :, :, :3], phi0[:, :, :, :3]) and np.array_equal(got[0], phi0[0])
    print(f"[parity] probe feature: column 3 of window 1 bit-equal; range {got[1, heads, :, 3].min():.3f}"
          f"..{got[1, heads, :, 3].max():.3f}", flush=True)
