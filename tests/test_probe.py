"""Eq. 3 probe error on the GPU (through the C ABI) against the oracle, plus
its closed forms on a cache whose rebuilt rows are exact in fp16."""
import numpy as np
import pytest

import oracle
import pins
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA70B_128K, Workload, generate

pytestmark = pytest.mark.gpu


def _refs(host, layer, heads, noise, seed):
    rng = np.random.default_rng(seed)
    K = np.stack([np.concatenate([oracle.reconstruct(host, layer, 0, h, b) for b in range(host.batch)])
                  for h in heads])
    V = np.stack([np.concatenate([oracle.reconstruct(host, layer, 1, h, b) for b in range(host.batch)])
                  for h in heads])
    if noise:
        K = K + rng.normal(0, noise, K.shape)
        V = V + rng.normal(0, noise, V.shape)
    return K.astype(np.float16), V.astype(np.float16)


def _run_probe(dc, layer, heads, K, V, eps=1e-6):
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    Vb = block_values(V)                       # values in the 16-token blocked layout
    pr = ProbeRef(list(heads), torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                  torch.from_numpy(Vb.view(np.uint16)).view(torch.float16).cuda(), eps)
    out, err, out_ref = dc.decode(layer, probe=pr)
    return out.cpu().numpy(), err.cpu().numpy(), out_ref.cpu().numpy()


class _Fixed:
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        if k.startswith("_"):
            raise AttributeError(k)
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


PROBE_CASES = [
    # name, G, r_b, levels, probs, lengths (None: ragged draw), split
    # general kernel (ranks to 32 at G = 4): one merge covers outputs and probe
    ("general-g4-ranks32", 4, 64, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), None, 512),
    # token-lane kernels: the wide merge's probed-head workgroups evaluate Eq. 3 per
    # channel chunk; the last chunk of a column adds the chunks' sums
    ("tl-g4", 4, 48, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), None, 512),
    ("tl-g8-empty-seq", 8, 64, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [0, 2100, 1700], 256),
    # groups of 1 and 2: the reference pass inside the split-K launch at those widths
    ("tl-g1", 1, 32, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), None, 256),
    ("tl-g2-tiny-seqs", 2, 16, (0, 8, 16), (0.8, 0.15, 0.05), [5, 1, 2300], 512),
    ("tl-g8-rb32", 8, 32, (0, 8, 32), (0.8, 0.15, 0.05), None, 256),
    # bases only (every rank 0): the kernels without the residual path
    ("tl-g4-bases-only", 4, 48, (0,), (1.0,), None, 512),
    ("general-g16-bases-only", 16, 32, (0,), (1.0,), None, 512),
]


@pytest.mark.parametrize("case", PROBE_CASES, ids=[c[0] for c in PROBE_CASES])
def test_probe_matches_oracle(case):
    torch_gpu()
    name, G, rb, levels, probs, lengths, split = case
    w = Workload(name="probe-" + name, batch=2 if lengths is None else len(lengths), n_layers=2, window=2,
                 n_kv_heads=4, n_q_heads=4 * G, head_dim=128, context=3000, basis_rank=rb, levels=levels,
                 probs=probs, q_dtype="bf16", seed=55, ragged=(1500, 3000))
    if lengths is not None:
        w = _Fixed(w, lengths)
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=split)
    heads = [3, 0, 2]
    K, V = _refs(host, 1, heads, 0.05, seed=3)
    announce(f"probe {name} layer 1, heads 3,0,2")
    out, err, out_ref = _run_probe(dc, 1, heads, K, V)
    e_ref = oracle.probe(host, 1, heads, K, V)
    assert np.abs(err - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max(), (err, e_ref)
    nonempty = [b for b in range(host.batch) if host.cu_seqlens[b + 1] > host.cu_seqlens[b]]
    assert e_ref[nonempty].min() > 0.01, "noise should give a visible probe error"
    # the compressed output is unchanged by probing
    compare(out, oracle.decode(host, 1), [(b, h) for b in range(host.batch) for h in range(4)], G,
            f"probe {name} out")
    # the reference output is plain attention over the dense reference cache
    for i, h in enumerate(heads):
        for b in nonempty:
            t0, t1 = int(host.cu_seqlens[b]), int(host.cu_seqlens[b + 1])
            q = oracle.q_to_f64(host.q_bits[1], "bf16")[b, h * G:(h + 1) * G]
            o, _ = oracle.attention(q, K[i, t0:t1].astype(np.float64), V[i, t0:t1].astype(np.float64),
                                    1 / np.sqrt(128))
            rel = np.linalg.norm(out_ref[b, i * G:(i + 1) * G] - o) / np.linalg.norm(o)
            assert rel < 1e-4, rel


def test_probe_closed_forms():
    """Rebuilt rows exact in fp16 (one-hot bases, small-integer coefficients,
    fp16-exact residuals): K_ref = K_hat, V_ref = V_hat gives e ~ 0, and
    V_ref = c V_hat gives e = |1-c| ||O|| / (|c| ||O|| + eps)."""
    torch_gpu()
    w = Workload(name="probe-exact", batch=1, n_layers=2, window=2, n_kv_heads=2, n_q_heads=4,
                 head_dim=128, context=700, basis_rank=16, levels=(0, 2), probs=(0.5, 0.5),
                 q_dtype="f16", seed=9)
    host = generate(w, threads=2)
    pins._perm_basis(host, 21)
    rng = np.random.default_rng(22)
    host.coef_k[:] = rng.integers(-3, 4, size=host.coef_k.shape).astype(np.float16)
    host.coef_v[:] = rng.integers(-3, 4, size=host.coef_v.shape).astype(np.float16)
    host.res_scale[:] = np.float16(0.5)
    dc = device_cache(host, split_tokens=256)
    K, V = _refs(host, 0, [0, 1], 0.0, 0)
    assert np.array_equal(K.astype(np.float64)[0], oracle.reconstruct(host, 0, 0, 0, 0)), "reference not fp16-exact"
    announce("probe exact reference")
    out, err, _ = _run_probe(dc, 0, [0, 1], K, V)
    assert err.max() < 2e-6, err
    for c in (2.0, -0.5):
        announce(f"probe scaled reference c={c}")
        out, err, _ = _run_probe(dc, 0, [0, 1], K, (c * V.astype(np.float64)).astype(np.float16))
        n = np.linalg.norm(oracle.decode(host, 0), axis=-1)       # [B, Hq]
        want = abs(1 - c) * n / (abs(c) * n + 1e-6)
        assert np.abs(err - want.reshape(err.shape)).max() < 1e-5, (err, want)


def test_probe_full_size_70b_shape():
    torch_gpu()
    wl = LLAMA70B_128K
    announce("generate 70b window for probe")
    host = generate(wl, layers=(0, 4))
    dc = device_cache(host)
    heads = [6, 1]
    K, V = _refs(host, 3, heads, 0.05, seed=8)
    announce("probe 70b layer 3")
    out, err, out_ref = _run_probe(dc, 3, heads, K, V)
    e_ref = oracle.probe(host, 3, heads, K, V)
    assert np.abs(err - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max(), (err, e_ref)


POS_CASES = [
    # name, G, r_b, levels, probs, lengths, split, positions
    # general kernel: a 1025-token sequence loses its last 256-token chunk
    # one position back; a 2-token one sees positions 0 and 1 only
    ("general-g4-p4", 4, 64, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [1025, 2, 1700], 256, 4),
    ("tl-g4-p3", 4, 48, (0, 4, 8, 16), (0.75, 0.12, 0.08, 0.05), [2049, 0, 1500], 512, 3),
    ("tl-g8-p8", 8, 64, (0, 4, 8, 16, 32), (0.7, 0.12, 0.1, 0.06, 0.02), [3, 1800, 7], 256, 8),
    # more sequences than the kernel-argument work table holds: the trimmed
    # passes walk the device sequence table
    ("tl-g4-20-seqs-p3", 4, 32, (0, 8), (0.7, 0.3), [1, 2, 0] + [37 + 23 * i for i in range(17)], 64, 3),
]


@pytest.mark.parametrize("case", POS_CASES, ids=[c[0] for c in POS_CASES])
def test_probe_positions_match_oracle(case):
    """Eq. 3 over several recent positions: the query j steps back attends to
    the first T_b - j tokens; the norms run over positions and d together."""
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    name, G, rb, levels, probs, lengths, split, P = case
    w = _Fixed(Workload(name="probepos-" + name, batch=len(lengths), n_layers=2, window=2, n_kv_heads=4,
                        n_q_heads=4 * G, head_dim=128, context=max(lengths), basis_rank=rb, levels=levels,
                        probs=probs, q_dtype="bf16", seed=61), lengths)
    host = generate(w, threads=4)
    dc = device_cache(host, split_tokens=split)
    heads, layer = [2, 0], 1
    K, V = _refs(host, layer, heads, 0.05, seed=5)
    rng = np.random.default_rng(7)
    q_prev = torch.from_numpy(rng.standard_normal((P - 1, host.batch, host.n_q_heads, 128)).astype(np.float32)
                              ).to(torch.bfloat16)
    qs = np.concatenate([oracle.q_to_f64(host.q_bits[layer], "bf16")[None],
                         q_prev.float().numpy().astype(np.float64)])
    pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                  torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda(), 1e-6,
                  q_prev=q_prev.cuda())
    announce(f"probe positions {name} P={P} layer {layer} heads 2,0 lengths {lengths} split {split}")
    out, err, _ = dc.decode(layer, probe=pr)
    err = err.cpu().numpy()
    e_ref = oracle.probe_positions(host, layer, heads, K, V, qs)
    assert np.abs(err - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max(), (err, e_ref)
    # the earlier positions change the error (they are not ignored)
    e_cur = oracle.probe(host, layer, heads, K, V)
    nonempty = [b for b in range(host.batch) if host.cu_seqlens[b + 1] - host.cu_seqlens[b] > 1]
    assert np.abs(e_cur - e_ref)[nonempty].max() > 10 * (1e-4 + 1e-3 * np.abs(e_ref).max())
    for b, L in enumerate(lengths):
        if L == 0:
            assert np.all(err[b] == 0)
    # the decode output is unchanged by probing
    compare(out.cpu().numpy(), oracle.decode(host, layer), [(b, h) for b in range(host.batch) for h in range(4)],
            G, f"probe positions {name} out")
    # two calls in a row agree bit for bit
    _, err2, _ = dc.decode(layer, probe=pr)
    assert np.array_equal(err, err2.cpu().numpy())


@pytest.mark.parametrize("positions", [1, 3])
def test_probe_two_phase_matches_one_phase(positions):
    """dwkv_decode_partials + dwkv_decode_merge with a probe (the reference
    passes in the first half, Eq. 3 in the second) equal dwkv_decode bit for
    bit, outputs and errors, on the token-lane kernel."""
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    host = generate(Workload(name="probe-two-phase", batch=2, n_layers=2, window=2, n_kv_heads=2, n_q_heads=8,
                             head_dim=128, context=2000, basis_rank=32, levels=(0, 8, 16), probs=(0.7, 0.2, 0.1),
                             q_dtype="bf16", seed=43, ragged=(1, 2000)), threads=4)
    dc = device_cache(host, split_tokens=256)
    heads = [1]
    K, V = _refs(host, 0, heads, 0.05, seed=9)
    q_prev = None
    if positions > 1:
        q_prev = torch.randn((positions - 1, host.batch, host.n_q_heads, 128)).to(torch.bfloat16).cuda()
    pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                  torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda(), 1e-6, q_prev=q_prev)
    announce(f"probe two-phase, {positions} position(s)")
    out1, err1, _ = dc.decode(0, probe=pr)
    ws = dc.new_workspace(pr)
    err2 = torch.empty_like(err1)
    dc.decode_partials(0, workspace=ws, probe=pr, err=err2)
    out2 = dc.decode_merge(0, workspace=ws, probe=pr, err=err2)
    torch.cuda.synchronize()
    assert np.array_equal(out1.cpu().numpy(), out2.cpu().numpy())
    assert np.array_equal(err1.cpu().numpy(), err2.cpu().numpy())


def test_probe_with_uninitialised_workspace():
    """The decode needs no initial workspace contents: a workspace whose bytes
    are all 0xFF (stale counters and partials) gives the clean workspace's
    outputs and probe errors bit for bit, on the token-lane path (the wide
    merge's counters) and the general one, with an empty sequence in the batch
    (its columns take e = 0 without counting in)."""
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    for G, rb in ((4, 32), (16, 32)):
        w = _Fixed(Workload(name=f"probe-stale-g{G}", batch=3, n_layers=2, window=2, n_kv_heads=2, n_q_heads=2 * G,
                            head_dim=128, context=1300, basis_rank=rb, levels=(0, 8), probs=(0.7, 0.3),
                            q_dtype="bf16", seed=19), [700, 0, 1300])
        host = generate(w, threads=4)
        dc = device_cache(host, split_tokens=256)
        heads = [1]
        K, V = _refs(host, 1, heads, 0.05, seed=5)
        pr = ProbeRef(heads, torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda(),
                      torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda())
        res = []
        for fill in (0, 0xFF, 0xFF):
            ws = dc.new_workspace(pr)
            ws.fill_(fill)
            announce(f"probe G {G} workspace filled with {fill:#x}")
            out, err, _ = dc.decode(1, probe=pr, workspace=ws)
            res.append((out.cpu().numpy(), err.cpu().numpy()))
        for out, err in res[1:]:
            assert np.array_equal(out, res[0][0]) and np.array_equal(err, res[0][1])
        assert np.all(res[0][1][1] == 0.0), "an empty sequence's probe error is 0"
        e_ref = oracle.probe(host, 1, heads, K, V)
        assert np.abs(res[0][1] - e_ref).max() <= 1e-4 + 1e-3 * np.abs(e_ref).max()
