"""The decode that appends (dwkv_decode_append) on the GPU through the C ABI.

Every non-empty sequence's last token is the new one: its key and value are
compressed into the cache (bit for bit the oracle's append/compress, reading
C5) and the layer's decode then attends to the whole cache with that token in
its compressed form (Eq. 1), within the decode tolerance of the float64
oracle.  One-launch path (token-lane query groups, fp16 coefficients): a
single sequence at automatic and explicit chunking, ragged batches with an
empty and a one-token sequence and per-token gates, groups of 1 and 8, rank-0
only caches; the two-step path (append/compress kernel per sequence, then the
decode): groups of 16 on the general kernel and int8 coefficients; and the
64K-token workload in the benchmark's launch configuration on sampled heads.
"""
import copy

import numpy as np
import pytest

import oracle
import oracle.compress as OC
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate

pytestmark = pytest.mark.gpu

WRITTEN = ("coef_k", "coef_v", "res_idx", "res_val", "res_scale")
WRITTEN_I8 = ("coef_k", "coef_v", "coef_scale_k", "coef_scale_v", "res_idx", "res_val", "res_scale")


class _Fixed:
    def __init__(self, w, lengths):
        self._w, self._lengths = w, list(lengths)

    def __getattr__(self, k):
        if k.startswith("_"):
            raise AttributeError(k)
        return getattr(self._w, k)

    def seqlens(self):
        return list(self._lengths)


def _device_arrays(dc):
    keys, values = dc.coef_host()
    if dc.coef_format == "int8":
        out = {"coef_k": keys.view(np.int8), "coef_v": values.view(np.int8),
               "coef_scale_k": dc.coef_scale_k.cpu().numpy().view(np.float16),
               "coef_scale_v": dc.coef_scale_v.cpu().numpy().view(np.float16)}
    else:
        out = {"coef_k": keys.view(np.float16), "coef_v": values.view(np.float16)}
    out["res_idx"] = dc.res_idx.cpu().numpy()
    out["res_val"] = dc.res_val.cpu().numpy()
    out["res_scale"] = dc.res_scale.cpu().numpy().view(np.float16)
    return out


def _assert_same(got, host, names, label):
    for name in names:
        want = np.ascontiguousarray(getattr(host, name))
        g = got[name].reshape(want.shape)
        if not np.array_equal(g.view(np.uint8), want.view(np.uint8)):
            diff = np.argwhere(g.view(np.uint8).reshape(-1) != want.view(np.uint8).reshape(-1))
            raise AssertionError(f"{label}: {name} differs from the oracle at byte(s) {diff[:5].ravel()}")


def _append_expected(host, layer, xk, xv, gate):
    """The oracle's cache after compressing every sequence's last token."""
    exp = copy.deepcopy(host)
    for b in range(host.batch):
        t1 = int(host.cu_seqlens[b + 1])
        if t1 == int(host.cu_seqlens[b]):
            continue
        g = None if gate is None else gate[:, :, b:b + 1]
        OC.compress(exp, layer, xk[b][None], xv[b][None], t1 - 1, t1, g)
    return exp


CASES = [
    # name, G, r_b, levels, probs, lengths, split, gate, coefficient format, launches
    ("one-seq-auto", 4, 48, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [3000], 0, False, "f16", 2),
    ("one-seq-split512", 4, 48, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [3000], 512, False, "f16", 2),
    ("ragged-g8-gate", 8, 64, (0, 4, 8, 16, 32), (0.5, 0.15, 0.15, 0.1, 0.1), [1700, 0, 1, 2049], 0, True, "f16", 2),
    ("ragged-g2-split256", 2, 32, (0, 2, 8, 16), (0.4, 0.2, 0.2, 0.2), [257, 256, 1025], 256, True, "f16", 2),
    ("g1-rank0", 1, 16, (0,), (1.0,), [900, 64], 0, False, "f16", 2),
    ("g16-general", 16, 64, (0, 8, 32), (0.5, 0.3, 0.2), [1200, 1], 0, True, "f16", 4),
    ("int8", 4, 48, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [2000], 0, False, "int8", 3),
    # more than 16 sequences: one compress launch per non-empty sequence, then the decode
    ("20-seqs", 4, 32, (0, 8), (0.7, 0.3), [0, 1] + [37 + 23 * i for i in range(18)], 64, True, "f16", 21),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_decode_append_matches_oracle(case):
    torch = torch_gpu()
    name, G, rb, levels, probs, lengths, split, with_gate, fmt, launches = case
    w = _Fixed(Workload(name="append-" + name, batch=len(lengths), n_layers=4, window=2, n_kv_heads=2,
                        n_q_heads=2 * G, head_dim=128, context=max(lengths), basis_rank=rb, levels=levels,
                        probs=probs, q_dtype="bf16", seed=71 + len(name), coef_format=fmt), lengths)
    host = generate(w, threads=4)
    rng = np.random.default_rng(17)
    Hk, B = host.n_kv_heads, host.batch
    xk = rng.standard_normal((B, Hk, 128)).astype(np.float16)
    xv = rng.standard_normal((B, Hk, 128)).astype(np.float16)
    gate = rng.uniform(0.0, 1.0, (2, Hk, B)).astype(np.float32) if with_gate else None
    layer = 3
    exp = _append_expected(host, layer, xk, xv, gate)
    dc = device_cache(host, split_tokens=split)
    assert dc.decode_append_launches == launches
    announce(f"decode append {name} layer {layer} lengths {lengths} split {split} launches {launches}")
    out = dc.decode_append(layer, torch.from_numpy(xk).cuda(), torch.from_numpy(xv).cuda(),
                           None if gate is None else torch.from_numpy(gate).cuda())
    out = out.cpu().numpy()
    torch.cuda.synchronize()
    _assert_same(_device_arrays(dc), exp, WRITTEN_I8 if fmt == "int8" else WRITTEN, name)
    pairs = [(b, h) for b in range(B) for h in range(Hk)]
    compare(out, oracle.decode(exp, layer), pairs, G, f"decode append {name}")
    for b, L in enumerate(lengths):
        if L == 0:
            assert np.all(out[b] == 0)
    # the plain decode over the appended cache agrees (same semantics)
    plain = dc.decode(layer).cpu().numpy()
    compare(plain, out, pairs, G, f"decode append {name} vs plain decode", rel_tol=1e-5, abs_tol=1e-5,
            regression=None)


def test_decode_append_64k_workload():
    """The 64K-token workload in the benchmark's launch configuration (one
    append item per KV head beside the split items); stored factors checked
    against the oracle bit for bit, outputs on two KV heads."""
    torch = torch_gpu()
    host = generate(LLAMA8B_64K.with_(n_layers=2, window=2), threads=8)
    rng = np.random.default_rng(23)
    Hk, B = host.n_kv_heads, host.batch
    xk = rng.standard_normal((B, Hk, 128)).astype(np.float16)
    xv = rng.standard_normal((B, Hk, 128)).astype(np.float16)
    layer = 1
    exp = _append_expected(host, layer, xk, xv, None)
    dc = device_cache(host)
    assert dc.decode_append_launches == 2
    announce("decode append 64K workload layer 1")
    out = dc.decode_append(layer, torch.from_numpy(xk).cuda(), torch.from_numpy(xv).cuda()).cpu().numpy()
    _assert_same(_device_arrays(dc), exp, WRITTEN, "64K append")
    G = host.n_q_heads // Hk
    heads = [(0, 0), (0, Hk - 1)]
    ref = oracle.decode(exp, layer, heads=heads)
    compare(out, ref, heads, G, "decode append 64K")
