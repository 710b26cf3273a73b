"""Decode parity when the residual scales span fp16's whole range.

The value-residual sums of Eq. 1 run in int64 fixed point whose unit follows
the largest value scale a wave has seen: a larger scale shifts the
accumulated sums down before it is added.  These cases drive that path with
scales from the fp16 subnormals to the top binade (2^15), zero scales among
them, and a ramp of the scale exponent within every run of tokens, so that
every wave meets its largest scale late (in its last tile) after sums are
already held.  Int8 block scales spanning several binades drive the 8-bit
coefficient path's per-block scaling.  Every output vector is compared with
the float64 oracle at the benchmark spec's tolerance and at the 1e-4 regression bar.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import Workload, generate

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
    # name, r_b, G, levels, probs, lengths, split, period, coefficient format, zero scales
    # token-lane kernel (fp16): ramps of 700 tokens over 512-token chunks
    ("tl-rb48-g4-ramp", 48, 4, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [3000, 517], 512, 700, "f16", False),
    # token-lane kernel at the benchmark's 2048-token chunks: the ramp's top is
    # the chunk's last token, each wave's scales grow tile by tile
    ("tl-rb48-g4-chunk-ramp", 48, 4, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [8192], 2048, 2048, "f16", False),
    ("tl-rb16-g1-short", 16, 1, (0, 2, 8), (0.4, 0.3, 0.3), [300, 65, 0], 64, 97, "f16", False),
    ("tl-rb64-g2-entry-heavy", 64, 2, (0, 16), (0.1, 0.9), [1500], 256, 300, "f16", False),
    ("tl-rb32-g4-all-zero", 32, 4, (0, 8, 16), (0.5, 0.3, 0.2), [1000], 256, 400, "f16", True),
    # token-lane kernel, 8-bit blockwise coefficients with wide block scales
    ("i8-rb48-g4-ramp", 48, 4, (0, 4, 8, 16), (0.55, 0.2, 0.15, 0.1), [3000, 517], 512, 700, "int8", False),
    ("i8-rb64-g4-ramp", 64, 4, (0, 8, 16), (0.5, 0.3, 0.2), [2500], 256, 600, "int8", False),
    # general kernel: groups of 8 and ranks to 32 (fixed point), groups of 16 at
    # r_b 128 (float accumulators)
    ("gen-rb64-g8-ramp", 64, 8, (0, 4, 8, 16, 32), (0.5, 0.15, 0.15, 0.1, 0.1), [2100, 400], 256, 500, "f16", False),
    ("gen-rb128-g16-ramp", 128, 16, (0, 8, 32), (0.5, 0.3, 0.2), [1200], 128, 333, "f16", False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_wide_scale_range(case):
    torch = torch_gpu()
    name, rb, G, levels, probs, lengths, split, period, fmt, zero = case
    base = Workload(name=name, batch=len(lengths), n_layers=2, window=2, n_kv_heads=2, n_q_heads=2 * G,
                    head_dim=128, context=max(lengths), basis_rank=rb, levels=levels, probs=probs,
                    q_dtype="bf16", seed=4000 + len(name), coef_format=fmt, scale_mode="wide",
                    scale_period=period, coef_scale_mode="wide" if fmt == "int8" else "narrow")
    host = generate(_Fixed(base, lengths), threads=4)
    if zero:
        host.res_scale[:] = 0
    else:
        s = host.res_scale.astype(np.float32)
        assert s.max() >= 2.0 ** 14 and np.any((s > 0) & (s < 2.0 ** -14)) and np.any(s == 0)
    dc = device_cache(host, split_tokens=split)
    pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
    for layer in range(host.n_layers):
        announce(f"wide-scale decode {name} layer={layer} split={dc.split_tokens}")
        out = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        compare(out, oracle.decode(host, layer), pairs, G, f"{name} layer {layer}")
        for b, L in enumerate(lengths):
            if L == 0:
                assert np.all(out[b] == 0)
