"""Helpers shared by the GPU parity tests."""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

# spec tolerance on decode outputs against float64
REL_L2_TOL = 1e-3       # per (sequence, layer, query head) output vector
MAX_ABS_TOL = 2e-3      # over all outputs compared
# the path computes scores and value sums to ~float32 accuracy (hi/lo fp16
# operands on MFMA, float32 accumulation); this tighter bar catches a
# precision regression long before the tolerance above would
REL_L2_REGRESSION = 1e-4


def torch_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def lib_ready():
    from paper_2607_06523_amd import binding, build
    if not os.path.exists(binding.LIB_PATH):
        build.build()
    return binding.load()


def announce(msg: str):
    """Print what the next GPU step is, flushed, so a failing run names its case."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def device_cache(host, split_tokens=0):
    lib_ready()
    from paper_2607_06523_amd import DeviceCache
    return DeviceCache(host, split_tokens=split_tokens)


def compare(gpu_out: np.ndarray, ref: np.ndarray, pairs, G: int, label: str,
            rel_tol=REL_L2_TOL, abs_tol=MAX_ABS_TOL, regression=REL_L2_REGRESSION):
    """Compare outputs of the query heads of the given (b, kv_head) pairs."""
    worst_rel, worst_abs = 0.0, 0.0
    for b, h in pairs:
        for g in range(G):
            hq = h * G + g
            r = ref[b, hq]
            o = gpu_out[b, hq]
            assert np.all(np.isfinite(o)), f"{label}: non-finite output b={b} hq={hq}"
            n = np.linalg.norm(r)
            rel = np.linalg.norm(o - r) / n if n > 0 else np.linalg.norm(o)
            worst_rel = max(worst_rel, rel)
            worst_abs = max(worst_abs, float(np.abs(o - r).max()))
    print(f"[parity] {label}: max rel-L2 {worst_rel:.3e}, max abs {worst_abs:.3e}", flush=True)
    assert worst_rel <= rel_tol, f"{label}: rel-L2 {worst_rel:.3e} > {rel_tol}"
    assert worst_abs <= abs_tol, f"{label}: max abs {worst_abs:.3e} > {abs_tol}"
    if regression is not None:
        assert worst_rel <= regression, f"{label}: rel-L2 {worst_rel:.3e} above regression bar {regression}"
    return worst_rel, worst_abs
