"""Budget-driven routing (dwkv_route_budget) on the GPU against the oracle,
bit for bit: rank codes and offsets, budgets from infeasible through exact to
generous, planted score ties (the lower token wins), a tail range continuing
an existing offset table, and the 64K-token shape."""
import numpy as np
import pytest

import oracle
import oracle.control as OCt
from gpu_util import announce, device_cache, torch_gpu
from synth import LLAMA8B_64K, TINY, Workload, generate, router_inputs

pytestmark = pytest.mark.gpu


def _run(dc, host, wl, entries, t0, t1, seed, ties=True, label=""):
    torch = torch_gpu()
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    phi, u, _ = router_inputs(wl, M, T)
    if ties:                                   # equal feature rows: equal scores
        rng = np.random.default_rng(seed)
        src = rng.integers(0, T, size=max(T // 20, 2))
        dst = rng.integers(0, T, size=src.size)
        phi[:, :, dst] = phi[:, :, src]
        phi[:, :, :3] = 0.0                    # three exact zero scores (+0 and -0 alike)
        phi[:, :, 1, 0] = -0.0
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    codes_ref = host.rank_code.copy()
    off_ref = host.res_off.copy()
    OCt.route_budget(phi, u, entries, host.levels, t0, t1, codes_ref, off_ref)
    announce(f"route_budget {label} [{t0},{t1})")
    codes, off = dc.route_budget(dev(phi), dev(u), dev(entries.astype(np.int64)), t0, t1)
    torch.cuda.synchronize()
    got_c = codes.cpu().numpy()
    got_o = off.cpu().numpy().view(np.uint32)
    assert np.array_equal(got_c, codes_ref), f"{label}: rank codes differ at {np.argwhere(got_c != codes_ref)[:5]}"
    assert np.array_equal(got_o, off_ref), f"{label}: offsets differ at {np.argwhere(got_o != off_ref)[:5]}"
    return codes_ref


def test_route_budget_small():
    torch_gpu()
    wl = TINY.with_(levels=(0, 8), probs=(0.7, 0.3))
    host = generate(wl)
    dc = device_cache(host)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    lo, hi = wl.levels
    for i, E in enumerate([0, T * lo + 7, 8 * 100, 8 * 1000 + 5, T * hi, T * hi + 1000]):
        entries = np.full((M, Hk), E, np.int64)
        entries[0, -1] = max(E - 8 * 37, 0)    # heads take different budgets
        codes = _run(dc, host, wl, entries, 0, T, seed=i, label=f"budget {E}")
        n = np.clip((entries - T * lo) // (hi - lo), 0, T)
        assert np.array_equal(codes.sum(axis=2), n), "promoted counts differ from the budget"


def test_route_budget_rank_floor_and_tail():
    """rho_min > 0 (infeasible budgets promote nobody) and a tail range that
    continues the offsets of the tokens before it."""
    torch_gpu()
    wl = Workload(name="budget-ragged", batch=3, n_layers=4, window=2, n_kv_heads=2, n_q_heads=8, head_dim=128,
                  context=3000, basis_rank=32, levels=(4, 16), probs=(0.5, 0.5), q_dtype="bf16", seed=9,
                  ragged=(1000, 3000))
    host = generate(wl, threads=4)
    dc = device_cache(host)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    t0 = T - 777
    N = T - t0
    entries = np.array([[N * 4 - 1, N * 4], [N * 4 + 12 * 50, N * 16]], np.int64)
    _run(dc, host, wl, entries, t0, T, seed=5, label="tail")
    entries = np.full((M, Hk), T * 4 + 12 * 333, np.int64)
    _run(dc, host, wl, entries, 0, T, seed=6, label="all")


def test_route_budget_full_size():
    torch_gpu()
    wl = LLAMA8B_64K.with_(levels=(0, 16), probs=(0.9, 0.1))
    host = generate(wl, layers=(0, 8), with_q=False)
    dc = device_cache(host)
    M, Hk, T = host.n_windows, host.n_kv_heads, host.total_tokens
    rng = np.random.default_rng(1)
    entries = rng.integers(0, T * 16 // 4, size=(M, Hk)).astype(np.int64)
    _run(dc, host, wl, entries, 0, T, seed=2, label="64k")
