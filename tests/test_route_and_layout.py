"""Bit-exact GPU checks of the integer parts of the path (through the C ABI):
router rank codes and residual offsets (Eq. 2), residual-entry decoding, and
the layout validator's verdicts on clean and corrupted caches."""
import copy

import numpy as np
import pytest

import oracle
from gpu_util import announce, device_cache, torch_gpu
from synth import LLAMA70B_128K, LLAMA8B_64K, TINY, BATCH16, generate, router_inputs

pytestmark = pytest.mark.gpu


def _route_both(dc, phi, u, theta, levels):
    torch = torch_gpu()
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    codes, off = dc.route(dev(phi), dev(u), dev(theta))
    c_ref, o_ref = oracle.route(phi, u, theta, levels)
    return codes.cpu().numpy(), off.cpu().numpy().view(np.uint32), c_ref, o_ref


@pytest.mark.parametrize("wl", [TINY, BATCH16.with_(n_layers=4), LLAMA70B_128K.with_(n_layers=4)],
                         ids=["tiny", "batch16-ragged", "llama70b-128k"])
def test_route_bit_exact(wl):
    torch_gpu()
    host = generate(wl, layers=(0, wl.window), with_q=False) if wl.n_layers > 2 else generate(wl)
    dc = device_cache(host)
    M = host.n_windows
    phi, u, theta = router_inputs(wl, M, host.total_tokens)
    # plant exact ties z == theta (the lower level must win) and far-off values
    z = oracle.router_score(phi[0, 0, :64], u[0])
    theta[0, 0] = z[7]
    phi[0, 1, 5] = [1e30, 0, 0, 0]
    announce(f"route {wl.name} T={host.total_tokens}")
    codes, off, c_ref, o_ref = _route_both(dc, phi, u, theta, host.levels)
    assert np.array_equal(codes, c_ref), f"rank codes differ at {np.argwhere(codes != c_ref)[:5]}"
    assert np.array_equal(off, o_ref), f"offsets differ at {np.argwhere(off != o_ref)[:5]}"
    assert len(set(codes.ravel().tolist())) == len(host.levels), "not every level was reached"


def test_route_infinite_thresholds():
    torch_gpu()
    host = generate(TINY)
    dc = device_cache(host)
    phi, u, theta = router_inputs(TINY, 1, host.total_tokens)
    for th, want in [(np.inf, 0), (-np.inf, len(TINY.levels) - 1)]:
        announce(f"route theta={th}")
        codes, off, c_ref, o_ref = _route_both(dc, phi, u, np.full_like(theta, th), host.levels)
        assert np.all(codes == want) and np.array_equal(off, o_ref)


def test_residual_map_bit_exact():
    torch_gpu()
    host = generate(TINY)
    dc = device_cache(host)
    for layer, z, h, t0, t1 in [(0, 0, 0, 0, 4096), (1, 1, 1, 37, 1000), (1, 0, 1, 4000, 4096),
                                (0, 1, 0, 63, 65), (1, 1, 0, 5, 5)]:
        announce(f"residual map l={layer} z={z} h={h} [{t0},{t1})")
        got = dc.residual_map(layer, z, h, t0, t1).cpu().numpy().astype(np.float64)
        ref = oracle.residual_map(host, layer, z, h, t0, t1)
        assert np.array_equal(got, ref), f"residual map differs at {np.argwhere(got != ref)[:5]}"


def test_residual_map_full_size_sampled():
    torch_gpu()
    host = generate(LLAMA8B_64K, layers=(28, 32), with_q=False)
    dc = device_cache(host)
    for layer, z, h, t0, t1 in [(3, 0, 7, 65000, 65536), (0, 1, 2, 31, 2100)]:
        announce(f"residual map 64k l={layer} z={z} h={h} [{t0},{t1})")
        got = dc.residual_map(layer, z, h, t0, t1).cpu().numpy().astype(np.float64)
        assert np.array_equal(got, oracle.residual_map(host, layer, z, h, t0, t1))


def _nibble(c, l, z, h, e):
    return (int(c.res_val[l, z, h, e // 2]) >> (4 * (e % 2))) & 0xF


def _set_entry(c, l, z, h, e, chan, nib):
    c.res_idx[l, z, h, e] = chan
    bb = int(c.res_val[l, z, h, e // 2])
    c.res_val[l, z, h, e // 2] = (bb & 0xF0) | nib if e % 2 == 0 else (bb & 0x0F) | (nib << 4)


def _corrupt(host, kind):
    c = copy.deepcopy(host)
    m, h = 0, 1
    off = c.res_off[m, h].astype(np.int64)
    t = int(np.nonzero(np.diff(off) >= 4)[0][3])         # a token with >= 4 entries
    e = int(off[t])
    if kind == 1:                                          # offset disagrees with the code
        c.rank_code[m, h, t] = 0
    elif kind == 2:
        c.rank_code[m, h, t] = len(c.levels)
    elif kind == 3:
        c.res_idx[1, 0, h, e] = 200
    elif kind == 4:
        c.res_idx[0, 1, h, e + 1] = c.res_idx[0, 1, h, e]
    elif kind == 5:
        byte = int(c.res_val[0, 0, h, e // 2])
        c.res_val[0, 0, h, e // 2] = (byte & 0xF0) | 0x8 if e % 2 == 0 else (byte & 0x0F) | 0x80
    elif kind == 6:                                        # swap two entries: breaks the order
        n0, n1 = _nibble(c, 0, 0, h, e), _nibble(c, 0, 0, h, e + 1)
        i0, i1 = c.res_idx[0, 0, h, e], c.res_idx[0, 0, h, e + 1]
        _set_entry(c, 0, 0, h, e, i1, n1)
        _set_entry(c, 0, 0, h, e + 1, i0, n0)
    return c, (m * host.n_kv_heads + h) * (host.total_tokens + 1) + t


def test_validate_clean_and_corrupted():
    torch_gpu()
    host = generate(TINY)
    announce("validate clean")
    ok, bad = device_cache(host).validate()
    assert ok and bad == -1
    for kind in (1, 2, 3, 4, 5, 6):
        c, flat = _corrupt(host, kind)
        announce(f"validate corruption kind {kind}")
        ok, bad = device_cache(c).validate()
        assert not ok, f"corruption kind {kind} not detected"
        assert bad & 7 == kind and bad >> 3 == flat, f"kind {kind}: reported {bad & 7} at {bad >> 3}, want {flat}"
    c = copy.deepcopy(host)
    c.res_stride = int(c.res_off.max()) + 256 - (int(c.res_off.max()) % 256)   # no tail pad
    c.res_idx = c.res_idx[..., :c.res_stride].copy()
    c.res_val = c.res_val[..., :c.res_stride // 2].copy()
    ok, bad = device_cache(c).validate()
    assert not ok and bad & 7 == 7
