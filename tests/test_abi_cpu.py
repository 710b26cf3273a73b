"""The C-ABI library on the CPU: it loads, exports every call include/dwkv.h
declares, and rejects bad arguments on the host before anything is enqueued
(no GPU needed: every case returns before the first HIP call)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_06523_amd import binding, build
    if not os.path.exists(binding.LIB_PATH):
        build.build()
    return binding.load()


def header_functions():
    text = open(os.path.join(ROOT, "include", "dwkv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dwkv_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), f"libdwkv.so does not export {n}"
    from paper_2607_06523_amd import binding
    assert sorted(binding.EXPORTS) == names


def test_abi_version_and_status_strings(lib):
    assert lib.dwkv_abi_version() == 4
    for s, text in [(0, b"ok"), (3, b"unsupported shape"), (5, b"malformed cache layout"),
                    (7, b"device pointer not 16-byte aligned")]:
        assert lib.dwkv_status_str(s) == text


def test_decode_rejects_misaligned_pointers(lib):
    d, keep = dims()
    assert decode_status(lib, d, q=FAKE + 8) == 7
    assert decode_status(lib, d, out=FAKE + 4) == 7
    from paper_2607_06523_amd import binding
    c = binding.Cache(*([FAKE] * 8))
    c.coef_v = FAKE + 2
    assert lib.dwkv_decode(C.byref(d), C.byref(c), 0, FAKE, 0, 0.0, FAKE, None, FAKE, 1 << 30, None) == 7
    assert lib.dwkv_decode(C.byref(d), C.byref(binding.Cache(*([FAKE] * 8))), 0, FAKE, 0, 0.0, FAKE, None,
                           FAKE + 32 + 8, 1 << 30, None) == 7


def dims(**kw):
    from paper_2607_06523_amd import binding
    base = dict(batch=2, n_layers=4, window=2, n_kv_heads=2, n_q_heads=8, head_dim=128,
                basis_rank=32, levels=(0, 8, 16), cu_seqlens_host=[0, 1000, 3000],
                cu_seqlens_dev_ptr=1, total_tokens=3000, res_stride=64 * 1024, split_tokens=0)
    base.update(kw)
    return binding.make_dims(**base)


FAKE = 1 << 20   # never dereferenced: every call below fails its host-side checks


def decode_status(lib, d, layer=0, qtype=0, ws=1 << 30, cache_ok=True, q=FAKE, out=FAKE, probe=None):
    from paper_2607_06523_amd import binding
    c = binding.Cache(*([FAKE] * 8)) if cache_ok else binding.Cache(FAKE, FAKE, 0, FAKE, FAKE, FAKE, FAKE, FAKE)
    return lib.dwkv_decode(C.byref(d), C.byref(c), layer, q, qtype, 0.0, out,
                           C.byref(probe) if probe is not None else None, FAKE, ws, None)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), 3),
    (dict(n_q_heads=7), 2),              # Hq % Hkv != 0
    (dict(n_q_heads=6), 3),              # G = 3
    (dict(n_q_heads=64, n_kv_heads=2), 3),   # G = 32
    (dict(n_kv_heads=65, n_q_heads=65), 3),  # more KV heads than a launch carries
    (dict(basis_rank=24), 3),
    (dict(basis_rank=144), 3),
    (dict(n_layers=5), 2),               # L % w != 0
    (dict(levels=(0, 3)), 2),            # odd level
    (dict(levels=(0, 8, 8)), 2),         # not ascending
    (dict(levels=(0, 130)), 2),          # > d
    (dict(levels=tuple(range(0, 18, 2))), 3),   # 9 levels
    (dict(total_tokens=2999), 2),        # cu[B] != T
    (dict(cu_seqlens_host=[1, 1000, 3000]), 2),
    (dict(cu_seqlens_host=[0, 3001, 3000]), 2),
    (dict(res_stride=1000), 2),          # not a multiple of 256
    (dict(res_stride=256), 2),           # below the tail pad
    (dict(split_tokens=100), 2),         # not a multiple of 64
    (dict(batch=0, cu_seqlens_host=[0]), 2),
    (dict(total_tokens=2**30, cu_seqlens_host=[0, 2**29, 2**30], levels=(0, 8)), 3),  # offsets overflow
])
def test_decode_rejects_bad_dims(lib, kw, status):
    d, keep = dims(**kw)
    assert decode_status(lib, d) == status


def test_decode_rejects_bad_call_arguments(lib):
    d, keep = dims()
    assert decode_status(lib, d, layer=4) == 2
    assert decode_status(lib, d, layer=-1) == 2
    assert decode_status(lib, d, qtype=2) == 2
    assert decode_status(lib, d, cache_ok=False) == 1
    assert decode_status(lib, d, q=0) == 1
    assert decode_status(lib, d, out=0) == 1
    need = lib.dwkv_workspace_bytes(C.byref(d), None)
    assert decode_status(lib, d, ws=need - 1) == 4
    assert lib.dwkv_decode(None, None, 0, FAKE, 0, 0.0, FAKE, None, FAKE, 1 << 30, None) == 1


def test_probe_argument_checks(lib):
    from paper_2607_06523_amd import binding
    d, keep = dims()
    heads = np.array([1, 1], dtype=np.int32)
    p = binding.Probe(2, heads.ctypes.data_as(C.POINTER(C.c_int32)), FAKE, FAKE, 1e-6, FAKE, 0)
    assert decode_status(lib, d, probe=p) == 2           # duplicate head
    heads[:] = [0, 2]
    assert decode_status(lib, d, probe=p) == 2           # out of range
    heads[:] = [1, 0]
    p.err = 0
    assert decode_status(lib, d, probe=p) == 1
    p.err = FAKE
    p.n_heads = 3
    assert decode_status(lib, d, probe=p) == 2
    p.n_heads = 2
    need = lib.dwkv_workspace_bytes(C.byref(d), C.byref(p))
    assert need > lib.dwkv_workspace_bytes(C.byref(d), None)
    assert decode_status(lib, d, probe=p, ws=need - 1) == 4
    # several positions: q_prev required and aligned, at most 8 positions,
    # per earlier position two more reference-sized regions and the sums
    p.n_pos = 3
    assert decode_status(lib, d, probe=p) == 1           # q_prev missing
    p.q_prev = FAKE + 2
    assert decode_status(lib, d, probe=p) == 7           # misaligned
    p.q_prev = FAKE
    for bad in (-1, 9):
        p.n_pos = bad
        assert decode_status(lib, d, probe=p) == 2
    p.n_pos = 3
    need3 = lib.dwkv_workspace_bytes(C.byref(d), C.byref(p))
    G = d.n_q_heads // d.n_kv_heads
    # reference partials: 256-token chunks (3000 tokens x 2 heads over 256
    # workgroups), 4 + 8 work items of the 1000- and 2000-token sequences
    ref = up256(12 * 2 * G * 132 * 4)
    # the wide merge's reference rows of the probed columns, and its counters
    assert need == lib.dwkv_workspace_bytes(C.byref(d), None) + ref + up256(d.batch * 2 * G * 128 * 4) \
        + up256(d.batch * 2 * G * 4)
    assert need3 == need + 2 * 2 * ref + up256(d.batch * 2 * G * 2 * 4)
    assert decode_status(lib, d, probe=p, ws=need3 - 1) == 4
    p.n_pos = 0
    assert lib.dwkv_workspace_bytes(C.byref(d), C.byref(p)) == need


def up256(n):
    return -(-n // 256) * 256


def test_workspace_and_split_plan(lib):
    # automatic chunk: ceil(T*Hkv/n) rounded up to 256, clamped to [256, 8192], with n = 256
    # workgroups for the token-lane kernel (groups of up to 4 with ranks <= 16, groups of 8 with
    # ranks <= 32; r_b <= 64) and 512 otherwise
    for T, Hk, want in [(4096, 2, 256), (32768, 8, 1024), (65536, 8, 2048), (262144, 8, 8192),
                        (10**6, 8, 8192)]:
        d, keep = dims(cu_seqlens_host=[0, T], batch=1, total_tokens=T, n_kv_heads=Hk, n_q_heads=4 * Hk,
                       res_stride=T * 16 + 512 + (-(T * 16 + 512)) % 256)
        assert lib.dwkv_split_tokens(C.byref(d)) == want
        n_work = -(-T // want)
        # token-lane partials (group of 4, r_b 32, ranks <= 16): d + 64 + 4 floats
        assert lib.dwkv_workspace_bytes(C.byref(d), None) == up256(n_work * Hk * 4 * 196 * 4)
    d, keep = dims(cu_seqlens_host=[0, 65536], batch=1, total_tokens=65536, n_kv_heads=8, n_q_heads=64,
                   res_stride=65536 * 16 + 512, levels=(0, 8, 32))
    assert lib.dwkv_split_tokens(C.byref(d)) == 2048      # group of 8, ranks <= 32: token-lane kernel
    d, keep = dims(cu_seqlens_host=[0, 65536], batch=1, total_tokens=65536, n_kv_heads=8, n_q_heads=128,
                   res_stride=65536 * 16 + 512)
    assert lib.dwkv_split_tokens(C.byref(d)) == 1024      # group of 16: general kernel
    d, keep = dims(split_tokens=640)
    assert lib.dwkv_split_tokens(C.byref(d)) == 640
    # ragged: per-sequence chunk counts, empty sequences contribute none
    d, keep = dims(batch=3, cu_seqlens_host=[0, 700, 700, 1300], total_tokens=1300, split_tokens=256)
    assert lib.dwkv_workspace_bytes(C.byref(d), None) == up256((3 + 3) * 2 * 4 * 196 * 4)
    # general kernel partials (group of 16): d + 4 floats
    d, keep = dims(batch=3, cu_seqlens_host=[0, 700, 700, 1300], total_tokens=1300, split_tokens=256,
                   n_q_heads=32)
    assert lib.dwkv_workspace_bytes(C.byref(d), None) == up256((3 + 3) * 2 * 16 * 132 * 4)


def test_route_and_map_argument_checks(lib):
    d, keep = dims()
    assert lib.dwkv_route(C.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, None) == 4
    need = lib.dwkv_route_workspace_bytes(C.byref(d))
    assert need > 0
    assert lib.dwkv_route(C.byref(d), FAKE, 0, FAKE, FAKE, FAKE, FAKE, need, None) == 1
    from paper_2607_06523_amd import binding
    c = binding.Cache(*([FAKE] * 8))
    assert lib.dwkv_residual_map(C.byref(d), C.byref(c), 0, 2, 0, 0, 10, FAKE, None) == 2
    assert lib.dwkv_residual_map(C.byref(d), C.byref(c), 0, 0, 0, 10, 5, FAKE, None) == 2
    assert lib.dwkv_residual_map(C.byref(d), C.byref(c), 0, 0, 0, 0, 3001, FAKE, None) == 2
    bad = C.c_int64(0)
    assert lib.dwkv_validate(C.byref(d), C.byref(c), C.byref(bad), FAKE, 8, None) == 4
    assert bad.value == -1


def test_decode_launch_count(lib):
    """The split-K pass and the merge; a probe adds its reference pass, inside
    the split-K launch on the token-lane kernel and as a launch of its own on
    the general kernel (the merge evaluates Eq. 3 on either)."""
    from paper_2607_06523_amd import binding
    for kw in (dict(), dict(n_q_heads=16), dict(batch=3, cu_seqlens_host=[0, 700, 700, 1300], total_tokens=1300)):
        d, keep = dims(**kw)
        assert lib.dwkv_decode_launches(C.byref(d), None) == 2
    heads = np.array([1], dtype=np.int32)
    p = binding.Probe(1, heads.ctypes.data_as(C.POINTER(C.c_int32)), FAKE, FAKE, 1e-6, FAKE, 0)
    d, keep = dims()                                  # G = 4, r_b 32: token-lane kernel
    assert lib.dwkv_decode_launches(C.byref(d), C.byref(p)) == 2
    d, keep = dims(n_q_heads=32)                      # G = 16: general kernel
    assert lib.dwkv_decode_launches(C.byref(d), C.byref(p)) == 3
    d, keep = dims(n_q_heads=7)
    assert lib.dwkv_decode_launches(C.byref(d), None) == -1
    # several positions: one launch per earlier position that still sees a
    # token, then one merge; lengths 700, 0 and 2 with 4 positions and 256-token
    # chunks: positions 1 and 2 see tokens (of the first sequences), 3 only of the first
    d, keep = dims(batch=3, cu_seqlens_host=[0, 700, 700, 702], total_tokens=702, split_tokens=256)
    p.n_pos, p.q_prev = 4, FAKE
    assert lib.dwkv_decode_launches(C.byref(d), C.byref(p)) == 2 + 3 + 1
    d, keep = dims(batch=2, cu_seqlens_host=[0, 2, 3], total_tokens=3, split_tokens=256)
    assert lib.dwkv_decode_launches(C.byref(d), C.byref(p)) == 2 + 1 + 1
    p.n_pos = 1
    assert lib.dwkv_decode_launches(C.byref(d), C.byref(p)) == 2


def test_route_range_and_compress_argument_checks(lib):
    """Both new calls reject bad ranges, null and misaligned pointers on the host."""
    from paper_2607_06523_amd import binding
    d, keep = dims()
    need = lib.dwkv_route_workspace_bytes(C.byref(d))
    rr = lambda t0, t1, ws=need, u=FAKE, phi=FAKE: lib.dwkv_route_range(
        C.byref(d), phi, u, FAKE, t0, t1, FAKE, FAKE, FAKE, ws, None)
    assert rr(10, 5) == 2
    assert rr(-1, 5) == 2
    assert rr(0, 3001) == 2
    assert rr(0, 10, ws=need - 1) == 4
    assert rr(0, 10, u=0) == 1
    assert rr(0, 10, phi=0) == 1
    assert rr(2999, 2999, phi=0) == 0         # empty range past the start: nothing to do
    c = binding.Cache(*([FAKE] * 8))
    cp = lambda layer=0, t0=2990, t1=3000, xk=FAKE, xv=FAKE, gate=None, cache=c: lib.dwkv_compress(
        C.byref(d), C.byref(cache), layer, xk, xv, gate, t0, t1, None)
    assert cp(layer=4) == 2
    assert cp(layer=-1) == 2
    assert cp(t0=5, t1=4) == 2
    assert cp(t1=3001) == 2
    assert cp(xk=0) == 1
    assert cp(t0=7, t1=7, xk=0, xv=0) == 0    # empty range
    assert cp(xv=FAKE + 8) == 7
    assert cp(gate=FAKE + 2) == 7
    c2 = binding.Cache(*([FAKE] * 8))
    c2.res_scale = FAKE + 1
    assert cp(cache=c2) == 7
    c3 = binding.Cache(*([FAKE] * 8))
    c3.coef_k = 0
    assert cp(cache=c3) == 1
    d2, keep2 = dims(head_dim=64)
    assert lib.dwkv_compress(C.byref(d2), C.byref(c), 0, FAKE, FAKE, None, 0, 1, None) == 3
    # the 8-bit blockwise form needs its block-scale arrays, 2-byte aligned
    d8, keep8 = dims(coef_format=1)
    assert lib.dwkv_compress(C.byref(d8), C.byref(c), 0, FAKE, FAKE, None, 0, 1, None) == 1
    c8 = binding.Cache(*([FAKE] * 8))
    c8.coef_k_scale, c8.coef_v_scale = FAKE, FAKE + 1
    assert lib.dwkv_compress(C.byref(d8), C.byref(c8), 0, FAKE, FAKE, None, 0, 1, None) == 7


def test_materialize_and_dense_argument_checks(lib):
    from paper_2607_06523_amd import binding
    d, keep = dims()
    c = binding.Cache(*([FAKE] * 8))
    assert lib.dwkv_materialize(C.byref(d), C.byref(c), 4, FAKE, FAKE, None) == 2
    assert lib.dwkv_materialize(C.byref(d), C.byref(c), 0, 0, FAKE, None) == 1
    assert lib.dwkv_materialize(C.byref(d), C.byref(c), 0, FAKE, FAKE + 8, None) == 7
    c.res_scale = FAKE + 1
    assert lib.dwkv_materialize(C.byref(d), C.byref(c), 0, FAKE, FAKE, None) == 7
    need = lib.dwkv_dense_workspace_bytes(C.byref(d))
    # general-kernel chunks: ceil(T*Hkv/512) rounded to 256 -> 256; (4 + 8) chunks x 2 heads x 4 x 132 floats
    assert need == up256((4 + 8) * 2 * 4 * 132 * 4)
    dd = lambda **kw: lib.dwkv_dense_decode(C.byref(d), kw.get("k", FAKE), FAKE, FAKE, kw.get("qt", 0), 0.0,
                                            kw.get("out", FAKE), FAKE, kw.get("ws", need), None)
    assert dd(ws=need - 1) == 4
    assert dd(k=0) == 1
    assert dd(qt=3) == 2
    assert dd(out=FAKE + 4) == 7
    d2, keep2 = dims(n_q_heads=7)
    assert lib.dwkv_dense_workspace_bytes(C.byref(d2)) == 0


def test_features_argument_checks(lib):
    from paper_2607_06523_amd import binding
    d, keep = dims()                          # groups of 4, r_b 32, ranks <= 16: token-lane path
    base = lib.dwkv_workspace_bytes(C.byref(d), None)
    need = lib.dwkv_features_workspace_bytes(C.byref(d))
    assert need == base + up256(8 * 3000 * 4) + up256(2 * 8 * 2 * 4)   # scores, then (m*, l*) per (b, hq)
    d8, keep8 = dims(n_q_heads=32)            # groups of 16: general kernel, no features
    assert lib.dwkv_features_workspace_bytes(C.byref(d8)) == 0
    c = binding.Cache(*([FAKE] * 8))
    f = lambda dd=d, **kw: lib.dwkv_decode_features(C.byref(dd), C.byref(c), kw.get("layer", 0), FAKE, 0, 0.0,
                                                    kw.get("out", FAKE), kw.get("phi", FAKE), FAKE,
                                                    kw.get("ws", need), None)
    assert f(ws=need - 1) == 4
    assert f(phi=0) == 1
    assert f(phi=FAKE + 4) == 7
    assert f(layer=4) == 2
    assert f(dd=d8, ws=1 << 30) == 3


def test_controller_update_matches_oracle(lib):
    """The host controller against the oracle's rule on random traces (bitwise:
    both step and clamp in float32)."""
    import oracle.control as OC
    from paper_2607_06523_amd import binding
    rng = np.random.default_rng(17)
    for trial in range(20):
        M, J = int(rng.integers(1, 6)), int(rng.integers(0, 4))
        ctl = binding.Controller(0.05, float(rng.uniform(0, 1)), float(rng.uniform(0, 1)), int(rng.integers(1, 4)),
                                 -3.0, 3.0)
        theta = np.sort(rng.uniform(-3, 3, size=(M, J)).astype(np.float32), axis=1)
        below = rng.integers(0, 3, size=M).astype(np.int32)
        th_ref, bl_ref = theta.copy(), below.astype(np.int64).copy()
        for step in range(12):
            err = rng.uniform(0, 0.1, size=M).astype(np.float32)
            err[rng.random(M) < 0.1] = np.nan
            st = lib.dwkv_controller_update(C.byref(ctl), M, J, err.ctypes.data, theta.ctypes.data,
                                            below.ctypes.data)
            assert st == 0
            OC.controller_update(th_ref, bl_ref, err, ctl.tol, ctl.step_down, ctl.step_up, ctl.patience,
                                 ctl.theta_min, ctl.theta_max)
            assert np.array_equal(theta.view(np.uint32), th_ref.astype(np.float32).view(np.uint32)), (trial, step)
            assert np.array_equal(below, bl_ref), (trial, step)
    bad = binding.Controller(0.1, -1.0, 0.5, 2, -1.0, 1.0)
    one = np.zeros(1, np.float32)
    assert lib.dwkv_controller_update(C.byref(bad), 1, 1, one.ctypes.data, one.ctypes.data,
                                      np.zeros(1, np.int32).ctypes.data) == 2


def test_route_budget_argument_checks(lib):
    d, keep = dims(levels=(0, 8))
    need = lib.dwkv_route_budget_workspace_bytes(C.byref(d))
    assert need == up256(2 * 2 * 3000 * 8)
    rb = lambda dd=d, **kw: lib.dwkv_route_budget(C.byref(dd), kw.get("phi", FAKE), FAKE, kw.get("ent", FAKE),
                                                  kw.get("t0", 0), kw.get("t1", 3000), FAKE, FAKE, FAKE,
                                                  kw.get("ws", need), None)
    assert rb(ws=need - 1) == 4
    assert rb(t1=3001) == 2
    assert rb(ent=0) == 1
    assert rb(ent=FAKE + 4) == 7
    assert rb(phi=FAKE + 8) == 7
    d3, keep3 = dims()                                   # three levels
    assert rb(dd=d3, ws=1 << 30) == 3


def test_sketch_argument_checks(lib):
    from paper_2607_06523_amd import binding
    d, keep = dims()
    need = lib.dwkv_sketch_workspace_bytes(C.byref(d), 5000)
    row = 2 * 2 * 32 * 128 * 8
    assert need == up256(3 * row) + up256(row)          # 10000 sketch rows: 3 chunks of 4096
    assert lib.dwkv_sketch_workspace_bytes(C.byref(d), 0) == 0
    c = binding.Cache(*([FAKE] * 8))
    sk = lambda **kw: lib.dwkv_sketch_basis(C.byref(d), C.byref(c), kw.get("win", 0), kw.get("seq", 0),
                                            kw.get("x", FAKE), FAKE, kw.get("n", 5000), FAKE, kw.get("ws", need),
                                            None)
    assert sk(ws=need - 1) == 4
    assert sk(win=2) == 2
    assert sk(seq=2) == 2
    assert sk(n=0) == 2
    assert sk(x=0) == 1
    assert sk(x=FAKE + 2) == 7


def test_hbm_read_rejects_bad_arguments(lib):
    blocks = lib.dwkv_hbm_read_blocks()
    assert blocks >= 256
    assert lib.dwkv_hbm_read(FAKE, 1024, None, blocks, None) == 1              # no sink
    assert lib.dwkv_hbm_read(None, 1024, FAKE, blocks, None) == 1              # no buffer
    assert lib.dwkv_hbm_read(FAKE, 1000, FAKE, blocks, None) == 2              # not a multiple of 16
    assert lib.dwkv_hbm_read(FAKE, 1024, FAKE, blocks - 1, None) == 4          # sink too small
    assert lib.dwkv_hbm_read(FAKE + 8, 1024, FAKE, blocks, None) == 7          # buffer alignment
    assert lib.dwkv_hbm_read(FAKE, 1024, FAKE + 2, blocks, None) == 7          # sink alignment


@pytest.mark.parametrize("lens,hk", [([65536], 8), ([32768], 8), ([131072], 8),
                                     ([8192 + 917 * i for i in range(16)], 8),     # ragged batch
                                     ([100, 20000, 3, 45000, 7777], 4), ([1] * 40, 8)])
def test_split_plan_fits_one_round(lib, lens, hk):
    """The automatic chunk is a multiple of 256 tokens and, on the token-lane
    path, the work items of every sequence (each rounded up) times the KV
    heads fit 256 workgroups whenever a chunk of at most 8192 tokens allows."""
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64).tolist()
    d, keep = dims(batch=len(lens), n_kv_heads=hk, n_q_heads=4 * hk, basis_rank=48, levels=(0, 4, 8, 16),
                   cu_seqlens_host=cu, total_tokens=cu[-1], res_stride=1 << 26)
    split = lib.dwkv_split_tokens(C.byref(d))
    assert split % 256 == 0 and 256 <= split <= 8192
    items = sum(-(-n // split) for n in lens)
    fits_at_max = sum(-(-n // 8192) for n in lens) * hk <= 256
    if fits_at_max:
        assert items * hk <= 256, f"split {split}: {items * hk} workgroups"
        if split > 256:                  # and the next smaller chunk would not fit
            assert sum(-(-n // (split - 256)) for n in lens) * hk > 256
    # an explicit split is taken as given
    d2, keep2 = dims(batch=len(lens), n_kv_heads=hk, n_q_heads=4 * hk, basis_rank=48, levels=(0, 4, 8, 16),
                     cu_seqlens_host=cu, total_tokens=cu[-1], res_stride=1 << 26, split_tokens=1024)
    assert lib.dwkv_split_tokens(C.byref(d2)) == 1024


def test_noalloc_refuses_beyond_static_scratch(lib):
    """dwkv_decode_noalloc checks its scratch need on the host before anything
    touches the GPU: dims whose workspace exceeds the static array get
    DWKV_E_SCRATCH."""
    from paper_2607_06523_amd import binding
    limit = int(lib.dwkv_static_scratch_bytes())
    assert limit == 16 << 20
    n = 40000
    cu = np.arange(n + 1, dtype=np.int32) * 64
    d, keep = binding.make_dims(batch=n, n_layers=1, window=1, n_kv_heads=8, n_q_heads=32, head_dim=128,
                                basis_rank=48, levels=(0,), cu_seqlens_host=cu, cu_seqlens_dev_ptr=16,
                                total_tokens=int(cu[-1]), res_stride=1024, split_tokens=64)
    assert lib.dwkv_workspace_bytes(C.byref(d), None) > limit
    cache = binding.Cache()
    st = lib.dwkv_decode_noalloc(C.byref(d), C.byref(cache), 0, C.c_void_p(16), 0,
                                 C.c_float(0.0), C.c_void_p(16), None, None)
    assert st == 8
    assert lib.dwkv_status_str(8) == b"needs more than the library's static scratch"


def test_decode_kernel_query(lib):
    """Which split kernel the plan picks: token-lane for groups of up to 4 with
    ranks up to 16 and groups of 8 with ranks up to 32 (r_b up to 64)."""
    for kw, want in [(dict(), 1), (dict(n_q_heads=16, levels=(0, 8, 32)), 1), (dict(levels=(0, 8, 32)), 0),
                     (dict(n_q_heads=32), 0), (dict(basis_rank=80), 0), (dict(n_q_heads=7), -1)]:
        d, keep = dims(**kw)
        assert lib.dwkv_decode_kernel(C.byref(d)) == want, kw


def test_probe_feature_argument_checks(lib):
    d, keep = dims()
    heads = np.array([1, 0], dtype=np.int32)
    hp = heads.ctypes.data_as(C.POINTER(C.c_int32))
    f = lambda layer=0, n=2, h=hp, err=FAKE, phi=FAKE: lib.dwkv_probe_feature(C.byref(d), layer, n, h, err, 1,
                                                                               phi, None)
    assert f(n=0) == 2 and f(n=3) == 2 and f(layer=4) == 2
    assert f(h=None) == 1 and f(err=0) == 1 and f(phi=0) == 1
    assert f(phi=FAKE + 4) == 7 and f(err=FAKE + 2) == 7
    dup = np.array([1, 1], dtype=np.int32)
    assert f(h=dup.ctypes.data_as(C.POINTER(C.c_int32))) == 2


def test_probe_schedule_matches_oracle(lib):
    """The host probe schedule against the oracle's rotation, and its argument checks."""
    import oracle.control as OC
    from paper_2607_06523_amd import probe_schedule
    for hk, n, p, P in ((8, 1, 1, 1), (8, 3, 4, 5), (5, 4, 2, 8), (64, 8, 16, 3), (8, 8, 1, 2)):
        for s in list(range(0, 70)) + [10**12, 10**12 + p * 7]:
            assert probe_schedule(s, p, n, hk, P) == OC.probe_schedule(s, p, n, hk, P), (hk, n, p, s)
    h = (C.c_int32 * 8)()
    npos = C.c_int32(0)
    for args in ((-1, 1, 1, 8, 1), (0, 0, 1, 8, 1), (0, 1, 0, 8, 1), (0, 1, 9, 8, 1), (0, 1, 1, 8, 0),
                 (0, 1, 1, 8, 9)):
        assert lib.dwkv_probe_schedule(*args, h, C.byref(npos)) == -1, args
    assert lib.dwkv_probe_schedule(0, 1, 1, 8, 1, None, C.byref(npos)) == -1


def test_decode_append_plan_and_argument_checks(lib):
    """The decode that appends: one launch plus the merge on token-lane dims
    (chunks sized so the split items and one append item per sequence and KV
    head fill one round of 256 workgroups), else one compress launch per
    non-empty sequence plus the decode; bad arguments refused on the host."""
    from paper_2607_06523_amd import binding
    T = 65536
    d, keep = dims(cu_seqlens_host=[0, T], batch=1, total_tokens=T, n_kv_heads=8, n_q_heads=32,
                   res_stride=T * 16 + 512, basis_rank=48, levels=(0, 4, 8, 16))
    assert lib.dwkv_decode_append_launches(C.byref(d)) == 2
    # chunks of 2176 tokens: 31 split items per head over 65535 tokens, + 1 append item
    assert lib.dwkv_decode_append_workspace_bytes(C.byref(d)) == up256((31 + 1) * 8 * 4 * 196 * 4)
    d, keep = dims(batch=3, cu_seqlens_host=[0, 700, 700, 1301], total_tokens=1301, split_tokens=256)
    # per head: ceil(699/256) + 1 and ceil(600/256) + 1 items; the empty sequence none
    assert lib.dwkv_decode_append_workspace_bytes(C.byref(d)) == up256((3 + 1 + 3 + 1) * 2 * 4 * 196 * 4)
    assert lib.dwkv_decode_append_launches(C.byref(d)) == 2
    d16, keep16 = dims(batch=3, cu_seqlens_host=[0, 700, 700, 1301], total_tokens=1301, n_q_heads=32)
    assert lib.dwkv_decode_append_launches(C.byref(d16)) == 2 + 2          # general kernel: per-sequence compress
    assert lib.dwkv_decode_append_workspace_bytes(C.byref(d16)) == lib.dwkv_workspace_bytes(C.byref(d16), None)
    bad, keepb = dims(n_q_heads=7)
    assert lib.dwkv_decode_append_launches(C.byref(bad)) == -1
    assert lib.dwkv_decode_append_workspace_bytes(C.byref(bad)) == 0
    c = binding.Cache(*([FAKE] * 8))
    need = lib.dwkv_decode_append_workspace_bytes(C.byref(d))

    def call(x_k=FAKE, x_v=FAKE, gate=None, ws=FAKE, ws_bytes=need, q=FAKE, out=FAKE, layer=0):
        return lib.dwkv_decode_append(C.byref(d), C.byref(c), layer, q, 0, 0.0, out, x_k, x_v, gate, ws, ws_bytes,
                                      None)
    assert call(x_k=None) == 1
    assert call(q=None) == 1
    assert call(x_v=FAKE + 8) == 7
    assert call(gate=FAKE + 2) == 7
    assert call(ws_bytes=need - 1) == 4
    assert call(layer=4) == 2
