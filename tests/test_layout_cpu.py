"""The host -> ABI coefficient layout conversions (paper_2607_06523_amd.layout)
against the element positions include/dwkv.h states, element by element, and
their round trips.  fp16 keys: token t, coefficient i at [t/16][i/8][t%16][i%8];
fp16 values: [t/8][i][t%8]; int8 keys: [t/16][i/16][t%16][i%16]; padding zero."""
import numpy as np
import pytest

from paper_2607_06523_amd import layout as Lo


@pytest.mark.parametrize("T,R", [(1, 16), (15, 48), (16, 48), (17, 64), (100, 32), (257, 128)])
def test_fp16_positions_and_round_trip(T, R):
    rng = np.random.default_rng(T * 131 + R)
    keys = rng.integers(1, 60000, size=(2, 3, T, R)).astype(np.uint16)
    T16 = -(-T // 16) * 16
    vals16 = np.zeros((2, 3, T16 // 16, R, 16), np.uint16)
    vals16[..., :] = rng.integers(1, 60000, size=vals16.shape)
    kt, vt = Lo.keys_to_abi(keys), Lo.values_to_abi(vals16)
    assert kt.shape == (2, 3, T16 // 16, R // 8, 16, 8) and vt.shape == (2, 3, T16 // 8, R, 8)
    flat_k, flat_v = kt.reshape(2, 3, -1), vt.reshape(2, 3, -1)
    for t in range(T16):
        for i in range(R):
            kpos = (((t // 16) * (R // 8) + i // 8) * 16 + t % 16) * 8 + i % 8
            vpos = ((t // 8) * R + i) * 8 + t % 8
            want_k = keys[:, :, t, i] if t < T else 0
            assert np.all(flat_k[:, :, kpos] == want_k)
            assert np.all(flat_v[:, :, vpos] == vals16[:, :, t // 16, i, t % 16])
    assert np.array_equal(Lo.keys_from_abi(kt, T), keys)
    assert np.array_equal(Lo.values_from_abi(vt), vals16)


@pytest.mark.parametrize("T,R", [(5, 16), (33, 48), (64, 64)])
def test_int8_key_positions(T, R):
    rng = np.random.default_rng(T + R)
    codes = rng.integers(-127, 128, size=(2, T, R)).astype(np.int8).view(np.uint8)
    kt = Lo.keys_to_abi(codes, group=16)
    T16 = -(-T // 16) * 16
    assert kt.shape == (2, T16 // 16, R // 16, 16, 16)
    flat = kt.reshape(2, -1)
    for t in range(T16):
        for i in range(R):
            pos = (((t // 16) * (R // 16) + i // 16) * 16 + t % 16) * 16 + i % 16
            assert np.all(flat[:, pos] == (codes[:, t, i] if t < T else 0))
    assert np.array_equal(Lo.keys_from_abi(kt, T), codes)
