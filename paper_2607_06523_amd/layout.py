"""The fp16 coefficient layouts of the C ABI, from and to the host layout.

Host layout (what ``DeviceCache`` takes and tests read back): keys row-major
``[L][Hkv][T][r_b]``; values in 16-token blocks ``[L][Hkv][T16/16][r_b][16]``,
token fastest (T16 = T rounded up to 16, padding zero).

ABI layout (``include/dwkv.h``), chosen so that every wave load instruction of
the decode reads whole 128-byte lines:
  keys   ``[L][Hkv][T16/16][r_b/8][16][8]``: tiles of 16 tokens x 8
         coefficients, coefficient fastest (int8 codes: 16 x 16 tiles,
         ``[L][Hkv][T16/16][r_b/16][16][16]``);
  values ``[L][Hkv][T16/8][r_b][8]``: 8-token blocks, token fastest (int8
         codes keep the host's 16-token blocks).
Argument marshalling only: element positions move, values do not change.
"""
from __future__ import annotations

import numpy as np


def keys_to_abi(rows: np.ndarray, group: int = 8) -> np.ndarray:
    """[..., T, R] -> [..., T16/16, R/group, 16, group] (tokens past T zero);
    group 8 for fp16 coefficients, 16 for int8 codes."""
    *lead, T, R = rows.shape
    T16 = -(-T // 16) * 16
    pad = np.zeros((*lead, T16, R), dtype=rows.dtype)
    pad[..., :T, :] = rows
    t = pad.reshape(*lead, T16 // 16, 16, R // group, group)
    return np.ascontiguousarray(np.swapaxes(t, -3, -2))


def keys_from_abi(tiles: np.ndarray, T: int) -> np.ndarray:
    """[..., T16/16, R/group, 16, group] -> [..., T, R]."""
    *lead, NB, G8, B16, E8 = tiles.shape
    rows = np.swapaxes(tiles, -3, -2).reshape(*lead, NB * B16, G8 * E8)
    return np.ascontiguousarray(rows[..., :T, :])


def values_to_abi(blocks16: np.ndarray) -> np.ndarray:
    """[..., T16/16, R, 16] -> [..., T16/8, R, 8]."""
    *lead, NB, R, B = blocks16.shape
    t = blocks16.reshape(*lead, NB, R, 2, 8)
    return np.ascontiguousarray(np.swapaxes(t, -3, -2).reshape(*lead, NB * 2, R, 8))


def values_from_abi(blocks8: np.ndarray) -> np.ndarray:
    """[..., T16/8, R, 8] -> [..., T16/16, R, 16]."""
    *lead, NB8, R, E = blocks8.shape
    t = blocks8.reshape(*lead, NB8 // 2, 2, R, 8)
    return np.ascontiguousarray(np.swapaxes(t, -3, -2).reshape(*lead, NB8 // 2, R, 16))
