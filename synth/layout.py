"""Storage layout helpers for value-side coefficient tiles.

Value coefficients (and the dense reference values a probe reads) are stored
in 16-token blocks, token index fastest: element (token t, channel i) of a
[T][R] matrix sits at [t // 16][i][t % 16] of a [ceil(T/16)][R][16] array;
tokens past T in the last block are zero.  Key coefficients stay row-major.
These helpers convert between the two views for input preparation and tests.
"""
from __future__ import annotations

import numpy as np

BLOCK = 16


def padded_tokens(T: int) -> int:
    return -(-T // BLOCK) * BLOCK


def block_values(rows: np.ndarray) -> np.ndarray:
    """[..., T, R] -> [..., ceil(T/16), R, 16] (zero padded)."""
    *lead, T, R = rows.shape
    Tp = padded_tokens(T)
    pad = np.zeros((*lead, Tp, R), dtype=rows.dtype)
    pad[..., :T, :] = rows
    return np.ascontiguousarray(pad.reshape(*lead, Tp // BLOCK, BLOCK, R).swapaxes(-1, -2))


def unblock_values(tiles: np.ndarray, T: int) -> np.ndarray:
    """[..., NB, R, 16] -> [..., T, R]."""
    *lead, NB, R, B = tiles.shape
    return tiles.swapaxes(-1, -2).reshape(*lead, NB * B, R)[..., :T, :]


def set_value_row(coef_v: np.ndarray, layer: int, h: int, t: int, row) -> None:
    coef_v[layer, h, t // BLOCK, :, t % BLOCK] = row


def value_row(coef_v: np.ndarray, layer: int, h: int, t: int) -> np.ndarray:
    return coef_v[layer, h, t // BLOCK, :, t % BLOCK]
