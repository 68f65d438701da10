"""Conversions between the row-major code store and the tiled store layout,
written from the layout's definition (include/eogp.h, eogp_sign_pack_tiled):
row r = 32 t + i, step s of S, 16-byte piece p of the step's 64 bytes sits at
byte (t * S + s) * 2048 + (p % 2) * 1024 + ((p // 2) * 32 + i) * 16."""
import numpy as np


def tiled_from_rows(rows: np.ndarray) -> np.ndarray:
    """uint8 [N, S*64] row-major codes -> the tiled store (rows past N zero)."""
    N, B = rows.shape
    assert B % 64 == 0
    S, T = B // 64, -(-N // 32)
    pad = np.zeros((T * 32, B), np.uint8)
    pad[:N] = rows
    # [t, i, s, hg, uc, j] -> [t, s, uc, hg, i, j]
    return np.ascontiguousarray(
        pad.reshape(T, 32, S, 2, 2, 16).transpose(0, 2, 4, 3, 1, 5)).reshape(-1)


def rows_from_tiled(tiled: np.ndarray, S: int) -> np.ndarray:
    """The tiled store of whole tiles -> uint8 [tiles*32, S*64] row-major."""
    T = tiled.size // (S * 2048)
    # [t, s, uc, hg, i, j] -> [t, i, s, hg, uc, j]
    return np.ascontiguousarray(
        tiled.reshape(T, S, 2, 2, 32, 16).transpose(0, 4, 1, 3, 2, 5)).reshape(T * 32, S * 64)
