"""Host definition of the library's tiled code layout (QL_LAYOUT_TILED in
include/qlinear.h): a storage order of the packed codes, not part of the
paper's computation.  Byte 16*hh + i of column n's group j (row-major byte
[n][64*j + 16*hh + i]) sits at tiled byte
16 * (64 * ((n // 16) * (K // 128) + j) + 16 * hh + n % 16) + i."""
import numpy as np


def tile_np(qw: np.ndarray) -> np.ndarray:
    """Row-major codes uint8 [N, K/2] -> tiled bytes (flat, N*K/2)."""
    N, H = qw.shape
    G = H // 64
    return np.ascontiguousarray(
        qw.reshape(N // 16, 16, G, 4, 16).transpose(0, 2, 3, 1, 4)).reshape(-1)


def untile_np(t: np.ndarray, N: int, K: int) -> np.ndarray:
    G = K // 128
    return np.ascontiguousarray(
        t.reshape(N // 16, G, 4, 16, 16).transpose(0, 3, 1, 2, 4)).reshape(N, K // 2)
