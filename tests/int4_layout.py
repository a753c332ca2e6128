"""The INT4 expert layout as the C header states it, written out element by
element (test helper).  Decoding a blob with these formulas and getting back
the integers and scales the weights were built from checks a packer against
the published byte layout, independently of the packer's own reshapes."""
from __future__ import annotations

import numpy as np


def matrix_bytes(rows: int, K: int) -> int:
    """M(rows, K) = rows*K/2 + rows*(K/64)*2."""
    return rows * K // 2 + rows * (K // 64) * 2


def nibble_location(r, k, K):
    """(byte offset, is_high_nibble) of element (r, k) of a [rows][K] matrix."""
    r = np.asarray(r, dtype=np.int64)
    k = np.asarray(k, dtype=np.int64)
    off = ((r // 16) * (K // 128) + k // 128) * 1024 + ((k % 64) // 16 * 16 + r % 16) * 16 \
        + ((k // 64) % 2) * 8 + ((k % 16) // 8) * 4 + k % 4
    return off, (k % 8) < 4


def scale_location(r, grp, rows, K):
    """Byte offset of the fp16 scale of row r and group grp, from the matrix start."""
    r = np.asarray(r, dtype=np.int64)
    grp = np.asarray(grp, dtype=np.int64)
    return rows * K // 2 + ((r // 16) * (K // 64) + grp) * 32 + (r % 16) * 2


def decode_matrix(mat: np.ndarray, rows: int, K: int):
    """(q [rows][K] int8, scales [rows][K/64] fp16) of one matrix's bytes."""
    mat = np.asarray(mat, dtype=np.uint8)
    rr, kk = np.meshgrid(np.arange(rows), np.arange(K), indexing="ij")
    off, high = nibble_location(rr, kk, K)
    b = mat[off].astype(np.int16)
    nib = np.where(high, b >> 4, b & 0xF)
    q = np.where(nib >= 8, nib - 16, nib).astype(np.int8)
    r2, g2 = np.meshgrid(np.arange(rows), np.arange(K // 64), indexing="ij")
    so = scale_location(r2, g2, rows, K)
    s = (mat[so].astype(np.uint16) | (mat[so + 1].astype(np.uint16) << 8)).view(np.float16)
    return q, s


def decode_blob(blob: np.ndarray, C: int, R: int):
    """((q, s) of gate, up, down) at offsets 0, M(R, C) and 2*M(R, C)."""
    m = matrix_bytes(R, C)
    return (decode_matrix(blob[0:m], R, C), decode_matrix(blob[m:2 * m], R, C),
            decode_matrix(blob[2 * m:3 * m], C, R))


# Marked elements (matrix, row, column, q) chosen so that each position
# differs from the others in a different part of the address: tile-row,
# column pair, group of the pair, 16-column run, row in the tile, 8-column
# half of the run, nibble and column in the quad.
MARKS = [
    ("gate", 0, 0, 1), ("gate", 1, 5, -3), ("gate", 2, 12, 2), ("gate", 3, 9, 5),
    ("gate", 17, 70, -7), ("gate", 30, 200, 4), ("gate", 46, 131, 6), ("gate", 63, 250, -1),
    ("up", 100, 150, -2), ("up", 127, 254, 3), ("up", 64, 16, -6), ("up", 81, 97, 7),
    ("down", 255, 126, 3), ("down", 40, 33, -5), ("down", 128, 64, 2), ("down", 9, 87, -4),
]
# (matrix, row, group) whose scale is twice the others
DOUBLE_SCALE = [("gate", 50, 2), ("up", 7, 1), ("down", 200, 0), ("down", 15, 1)]


def marked_weights(C: int = 256, R: int = 128, unit: float = 2.0 ** -7):
    """fp32 weights (gate [R][C], up [R][C], down [C][R]) and the integers
    and scales the INT4 format must store for them.  Every row and group
    holds a 7 at its last column, so its scale is exactly unit (or 2*unit for
    the DOUBLE_SCALE groups, whose anchor is 7*2*unit): the marks quantize to
    themselves."""
    shapes = {"gate": (R, C), "up": (R, C), "down": (C, R)}
    q = {m: np.zeros(s, dtype=np.int8) for m, s in shapes.items()}
    sc = {m: np.full((s[0], s[1] // 64), unit, dtype=np.float64) for m, s in shapes.items()}
    for m, (rows, K) in shapes.items():
        q[m][:, 63::64] = 7
    for m, r, g in DOUBLE_SCALE:
        sc[m][r, g] = 2 * unit
    for m, r, k, v in MARKS:
        assert k % 64 != 63
        q[m][r, k] = v
    w = {}
    for m in shapes:
        s = np.repeat(sc[m], 64, axis=1)
        w[m] = (q[m].astype(np.float64) * s).astype(np.float32)
        # the DOUBLE_SCALE groups' marks are 0, so q = w / (2*unit) is still q
    return (w["gate"], w["up"], w["down"]), q, sc
