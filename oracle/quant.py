"""Group-quantised expert weights decoded to fp64 (test infrastructure only).

Sec. 5.1: the experts of the measured model were stored as 2-bit codes in
groups of 16 weights, with compressed zero points.  The byte format read here
(a reading; the paper gives no format) stores a matrix [rows x cols] as three
planes, back to back:

* codes: rows x cols/4 bytes; column c of a row sits in bits 2 (c mod 4) and
  2 (c mod 4) + 1 of byte floor(c / 4) of that row;
* scales: one IEEE fp16 per group of 16 consecutive columns, rows x cols/16;
* zero codes: one byte per group, the zero point being code / 64.

The weight is (q - zero) * scale.  An expert is W1 [d_ff x d] | W3 [d_ff x d] |
W2 [d x d_ff], each stored this way.
"""
from __future__ import annotations

import numpy as np

GROUP = 16
ZERO_STEPS = 64


def matrix_bytes(rows: int, cols: int) -> int:
    """Stored size: 2 bits + 16/16 + 8/16 bits per weight = 7 bytes per 16 weights."""
    return rows * cols // 4 + rows * cols // 8 + rows * cols // 16


def dequantize(buf: np.ndarray, rows: int, cols: int) -> np.ndarray:
    """fp64 [rows x cols] from one stored matrix (uint8 buffer)."""
    buf = np.asarray(buf, dtype=np.uint8)
    n = rows * cols
    assert cols % GROUP == 0 and buf.size == matrix_bytes(rows, cols)
    codes = buf[:n // 4].reshape(rows, cols // 4)
    scale = buf[n // 4:n // 4 + n // 8].copy().view("<f2").astype(np.float64).reshape(rows, cols // GROUP)
    zero = buf[n // 4 + n // 8:].astype(np.float64).reshape(rows, cols // GROUP) / ZERO_STEPS
    q = np.empty((rows, cols), dtype=np.float64)
    for t in range(4):  # column 4 j + t is field t of byte j
        q[:, t::4] = (codes >> np.uint8(2 * t)) & np.uint8(3)
    return (q - np.repeat(zero, GROUP, axis=1)) * np.repeat(scale, GROUP, axis=1)


def split_expert(flat: np.ndarray, d: int, d_ff: int):
    """W1 [d_ff x d], W3 [d_ff x d], W2 [d x d_ff] in fp64 from a stored expert."""
    flat = np.asarray(flat, dtype=np.uint8)
    m = matrix_bytes(d_ff, d)
    assert flat.size == 3 * m
    return (dequantize(flat[:m], d_ff, d), dequantize(flat[m:2 * m], d_ff, d),
            dequantize(flat[2 * m:], d, d_ff))
