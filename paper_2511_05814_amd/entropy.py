"""Entropy-coded bf16 experts for the host store (MOE_HOST_ENTROPY).

At batch-1 decode every miss moves a whole expert over the host link, and
the link is the bound, so every bit a weight costs in host memory is time.
A bf16 weight is a sign, an 8-bit exponent and a 7-bit mantissa.  Sign and
mantissa of N(0, sigma) weights are close to uniform, but the exponent takes
only a handful of values with a steeply falling distribution: its entropy is
about 2.5 bits.  The format keeps sign and mantissa as one byte and codes
the exponent with a canonical prefix code of at most 8 bits built for each
matrix, so a weight costs about 10.9 bits instead of 16; the GPU rebuilds the
identical bf16 bits after the copy.  The byte layout is documented with
MOE_HOST_ENTROPY in include/moe_offload.h; the encoder is the library's
moe_entropy_pack (host code, one matrix per call, safe to run in parallel).
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import binding as b

SPAN = 32768     # weights per span: 64 lane streams x 64 steps x 8 weights
LANES = 64
MAX_LEN = 8
TABLE_BYTES = 2 << MAX_LEN


def spans(n: int) -> int:
    return (n + SPAN - 1) // SPAN


def starts_bytes(n: int) -> int:
    """Bytes of the span-start table (one uint32 per span, padded to 16)."""
    return (4 * spans(n) + 15) // 16 * 16


def matrix_capacity(n: int, cap_words: int) -> int:
    """Bytes of one matrix of n weights with cap_words stream words."""
    if n <= 0 or n % 512:
        raise ValueError("entropy-coded matrices need a positive multiple of 512 weights")
    return (TABLE_BYTES + starts_bytes(n) + n + 4 * cap_words + 15) // 16 * 16


def default_cap_words(n: int) -> int:
    """Stream words that hold the exponents of N(0, sigma) bf16 weights with
    room to spare: 3 bits a weight (they take about 2.75 with the padding of
    every span to its longest lane stream)."""
    return (3 * n + 31) // 32 + 64 * spans(n)


def pack_matrix(bits: np.ndarray, cap_words: int, out: np.ndarray) -> int:
    """Encode flat bf16 bit patterns (n of them) into `out` (uint8, exactly
    matrix_capacity(n, cap_words) bytes, any host memory).  Returns the stream
    words used; raises binding.MoeError if they exceed cap_words."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16).reshape(-1)
    n = bits.size
    if out.dtype != np.uint8 or out.size != matrix_capacity(n, cap_words) or not out.flags.c_contiguous:
        raise ValueError("out must be a contiguous uint8 array of matrix_capacity(n, cap_words) bytes")
    return b.moe_entropy_pack(bits.ctypes.data_as(ctypes.c_void_p).value, n, cap_words,
                              out.ctypes.data_as(ctypes.c_void_p).value)
