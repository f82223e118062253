"""Lossless packing of bf16 experts for the host store.

The experts are fetched over the host link on every miss, and at batch-1
decode that transfer is the bound.  A bf16 weight is a sign, an 8-bit
exponent and a 7-bit mantissa; sign and mantissa are close to random, but
within a small group of weights the exponents span only a few binades.  The
packed form keeps sign and mantissa as one byte and the exponent as a 4-bit
offset below the group's largest exponent, so a weight costs about 12.25 bits
instead of 16 and the GPU rebuilds the identical bf16 bits after the copy.

Format of one matrix of n weights (row-major, as in the plain store), cut
into blocks of 8192 weights (256 groups of 32; the last block is padded):

  block (12560 bytes)
    header  16 bytes   uint32 first exception of the block (index into the
                       matrix's list), uint32 number of exceptions, 8 zero bytes
    sm      8192 bytes weight i: (sign << 7) | mantissa
    off     4096 bytes weight i: 4-bit offset, low nibble for even i
    base     256 bytes group g: largest exponent of its 32 weights
  exceptions  uint32 entries ((index within block) << 8) | exponent, in block
              and index order, for every weight whose offset would be 15 or
              more (stored offset 15): exact zeros, subnormals, tiny values

The matrix is padded to a capacity of blocks * 12560 + 4 * exc_cap bytes
(rounded up to 16), and an expert is W1 | W3 | W2 at that capacity each.
"""
from __future__ import annotations

import numpy as np

BLOCK = 8192
GROUP = 32
BLOCK_BYTES = 16 + BLOCK + BLOCK // 2 + BLOCK // GROUP  # 12560
ESC = 15


def blocks(n: int) -> int:
    return (n + BLOCK - 1) // BLOCK


def matrix_capacity(n: int, exc_cap: int) -> int:
    return (blocks(n) * BLOCK_BYTES + 4 * exc_cap + 15) // 16 * 16


def expert_capacity(n: int, exc_cap: int) -> int:
    return 3 * matrix_capacity(n, exc_cap)


def pack_matrix(bits: np.ndarray, exc_cap: int, out: np.ndarray = None):
    """Pack flat bf16 bit patterns (uint16, n of them).  Returns (packed bytes
    of matrix_capacity(n, exc_cap), number of exceptions); raises if the
    exceptions exceed exc_cap."""
    bits = np.asarray(bits, dtype=np.uint16).reshape(-1)
    n = bits.size
    nb = blocks(n)
    cap = matrix_capacity(n, exc_cap)
    if out is None:
        out = np.zeros(cap, dtype=np.uint8)
    else:
        assert out.size == cap and out.dtype == np.uint8
        out[:] = 0
    pad = np.zeros(nb * BLOCK, dtype=np.uint16)
    pad[:n] = bits
    w = pad.reshape(nb, BLOCK // GROUP, GROUP)
    expo = ((w >> np.uint16(7)) & np.uint16(0xFF)).astype(np.int32)
    sm = (((w >> np.uint16(8)) & np.uint16(0x80)) | (w & np.uint16(0x7F))).astype(np.uint8)
    base = expo.max(axis=2)
    off = base[..., None] - expo
    valid = (np.arange(nb * BLOCK) < n).reshape(nb, BLOCK // GROUP, GROUP)
    esc = (off >= ESC) & valid
    off4 = np.where(off >= ESC, ESC, off).astype(np.uint8)
    offb = (off4[..., 0::2] | (off4[..., 1::2] << np.uint8(4))).astype(np.uint8)
    # exceptions: (index within block << 8) | exponent, block by block
    esc_flat = esc.reshape(nb, BLOCK)
    counts = esc_flat.sum(axis=1)
    total = int(counts.sum())
    if total > exc_cap:
        raise ValueError(f"{total} exceptions exceed the capacity {exc_cap}")
    first = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.uint32)
    blk, idx = np.nonzero(esc_flat)
    entries = ((idx.astype(np.uint32) << np.uint32(8)) |
               expo.reshape(nb, BLOCK)[blk, idx].astype(np.uint32)).astype("<u4")
    body = out[:nb * BLOCK_BYTES].reshape(nb, BLOCK_BYTES)
    hdr = np.zeros((nb, 4), dtype="<u4")
    hdr[:, 0] = first
    hdr[:, 1] = counts
    body[:, :16] = hdr.view(np.uint8).reshape(nb, 16)
    body[:, 16:16 + BLOCK] = sm.reshape(nb, BLOCK)
    body[:, 16 + BLOCK:16 + BLOCK + BLOCK // 2] = offb.reshape(nb, BLOCK // 2)
    body[:, 16 + BLOCK + BLOCK // 2:] = base.astype(np.uint8)
    ex = out[nb * BLOCK_BYTES:nb * BLOCK_BYTES + 4 * total]
    ex[:] = entries.view(np.uint8)
    return out, total


def exceptions_needed(bits: np.ndarray) -> int:
    """Exceptions pack_matrix would record for these bf16 bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16).reshape(-1)
    n = bits.size
    pad = np.zeros(blocks(n) * BLOCK, dtype=np.uint16)
    pad[:n] = bits
    expo = ((pad >> np.uint16(7)) & np.uint16(0xFF)).astype(np.int32).reshape(-1, GROUP)
    off = expo.max(axis=1, keepdims=True) - expo
    valid = (np.arange(pad.size) < n).reshape(-1, GROUP)
    return int(((off >= ESC) & valid).sum())
