"""Lossless packing of bf16 experts: an independent unpacking written from the
documented format must give back every bit pattern, for random weights and
for the awkward ones (zeros, subnormals, infinities, NaN, a partial block)."""
import numpy as np
import pytest

from paper_2511_05814_amd import pack
from paper_2511_05814_amd import workload as wl


def unpack(buf, n):
    """Rebuild n bf16 bit patterns from one packed matrix, entry by entry."""
    buf = np.asarray(buf, dtype=np.uint8)
    out = np.empty(n, dtype=np.uint16)
    nb = (n + 8191) // 8192
    exc = buf[nb * 12560:].view("<u4")
    for b in range(nb):
        blk = buf[b * 12560:(b + 1) * 12560]
        first, count = (int(v) for v in blk[:8].view("<u4"))
        sm, offb, base = blk[16:8208], blk[8208:12304], blk[12304:12560]
        table = {int(e) >> 8: int(e) & 0xFF for e in exc[first:first + count]}
        for i in range(min(8192, n - b * 8192)):
            o = (int(offb[i // 2]) >> (4 * (i % 2))) & 0xF
            e = table[i] if o == 15 else int(base[i // 32]) - o
            s = int(sm[i])
            out[b * 8192 + i] = ((s & 0x80) << 8) | (e << 7) | (s & 0x7F)
    return out


def roundtrip(bits, exc_cap=None):
    need = pack.exceptions_needed(bits)
    buf, total = pack.pack_matrix(bits, need if exc_cap is None else exc_cap)
    assert total == need and buf.size == pack.matrix_capacity(bits.size, need if exc_cap is None else exc_cap)
    assert np.array_equal(unpack(buf, bits.size), bits)
    return buf, total


def test_random_weights_round_trip():
    rng = np.random.default_rng(3)
    bits = wl.f32_to_bf16_bits((rng.standard_normal(20000) * 0.02).astype(np.float32))
    _, total = roundtrip(bits)
    assert total < 20


def test_special_values_round_trip():
    special = np.array([0x0000, 0x8000, 0x0001, 0x807F, 0x7F80, 0xFF80, 0x7FC1, 0x3F80, 0x0080, 0x7F7F],
                       dtype=np.uint16)
    rng = np.random.default_rng(4)
    bits = rng.integers(0, 1 << 16, size=9000, dtype=np.uint16)  # every exponent, NaNs included
    bits[::97] = special[np.arange(bits[::97].size) % special.size]
    _, total = roundtrip(bits)
    assert total > 100  # many offsets of 15 or more


def test_partial_block_and_capacity():
    bits = np.full(8192 + 100, 0x3C00, dtype=np.uint16)
    bits[5] = 0
    bits[8192 + 99] = 0
    buf, total = roundtrip(bits, exc_cap=7)
    assert total == 2 and buf.size % 16 == 0
    with pytest.raises(ValueError):
        pack.pack_matrix(bits, 1)


def test_mixtral_shaped_weights_pack_to_about_12_bits():
    cfg = wl.CONFIGS["tiny-stack"].with_(dtype="bf16")
    w = wl.expert_weights(cfg, 0, 0)
    n = cfg.matrix_elems
    for m in range(3):
        need = pack.exceptions_needed(w[m * n:(m + 1) * n])
        assert pack.matrix_capacity(n, need) * 8 / n < 12.4
