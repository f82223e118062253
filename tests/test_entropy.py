"""The entropy-coded host format (CPU only): the library's encoder output,
read back by an independent decoder written here from the layout documented
in moe_offload.h, gives the input bf16 bits exactly; its codes are prefix
codes of at most 8 bits, optimal where an unrestricted Huffman code already
fits in 8 bits; capacity and shape errors are reported."""
import heapq

import numpy as np
import pytest

from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import entropy as en
from paper_2511_05814_amd import workload as wl


def decode(buf: np.ndarray, n: int) -> np.ndarray:
    """bf16 bit patterns from one coded matrix, one code at a time."""
    nspans = (n + 32767) // 32768
    sb = (4 * nspans + 15) // 16 * 16
    table = buf[:512].view("<u2")
    starts = buf[512:512 + 4 * nspans].view("<u4")
    sm = buf[512 + sb:512 + sb + n]
    streams = buf[512 + sb + n:]
    streams = streams[:streams.size // 4 * 4].view("<u4")
    expo = np.zeros(n, dtype=np.uint16)
    for s in range(nspans):
        steps = min(64, (n - 32768 * s) // 512)
        for lane in range(64):
            k = 0  # word of this lane stream
            acc, nb = 0, 0
            for j in range(steps):
                for u in range(8):
                    while nb < 8:
                        at = int(starts[s]) + 64 * k + lane
                        acc |= int(streams[at]) << nb if at < streams.size else 0
                        k += 1
                        nb += 32
                    ent = int(table[acc & 0xFF])
                    length = ent >> 8
                    assert length > 0, "stream bits that start no code"
                    expo[32768 * s + 512 * j + 8 * lane + u] = ent & 0xFF
                    acc >>= length
                    nb -= length
    smu = sm.astype(np.uint16)
    return ((smu & 0x80) << 8) | (expo << 7) | (smu & 0x7F)


def encode(bits, cap_words=None):
    n = bits.size
    cap = en.default_cap_words(n) if cap_words is None else cap_words
    out = np.full(en.matrix_capacity(n, cap), 0xAB, dtype=np.uint8)
    used = en.pack_matrix(bits, cap, out)
    return out, used


def code_of(table: np.ndarray):
    """(code bits first-bit-lowest, length) per symbol, read off the table."""
    codes = {}
    for w, ent in enumerate(table.view("<u2")):
        if ent:
            s, l = int(ent) & 0xFF, int(ent) >> 8
            c = w & ((1 << l) - 1)
            assert codes.setdefault(s, (c, l)) == (c, l), "inconsistent table"
    return codes


def huffman_cost(freq):
    h = [int(f) for f in freq if f > 0]
    if len(h) < 2:
        return sum(h)
    heapq.heapify(h)
    cost = 0
    while len(h) > 1:
        a, c = heapq.heappop(h), heapq.heappop(h)
        cost += a + c
        heapq.heappush(h, a + c)
    return cost


def bf16(x):
    return wl.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def check_roundtrip(bits, cap_words=None):
    buf, used = encode(bits, cap_words)
    assert np.array_equal(decode(buf, bits.size), bits)
    codes = code_of(buf[:512])
    lengths = {s: l for s, (c, l) in codes.items()}
    assert max(lengths.values()) <= 8
    present = set(((bits >> 7) & 0xFF).tolist())
    assert set(lengths) == present
    if len(present) > 1:
        assert sum(2.0 ** -l for l in lengths.values()) == 1.0  # complete prefix code
    # no code is a prefix of another
    items = sorted(codes.items(), key=lambda kv: kv[1][1])
    for i, (s, (c, l)) in enumerate(items):
        for t, (c2, l2) in items[i + 1:]:
            assert (c2 & ((1 << l) - 1)) != c, (s, t)
    return buf, used, lengths


def test_gaussian_weights_ragged_last_span():
    rng = np.random.default_rng(1)
    n = 32768 + 56 * 512   # the second span has 56 of 64 steps
    bits = bf16(rng.normal(0, 0.02, n))
    buf, used, lengths = check_roundtrip(bits)
    expo = (bits >> 7) & 0xFF
    freq = np.bincount(expo, minlength=256)
    p = freq[freq > 0] / n
    entropy = float(-(p * np.log2(p)).sum())
    avg = sum(freq[s] * l for s, l in lengths.items()) / n
    assert entropy <= avg < entropy + 0.15  # 8-bit codes cost ~0.07 bits more than Huffman
    assert used * 32 / n < 2.85


def test_special_values_and_every_exponent():
    # zeros, subnormals, infinities, NaNs, both signs, and all 256 exponents
    rng = np.random.default_rng(2)
    bits = rng.integers(0, 1 << 16, size=2048, dtype=np.uint16)
    bits[:8] = [0x0000, 0x8000, 0x0001, 0x807F, 0x7F80, 0xFF80, 0x7FC1, 0xFFFF]
    bits[8:264] = (np.arange(256, dtype=np.uint16) << 7) | (bits[8:264] & 0x807F)
    _, used, lengths = check_roundtrip(bits, cap_words=2048 * 12 // 32 + 64)
    assert len(lengths) == 256


def test_single_and_two_symbol_matrices():
    bits = np.full(1024, bf16(1.0), dtype=np.uint16)
    bits[::3] |= 0x8000  # sign and mantissa vary, the exponent does not
    bits[::5] |= 0x0055
    _, used, lengths = check_roundtrip(bits)
    assert lengths == {127: 1} and used == 64   # 16 one-bit codes per lane stream: one row of 64 words
    bits[::7] = bf16(2.0)
    _, _, lengths = check_roundtrip(bits)
    assert lengths == {127: 1, 128: 1}


def test_length_limit_and_optimality():
    # geometric exponent frequencies: an unrestricted Huffman code would need
    # 20-bit codes; the encoder must stay within 8 bits
    sizes = [2 ** (19 - i) for i in range(20)]
    expo = np.concatenate([np.full(sz, 100 + i) for i, sz in enumerate(sizes)])
    pad = (-expo.size) % 512
    expo = np.concatenate([expo, np.full(pad, 100)])
    rng = np.random.default_rng(3)
    expo = rng.permutation(expo)
    bits = (expo.astype(np.uint16) << 7) | rng.integers(0, 128, expo.size).astype(np.uint16)
    _, _, lengths = check_roundtrip(bits, cap_words=expo.size * 12 // 32 + 64)
    assert max(lengths.values()) == 8
    # a distribution whose Huffman code fits in 8 bits: same cost as Huffman
    p = np.array([40, 30, 12, 9, 5, 3, 1])
    expo = np.repeat(np.arange(120, 127), p * 512)
    bits = (rng.permutation(expo).astype(np.uint16) << 7)
    _, _, lengths = check_roundtrip(bits, cap_words=expo.size * 12 // 32 + 64)
    freq = np.bincount((bits >> 7) & 0xFF, minlength=256)
    assert sum(freq[s] * l for s, l in lengths.items()) == huffman_cost(freq)


def test_capacity_and_shape_errors():
    rng = np.random.default_rng(4)
    bits = bf16(rng.normal(0, 0.02, 4096))
    with pytest.raises(b.MoeError) as e:
        encode(bits, cap_words=64)
    assert e.value.code == b.MOE_ERR_ARG and "capacity" in str(e.value)
    assert b.moe_entropy_matrix_bytes(1000, 100) == 0
    assert b.moe_entropy_matrix_bytes(0, 100) == 0
    with pytest.raises(ValueError):
        en.matrix_capacity(1000, 100)
    for n, cap in ((512, 1), (32768, 5000), (32768 * 3 + 512, 77)):
        assert b.moe_entropy_matrix_bytes(n, cap) == en.matrix_capacity(n, cap)


def test_expert_of_the_workload():
    # one matrix of a 64-expert-shaped expert (d 2048, d_ff 1408 is not tiny,
    # so only its first 2 spans are decoded here; the sizes are checked whole)
    cfg = wl.CONFIGS["fine-grained"]
    w = wl.expert_weights(cfg, 0, 0)
    n = cfg.matrix_elems
    buf, used = encode(w[:n])
    assert used * 32 / n < 2.85
    head = 65536
    sub, _ = encode(w[:head])
    assert np.array_equal(decode(sub, head), w[:head])
