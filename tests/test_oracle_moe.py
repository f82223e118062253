"""Pins for the fp64 MoE math of the oracle (CPU only).

Each check rests on something outside the oracle's own code: a closed form,
a known constant, a library routine for a special case, exact rational
arithmetic, or a structured input whose answer is known by inspection.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import expit

from oracle import moe


# ---- bf16 widening -----------------------------------------------------------
@pytest.mark.parametrize("bits,value", [
    (0x3F80, 1.0), (0xC000, -2.0), (0x3E80, 0.25), (0x0000, 0.0),
    (0x8000, -0.0), (0x0001, 2.0 ** -133), (0x7F7F, (2 - 2 ** -7) * 2.0 ** 127),
    (0x3FC0, 1.5), (0x4049, 3.140625),
])
def test_bf16_widening_known_patterns(bits, value):
    assert moe.bf16_bits_to_f64(np.array([bits], np.uint16))[0] == value


# ---- rms ---------------------------------------------------------------------
def test_rms_constant_vector():
    h = np.full(100, 3.0)
    assert moe.rms(h) == pytest.approx(math.sqrt(9.0 + 1e-5), rel=1e-15)


def test_rms_scale():
    rng = np.random.default_rng(0)
    h = rng.standard_normal(64)
    ms = sum(float(v) ** 2 for v in h) / 64
    assert moe.rms(h) == pytest.approx(math.sqrt(ms + 1e-5), rel=1e-14)


# ---- softmax / top-k / combine weights ----------------------------------------
def test_softmax_sums_to_one_and_shift_invariant():
    rng = np.random.default_rng(1)
    for _ in range(50):
        v = rng.standard_normal(rng.integers(1, 70)) * 30
        p = moe.softmax(v)
        assert abs(p.sum() - 1.0) < 1e-12
        assert np.all(p > 0)
        np.testing.assert_allclose(moe.softmax(v + 1234.5), p, rtol=1e-12, atol=0)


def test_softmax_two_way_is_logistic():
    for a, b in [(0.0, 0.0), (1.0, -1.0), (5.0, 2.0), (-40.0, 3.0)]:
        p = moe.softmax(np.array([a, b]))
        assert p[0] == pytest.approx(expit(a - b), rel=1e-14, abs=1e-300)


def _brute_topk(z, k):
    # full sort of (logit desc, id asc) written as an exhaustive selection
    remaining = list(range(len(z)))
    out = []
    for _ in range(k):
        best = remaining[0]
        for e in remaining[1:]:
            if z[e] > z[best] or (z[e] == z[best] and e < best):
                best = e
        out.append(best)
        remaining.remove(best)
    return out


def test_topk_matches_bruteforce():
    rng = np.random.default_rng(2)
    for _ in range(500):
        E = int(rng.integers(1, 65))
        k = int(rng.integers(1, E + 1))
        z = rng.integers(-3, 4, size=E).astype(np.float64)  # many exact ties
        if rng.random() < 0.5:
            z = rng.standard_normal(E)
        assert list(moe.topk(z, k)) == _brute_topk(z, k)


def test_topk_duplicate_gate_rows_tie_to_lower_id():
    rng = np.random.default_rng(3)
    h = rng.standard_normal(32)
    w = rng.standard_normal((8, 32)) * 0.01
    w[2] = 10 * h / np.linalg.norm(h)   # experts 2 and 5 share one gate row that
    w[5] = w[2]                         # dominates every other row
    z = moe.gate_logits(w, h)
    assert z[2] == z[5] and z[2] > np.max(np.delete(z, [2, 5]))
    assert list(moe.topk(z, 1)) == [2]
    assert list(moe.topk(z, 2)) == [2, 5]


def test_combine_weights_k2_is_logistic_and_sums_to_one():
    rng = np.random.default_rng(4)
    for _ in range(100):
        z = rng.standard_normal(8) * 4
        r = float(rng.uniform(0.5, 5))
        ids = moe.topk(z, 2)
        g = moe.combine_weights(z, ids, r)
        assert abs(g.sum() - 1) < 1e-14
        assert g[0] == pytest.approx(expit((z[ids[0]] - z[ids[1]]) / r), rel=1e-13)
        assert g[0] >= g[1]


def test_combine_weights_k_equals_E_is_full_softmax_and_k1_is_one():
    z = np.array([0.3, -1.0, 2.5, 0.0])
    ids = moe.topk(z, 4)
    g = moe.combine_weights(z, ids, 2.0)
    full = np.exp(z / 2.0) / np.exp(z / 2.0).sum()
    np.testing.assert_allclose(g, full[ids], rtol=1e-14)
    assert moe.combine_weights(z, moe.topk(z, 1), 2.0)[0] == 1.0


def test_topk_of_softmax_equals_topk_of_logits():
    rng = np.random.default_rng(5)
    for _ in range(100):
        z = rng.standard_normal(16)
        p = moe.softmax(z / 1.7)
        assert list(moe.topk(p, 4)) == list(moe.topk(z, 4))


# ---- fp64 logit error bound and certification ----------------------------------
def test_logit_error_bound_covers_exact_dot():
    rng = np.random.default_rng(6)
    for _ in range(20):
        d = int(rng.integers(8, 300))
        w = rng.standard_normal((3, d)) * 0.02
        h = rng.standard_normal(d) * 10
        z = moe.gate_logits(w, h)
        tau = moe.logit_error_bound(w, h)
        for e in range(3):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(w[e], h))
            assert abs(Fraction(float(z[e])) - exact) <= Fraction(float(tau[e])) / 2


def test_certification_rejects_near_ties():
    z = np.array([1.0, 1.0 + 1e-15, -3.0])
    tau = np.full(3, 1e-12)
    ids = moe.topk(z, 1)
    assert not moe.topk_certified(z, ids, tau)
    z2 = np.array([1.0, 0.5, -3.0])
    assert moe.topk_certified(z2, moe.topk(z2, 2), tau)


# ---- SiLU and the SwiGLU expert ---------------------------------------------------
def test_silu_constants_and_identity():
    assert moe.silu(np.array([0.0]))[0] == 0.0
    assert moe.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert moe.silu(np.array([1.0]))[0] == pytest.approx(0.7310585786300049, rel=1e-15)
    a = np.linspace(-30, 30, 121)
    np.testing.assert_allclose(moe.silu(-a), moe.silu(a) - a, atol=1e-12)
    np.testing.assert_allclose(moe.silu(a), a * expit(a), rtol=1e-13, atol=1e-300)


def test_split_expert_layout():
    d, dff = 3, 5
    flat = np.arange(3 * d * dff, dtype=np.float64)
    w1, w3, w2 = moe.split_expert(flat, d, dff)
    assert w1.shape == (dff, d) and w3.shape == (dff, d) and w2.shape == (d, dff)
    assert w1[4, 2] == 4 * d + 2
    assert w3[1, 0] == d * dff + 1 * d
    assert w2[2, 4] == 2 * d * dff + 2 * dff + 4


def test_expert_ffn_one_hot_structure():
    # d = 2, d_ff = 3.  W1 picks x_0 into hidden unit 1 with gain 1, W3 picks
    # x_1 into the same unit with gain 3, W2 sends hidden unit 1 to output 1
    # with gain 0.5: y = [0, 0.5 * SiLU(1 * x_0) * (3 * x_1)].
    w1 = np.zeros((3, 2)); w1[1, 0] = 1.0
    w3 = np.zeros((3, 2)); w3[1, 1] = 3.0
    w2 = np.zeros((2, 3)); w2[1, 1] = 0.5
    x = np.array([1.0, 2.0])
    y = moe.expert_ffn(w1, w3, w2, x)
    assert y[0] == 0.0
    assert y[1] == pytest.approx(0.5 * 0.7310585786300049 * 6.0, rel=1e-15)


def test_expert_ffn_special_cases():
    rng = np.random.default_rng(7)
    w1, w3, w2 = (rng.standard_normal(s) for s in [(6, 4), (6, 4), (4, 6)])
    assert np.all(moe.expert_ffn(w1, w3, w2, np.zeros(4)) == 0)
    assert np.all(moe.expert_ffn(w1, w3, np.zeros((4, 6)), rng.standard_normal(4)) == 0)
    # W3 = 0 kills the gate product
    assert np.all(moe.expert_ffn(w1, np.zeros((6, 4)), w2, rng.standard_normal(4)) == 0)


def test_moe_output_identical_experts_independent_of_routing():
    rng = np.random.default_rng(8)
    w = tuple(rng.standard_normal(s) * 0.3 for s in [(16, 8), (16, 8), (8, 16)])
    x = rng.standard_normal(8)
    base = moe.expert_ffn(*w, x)
    for ids in ([0, 1], [3, 7], [5, 2]):
        g = moe.softmax(rng.standard_normal(2))
        np.testing.assert_allclose(moe.moe_output(lambda e: w, ids, g, x), base, rtol=1e-13)


def test_moe_layer_k1_and_residual():
    rng = np.random.default_rng(9)
    E, d, dff = 4, 8, 12
    ex = [tuple(rng.standard_normal(s) * 0.2 for s in [(dff, d), (dff, d), (d, dff)])
          for _ in range(E)]
    gate = rng.standard_normal((E, d))
    h = rng.standard_normal(d) * 3
    h2, ids, g, _ = moe.moe_layer(gate, lambda e: ex[e], h, 1)
    assert g[0] == 1.0
    r = math.sqrt(float(np.mean(h * h)) + 1e-5)
    np.testing.assert_allclose(h2 - h, moe.expert_ffn(*ex[ids[0]], h / r), rtol=1e-12, atol=1e-14)
    assert ids[0] == int(np.argmax(gate @ h))
