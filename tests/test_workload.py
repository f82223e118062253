"""The seeded input generator: determinism, bf16 rounding, layout, statistics."""
import hashlib

import numpy as np
import pytest
import torch

from paper_2511_05814_amd import workload as wl


def _small(name="tiny-stack", **kw):
    return wl.CONFIGS[name].with_(**kw)


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 0.02,
                        rng.standard_normal(1000).astype(np.float32) * 1e30,
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8,
                                  0.0, -0.0, 1e-40], np.float32)])
    ours = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_same_seed_same_bytes_and_distinct_streams():
    cfg = _small()
    a = wl.expert_weights(cfg, 1, 3)
    b = wl.expert_weights(cfg, 1, 3)
    assert hashlib.sha256(a.tobytes()).digest() == hashlib.sha256(b.tobytes()).digest()
    c = wl.expert_weights(cfg, 1, 4)
    assert not np.array_equal(a, c)
    assert np.array_equal(wl.hidden_states(cfg, 10), wl.hidden_states(cfg, 10))
    assert np.array_equal(wl.gate_weights(cfg), wl.gate_weights(cfg))


def test_host_store_layout_matches_per_expert_draws():
    cfg = _small(layers=2, experts=3, d_model=16, d_ff=24, dtype="bf16")
    buf = np.empty(cfg.layers * cfg.experts * cfg.expert_bytes, np.uint8)
    wl.fill_host_store(cfg, buf, workers=3)
    v = buf.view(np.uint16).reshape(cfg.layers, cfg.experts, -1)
    for l in range(cfg.layers):
        for e in range(cfg.experts):
            assert np.array_equal(v[l, e], wl.expert_weights(cfg, l, e))


def test_weight_statistics():
    cfg = _small()
    w = wl.expert_weights(cfg, 0, 0)
    assert w.dtype == np.float32 and w.size == 3 * 256 * 512
    assert abs(float(w.std()) - 0.02) < 0.0005 and abs(float(w.mean())) < 0.0005


def test_zipf_closed_form():
    p = wl.zipf_probabilities(8, 1.1)
    h = sum(r ** -1.1 for r in range(1, 9))
    assert p[0] == pytest.approx(1 / h, rel=1e-14)
    assert p[1] / p[0] == pytest.approx(2 ** -1.1, rel=1e-14)
    assert p.sum() == pytest.approx(1.0, rel=1e-15)


def test_concept_chain_statistics():
    cfg = _small(experts=8, zipf_s=1.1, markov_p=0.6)
    c = wl.concept_chain(cfg, 40000)
    p = wl.zipf_probabilities(8, 1.1)
    # stationary law is the Zipf law; repeat rate is p + (1-p) sum p_i^2
    freq = np.bincount(c, minlength=8) / len(c)
    np.testing.assert_allclose(freq, p, atol=0.02)
    rep = float(np.mean(c[1:] == c[:-1]))
    assert rep == pytest.approx(0.6 + 0.4 * float((p ** 2).sum()), abs=0.02)


def test_hidden_state_shape_and_amplitude():
    cfg = _small()
    h = wl.hidden_states(cfg, 256)
    assert h.shape == (256, 256) and h.dtype == np.float32
    u = wl.concept_directions(cfg)
    np.testing.assert_allclose(np.linalg.norm(u, axis=1), 1.0, rtol=1e-6)
    c = wl.concept_chain(cfg, 256)
    proj = np.einsum("td,td->t", h.astype(np.float64), u[c].astype(np.float64))
    assert abs(float(proj.mean()) - cfg.alpha) < 0.5


def test_configs_sizes():
    c2 = wl.CONFIGS["mixtral-layer"]
    assert c2.expert_bytes == 352_321_536
    c5 = wl.CONFIGS["fine-grained"]
    assert c5.expert_bytes == 17_301_504
    assert c5.layers * c5.experts * c5.expert_bytes == 26_575_110_144
    assert wl.CONFIGS["tiny-stack"].expert_bytes == 1_572_864
