"""Pins for the oracle's residual stack, teacher-forced replay and prefill (CPU only)."""
import numpy as np
import pytest

from oracle import moe, stack
from oracle.cache import KIND_ACCESS, make_caches
from paper_2511_05814_amd import workload as wl


def _model(cfg):
    gates = wl.gate_weights(cfg)
    return stack.Model(gates, lambda l, e: wl.expert_weights(cfg, l, e),
                       cfg.d_model, cfg.d_ff, cfg.dtype)


@pytest.fixture(scope="module")
def tiny():
    cfg = wl.CONFIGS["tiny-stack"].with_(d_model=64, d_ff=96)
    return cfg, _model(cfg), wl.hidden_states(cfg, 24).astype(np.float64)


def test_free_run_residual_and_norm(tiny):
    cfg, m, h0 = tiny
    hs, recs, caches, unc = stack.decode_free(m, h0, cfg.top_k, "lfu", 4)
    assert unc == 0
    for t in range(3):
        for l in range(cfg.layers):
            h = hs[t, l]
            st = stack.layer_step(m, l, h, cfg.top_k)
            np.testing.assert_allclose(hs[t, l + 1] - h, st["y"], rtol=1e-12, atol=1e-13)
    assert sum(1 for r in recs if r.kind == KIND_ACCESS) == 24 * cfg.layers * cfg.top_k


def test_routing_uses_the_scale_free_logits(tiny):
    # scaling h by a positive constant must not change the selected experts
    cfg, m, h0 = tiny
    for t in range(10):
        a = stack.layer_step(m, 0, h0[t], cfg.top_k, with_ffn=False)
        b = stack.layer_step(m, 0, 7.5 * h0[t], cfg.top_k, with_ffn=False)
        assert list(a["ids"]) == list(b["ids"])
        np.testing.assert_allclose(a["g"], b["g"], rtol=1e-6)


def test_replay_of_free_run_routing_gives_the_same_trace(tiny):
    cfg, m, h0 = tiny
    hs, recs, _, _ = stack.decode_free(m, h0, cfg.top_k, "lru", 4, prefetch=True, prefetch_max=2)
    ids = [[stack.layer_step(m, l, hs[t, l], cfg.top_k, with_ffn=False)["ids"]
            for l in range(cfg.layers)] for t in range(len(h0))]
    gs = [[stack.layer_step(m, l, hs[t, l], cfg.top_k, with_ffn=False, guess=True).get("guesses")
           for l in range(cfg.layers)] for t in range(len(h0))]
    recs2, _ = stack.replay(ids, gs, cfg.layers, cfg.experts, 4, "lru", 2)
    assert [r.astuple() for r in recs] == [r.astuple() for r in recs2]


def test_prefill_rows_equal_decode_rows(tiny):
    cfg, m, h0 = tiny
    cache = make_caches(1, cfg.experts, 4, "lfu")[0]
    out, ids, g, cert, recs = stack.prefill_layer(m, 0, h0[:12], cfg.top_k, cache)
    for t in range(12):
        st = stack.layer_step(m, 0, h0[t], cfg.top_k)
        assert list(st["ids"]) == list(ids[t])
        np.testing.assert_allclose(out[t], h0[t] + st["y"], rtol=1e-13, atol=1e-13)
    assert sum(r.rank for r in recs) == 12 * cfg.top_k


def test_bf16_model_reads_exact_stored_values():
    cfg = wl.CONFIGS["tiny-stack"].with_(d_model=32, d_ff=48, dtype="bf16", layers=1)
    m = _model(cfg)
    raw = wl.expert_weights(cfg, 0, 2)
    w1, _, _ = m.expert(0, 2)
    # every widened weight re-rounds to its own bf16 pattern
    assert np.array_equal(wl.f32_to_bf16_bits(w1.astype(np.float32).reshape(-1)),
                          raw[:32 * 48])
    assert np.array_equal(moe.bf16_bits_to_f64(raw[:32 * 48]).reshape(48, 32), w1)
