"""Parity on the metric's headline cell: the 32-layer Mixtral-shaped stack
(8 bf16 experts per layer, d 4096, d_ff 14336, its own seed) at 4 slots per
layer without speculation, under LRU (Sec. 3.1) and LFU (Sec. 4.2, Table 2's
comparison), on the first 16 decode tokens from the warm start (needs an
MI355X).  The store pins 24 distinct layers; layers 24..31 reuse the pages of
layers 0..7 (see offload.HostStore), gates are distinct for every layer.

Every routing decision and trace record is compared bit for bit, the final
tables of sampled layers too; layer outputs of every token at four layers and
of every layer for two tokens against the fp64 oracle.  The trace analytics
(hit rates, activation histograms, repeat rates) computed from the device
trace must equal the oracle's metrics on the oracle's own trace.
"""
import numpy as np
import pytest

from oracle import metrics, stack
from paper_2511_05814_amd import analysis
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import LazyRig, _say, _tol
from tests._parity import check_decode, check_y_by_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOKENS = 16


@pytest.fixture(scope="module")
def stack_c3():
    cfg = wl.CONFIGS["mixtral-stack"].with_(tokens=TOKENS)
    _say("mixtral-stack (4 slots, no prefetch) host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    rig = LazyRig(cfg)
    yield rig
    rig.store.close()


@pytest.mark.parametrize("policy", ["lfu", "lru"])
def test_mixtral_stack_four_slots(stack_c3, policy):
    rig = stack_c3
    cfg = rig.cfg
    _say("mixtral-stack 4 slots", policy, cfg.tokens, "tokens")
    moe = rig.cache(4, policy)
    hs, recs, _ = rig.run(moe, cfg.tokens)
    want = []
    worst, unc, caches = check_decode(cfg, rig.model, hs, recs, 4, policy, y_tokens=[0, TOKENS - 1],
                                      tol=_tol(cfg), records_out=want)
    ymodel = stack.Model(rig.gates.host, lambda l, e: rig.store.expert(l, e), cfg.d_model, cfg.d_ff, cfg.dtype)
    w_all = check_y_by_layer(ymodel, hs, [0, 10, 21, 31], cfg.top_k, _tol(cfg))
    _say("worst", worst, "every token at layers 0/10/21/31", w_all, "uncertified", unc)
    for l in (0, 13, 31):
        assert moe.state(l) == caches[l].state()
    st = moe.stats()
    assert sum(s["hits"] for s in st) == sum(c.stats.hits for c in caches)
    assert sum(s["misses"] for s in st) == sum(c.stats.misses for c in caches)
    # analytics from the device trace = the oracle's metrics on its own trace
    rep = analysis.report(recs, cfg.layers, cfg.experts, cfg.top_k)
    assert rep["per_layer_hit_rate"] == [round(v, 4) for v in metrics.per_layer_hit_rate(want).values()]
    for key, h in rep["activation_histograms"].items():
        assert h == metrics.activation_histogram(want, int(key) - 1, cfg.experts)
    assert rep["repeat_rate"]["per_layer"] == [round(metrics.repeat_rate(want, l), 4) for l in range(cfg.layers)]
    assert rep["top1_repeat_rate"]["per_layer"] == [round(metrics.top1_repeat_rate(want, l), 4)
                                                    for l in range(cfg.layers)]
    assert analysis.hit_rate(recs) == metrics.hit_rate(want)
    assert analysis.cache_precision_recall(recs, 4) == metrics.cache_pr(want, 4)
    _say(policy, "hit rate", analysis.hit_rate(recs), "top-1 repeat", rep["top1_repeat_rate"]["mean"])
    moe.close()
