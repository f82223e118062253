"""GPU parity of decode on group-quantised experts (2-bit codes, groups of 16,
fp16 scales, 8-bit zero codes; the paper's expert setting, Sec. 5.1) against
the fp64 oracle, which decodes the same stored bytes.  Routing, guesses and the
cache trace bit for bit; layer outputs within 1e-5 relative L2 (the dequantised
weights are exact fp32 numbers on both sides)."""
import numpy as np
import pytest

from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import Rig, _say, _tol
from tests._parity import check_decode

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def tq():
    cfg = wl.CONFIGS["tiny-q2"]
    _say("tiny-q2", cfg)
    return Rig(cfg)


@pytest.mark.parametrize("policy", ["lru", "lfu"])
def test_q2_decode_parity(tq, policy):
    cfg = tq.cfg
    _say("q2 decode", policy)
    moe = tq.cache(4, policy)
    hs, recs, _ = tq.run(moe, cfg.tokens)
    worst, unc, caches = check_decode(cfg, tq.model, hs, recs, 4, policy, tol=_tol(cfg))
    _say("worst y rel L2", worst, "uncertified", unc)
    st = moe.stats()
    for l in range(cfg.layers):
        o = caches[l].stats
        assert (st[l]["hits"], st[l]["misses"]) == (o.hits, o.misses)
        assert st[l]["bytes_fetched"] == o.misses * cfg.expert_bytes
    moe.close()


def test_q2_prefetch_parity_all_fetch_modes(tq):
    cfg = tq.cfg
    outs = []
    for mode in (b.MOE_FETCH_KERNEL, b.MOE_FETCH_DMA, b.MOE_FETCH_SPLIT):
        _say("q2 lfu + prefetch 2, fetch mode", mode)
        moe = tq.cache(4, "lfu", prefetch_max=2, fetch_mode=mode)
        hs, recs, H = tq.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
        worst, unc, _ = check_decode(cfg, tq.model, hs, recs, 4, "lfu", prefetch=True, pmax=2, tol=_tol(cfg))
        _say("worst", worst, "uncertified", unc)
        outs.append((H.tobytes(), recs))
        moe.close()
    assert outs[0] == outs[1] == outs[2]


def test_q2_ragged_shape():
    # rows and columns that fill neither a wave step nor a row block: the
    # clamped loads and partial chunks
    cfg = wl.CONFIGS["tiny-q2"].with_(layers=3, experts=5, top_k=3, d_model=192, d_ff=320, tokens=24)
    _say("q2 ragged", cfg)
    rig = Rig(cfg)
    moe = rig.cache(3, "lru", prefetch_max=1)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    worst, unc, _ = check_decode(cfg, rig.model, hs, recs, 3, "lru", prefetch=True, pmax=1, tol=_tol(cfg))
    _say("worst", worst, "uncertified", unc)
    moe.close()
    rig.store.close()


def test_q2_mixtral_layer_full_size():
    # the Mixtral-shaped layer (d 4096, d_ff 14336) at full size: 48 tokens
    cfg = wl.CONFIGS["mixtral-layer-q2"].with_(tokens=48)
    _say("mixtral-layer-q2 host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    rig = Rig(cfg)
    moe = rig.cache(4, "lfu")
    hs, recs, _ = rig.run(moe, cfg.tokens)
    worst, unc, caches = check_decode(cfg, rig.model, hs, recs, 4, "lfu", tol=_tol(cfg))
    _say("worst y rel L2", worst, "uncertified", unc, "hits", caches[0].stats.hits)
    moe.close()
    rig.store.close()
