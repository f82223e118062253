"""Parity at the full size of the 32-layer Mixtral-shaped stack (needs an
MI355X): 32 layers of 8 bf16 experts (d 4096, d_ff 14336), each fetch a whole
352 MB expert over the host link.  The driver pins at most about 70 GB, so the
store pins 24 distinct layers and layers 24..31 reuse the pages of layers
0..7 (see offload.HostStore); gates are distinct for every layer.

* next-layer prefetch with 4 slots, LFU, on a token prefix;
* 2 slots with LRU and 6 slots with LFU on a shorter prefix.

Routing, guesses, every trace record and sampled tables are compared bit for
bit; layer outputs on sampled tokens against the fp64 oracle.
"""
import numpy as np
import pytest

from oracle import moe as omoe
from oracle import stack
from oracle.cache import make_caches
from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import LazyRig, _say, _tol
from tests._parity import check_decode, check_y_by_layer, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def mixtral_stack():
    cfg = wl.CONFIGS["mixtral-stack-prefetch"].with_(tokens=24)
    _say("mixtral-stack host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    rig = LazyRig(cfg)
    yield rig
    rig.store.close()


def test_mixtral_stack_prefetch_full_size(mixtral_stack):
    rig = mixtral_stack
    cfg = rig.cfg
    _say("mixtral-stack prefetch, 4 slots, lfu,", cfg.tokens, "tokens")
    moe = rig.cache(4, "lfu", prefetch_max=2)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    # outputs at sampled layers; traces for every (token, layer)
    worst, unc, caches = check_decode(cfg, rig.model, hs, recs, 4, "lfu", prefetch=True, pmax=2,
                                      y_tokens=[0, 23], tol=_tol(cfg))
    ymodel = stack.Model(rig.gates.host, lambda l, e: rig.store.expert(l, e), cfg.d_model, cfg.d_ff, cfg.dtype)
    w_all = check_y_by_layer(ymodel, hs, [0, 16, 31], cfg.top_k, _tol(cfg))
    _say("worst", worst, "every token at layers 0/16/31", w_all, "uncertified", unc)
    for l in (0, 17, 31):
        assert moe.state(l) == caches[l].state()
    moe.close()


@pytest.mark.parametrize("slots,policy", [(2, "lru"), (6, "lfu")])
def test_mixtral_stack_slot_sweep(mixtral_stack, slots, policy):
    rig = mixtral_stack
    cfg = rig.cfg.with_(tokens=10)
    _say("mixtral-stack", slots, "slots", policy)
    moe = rig.cache(slots, policy)
    hs, recs, _ = rig.run(moe, cfg.tokens)
    check_decode(cfg, rig.model, hs, recs, slots, policy, y_tokens=[], tol=_tol(cfg))
    moe.close()
