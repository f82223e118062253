"""Free-running parity (needs an MI355X): the GPU decodes with its own fp32
hidden states from layer to layer, the oracle with its own fp64 ones from
the same inputs, and the two are compared without teacher forcing: routing
and cache traces must agree record for record (if a near-tie ever sent them
apart, the test names the first (token, layer) where they part), and the
final hidden states within the FFN tolerance of the weight type.

Workloads: the tiny two-layer fp32 stack (all 64 tokens, LRU and LFU with
next-layer prefetch) and the Mixtral-shaped bf16 layer (all 256 tokens)."""
import numpy as np
import pytest

from oracle import stack
from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import Rig, _say, _tol
from tests._parity import rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def first_divergence(got, want):
    for i, (a, w) in enumerate(zip(got, want)):
        if a != w:
            return i, a, w
    if len(got) != len(want):
        return min(len(got), len(want)), None, None
    return None


def free_run(rig, slots, policy, prefetch_max, tol):
    cfg = rig.cfg
    flags = b.MOE_PREFETCH_NEXT if prefetch_max else 0
    moe = rig.cache(slots, policy, prefetch_max=prefetch_max)
    hs, recs, H = rig.run(moe, cfg.tokens, flags=flags)
    moe.close()
    h0 = wl.hidden_states(cfg, cfg.tokens).astype(np.float64)
    ohs, orecs, _, unc = stack.decode_free(rig.model, h0, cfg.top_k, policy, slots,
                                           prefetch=bool(prefetch_max), prefetch_max=prefetch_max)
    want = [r.astuple() for r in orecs]
    div = first_divergence(recs, want)
    assert div is None, f"routing or trace parts at record {div[0]}: gpu {div[1]} oracle {div[2]}"
    worst = max(rel_l2(H[t] - h0[t], ohs[t, cfg.layers] - h0[t]) for t in range(cfg.tokens))
    _say(cfg.name, policy, "free-running: traces identical, worst rel L2 of h_L - h_0", worst,
         "uncertified oracle decisions", unc)
    assert worst <= tol, worst


@pytest.mark.parametrize("policy,pmax", [("lru", 0), ("lfu", 2)])
def test_tiny_stack_free_running(policy, pmax):
    cfg = wl.CONFIGS["tiny-stack"]
    rig = Rig(cfg)
    free_run(rig, 4, policy, pmax, _tol(cfg))
    rig.store.close()


def test_mixtral_layer_free_running():
    cfg = wl.CONFIGS["mixtral-layer"]
    rig = Rig(cfg)  # the oracle keeps the 8 experts widened to fp64 (11 GB of host memory)
    free_run(rig, 4, "lfu", 0, _tol(cfg))
    rig.store.close()
