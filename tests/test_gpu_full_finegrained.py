"""Parity at the full size of the 64-expert stack (needs an MI355X): the whole
4096-token prefill through all 24 layers (26.6 GB pinned host store, 16 slots,
LFU), then its 256 decode tokens with next-layer prefetch.

Routing, every prefill and decode trace record are compared bit for bit; layer
outputs on sampled rows and tokens against the fp64 oracle.
"""
import numpy as np
import pytest

from oracle import moe as omoe
from oracle import stack
from oracle.cache import make_caches
from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import LazyRig, _say
from tests._parity import check_decode, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def test_fine_grained_full_prefill_and_decode():
    cfg = wl.CONFIGS["fine-grained"]
    T, K, L = cfg.prefill_tokens, cfg.top_k, cfg.layers
    _say("fine-grained full: prefill", T, "decode", cfg.tokens, "layers", L)
    rig = LazyRig(cfg)
    moe = rig.cache(16, "lfu", prefetch_max=cfg.prefetch_max, max_prefill_tokens=T)
    h = wl.hidden_states(cfg)
    H = torch.from_numpy(np.ascontiguousarray(h[:T])).to("cuda")
    caches = make_caches(L, cfg.experts, 16, "lfu")
    worst = 0.0
    torch.cuda.synchronize()
    sample = {0: [0, 4095], 11: [1234], 23: [77, 2048]}
    for l in range(L):
        hin = H.cpu().numpy().astype(np.float64)
        with torch.cuda.stream(moe.compute):
            b.moe_prefill_layer(moe.handle, l, H.data_ptr(), T)
        moe.sync()
        gids, _, n = b.moe_cache_last_routing(moe.handle, T * K)
        gids = np.array(gids).reshape(T, K)
        _, ids, g, cert, _ = stack.prefill_layer(rig.model, l, hin, K, None, with_ffn=False)
        assert np.array_equal(ids[cert], gids[cert]), l
        merged = np.where(cert[:, None], ids, gids)
        want = caches[l].prefill(merged)
        got = [r for r in moe.trace_records()[0] if r[0] == 2 and r[2] == l]
        assert got == [w.astuple() for w in want], l
        if l in sample:
            hout = H.cpu().numpy().astype(np.float64)
            for t in sample[l]:
                y = omoe.moe_output(lambda e: rig.model.expert(l, e), merged[t], g[t],
                                    hin[t] / omoe.rms(hin[t]))
                worst = max(worst, rel_l2(hout[t] - hin[t], y))
    _say("prefill worst", worst)
    assert worst < 2e-2
    # decode continues from the prefilled caches with prefetch
    Hd = torch.from_numpy(np.ascontiguousarray(h[T:])).to("cuda")
    snaps = torch.empty((cfg.tokens, L + 1, cfg.d_model), device="cuda")
    moe.decode(Hd, flags=b.MOE_PREFETCH_NEXT, snapshots=snaps)
    moe.sync()
    dec = [r for r in moe.trace_records()[0] if r[0] != 2]
    w2, unc, _ = check_decode(cfg, rig.model, snaps.cpu().numpy().astype(np.float64), dec, 16, "lfu",
                              prefetch=True, pmax=cfg.prefetch_max, y_tokens=[0, 255], tol=2e-2,
                              caches=caches)
    _say("decode worst", w2, "uncertified", unc)
    moe.close()
    rig.store.close()
