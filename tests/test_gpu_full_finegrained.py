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
from tests._gpu_rig import LazyRig, _batch_tol, _say, _tol
from tests._parity import check_decode, check_y_by_layer, rel_l2

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
    # rows checked against the fp64 SwiGLU: every 32nd row and the last at
    # three layers, with each layer's experts widened once
    rows = list(range(0, T, 32)) + [T - 1]
    sample = {0: rows, 11: rows, 23: rows}
    ymodel = stack.Model(rig.gates.host, lambda l, e: rig.store.expert(l, e), cfg.d_model, cfg.d_ff, cfg.dtype)
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
                y = omoe.moe_output(lambda e: ymodel.expert(l, e), merged[t], g[t],
                                    hin[t] / omoe.rms(hin[t]))
                worst = max(worst, rel_l2(hout[t] - hin[t], y))
            ymodel.forget()
    _say("prefill worst", worst)
    assert worst <= _batch_tol(cfg)
    # decode continues from the prefilled caches with prefetch
    Hd = torch.from_numpy(np.ascontiguousarray(h[T:])).to("cuda")
    snaps = torch.empty((cfg.tokens, L + 1, cfg.d_model), device="cuda")
    moe.decode(Hd, flags=b.MOE_PREFETCH_NEXT, snapshots=snaps)
    moe.sync()
    dec = [r for r in moe.trace_records()[0] if r[0] != 2]
    hs = snaps.cpu().numpy().astype(np.float64)
    w2, unc, _ = check_decode(cfg, rig.model, hs, dec, 16, "lfu", prefetch=True, pmax=cfg.prefetch_max,
                              y_tokens=[0, 255], tol=_tol(cfg), caches=caches)
    # every decode token at three layers
    w3 = check_y_by_layer(ymodel, hs, [0, 12, 23], K, _tol(cfg))
    _say("decode worst", w2, "all tokens at layers 0/12/23", w3, "uncertified", unc)
    moe.close()
    rig.store.close()
