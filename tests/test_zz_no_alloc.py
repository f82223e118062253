"""moe_decode_layer_noalloc, the decode entry point for callers that cannot
allocate (its scratch is a static device array instead of the bound
workspace), against moe_decode_layer through the C ABI (needs an MI355X).

Two calls in a row on one device, the second on a smaller model, so the
second reads a scratch array that still holds the first call's contents:
each must give bit for bit the hidden states, routing and trace records of
moe_decode_layer on the same inputs, and match the fp64 oracle like any
decode run.  A model that needs more scratch than the array holds is
rejected on the host before any device work.
"""
import numpy as np
import pytest

from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import Rig, _say, _tol
from tests._parity import check_decode

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _decode(moe, H, entry, flags):
    cfg = moe.cfg
    T, L = H.shape[0], cfg.layers
    snaps = torch.empty((T, L + 1, cfg.d_model), device="cuda")
    moe.compute.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(moe.compute):
        for t in range(T):
            row = H[t]
            for l in range(L):
                snaps[t, l].copy_(row)
                entry(moe.handle, l, row.data_ptr(), flags)
            snaps[t, L].copy_(row)
    moe.sync()
    recs, dropped = moe.trace_records()
    assert dropped == 0
    return snaps.cpu().numpy(), recs


def _compare_entry_points(cfg, slots, policy, pmax):
    rig = Rig(cfg)
    h0 = np.ascontiguousarray(wl.hidden_states(cfg, cfg.tokens))
    flags = b.MOE_PREFETCH_NEXT if pmax else 0
    out = {}
    for name, entry in (("workspace", b.moe_decode_layer), ("noalloc", b.moe_decode_layer_noalloc)):
        moe = rig.cache(slots, policy, prefetch_max=pmax)
        if name == "noalloc":
            b.moe_cache_set_timing(moe.handle, b.MOE_TIMING_ALL)
            h = torch.zeros(cfg.d_model, device="cuda")
            with pytest.raises(b.MoeError) as e:   # timed spans would create events
                b.moe_decode_layer_noalloc(moe.handle, 0, h.data_ptr(), flags)
            assert e.value.code == b.MOE_ERR_STATE
            b.moe_cache_set_timing(moe.handle, b.MOE_TIMING_OFF)
        H = torch.from_numpy(h0).to("cuda")
        snaps, recs = _decode(moe, H, entry, flags)
        out[name] = (H.cpu().numpy(), snaps, recs, moe.stats())
        moe.close()
    (Hw, sw, rw, stw), (Hn, sn, rn, stn) = out["workspace"], out["noalloc"]
    assert np.array_equal(Hw.view(np.uint32), Hn.view(np.uint32)), "final hidden states differ"
    assert np.array_equal(sw.view(np.uint32), sn.view(np.uint32)), "per-layer hidden states differ"
    assert rw == rn, "trace records differ"
    assert stw == stn, "statistics differ"
    worst, unc, _ = check_decode(cfg, rig.model, sn.astype(np.float64), rn, slots, policy,
                                 prefetch=bool(pmax), pmax=pmax, tol=_tol(cfg))
    _say(cfg.name, "noalloc = workspace entry point bit for bit; oracle worst", worst, "uncertified", unc)
    rig.store.close()


def test_noalloc_matches_decode_layer_two_calls_second_smaller():
    # first: the 64-expert shape (d 2048, d_ff 1408, top-8, bf16) with
    # next-layer prefetch; second: the fp32 tiny stack (d 256, d_ff 512, top-2)
    _compare_entry_points(wl.CONFIGS["fine-grained"].with_(layers=2, tokens=6, prefill_tokens=0), 16, "lfu", 2)
    _compare_entry_points(wl.CONFIGS["tiny-stack"].with_(tokens=8), 4, "lru", 0)


def test_noalloc_rejects_a_model_beyond_its_scratch():
    # top-16 of 16 experts with d_ff = 65544: 16 * 65544 fp32 activations alone
    # exceed the 4 MiB array; the workspace entry point is the one to use
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=1, experts=16, top_k=16, d_model=8, d_ff=65544,
                                         dtype="bf16", tokens=1)
    rig = Rig(cfg)
    moe = rig.cache(16, "lfu")
    h = torch.zeros(cfg.d_model, device="cuda")
    with pytest.raises(b.MoeError) as e:
        b.moe_decode_layer_noalloc(moe.handle, 0, h.data_ptr(), 0)
    assert e.value.code == b.MOE_ERR_ARG and "scratch" in str(e.value)
    moe.sync()
    assert all(s["lookups"] == 0 for s in moe.stats())  # nothing was enqueued
    moe.close()
    rig.store.close()
