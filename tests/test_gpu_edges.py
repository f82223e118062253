"""Degenerate and boundary cases of the decode and batch paths against the
oracle: top-1 with one slot, every expert resident, the largest top-K, a trace
ring that overflows, an all-zero hidden state (every logit ties), and batches
of one token and of the full batch capacity."""
import numpy as np
import pytest

from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import Rig, _say, _tol
from tests._parity import check_decode
from tests.test_gpu_prefill import prefill_and_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.mark.parametrize("policy", ["lru", "lfu"])
def test_top1_single_slot(policy):
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=2, experts=4, top_k=1, d_model=64, d_ff=128,
                                         dtype="bf16", tokens=40)
    _say("top-1, one slot", policy)
    rig = Rig(cfg)
    moe = rig.cache(1, policy, prefetch_max=1)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    check_decode(cfg, rig.model, hs, recs, 1, policy, prefetch=True, pmax=1, tol=_tol(cfg))
    moe.close()
    rig.store.close()


def test_every_expert_resident():
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=2, experts=8, top_k=2, d_model=128, d_ff=256,
                                         dtype="bf16", tokens=30)
    _say("slots = experts")
    rig = Rig(cfg)
    moe = rig.cache(8, "lfu")
    hs, recs, _ = rig.run(moe, cfg.tokens)
    check_decode(cfg, rig.model, hs, recs, 8, "lfu", tol=_tol(cfg))
    assert all(r[5] & 1 for r in recs if r[0] == 0)  # every access hits
    for st in moe.stats():
        assert st["misses"] == 0 and st["bytes_fetched"] == 0 and st["evictions"] == 0
    moe.close()
    rig.store.close()


def test_largest_top_k():
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=2, experts=64, top_k=16, d_model=128, d_ff=256,
                                         dtype="bf16", tokens=12)
    _say("64 experts, top-16, 16 slots")
    rig = Rig(cfg)
    moe = rig.cache(16, "lru", prefetch_max=4)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    worst, unc, _ = check_decode(cfg, rig.model, hs, recs, 16, "lru", prefetch=True, pmax=4, tol=_tol(cfg))
    _say("worst", worst, "uncertified", unc)
    moe.close()
    rig.store.close()


@pytest.mark.parametrize("dtype,d_model", [("bf16", 1536), ("f32", 768)])
def test_rows_of_fewer_steps_than_the_up_kernel_width(dtype, d_model):
    # three 16-byte steps a lane while the up kernel is built for four: the
    # fourth step must read zeros, not the next row and h past its end
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=2, experts=4, top_k=2, d_model=d_model, d_ff=256,
                                         dtype=dtype, tokens=10)
    _say("d_model", d_model, dtype)
    rig = Rig(cfg)
    moe = rig.cache(4, "lfu")
    hs, recs, _ = rig.run(moe, cfg.tokens)
    worst, _, _ = check_decode(cfg, rig.model, hs, recs, 4, "lfu", tol=_tol(cfg))
    _say("worst", worst)
    moe.close()
    rig.store.close()


def test_trace_ring_overflow_keeps_the_newest_records():
    cfg = wl.CONFIGS["tiny-stack"].with_(tokens=16)
    rig = Rig(cfg)
    full = rig.cache(4, "lru")
    _, recs_full, _ = rig.run(full, cfg.tokens)
    full.close()
    moe = rig.cache(4, "lru", trace_cap=20)
    H = torch.from_numpy(np.ascontiguousarray(wl.hidden_states(cfg, cfg.tokens))).to("cuda")
    moe.decode(H)
    moe.sync()
    recs, dropped = moe.trace_records()
    assert len(recs_full) == cfg.tokens * cfg.layers * cfg.top_k
    assert dropped == len(recs_full) - 20 and recs == recs_full[-20:]
    moe.close()
    rig.store.close()


@pytest.mark.parametrize("experts,top_k,d_model,slots,flags", [
    (8, 2, None, 4, 0),
    # with speculation (both roles, two workgroups), 16 and 64 experts
    (16, 2, 128, 4, b.MOE_PREFETCH_NEXT),
    (64, 8, 2048, 16, b.MOE_PREFETCH_NEXT),
])
def test_zero_hidden_state_ties_to_the_lowest_ids(experts, top_k, d_model, slots, flags):
    # h = 0: every logit is exactly 0, the tie rule picks experts 0..K-1, the
    # combine weights are uniform and the layer output is exactly zero
    cfg = wl.CONFIGS["tiny-stack"].with_(dtype="bf16", tokens=3, experts=experts, top_k=top_k,
                                         d_model=d_model or wl.CONFIGS["tiny-stack"].d_model)
    _say("zero h", experts, top_k, cfg.d_model)
    rig = Rig(cfg)
    moe = rig.cache(slots, "lfu", prefetch_max=2 if flags else 0)
    hs, recs, H = rig.run(moe, 3, flags=flags, h0=np.zeros((3, cfg.d_model), np.float32))
    assert np.all(H == 0.0)
    for r in recs:
        assert r[4] == r[3]  # rank r -> expert r
    ids, g, n = b.moe_cache_last_routing(moe.handle, cfg.top_k)
    assert list(ids) == list(range(cfg.top_k)) and np.allclose(g, 1.0 / cfg.top_k)
    moe.close()
    rig.store.close()


@pytest.mark.parametrize("T", [1, 64])
def test_batch_of_one_and_of_full_capacity(T):
    cfg = wl.CONFIGS["fine-grained"].with_(layers=2, tokens=2, prefill_tokens=T)
    _say("batch path, T =", T)
    rig = Rig(cfg)
    moe = rig.cache(16, "lfu", max_prefill_tokens=64)
    _, _, worst, _ = prefill_and_check(rig, moe, "lfu", 16, T, sorted({0, T - 1}))
    _say("worst", worst)
    moe.close()
    rig.store.close()


def test_hbm_read_probe():
    # calibration call beside the path: a plausible rate on 512 MiB, and its
    # argument errors (a misaligned pointer, a size that is not a multiple of 16)
    _say("hbm read probe, 512 MiB, 3 reps")
    nbytes = 512 << 20
    buf = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream().cuda_stream
    gbps = b.moe_probe_hbm_read(buf.data_ptr(), nbytes, 3, stream)
    assert 1000.0 < gbps < 10000.0
    assert int(buf.sum().item()) == 0  # read only
    for ptr, n in ((buf.data_ptr() + 4, 1024), (buf.data_ptr(), 1000)):
        with pytest.raises(b.MoeError) as e:
            b.moe_probe_hbm_read(ptr, n, 1, stream)
        assert e.value.code == b.MOE_ERR_ARG
