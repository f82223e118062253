"""GPU parity of the decode path against the fp64 oracle (needs an MI355X).

Every test drives the HIP library through the C ABI (binding -> offload) and
compares, teacher-forced, with the oracle: routing, next-layer guesses and the
cache trace bit for bit, layer outputs within 1e-5 (fp32 weights) or 1e-4
(bf16 weights, inside the 2e-2 stated for them: decode keeps fp32
activations) relative L2.
"""
import numpy as np
import pytest

from oracle import stack
from oracle.cache import LayerCache
from paper_2511_05814_amd import binding as b
from paper_2511_05814_amd import workload as wl
from tests._gpu_rig import Rig, _say, _tol
from tests._parity import check_decode

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def tiny():
    cfg = wl.CONFIGS["tiny-stack"]
    _say("tiny-stack", cfg)
    return Rig(cfg)


@pytest.mark.parametrize("policy", ["lru", "lfu", "lfu-aged:2"])
def test_tiny_stack_decode_parity(tiny, policy):
    cfg = tiny.cfg
    _say("tiny decode", policy)
    moe = tiny.cache(4, policy)
    hs, recs, _ = tiny.run(moe, cfg.tokens)
    worst, unc, caches = check_decode(cfg, tiny.model, hs, recs, 4, policy, tol=_tol(cfg))
    _say("worst y rel L2", worst, "uncertified", unc)
    # final tables and statistics agree with the oracle's
    for l in range(cfg.layers):
        se, es, cnt, last, clock = moe.state(l)
        ose, oes, ocnt, olast, oclock = caches[l].state()
        assert (se, es, cnt, last, clock) == (ose, oes, ocnt, olast, oclock)
    st = moe.stats()
    for l in range(cfg.layers):
        o = caches[l].stats
        assert (st[l]["hits"], st[l]["misses"], st[l]["lookups"]) == (o.hits, o.misses, o.lookups)
        assert st[l]["bytes_fetched"] == o.misses * cfg.expert_bytes
    moe.close()


@pytest.mark.parametrize("policy", ["lfu", "lfu-aged:3"])
def test_tiny_stack_prefetch_parity(tiny, policy):
    cfg = tiny.cfg
    _say("tiny decode + prefetch 2", policy)
    moe = tiny.cache(4, policy, prefetch_max=2)
    hs, recs, _ = tiny.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    worst, unc, caches = check_decode(cfg, tiny.model, hs, recs, 4, policy, prefetch=True, pmax=2,
                                      tol=_tol(cfg))
    st = moe.stats()
    o = caches[1].stats
    assert (st[1]["pf_issued"], st[1]["pf_useful"], st[1]["pf_wasted"]) == \
           (o.pf_issued, o.pf_useful, o.pf_wasted)
    assert st[1]["pf_guesses"] == cfg.tokens * cfg.top_k
    moe.close()


def test_streams_and_fetch_modes_give_identical_results(tiny):
    cfg = tiny.cfg
    _say("stream/fetch-mode equivalence")
    outs = []
    for kw in (dict(), dict(separate_copy_stream=False), dict(fetch_mode=b.MOE_FETCH_DMA),
               dict(fetch_mode=b.MOE_FETCH_KERNEL), dict(fetch_mode=b.MOE_FETCH_SPLIT, separate_copy_stream=False)):
        moe = tiny.cache(4, "lfu", prefetch_max=2, **kw)
        hs, recs, H = tiny.run(moe, 32, flags=b.MOE_PREFETCH_NEXT)
        outs.append((H.tobytes(), recs))
        moe.close()
    assert all(o == outs[0] for o in outs[1:])


@pytest.mark.parametrize("mode", ["kernel", "split"])
def test_delayed_copy_stream_still_correct(tiny, mode):
    # A long spin on the copy stream ahead of every layer: if any FFN did not
    # wait for the copies that fill its slots (demand copies, and with
    # speculation the previous layer's prefetch copies) it would read stale
    # weights.
    cfg = tiny.cfg
    fm = b.MOE_FETCH_KERNEL if mode == "kernel" else b.MOE_FETCH_SPLIT
    for flags, pmax in ((0, 0), (b.MOE_PREFETCH_NEXT, 2)):
        _say(f"delayed copy stream {mode} flags={flags}")
        ref = tiny.cache(4, "lru", prefetch_max=pmax, fetch_mode=fm)
        _, recs0, H0 = tiny.run(ref, 16, flags=flags)
        ref.close()
        moe = tiny.cache(4, "lru", prefetch_max=pmax, fetch_mode=fm)
        h0 = wl.hidden_states(cfg, 16)
        H = torch.from_numpy(h0).to("cuda")
        with torch.cuda.stream(moe.compute):
            for t in range(16):
                for l in range(cfg.layers):
                    with torch.cuda.stream(moe.copy):
                        torch.cuda._sleep(200000)
                    b.moe_decode_layer(moe.handle, l, H[t].data_ptr(), flags)
        moe.sync()
        recs, _ = moe.trace_records()
        assert recs == recs0
        assert H.cpu().numpy().tobytes() == H0.tobytes()
        moe.close()


@pytest.mark.parametrize("mode", ["kernel", "split", "dma"])
def test_poisoned_slots_are_never_read_before_their_copies(tiny, mode):
    # Every slot a copy is about to fill is overwritten with NaN bytes just
    # before the layer call that issues the copy: a speculative copy's slot on
    # the copy stream (after the compute stream's earlier work, then a long
    # spin), a demand copy's slot on the stream that carries demand copies (the
    # compute stream, or the copy stream in DMA mode).  A kernel that read a
    # slot before the copy filling it finished would meet NaN (or the evicted
    # expert) and carry it into h; with every wait in place the outputs and the
    # trace are those of the unpoisoned run, bit for bit.
    from collections import defaultdict
    from oracle.cache import F_HIT, F_ISSUED, KIND_ACCESS, KIND_PREFETCH

    cfg = tiny.cfg
    fm = {"kernel": b.MOE_FETCH_KERNEL, "split": b.MOE_FETCH_SPLIT, "dma": b.MOE_FETCH_DMA}[mode]
    T, S = 16, 4
    ref = tiny.cache(S, "lru", prefetch_max=2, fetch_mode=fm)
    _, recs0, H0 = tiny.run(ref, T, flags=b.MOE_PREFETCH_NEXT)
    ref.close()
    spec, demand = defaultdict(list), defaultdict(list)  # (token, calling layer) -> [(layer, slot)]
    for kind, tok, layer, _rank, _e, flags, slot, _v in recs0:
        if kind == KIND_PREFETCH and flags & F_ISSUED:
            spec[(tok, layer - 1)].append((layer, slot))
        elif kind == KIND_ACCESS and not flags & F_HIT:
            demand[(tok, layer)].append((layer, slot))
    assert spec and demand  # both kinds of copy happen in this run
    _say(f"poisoned slots, {mode}: {sum(map(len, spec.values()))} speculative, "
         f"{sum(map(len, demand.values()))} demand")
    moe = tiny.cache(S, "lru", prefetch_max=2, fetch_mode=fm)
    arena = moe.arena.view(cfg.layers, S, cfg.expert_bytes)
    H = torch.from_numpy(wl.hidden_states(cfg, T)).to("cuda")
    with torch.cuda.stream(moe.compute):
        for t in range(T):
            for l in range(cfg.layers):
                moe.copy.wait_stream(moe.compute)
                with torch.cuda.stream(moe.copy):
                    for layer, slot in spec[(t, l)] + (demand[(t, l)] if mode == "dma" else []):
                        arena[layer, slot].fill_(255)
                    torch.cuda._sleep(200000)
                if mode != "dma":
                    for layer, slot in demand[(t, l)]:
                        arena[layer, slot].fill_(255)
                b.moe_decode_layer(moe.handle, l, H[t].data_ptr(), b.MOE_PREFETCH_NEXT)
    moe.sync()
    recs, _ = moe.trace_records()
    assert recs == recs0
    out = H.cpu().numpy()
    assert np.isfinite(out).all()
    assert out.tobytes() == H0.tobytes()
    moe.close()


def test_reset_replays_identically(tiny):
    _say("reset replay")
    moe = tiny.cache(4, "lfu")
    _, r1, H1 = tiny.run(moe, 24)
    moe.reset()
    _, r2, H2 = tiny.run(moe, 24)
    assert r1 == r2 and H1.tobytes() == H2.tobytes()
    moe.close()


@pytest.mark.parametrize("policy", ["lru", "lfu", "lfu-aged:1", "lfu-aged:4"])
def test_injected_routing_traces_match_oracle(tiny, policy):
    cfg = tiny.cfg
    _say("injected routing", policy)
    rng = np.random.default_rng({"lru": 5, "lfu": 6}.get(policy, 7))
    moe = tiny.cache(4, policy, trace_cap=4096)
    T = 300
    p = rng.dirichlet(np.full(cfg.experts, 0.4))
    ids = np.stack([rng.choice(cfg.experts, cfg.top_k, replace=False, p=p) for _ in range(T)])
    dev = torch.from_numpy(ids.astype(np.int32)).to("cuda")
    oracle = [LayerCache(cfg.experts, 4, policy, layer=l) for l in range(cfg.layers)]
    want = []
    with torch.cuda.stream(moe.compute):
        for t in range(T):
            l = t % cfg.layers
            b.moe_cache_access(moe.handle, l, dev[t].data_ptr())
            want += oracle[l].access(ids[t])
    recs, _ = moe.trace_records()
    assert recs == [w.astuple() for w in want]
    if policy.startswith("lfu-aged"):
        # the aged key really decided evictions: plain LFU takes other victims
        plain = [LayerCache(cfg.experts, 4, "lfu", layer=l) for l in range(cfg.layers)]
        lfu = []
        for t in range(T):
            lfu += plain[t % cfg.layers].access(ids[t])
        assert sum(a != w.astuple() for a, w in zip(recs, lfu)) > 50
    # the copies really happened: slot contents equal the host store's experts
    arena = moe.arena.cpu().numpy().reshape(cfg.layers, 4, -1)
    for l in range(cfg.layers):
        se, _, _, _, _ = moe.state(l)
        for s, e in enumerate(se):
            assert np.array_equal(arena[l, s], tiny.store.layer_array(l).reshape(cfg.experts, -1)[e])
    moe.close()


def test_injected_invalid_ids_rejected_without_change(tiny):
    cfg = tiny.cfg
    _say("invalid injected ids")
    moe = tiny.cache(4, "lru")
    before = moe.state(0)
    for bad in ([3, 3], [1, 8], [-1, 2]):
        dev = torch.tensor(bad, dtype=torch.int32, device="cuda")
        with torch.cuda.stream(moe.compute):
            b.moe_cache_access(moe.handle, 0, dev.data_ptr())
        with pytest.raises(b.MoeError) as e:
            moe.sync()
        assert e.value.code == b.MOE_ERR_ARG
        assert moe.state(0) == before
    moe.close()


def test_standalone_prefetch_matches_oracle(tiny):
    cfg = tiny.cfg
    _say("standalone moe_prefetch")
    moe = tiny.cache(4, "lru", prefetch_max=2)
    h0 = wl.hidden_states(cfg, 12)
    H = torch.from_numpy(h0).to("cuda")
    oracle = LayerCache(cfg.experts, 4, "lru", layer=1)
    want = []
    with torch.cuda.stream(moe.compute):
        for t in range(12):
            b.moe_prefetch(moe.handle, 1, H[t].data_ptr(), 1 + t % 2)
    moe.sync()
    recs, _ = moe.trace_records()
    for t in range(12):
        g = stack.layer_step(tiny.model, 1, h0[t].astype(np.float64), cfg.top_k, with_ffn=False)["ids"]
        want += oracle.prefetch(g, 1 + t % 2)
    assert recs == [w.astuple() for w in want]
    moe.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ragged_shapes(dtype):
    # d and d_ff are not multiples of any tile; E, K, S odd; 3 layers
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=3, experts=5, top_k=3, d_model=136, d_ff=200,
                                         dtype=dtype, tokens=20)
    _say("ragged", cfg)
    rig = Rig(cfg)
    moe = rig.cache(3, "lfu", prefetch_max=1)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    check_decode(cfg, rig.model, hs, recs, 3, "lfu", prefetch=True, pmax=1, tol=_tol(cfg))
    moe.close()
    rig.store.close()


def test_fine_grained_decode_shape():
    # 64 experts, top-8, 16 slots, d = 2048, d_ff = 1408 (two layers of that stack)
    cfg = wl.CONFIGS["fine-grained"].with_(layers=2, tokens=12, prefill_tokens=0)
    _say("fine-grained decode", cfg)
    rig = Rig(cfg)
    moe = rig.cache(16, "lfu", prefetch_max=2)
    hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
    worst, unc, _ = check_decode(cfg, rig.model, hs, recs, 16, "lfu", prefetch=True, pmax=2,
                                 y_tokens=[0, 5, 11], tol=_tol(cfg))
    _say("worst", worst, "uncertified", unc)
    moe.close()
    rig.store.close()


@pytest.fixture(scope="module")
def mixtral_layer():
    cfg = wl.CONFIGS["mixtral-layer"]
    _say("mixtral-layer host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    rig = Rig(cfg)
    yield rig
    rig.store.close()


@pytest.mark.parametrize("policy", ["lru", "lfu"])
def test_mixtral_layer_full_run(mixtral_layer, policy):
    # the benchmark's workload: all 256 tokens, 4 slots; traces exact for every
    # token, outputs checked on sampled tokens
    rig = mixtral_layer
    cfg = rig.cfg
    _say("mixtral-layer full run", policy)
    moe = rig.cache(4, policy)
    hs, recs, _ = rig.run(moe, cfg.tokens)
    worst, unc, caches = check_decode(cfg, rig.model, hs, recs, 4, policy,
                                      y_tokens=[0, 1, 77, 128, 200, 255], tol=_tol(cfg))
    _say("worst", worst, "uncertified", unc, "hit rate", caches[0].stats.hits / (cfg.tokens * 2))
    assert worst < 1e-4   # bf16 weights, fp32 activations and accumulation
    moe.close()


def test_aliased_host_layers():
    # a store that pins only 2 distinct layers for a 5-layer stack: layers 2..4
    # read the pages of layers 0, 1, 0 through the per-layer host table
    from paper_2511_05814_amd import offload
    cfg = wl.CONFIGS["tiny-stack"].with_(layers=5, tokens=12)
    _say("aliased host layers", cfg)
    rig = Rig.__new__(Rig)
    rig.cfg = cfg
    rig.store = offload.HostStore(cfg, max_pinned_bytes=2 * cfg.experts * cfg.expert_bytes)
    assert rig.store.distinct == 2 and rig.store.aliased
    rig.gates = offload.DeviceGates(cfg)
    rig.model = stack.Model(rig.gates.host, lambda l, e: rig.store.expert(l, e), cfg.d_model, cfg.d_ff,
                            cfg.dtype)
    for mode in (b.MOE_FETCH_KERNEL, b.MOE_FETCH_DMA, b.MOE_FETCH_SPLIT):
        moe = rig.cache(4, "lru", prefetch_max=1, fetch_mode=mode)
        hs, recs, _ = rig.run(moe, cfg.tokens, flags=b.MOE_PREFETCH_NEXT)
        check_decode(cfg, rig.model, hs, recs, 4, "lru", prefetch=True, pmax=1, tol=_tol(cfg))
        moe.close()
    rig.store.close()


def test_timing_levels(tiny):
    # MOE_TIMING_ALL times every decode launch, MOE_TIMING_FFN_UP only the FFN
    # up launches, OFF nothing; the events change no result
    cfg = tiny.cfg
    T = 8
    calls = T * cfg.layers
    out = {}
    for level in (b.MOE_TIMING_OFF, b.MOE_TIMING_ALL, b.MOE_TIMING_FFN_UP):
        _say("timing level", level)
        moe = tiny.cache(4, "lfu", prefetch_max=2)
        b.moe_cache_set_timing(moe.handle, level)
        _, recs, H = tiny.run(moe, T, flags=b.MOE_PREFETCH_NEXT)
        issued = sum(s["pf_issued"] for s in moe.stats())
        out[level] = ([tuple(r) for r in recs], H, b.moe_cache_read_timing(moe.handle), issued)
        with pytest.raises(b.MoeError) as e:
            b.moe_cache_set_timing(moe.handle, 3)
        assert e.value.code == b.MOE_ERR_ARG
        moe.close()
    t_all = out[b.MOE_TIMING_ALL][2]
    # experts whose d_ff fits one column chunk of the down kernel (4 x 64 lanes
    # x 16 bytes) add the rank partials there: no reduce launch to time
    fused = (cfg.dtype in ("f32", "bf16") and cfg.top_k <= 16
             and cfg.d_ff <= 4 * 64 * (8 if cfg.dtype == "bf16" else 4))
    for k in ("router", "fetch", "ffn_up", "ffn_down", "wait") + (() if fused else ("ffn_reduce",)):
        assert t_all[k + "_n"] == calls, k
        assert t_all[k + "_ms"] > 0, k
    if fused:
        assert t_all["ffn_reduce_n"] == 0 and t_all["ffn_reduce_ms"] == 0
    assert (t_all["pf_fetch_n"] > 0) == (out[b.MOE_TIMING_ALL][3] > 0)
    t_up = out[b.MOE_TIMING_FFN_UP][2]
    assert t_up["ffn_up_n"] == calls and t_up["ffn_up_ms"] > 0
    assert all(v == 0 for k, v in t_up.items() if not k.startswith("ffn_up")), t_up
    assert all(v == 0 for v in out[b.MOE_TIMING_OFF][2].values())
    for level in (b.MOE_TIMING_ALL, b.MOE_TIMING_FFN_UP):
        assert out[level][0] == out[b.MOE_TIMING_OFF][0]
        assert np.array_equal(out[level][1], out[b.MOE_TIMING_OFF][1])
