"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments on the host (no GPU work is started by any call here)."""
import ctypes
import os
import re

import pytest

from paper_2511_05814_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe_offload.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_functions():
    assert _declared() == sorted(b.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = b.lib()
    for name in _declared():
        assert hasattr(lib, name), name
    nm = os.popen(f"nm -D --defined-only {b.LIB_PATH}").read()
    for name in _declared():
        assert re.search(rf"\bT {name}$", nm, flags=re.M), name


def test_struct_sizes_match_the_header_layout():
    assert ctypes.sizeof(b.moe_trace_rec) == 32
    assert ctypes.sizeof(b.moe_layer_stats) == 9 * 8
    assert ctypes.sizeof(b.moe_model_desc) == 8 * 4 + 10 * 8 + 2 * 4


@pytest.mark.parametrize("args", [
    (0, 8, 4, 0), (2, 0, 1, 0), (2, 65, 4, 0), (2, 8, 0, 0), (2, 8, 9, 0), (2, 8, 4, 3), (2, 8, 4, -1),
])
def test_create_rejects_bad_arguments(args):
    with pytest.raises(b.MoeError) as e:
        b.moe_cache_create(*args)
    assert e.value.code == b.MOE_ERR_ARG
    assert b.moe_last_error()


def _desc(**kw):
    d = b.moe_model_desc()
    d.d_model, d.d_ff, d.top_k, d.dtype = 64, 64, 2, b.MOE_DTYPE_BF16
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def test_workspace_query_and_bind_validation_without_gpu():
    h = b.moe_cache_create(2, 8, 4, b.MOE_POLICY_LFU)
    try:
        assert b.moe_cache_workspace_bytes(h, _desc()) > 0
        for bad in (dict(d_model=60), dict(d_ff=0), dict(top_k=0), dict(top_k=5), dict(dtype=7),
                    dict(prefetch_max=3), dict(fetch_mode=9), dict(max_prefill_tokens=-1)):
            assert b.moe_cache_workspace_bytes(h, _desc(**bad)) == 0, bad
            with pytest.raises(b.MoeError) as e:
                b.moe_cache_bind(h, _desc(**bad))
            assert e.value.code == b.MOE_ERR_ARG
        # NULL buffers are rejected before any device call
        with pytest.raises(b.MoeError) as e:
            b.moe_cache_bind(h, _desc())
        assert e.value.code == b.MOE_ERR_ARG
        # calls before bind are state errors
        for f, args in ((b.moe_decode_layer, (0, 16, 0)), (b.moe_cache_sync, ()),
                        (b.moe_prefetch, (1, 16, 1)), (b.moe_cache_reset, ())):
            with pytest.raises(b.MoeError) as e:
                f(h, *args)
            assert e.value.code == b.MOE_ERR_STATE
    finally:
        b.moe_cache_destroy(h)
    b.moe_cache_destroy(0)  # NULL-safe


def test_group_quantised_shape_rules():
    h = b.moe_cache_create(2, 8, 4, b.MOE_POLICY_LFU)
    try:
        assert b.moe_cache_workspace_bytes(h, _desc(dtype=b.MOE_DTYPE_Q2G16)) > 0
        for bad in (dict(d_model=72), dict(d_ff=200), dict(d_model=8256, d_ff=64), dict(max_prefill_tokens=16)):
            assert b.moe_cache_workspace_bytes(h, _desc(dtype=b.MOE_DTYPE_Q2G16, **bad)) == 0, bad
    finally:
        b.moe_cache_destroy(h)


def test_slots_below_top_k_rejected():
    h = b.moe_cache_create(1, 8, 2, b.MOE_POLICY_LRU)
    try:
        assert b.moe_cache_workspace_bytes(h, _desc(top_k=3)) == 0
    finally:
        b.moe_cache_destroy(h)


def test_aged_lfu_needs_a_period():
    h = b.moe_cache_create(2, 8, 4, b.MOE_POLICY_LFU_AGED)
    try:
        for bad in (0, -3):
            assert b.moe_cache_workspace_bytes(h, _desc(aging_ticks=bad)) == 0
            with pytest.raises(b.MoeError) as e:
                b.moe_cache_bind(h, _desc(aging_ticks=bad))
            assert e.value.code == b.MOE_ERR_ARG
        assert b.moe_cache_workspace_bytes(h, _desc(aging_ticks=1)) > 0
    finally:
        b.moe_cache_destroy(h)
    # the other policies ignore the field
    h = b.moe_cache_create(2, 8, 4, b.MOE_POLICY_LFU)
    try:
        assert b.moe_cache_workspace_bytes(h, _desc(aging_ticks=0)) > 0
    finally:
        b.moe_cache_destroy(h)


def test_policy_names():
    assert b.parse_policy("lru") == (b.MOE_POLICY_LRU, 0)
    assert b.parse_policy("lfu") == (b.MOE_POLICY_LFU, 0)
    assert b.parse_policy("lfu-aged:32") == (b.MOE_POLICY_LFU_AGED, 32)
    for bad in ("lfu-aged", "lfu-aged:0", "lfu:3", "mru"):
        with pytest.raises(ValueError):
            b.parse_policy(bad)
