"""ctypes binding of the C ABI in include/moe_offload.h.

Argument marshalling only: every function has the name of the C function it
calls, takes plain integers for pointers (device addresses, pinned host
addresses, stream handles) and raises MoeError when the C call returns a
negative status.  No compute happens here.  The shared library is built by
`__graft_entry__.build()`; `lib()` raises if it is missing, so nothing can
silently run without the HIP kernels.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libmoe_offload.so")

MOE_POLICY_LRU, MOE_POLICY_LFU, MOE_POLICY_LFU_AGED = 0, 1, 2
MOE_DTYPE_F32, MOE_DTYPE_BF16, MOE_DTYPE_Q2G16 = 0, 1, 2
MOE_OK, MOE_ERR_ARG, MOE_ERR_STATE, MOE_ERR_HIP, MOE_ERR_NOMEM = 0, -1, -2, -3, -4
MOE_PREFETCH_NEXT = 1
MOE_FETCH_KERNEL, MOE_FETCH_DMA, MOE_FETCH_SPLIT = 0, 1, 2
MOE_HOST_PLAIN, MOE_HOST_PACKED, MOE_HOST_ENTROPY = 0, 1, 2
MOE_TIMING_OFF, MOE_TIMING_ALL, MOE_TIMING_FFN_UP = 0, 1, 2
MOE_MAX_EXPERTS, MOE_MAX_TOPK = 64, 16

POLICIES = {"lru": MOE_POLICY_LRU, "lfu": MOE_POLICY_LFU, "lfu-aged": MOE_POLICY_LFU_AGED}


def parse_policy(spec: str):
    """'lru', 'lfu' or 'lfu-aged:A' -> (MOE_POLICY_*, aging_ticks)."""
    name, _, arg = spec.partition(":")
    if name == "lfu-aged":
        if not arg.isdigit() or int(arg) < 1:
            raise ValueError(f"aged LFU needs a period of at least one tick: {spec!r}")
        return MOE_POLICY_LFU_AGED, int(arg)
    if name not in POLICIES or arg:
        raise ValueError(f"unknown policy {spec!r}")
    return POLICIES[name], 0
DTYPES = {"f32": MOE_DTYPE_F32, "bf16": MOE_DTYPE_BF16, "q2g16": MOE_DTYPE_Q2G16}


class MoeError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where} failed with {code}: {msg}")
        self.code = code


class moe_model_desc(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int), ("d_ff", ctypes.c_int), ("top_k", ctypes.c_int),
        ("dtype", ctypes.c_int), ("prefetch_max", ctypes.c_int), ("fetch_mode", ctypes.c_int),
        ("max_prefill_tokens", ctypes.c_int), ("host_format", ctypes.c_int),
        ("gate_w", ctypes.c_void_p), ("host_experts", ctypes.c_void_p),
        ("arena", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t), ("trace", ctypes.c_void_p),
        ("trace_cap", ctypes.c_size_t), ("compute_stream", ctypes.c_void_p),
        ("copy_stream", ctypes.c_void_p), ("host_layers", ctypes.POINTER(ctypes.c_void_p)),
        ("packed_cap", ctypes.c_int), ("aging_ticks", ctypes.c_int),
    ]


class moe_trace_rec(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("kind", "token", "layer", "rank", "expert", "flags", "slot", "victim")]


class moe_layer_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in
                ("hits", "misses", "evictions", "pf_guesses", "pf_issued", "pf_useful",
                 "pf_wasted", "lookups", "bytes_fetched")]


class moe_timing(ctypes.Structure):
    _fields_ = ([(n, ctypes.c_double) for n in
                 ("router_ms", "fetch_ms", "ffn_up_ms", "ffn_down_ms", "prefill_ms", "gemm_up_ms",
                  "gemm_down_ms", "ffn_reduce_ms")]
                + [(n, ctypes.c_uint64) for n in
                   ("router_n", "fetch_n", "ffn_up_n", "ffn_down_n", "prefill_n", "gemm_up_n",
                    "gemm_down_n", "ffn_reduce_n")]
                + [(n, ctypes.c_double) for n in ("gemm_up_flop", "gemm_down_flop", "unpack_ms")]
                + [("unpack_n", ctypes.c_uint64), ("wait_ms", ctypes.c_double), ("wait_n", ctypes.c_uint64),
                   ("pf_fetch_ms", ctypes.c_double), ("pf_fetch_n", ctypes.c_uint64)])


# (name, restype, argtypes) of every exported function, in header order
_SIGNATURES = [
    ("moe_cache_create", ctypes.c_int,
     [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_void_p)]),
    ("moe_cache_workspace_bytes", ctypes.c_size_t, [ctypes.c_void_p, ctypes.POINTER(moe_model_desc)]),
    ("moe_cache_bind", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(moe_model_desc)]),
    ("moe_cache_reset", ctypes.c_int, [ctypes.c_void_p]),
    ("moe_decode_layer", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int]),
    ("moe_decode_layer_noalloc", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int]),
    ("moe_prefetch", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int]),
    ("moe_prefill_layer", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int]),
    ("moe_cache_access", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]),
    ("moe_cache_sync", ctypes.c_int, [ctypes.c_void_p]),
    ("moe_cache_stats", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(moe_layer_stats), ctypes.c_int]),
    ("moe_cache_read_trace", ctypes.c_int,
     [ctypes.c_void_p, ctypes.POINTER(moe_trace_rec), ctypes.c_size_t,
      ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_uint64)]),
    ("moe_cache_read_state", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
      ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]),
    ("moe_cache_last_routing", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
      ctypes.POINTER(ctypes.c_size_t)]),
    ("moe_cache_set_timing", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    ("moe_cache_read_timing", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(moe_timing)]),
    ("moe_cache_destroy", None, [ctypes.c_void_p]),
    ("moe_host_alloc", ctypes.c_int, [ctypes.c_size_t, ctypes.POINTER(ctypes.c_void_p)]),
    ("moe_host_free", ctypes.c_int, [ctypes.c_void_p]),
    ("moe_entropy_matrix_bytes", ctypes.c_size_t, [ctypes.c_size_t, ctypes.c_size_t]),
    ("moe_entropy_pack", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_void_p, ctypes.POINTER(ctypes.c_size_t)]),
    ("moe_probe_hbm_read", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
    ("moe_probe_h2d_copy", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
      ctypes.POINTER(ctypes.c_double)]),
    ("moe_probe_mfma_bf16", ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
    ("moe_last_error", ctypes.c_char_p, []),
]
EXPORTED = [s[0] for s in _SIGNATURES]

_lib = None


def lib():
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        h = ctypes.CDLL(LIB_PATH)
        for name, res, args in _SIGNATURES:
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _lib = h
    return _lib


def moe_last_error() -> str:
    return lib().moe_last_error().decode()


def _check(rc: int, where: str) -> None:
    if rc != MOE_OK:
        raise MoeError(rc, where, moe_last_error())


def moe_cache_create(layers: int, experts: int, slots: int, policy: int) -> int:
    out = ctypes.c_void_p()
    _check(lib().moe_cache_create(layers, experts, slots, policy, ctypes.byref(out)), "moe_cache_create")
    return out.value


def moe_cache_workspace_bytes(cache: int, desc: moe_model_desc) -> int:
    return lib().moe_cache_workspace_bytes(cache, ctypes.byref(desc))


def moe_cache_bind(cache: int, desc: moe_model_desc) -> None:
    _check(lib().moe_cache_bind(cache, ctypes.byref(desc)), "moe_cache_bind")


def moe_cache_reset(cache: int) -> None:
    _check(lib().moe_cache_reset(cache), "moe_cache_reset")


def moe_decode_layer(cache: int, layer: int, h: int, flags: int = 0) -> None:
    _check(lib().moe_decode_layer(cache, layer, h, flags), "moe_decode_layer")


def moe_decode_layer_noalloc(cache: int, layer: int, h: int, flags: int = 0) -> None:
    _check(lib().moe_decode_layer_noalloc(cache, layer, h, flags), "moe_decode_layer_noalloc")


def moe_prefetch(cache: int, next_layer: int, h: int, max_experts: int) -> None:
    _check(lib().moe_prefetch(cache, next_layer, h, max_experts), "moe_prefetch")


def moe_prefill_layer(cache: int, layer: int, H: int, tokens: int) -> None:
    _check(lib().moe_prefill_layer(cache, layer, H, tokens), "moe_prefill_layer")


def moe_cache_access(cache: int, layer: int, ids: int) -> None:
    _check(lib().moe_cache_access(cache, layer, ids), "moe_cache_access")


def moe_cache_sync(cache: int) -> None:
    _check(lib().moe_cache_sync(cache), "moe_cache_sync")


def moe_cache_stats(cache: int, layers: int):
    arr = (moe_layer_stats * layers)()
    _check(lib().moe_cache_stats(cache, arr, layers), "moe_cache_stats")
    return [{n: getattr(s, n) for n, _ in moe_layer_stats._fields_} for s in arr]


def moe_cache_read_trace(cache: int, cap: int):
    """Returns (records as a list of 8-tuples, dropped count)."""
    arr = (moe_trace_rec * max(cap, 1))()
    n = ctypes.c_size_t()
    dropped = ctypes.c_uint64()
    _check(lib().moe_cache_read_trace(cache, arr, cap, ctypes.byref(n), ctypes.byref(dropped)),
           "moe_cache_read_trace")
    names = [f for f, _ in moe_trace_rec._fields_]
    return [tuple(getattr(arr[i], f) for f in names) for i in range(n.value)], dropped.value


def moe_cache_read_state(cache: int, layer: int, slots: int, experts: int):
    se = (ctypes.c_int32 * slots)()
    es = (ctypes.c_int32 * experts)()
    cnt = (ctypes.c_uint32 * experts)()
    last = (ctypes.c_int64 * experts)()
    clock = ctypes.c_int64()
    _check(lib().moe_cache_read_state(cache, layer, se, es, cnt, last, ctypes.byref(clock)),
           "moe_cache_read_state")
    return list(se), list(es), list(cnt), list(last), clock.value


def moe_cache_last_routing(cache: int, cap: int):
    ids = (ctypes.c_int32 * max(cap, 1))()
    g = (ctypes.c_float * max(cap, 1))()
    n = ctypes.c_size_t()
    _check(lib().moe_cache_last_routing(cache, ids, g, cap, ctypes.byref(n)), "moe_cache_last_routing")
    m = min(n.value, cap)
    return list(ids[:m]), list(g[:m]), n.value


def moe_cache_set_timing(cache: int, level) -> None:
    """level: a MOE_TIMING_* value (False/True are OFF/ALL)."""
    _check(lib().moe_cache_set_timing(cache, int(level)), "moe_cache_set_timing")


def moe_cache_read_timing(cache: int) -> dict:
    t = moe_timing()
    _check(lib().moe_cache_read_timing(cache, ctypes.byref(t)), "moe_cache_read_timing")
    return {n: getattr(t, n) for n, _ in moe_timing._fields_}


def moe_cache_destroy(cache: int) -> None:
    if cache:
        lib().moe_cache_destroy(cache)


def moe_host_alloc(nbytes: int) -> int:
    out = ctypes.c_void_p()
    _check(lib().moe_host_alloc(nbytes, ctypes.byref(out)), "moe_host_alloc")
    return out.value


def moe_host_free(ptr: int) -> None:
    _check(lib().moe_host_free(ptr), "moe_host_free")


def moe_entropy_matrix_bytes(n: int, cap_words: int) -> int:
    return lib().moe_entropy_matrix_bytes(n, cap_words)


def moe_probe_hbm_read(buf_ptr: int, nbytes: int, reps: int, stream: int) -> float:
    """Streaming read rate (GB/s) of nbytes of device memory at buf_ptr."""
    out = ctypes.c_double()
    _check(lib().moe_probe_hbm_read(buf_ptr, nbytes, reps, stream, ctypes.byref(out)), "moe_probe_hbm_read")
    return out.value


def moe_probe_h2d_copy(host_ptr: int, dev_ptr: int, nbytes: int, workgroups: int, reps: int, stream: int) -> float:
    """Host-to-device shader-copy rate (GB/s) from pinned host_ptr to dev_ptr."""
    out = ctypes.c_double()
    _check(lib().moe_probe_h2d_copy(host_ptr, dev_ptr, nbytes, workgroups, reps, stream, ctypes.byref(out)),
           "moe_probe_h2d_copy")
    return out.value


def moe_probe_mfma_bf16(shape: int, iters: int, stream: int) -> float:
    """bf16 matrix-core rate (TFLOP/s) of a register-only MFMA loop."""
    out = ctypes.c_double()
    _check(lib().moe_probe_mfma_bf16(shape, iters, stream, ctypes.byref(out)), "moe_probe_mfma_bf16")
    return out.value


def moe_entropy_pack(w_ptr: int, n: int, cap_words: int, out_ptr: int) -> int:
    """Encode n bf16 weights at host address w_ptr into out_ptr; returns the
    stream words used."""
    used = ctypes.c_size_t()
    _check(lib().moe_entropy_pack(w_ptr, n, cap_words, out_ptr, ctypes.byref(used)), "moe_entropy_pack")
    return used.value
