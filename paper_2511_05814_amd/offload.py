"""Buffers and streams around the C ABI, allocated with PyTorch (plumbing only).

* `HostStore`  pinned host memory holding every expert, [L][E][W1|W3|W2]
* `DeviceGates` the gate tensor [L][E][d] in HBM
* `OffloadedMoE` one cache handle: its HBM slot arena, workspace, trace ring
  and two streams (compute and copy), plus thin loops that call
  moe_decode_layer / moe_prefill_layer for every layer.

All arithmetic of the decode path runs in the HIP library; this module only
allocates, fills inputs and calls the binding.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import numpy as np

from . import binding as b
from . import entropy, pack
from . import workload as wl


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("a ROCm GPU is required for the HIP decode path")
    return torch


class HostStore:
    """Pinned host store of all experts, one allocation per layer, filled from
    the seeded generator.

    The GPU driver caps how much host memory can be pinned (about 70 GB on an
    MI355X machine with 295 GB of RAM), below the 90 GB a 32-layer Mixtral-shaped
    stack needs.  When the store would exceed `max_pinned_bytes`, only the
    first `distinct` layers get pages of their own and layer l uses the pages
    of layer l mod distinct: every fetch still moves a whole expert over the
    host link, only the weight values repeat (gates stay per layer).

    fmt selects how bf16 experts are held (the GPU rebuilds identical bf16
    weights after each copy, so fewer bytes cross the host link per miss):
    "plain" (as stored in HBM), "packed" (paper_2511_05814_amd.pack, about
    12.25 bits a weight; `cap` = exception entries per matrix, default
    n / 4096 + 64, about three times what N(0, sigma) weights need) or
    "entropy" (paper_2511_05814_amd.entropy, about 10.9 bits a weight; `cap`
    = stream words per matrix, by default 1% above what the first matrix of
    the store needs).
    packed=True is the same as fmt="packed"."""

    FORMATS = ("plain", "packed", "entropy")

    def __init__(self, cfg: wl.Config, fill: bool = True, workers: Optional[int] = None,
                 max_pinned_bytes: int = 64 << 30, packed: bool = False, fmt: Optional[str] = None,
                 cap: Optional[int] = None):
        self.cfg = cfg
        fmt = fmt or ("packed" if packed else "plain")
        if fmt not in self.FORMATS:
            raise ValueError(f"unknown host store format {fmt!r}")
        self.fmt = fmt
        self.packed = fmt != "plain"   # a coded store: copies move coded bytes
        n = cfg.matrix_elems
        if self.packed and cfg.dtype != "bf16":
            raise ValueError("a coded host store holds bf16 experts")
        if fmt == "packed":
            self.cap = cap if cap is not None else n // 4096 + 64
            self.matrix_stride = pack.matrix_capacity(n, self.cap)
        elif fmt == "entropy":
            self.cap = cap if cap is not None else self._entropy_cap(cfg)
            self.matrix_stride = entropy.matrix_capacity(n, self.cap)
        else:
            self.cap = 0
            self.matrix_stride = cfg.matrix_bytes
        self.expert_stride = 3 * self.matrix_stride
        self.layer_bytes = cfg.experts * self.expert_stride
        self.distinct = int(max(1, min(cfg.layers, max_pinned_bytes // self.layer_bytes)))
        self.nbytes = self.distinct * self.layer_bytes
        self.ptrs = []
        self.arrays = []
        try:
            for _ in range(self.distinct):
                p = b.moe_host_alloc(self.layer_bytes)
                self.ptrs.append(p)
                self.arrays.append(np.ctypeslib.as_array((ctypes.c_uint8 * self.layer_bytes).from_address(p)))
        except Exception:
            self.close()
            raise
        self.layer_src = [l % self.distinct for l in range(cfg.layers)]
        self.layer_ptrs = (ctypes.c_void_p * cfg.layers)(*[self.ptrs[s] for s in self.layer_src])
        if fill:
            self._fill(workers)

    def _fill(self, workers):
        import os
        from concurrent.futures import ThreadPoolExecutor
        cfg = self.cfg
        sdt = cfg.storage_dtype
        todo = [(l, e) for l in range(self.distinct) for e in range(cfg.experts)]

        def one(le):
            l, e = le
            if self.packed:
                raw = wl.expert_weights(cfg, l, e)
                n = cfg.matrix_elems
                row = self.arrays[l].reshape(cfg.experts, self.expert_stride)[e]
                for m in range(3):
                    dst = row[m * self.matrix_stride:(m + 1) * self.matrix_stride]
                    if self.fmt == "entropy":
                        entropy.pack_matrix(raw[m * n:(m + 1) * n], self.cap, dst)
                    else:
                        pack.pack_matrix(raw[m * n:(m + 1) * n], self.cap, out=dst)
                return
            view = self.arrays[l].view(sdt).reshape(cfg.experts, cfg.expert_storage_len)
            wl.fill_expert(cfg, l, e, view[e])

        workers = workers or max(1, min(16, os.cpu_count() or 1))
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(one, todo))

    @staticmethod
    def _entropy_cap(cfg: wl.Config) -> int:
        """Stream words per matrix: what W1 of expert (0, 0) needs plus 2% and
        one row (64 words) per span.  Every matrix of the generator has the
        same distribution; what varies is mostly the padding of each span to
        its longest lane stream, well within that margin."""
        n = cfg.matrix_elems
        probe = entropy.default_cap_words(n)
        buf = np.empty(entropy.matrix_capacity(n, probe), dtype=np.uint8)
        used = entropy.pack_matrix(wl.expert_matrix(cfg, 0, 0, 0), probe, buf)
        return used + used // 50 + 64 * entropy.spans(n)

    @property
    def aliased(self) -> bool:
        return self.distinct < self.cfg.layers

    def expert(self, layer: int, expert: int) -> np.ndarray:
        """Storage-dtype view of one expert (W1|W3|W2).  A packed store holds
        an exact encoding of the generator's bf16 weights, so those are
        returned (drawn again) rather than the packed bytes."""
        cfg = self.cfg
        if self.packed:
            return wl.expert_weights(cfg, self.layer_src[layer], expert)
        off = expert * cfg.expert_bytes
        raw = self.arrays[self.layer_src[layer]][off:off + cfg.expert_bytes]
        return raw.view(cfg.storage_dtype)

    def layer_array(self, layer: int) -> np.ndarray:
        return self.arrays[self.layer_src[layer]]

    def close(self):
        self.arrays = []
        for p in self.ptrs:
            b.moe_host_free(p)
        self.ptrs = []

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DeviceGates:
    def __init__(self, cfg: wl.Config, gates: Optional[np.ndarray] = None):
        torch = _torch()
        self.host = gates if gates is not None else wl.gate_weights(cfg)
        raw = np.ascontiguousarray(self.host).view(np.uint8).reshape(-1)
        self.tensor = torch.from_numpy(raw.copy()).to("cuda")

    @property
    def ptr(self) -> int:
        return self.tensor.data_ptr()


class OffloadedMoE:
    """One expert cache over a whole stack (one handle of the C ABI)."""

    def __init__(self, cfg: wl.Config, store: HostStore, gates: DeviceGates, slots: int,
                 policy: str, prefetch_max: int = 0, fetch_mode: int = b.MOE_FETCH_SPLIT,
                 trace_cap: Optional[int] = None, max_prefill_tokens: int = 0,
                 separate_copy_stream: bool = True):
        torch = _torch()
        self.cfg, self.store, self.gates = cfg, store, gates
        self.L, self.E, self.S, self.K = cfg.layers, cfg.experts, slots, cfg.top_k
        policy_id, aging = b.parse_policy(policy)
        self.handle = b.moe_cache_create(cfg.layers, cfg.experts, slots, policy_id)
        try:
            self.compute = torch.cuda.Stream()
            self.copy = torch.cuda.Stream() if separate_copy_stream else self.compute
            self.arena = torch.empty(cfg.layers * slots * cfg.expert_bytes, dtype=torch.uint8,
                                     device="cuda")
            if trace_cap is None:
                trace_cap = max(1024, 2 * self.K * self.L * (cfg.tokens + cfg.prefill_tokens + 8))
            self.trace_cap = trace_cap
            self.trace = (torch.empty(trace_cap * 32, dtype=torch.uint8, device="cuda")
                          if trace_cap > 0 else None)
            d = b.moe_model_desc()
            d.d_model, d.d_ff, d.top_k = cfg.d_model, cfg.d_ff, cfg.top_k
            d.dtype = b.DTYPES[cfg.dtype]
            d.prefetch_max = prefetch_max
            d.fetch_mode = fetch_mode
            d.max_prefill_tokens = max_prefill_tokens
            d.host_format = {"plain": b.MOE_HOST_PLAIN, "packed": b.MOE_HOST_PACKED,
                             "entropy": b.MOE_HOST_ENTROPY}[store.fmt]
            d.packed_cap = store.cap
            d.aging_ticks = aging
            d.gate_w = gates.ptr
            d.host_experts = None
            d.host_layers = ctypes.cast(store.layer_ptrs, ctypes.POINTER(ctypes.c_void_p))
            d.arena = self.arena.data_ptr()
            d.trace = self.trace.data_ptr() if self.trace is not None else None
            d.trace_cap = trace_cap if self.trace is not None else 0
            d.compute_stream = self.compute.cuda_stream
            d.copy_stream = self.copy.cuda_stream
            ws = b.moe_cache_workspace_bytes(self.handle, d)
            if ws == 0:
                raise b.MoeError(b.MOE_ERR_ARG, "moe_cache_workspace_bytes", b.moe_last_error())
            self.workspace = torch.empty(ws, dtype=torch.uint8, device="cuda")
            d.workspace = self.workspace.data_ptr()
            d.workspace_bytes = ws
            self.desc = d
            torch.cuda.synchronize()
            b.moe_cache_bind(self.handle, d)
            b.moe_cache_reset(self.handle)
        except Exception:
            b.moe_cache_destroy(self.handle)
            self.handle = 0
            raise

    # -- driving the stack ------------------------------------------------------
    def reset(self):
        b.moe_cache_reset(self.handle)

    def decode(self, H, flags: int = 0, snapshots=None):
        """Decode tokens H [T][d] (fp32, device) in place, token by token.

        snapshots (optional, device [T][L+1][d]) receives h entering every layer
        and the final output, copied on the compute stream."""
        torch = _torch()
        self.compute.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(self.compute):
            for t in range(H.shape[0]):
                row = H[t]
                p = row.data_ptr()
                for l in range(self.L):
                    if snapshots is not None:
                        snapshots[t, l].copy_(row)
                    b.moe_decode_layer(self.handle, l, p, flags)
                if snapshots is not None:
                    snapshots[t, self.L].copy_(row)

    def decode_layer(self, layer: int, h, flags: int = 0):
        b.moe_decode_layer(self.handle, layer, h.data_ptr(), flags)

    def prefill(self, H, snapshots=None):
        """All layers over the token batch H [T][d] (fp32, device) in place."""
        torch = _torch()
        self.compute.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(self.compute):
            for l in range(self.L):
                if snapshots is not None:
                    snapshots[l].copy_(H)
                b.moe_prefill_layer(self.handle, l, H.data_ptr(), H.shape[0])
            if snapshots is not None:
                snapshots[self.L].copy_(H)

    def decode_batched(self, H, batch: int):
        """Decode tokens H [T][d] (fp32, device) in place, `batch` tokens at a
        time: each group of tokens goes through all layers as one batch
        (moe_prefill_layer: batched routing, the batch residency rule and the
        grouped GEMMs), which is batched decode of `batch` sequences."""
        for g in range(0, H.shape[0], batch):
            self.prefill(H[g:g + batch])

    def sync(self):
        b.moe_cache_sync(self.handle)

    def stats(self):
        return b.moe_cache_stats(self.handle, self.L)

    def trace_records(self):
        recs, dropped = b.moe_cache_read_trace(self.handle, self.trace_cap)
        return recs, dropped

    def state(self, layer: int):
        return b.moe_cache_read_state(self.handle, layer, self.S, self.E)

    def close(self):
        if self.handle:
            b.moe_cache_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
