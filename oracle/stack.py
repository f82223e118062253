"""The residual MoE stack run token by token in fp64 (test infrastructure only).

Batch-1 autoregressive decode (Sec. 4.1): tokens pass one after another and
each token visits layers 0..L-1 in order.  There is no attention in this
stack, so the hidden state that enters layer l is h_l and
h_{l+1} = h_l + MoE_l(h_l / rms(h_l)).  At each layer the router's selection
drives that layer's cache (Sec. 3.1, Sec. 4.2); with speculation on, layer
l+1's gate applied to h_l gives the guesses that are prefetched into layer
l+1's cache before that layer's own lookup (Sec. 3.2, Sec. 4.3).
"""
from __future__ import annotations

from typing import Callable, Dict, Optional

import numpy as np

from . import moe, quant
from .cache import LayerCache, make_caches


class Model:
    """fp64 view of stored weights (fp32, bf16 bit patterns, or group-quantised
    bytes); experts are widened on first use and kept."""

    def __init__(self, gates: np.ndarray, expert_source: Callable[[int, int], np.ndarray],
                 d_model: int, d_ff: int, dtype: str, keep: bool = True):
        self.gates = gates
        self.L, self.E = gates.shape[0], gates.shape[1]
        self.d, self.d_ff, self.dtype = d_model, d_ff, dtype
        self._src = expert_source
        self._keep = keep
        self._experts: Dict[tuple, tuple] = {}
        self._gates: Dict[int, np.ndarray] = {}

    def forget(self) -> None:
        """Drop the widened experts kept so far (bounds memory in long checks)."""
        self._experts.clear()

    def gate(self, l: int) -> np.ndarray:
        # the gate of a group-quantised model stays bf16
        if l not in self._gates:
            self._gates[l] = moe.to_f64(self.gates[l], "bf16" if self.dtype == "q2g16" else self.dtype)
        return self._gates[l]

    def expert(self, l: int, e: int):
        key = (l, e)
        if key in self._experts:
            return self._experts[key]
        if self.dtype == "q2g16":
            w = quant.split_expert(self._src(l, e), self.d, self.d_ff)
        else:
            w = moe.split_expert(moe.to_f64(self._src(l, e), self.dtype), self.d, self.d_ff)
        if self._keep:
            self._experts[key] = w
        return w


def layer_step(model: Model, l: int, h: np.ndarray, k: int, with_ffn: bool = True,
               guess: bool = False):
    """One token at one layer from hidden state h (teacher forcing uses the
    device's h here).  Returns a dict with ids, g, certified, y (if asked) and,
    when `guess` is set and l+1 exists, the next-layer guesses."""
    h = np.asarray(h, np.float64)
    ids, g, z, r, cert = moe.route(model.gate(l), h, k)
    out = {"ids": ids, "g": g, "z": z, "r": r, "certified": cert}
    if with_ffn:
        out["y"] = moe.moe_output(lambda e: model.expert(l, e), ids, g, h / r)
    if guess and l + 1 < model.L:
        gw = model.gate(l + 1)
        z2 = moe.gate_logits(gw, h)
        gids = moe.topk(z2, k)
        out["guesses"] = gids
        out["guess_certified"] = moe.topk_certified(z2, gids, moe.logit_error_bound(gw, h))
    return out


def decode_free(model: Model, h0: np.ndarray, k: int, policy: str, slots: int,
                prefetch: bool = False, prefetch_max: int = 0, caches=None,
                with_ffn: bool = True):
    """Free-running decode of h0 [T][d].  Returns (h per (t, l) [T][L+1][d],
    records, caches, uncertified-decision count)."""
    L = model.L
    caches = caches if caches is not None else make_caches(L, model.E, slots, policy)
    T = h0.shape[0]
    hs = np.empty((T, L + 1, model.d))
    recs = []
    uncertified = 0
    for t in range(T):
        h = np.asarray(h0[t], np.float64)
        for l in range(L):
            hs[t, l] = h
            st = layer_step(model, l, h, k, with_ffn=with_ffn, guess=prefetch)
            uncertified += not st["certified"]
            recs += caches[l].access(st["ids"])
            if prefetch and l + 1 < L:
                uncertified += not st["guess_certified"]
                recs += caches[l + 1].prefetch(st["guesses"], prefetch_max)
            if with_ffn:
                h = h + st["y"]
        hs[t, L] = h
    return hs, recs, caches, uncertified


def replay(ids_tl, guesses_tl, L: int, E: int, slots: int, policy: str,
           prefetch_max: int = 0, caches=None):
    """Drive the caches with given routing: ids_tl[t][l] (rank order) and, when
    speculation is on, guesses_tl[t][l] = guesses for layer l+1 made at layer l
    (None for no speculation)."""
    caches = caches if caches is not None else make_caches(L, E, slots, policy)
    recs = []
    for t in range(len(ids_tl)):
        for l in range(L):
            recs += caches[l].access(ids_tl[t][l])
            if guesses_tl is not None and l + 1 < L and guesses_tl[t][l] is not None:
                recs += caches[l + 1].prefetch(guesses_tl[t][l], prefetch_max)
    return recs, caches


def prefill_layer(model: Model, l: int, H: np.ndarray, k: int, cache: Optional[LayerCache],
                  with_ffn: bool = True, rows: Optional[np.ndarray] = None):
    """A batch of T tokens through layer l at once: every row is routed and
    computed exactly as a decode token would be; the cache sees the whole
    batch's routing through its prefill rule.  `rows` restricts the FFN to a
    subset of rows (the others are returned unchanged)."""
    H = np.asarray(H, np.float64)
    T = H.shape[0]
    ids = np.empty((T, k), np.int64)
    g = np.empty((T, k))
    cert = np.empty(T, bool)
    for t in range(T):
        i, gg, _, _, c = moe.route(model.gate(l), H[t], k)
        ids[t], g[t], cert[t] = i, gg, c
    out = H.copy()
    if with_ffn:
        for t in (range(T) if rows is None else rows):
            r = moe.rms(H[t])
            out[t] = H[t] + moe.moe_output(lambda e: model.expert(l, e), ids[t], g[t], H[t] / r)
    recs = cache.prefill(ids) if cache is not None else []
    return out, ids, g, cert, recs
