"""Teacher-forced comparison of a GPU decode run with the fp64 oracle.

The GPU run records the hidden state entering every layer of every token.
The oracle recomputes each layer from those exact fp32 values: routing ids
and next-layer guesses must match exactly wherever the fp64 decision is
certified (logit gaps above the two sides' rounding bound); the cache trace
must match record for record; the layer output y = h_out - h_in must match
the oracle's fp64 y within a relative L2 tolerance.
"""
from __future__ import annotations

import numpy as np

from oracle import stack
from oracle.cache import make_caches


def rel_l2(a, b):
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / max(np.linalg.norm(b), 1e-300))


def check_decode(cfg, model, hs, gpu_recs, slots, policy, prefetch=False, pmax=0,
                 y_tokens=None, tol=1e-5, caches=None, records_out=None):
    """Returns (worst relative L2 of y, uncertified decisions, oracle caches);
    the oracle's records are appended to records_out when it is a list."""
    L, K = cfg.layers, cfg.top_k
    gpu_ids = {}
    gpu_guess = {}
    for r in gpu_recs:
        if r[0] == 0:
            gpu_ids.setdefault((r[1], r[2]), []).append(r[4])
        elif r[0] == 1:
            gpu_guess.setdefault((r[1], r[2]), []).append(r[4])
    caches = caches if caches is not None else make_caches(L, cfg.experts, slots, policy)
    want = []
    worst = 0.0
    unc = 0
    T = hs.shape[0]
    ys = set(range(T)) if y_tokens is None else set(y_tokens)
    for t in range(T):
        for l in range(L):
            with_ffn = t in ys
            st = stack.layer_step(model, l, hs[t, l], K, with_ffn=with_ffn, guess=prefetch)
            if st["certified"]:
                ids = st["ids"]
            else:
                unc += 1
                ids = gpu_ids[(caches[l].lookups, l)]
            want += caches[l].access(ids)
            if prefetch and l + 1 < L:
                if st["guess_certified"]:
                    g = st["guesses"]
                else:
                    unc += 1
                    g = gpu_guess[(caches[l + 1].lookups, l + 1)]
                want += caches[l + 1].prefetch(g, pmax)
            if with_ffn:
                worst = max(worst, rel_l2(hs[t, l + 1] - hs[t, l], st["y"]))
    if records_out is not None:
        records_out.extend(want)
    got = [tuple(int(v) for v in r) for r in gpu_recs]
    exp = [w.astuple() for w in want]
    if got != exp:
        for i, (a, e) in enumerate(zip(got, exp)):
            if a != e:
                raise AssertionError(f"trace differs at record {i}: gpu {a} oracle {e}")
        raise AssertionError(f"trace length differs: gpu {len(got)} oracle {len(exp)}")
    assert worst <= tol, f"y relative L2 {worst:.3e} > {tol:.1e}"
    return worst, unc, caches


def check_y_by_layer(model, hs, layers, k, tol):
    """y = h_{l+1} - h_l of every token at each of `layers` against the fp64
    oracle (teacher-forced from the device's h_l).  `model` keeps widened
    experts; they are dropped after each layer, so a layer's experts are
    widened once however many tokens use them.  Returns the worst relative L2."""
    worst = 0.0
    for l in layers:
        for t in range(hs.shape[0]):
            st = stack.layer_step(model, l, hs[t, l], k)
            worst = max(worst, rel_l2(hs[t, l + 1] - hs[t, l], st["y"]))
        model.forget()
    assert worst <= tol, f"y relative L2 {worst:.3e} > {tol:.1e}"
    return worst
