"""fp64 MoE layer math, written from its plain definitions (test infrastructure only).

Sec. 2.2: an MoE layer is a gating network plus several FFN experts, and only
the experts the gate selects run for a token.  Sec. 4.3: the gate is a linear
map [len_hidden, num_experts]; its output goes through a softmax and a top-K
(K = 2 for Mixtral).  The paper states neither the expert form, the tie rule,
the normalisation nor whether the top-K weights are renormalised; the readings
taken here are:

* pre-norm: x = h / sqrt(mean(h^2) + 1e-5)  (unit-weight RMSNorm);
* logits z = W_g h on the raw residual h (top-K ranks do not depend on the
  positive scale 1/r, so routing is independent of the norm);
* top-K = first K of a stable sort by (z descending, expert id ascending);
* combine weights g = softmax over the K selected logits z/r (renormalised);
* expert = SwiGLU: y = W2 (SiLU(W1 x) * (W3 x)), SiLU(a) = a / (1 + e^-a).
"""
from __future__ import annotations

import numpy as np

EPS = 1e-5
U64 = 2.0 ** -53  # unit roundoff of fp64


def bf16_bits_to_f64(u16: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns: the bits are the top half of an fp32."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def to_f64(w: np.ndarray, dtype: str) -> np.ndarray:
    """Storage-dtype array ('bf16' as uint16 bits, or 'f32') -> fp64, exactly."""
    if dtype == "bf16":
        return bf16_bits_to_f64(w)
    return np.asarray(w, dtype=np.float32).astype(np.float64)


def rms(h: np.ndarray) -> float:
    """r = sqrt(mean(h^2) + eps): the pre-norm scale (reading: unit-weight RMSNorm)."""
    h = np.asarray(h, dtype=np.float64)
    return float(np.sqrt(np.mean(h * h) + EPS))


def gate_logits(w_gate: np.ndarray, h: np.ndarray) -> np.ndarray:
    """z = W_g h for one layer's gate W_g [E x d] (Sec. 4.3), in fp64."""
    return np.asarray(w_gate, np.float64) @ np.asarray(h, np.float64)


def logit_error_bound(w_gate: np.ndarray, h: np.ndarray) -> np.ndarray:
    """Per-logit bound on |computed - exact| for a length-d fp64 dot product
    evaluated by either side in any order: tau_e = 2 d u sum_i |w_ei h_i|.
    Used to certify that a top-K decision cannot flip between two correct
    fp64 evaluations."""
    d = np.asarray(h).shape[-1]
    a = np.abs(np.asarray(w_gate, np.float64)) @ np.abs(np.asarray(h, np.float64))
    return 2.0 * d * U64 * a


def topk(z: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest logits in rank order; ties go to the lower id.

    A stable sort on -z keeps equal logits in ascending id order."""
    order = np.argsort(-np.asarray(z, np.float64), kind="stable")
    return order[:k].astype(np.int64)


def topk_certified(z: np.ndarray, ids: np.ndarray, tau: np.ndarray) -> bool:
    """True when every decision that fixes `ids` (membership and rank order)
    has a logit gap larger than the two sides' combined error bound."""
    z = np.asarray(z, np.float64)
    k = len(ids)
    chosen = list(ids)
    for a, b in zip(chosen[:-1], chosen[1:]):           # order inside the top-k
        if z[a] - z[b] <= tau[a] + tau[b]:
            return False
    rest = [e for e in range(len(z)) if e not in set(chosen)]
    if rest and k > 0:
        last = chosen[-1]
        for e in rest:                                    # membership
            if z[last] - z[e] <= tau[last] + tau[e]:
                return False
    return True


def softmax(v: np.ndarray) -> np.ndarray:
    """exp(v - max v) / sum exp(v - max v), fp64."""
    v = np.asarray(v, np.float64)
    e = np.exp(v - np.max(v))
    return e / np.sum(e)


def combine_weights(z: np.ndarray, ids: np.ndarray, r: float) -> np.ndarray:
    """g_r = softmax over the selected logits z_{i_r} / r (renormalised top-K)."""
    return softmax(np.asarray(z, np.float64)[np.asarray(ids)] / r)


def route(w_gate: np.ndarray, h: np.ndarray, k: int):
    """Router of one layer for one token: (ids, g, z, r, certified)."""
    h = np.asarray(h, np.float64)
    z = gate_logits(w_gate, h)
    ids = topk(z, k)
    r = rms(h)
    g = combine_weights(z, ids, r)
    cert = topk_certified(z, ids, logit_error_bound(w_gate, h))
    return ids, g, z, r, cert


def silu(a: np.ndarray) -> np.ndarray:
    """SiLU(a) = a / (1 + exp(-a))."""
    a = np.asarray(a, np.float64)
    return a / (1.0 + np.exp(-a))


def split_expert(flat: np.ndarray, d: int, d_ff: int):
    """Views W1 [d_ff x d], W3 [d_ff x d], W2 [d x d_ff] of a W1|W3|W2 expert."""
    m = d * d_ff
    return (flat[:m].reshape(d_ff, d), flat[m:2 * m].reshape(d_ff, d),
            flat[2 * m:3 * m].reshape(d, d_ff))


def expert_ffn(w1: np.ndarray, w3: np.ndarray, w2: np.ndarray, x: np.ndarray) -> np.ndarray:
    """SwiGLU expert: W2 (SiLU(W1 x) * (W3 x)), fp64."""
    x = np.asarray(x, np.float64)
    return np.asarray(w2, np.float64) @ (silu(np.asarray(w1, np.float64) @ x)
                                         * (np.asarray(w3, np.float64) @ x))


def moe_output(experts, ids, g, x) -> np.ndarray:
    """y = sum_r g_r FFN_{i_r}(x); `experts(e)` returns (W1, W3, W2) in fp64."""
    y = None
    for r, e in enumerate(ids):
        w1, w3, w2 = experts(int(e))
        t = g[r] * expert_ffn(w1, w3, w2, x)
        y = t if y is None else y + t
    return y


def moe_layer(w_gate, experts, h, k):
    """One residual pre-norm MoE layer: h' = h + sum_r g_r FFN_{i_r}(h / r).

    Returns (h', ids, g, certified)."""
    h = np.asarray(h, np.float64)
    ids, g, _, r, cert = route(w_gate, h, k)
    y = moe_output(experts, ids, g, h / r)
    return h + y, ids, g, cert
