"""Seeded synthetic inputs for the MoE-offloading decode path.

This module only draws random numbers and lays bytes out; it holds none of the
method's arithmetic (no routing, no caching, no FFN).  Both the HIP path and
the fp64 oracle read the bytes it produces, so they see identical inputs.

The paper ran Mixtral-8x7B on one chat prompt and an MMLU subset (Sec. 4.1).
Neither the weights nor the prompts are available, so these inputs stand in
for them:

* every gate and expert matrix is N(0, 0.02^2), drawn in fp32 and rounded to
  bf16 with round-to-nearest-even (fp32 workloads keep the fp32 draw);
* a token's hidden state is alpha * u_c + n, where u_c is one of E random unit
  "concept" directions, c follows a Zipf(s) law over concepts with Markov
  persistence p (the same concept as the previous token with probability p),
  and n ~ N(0, I).  Zipf skew models the expert imbalance and Markov
  persistence models the temporal locality the paper reports (Sec. 3.1,
  Sec. 5.2, Sec. 6.1);
* alpha = sqrt(d_model).

Expert storage layout (host store and HBM slots alike): per expert the three
matrices W1 [d_ff x d], W3 [d_ff x d] and W2 [d x d_ff], each row-major
(out x in), stored back to back as W1 | W3 | W2.  The host store is
[layers][experts][expert bytes]; the gate tensor is [layers][experts][d].
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

# sub-stream tags for np.random.SeedSequence(seed, spawn_key=(tag, ...))
TAG_GATE, TAG_W1, TAG_W3, TAG_W2, TAG_DIR, TAG_CHAIN, TAG_NOISE = range(7)

WEIGHT_STD = 0.02
_CHUNK = 1 << 22  # elements generated per call, bounds temporary memory


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    seed: int
    layers: int
    experts: int
    top_k: int
    d_model: int
    d_ff: int
    dtype: str            # "f32" or "bf16" (storage type of gates and experts)
    tokens: int           # batch-1 decode tokens
    slots: tuple          # cache slots per layer to run
    policies: tuple       # ("lru", "lfu") subset
    zipf_s: float
    markov_p: float
    prefetch_max: int = 0
    prefill_tokens: int = 0

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def matrix_elems(self) -> int:
        return self.d_model * self.d_ff

    @property
    def expert_elems(self) -> int:
        return 3 * self.matrix_elems

    @property
    def expert_bytes(self) -> int:
        return self.expert_elems * self.elem_bytes

    @property
    def alpha(self) -> float:
        return math.sqrt(self.d_model)

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads.  Seeds are 251100 + i for the i-th workload.
CONFIGS = {
    # 2 layers x 8 experts, top-2, d=256, d_ff=512, fp32, 64 tokens, 4 slots
    "tiny-stack": Config("tiny-stack", 251101, 2, 8, 2, 256, 512, "f32", 64,
                         (4,), ("lru", "lfu"), 1.1, 0.6),
    # one Mixtral-8x7B-shaped layer, bf16, 256 tokens, 4 slots
    "mixtral-layer": Config("mixtral-layer", 251102, 1, 8, 2, 4096, 14336, "bf16",
                            256, (4,), ("lru", "lfu"), 1.1, 0.6),
    # 32 Mixtral-shaped layers, 512 tokens, 2/4/6 slots
    "mixtral-stack": Config("mixtral-stack", 251103, 32, 8, 2, 4096, 14336, "bf16",
                            512, (2, 4, 6), ("lru", "lfu"), 1.1, 0.6),
    # the same stack with next-layer speculative prefetch of up to 2 experts
    "mixtral-stack-prefetch": Config("mixtral-stack-prefetch", 251104, 32, 8, 2, 4096,
                                     14336, "bf16", 512, (4,), ("lfu",), 1.1, 0.6,
                                     prefetch_max=2),
    # 24 layers x 64 experts, top-8, d=2048, d_ff=1408; 4096-token prefill then
    # 256 decode tokens; 16 slots, LFU + prefetch
    "fine-grained": Config("fine-grained", 251105, 24, 64, 8, 2048, 1408, "bf16", 256,
                           (16,), ("lfu",), 1.2, 0.6, prefetch_max=2, prefill_tokens=4096),
}


def _rng(cfg: Config, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(cfg.seed, spawn_key=tuple(key)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _storage_dtype(cfg: Config):
    return np.float32 if cfg.dtype == "f32" else np.uint16


def _draw_into(rng: np.random.Generator, out: np.ndarray, cfg: Config) -> None:
    """Fill flat `out` (storage dtype) with N(0, 0.02^2) drawn in fp32."""
    n = out.size
    std = np.float32(WEIGHT_STD)
    for i in range(0, n, _CHUNK):
        m = min(_CHUNK, n - i)
        v = rng.standard_normal(m, dtype=np.float32)
        v *= std
        out[i:i + m] = v if cfg.dtype == "f32" else f32_to_bf16_bits(v)


def gate_weights(cfg: Config) -> np.ndarray:
    """Gate tensor [layers][experts][d_model] in the storage dtype."""
    g = np.empty((cfg.layers, cfg.experts, cfg.d_model), dtype=_storage_dtype(cfg))
    for l in range(cfg.layers):
        _draw_into(_rng(cfg, TAG_GATE, l), g[l].reshape(-1), cfg)
    return g


def fill_expert(cfg: Config, layer: int, expert: int, out: np.ndarray) -> None:
    """Write expert (layer, expert) as W1 | W3 | W2 into flat `out` (storage dtype)."""
    m = cfg.matrix_elems
    assert out.size == 3 * m
    for j, tag in enumerate((TAG_W1, TAG_W3, TAG_W2)):
        _draw_into(_rng(cfg, tag, layer, expert), out[j * m:(j + 1) * m], cfg)


def expert_weights(cfg: Config, layer: int, expert: int) -> np.ndarray:
    out = np.empty(cfg.expert_elems, dtype=_storage_dtype(cfg))
    fill_expert(cfg, layer, expert, out)
    return out


def fill_host_store(cfg: Config, out: np.ndarray, workers: Optional[int] = None,
                    layers: Optional[range] = None) -> None:
    """Fill a flat byte buffer laid out [layers][experts][W1|W3|W2].

    `out` may be a view of pinned host memory; it is written in place.
    `layers` restricts the fill to a subset of layers (offsets are unchanged).
    """
    view = out.view(_storage_dtype(cfg)).reshape(cfg.layers, cfg.experts, cfg.expert_elems)
    todo = [(l, e) for l in (layers if layers is not None else range(cfg.layers))
            for e in range(cfg.experts)]
    if workers is None:
        workers = max(1, min(16, os.cpu_count() or 1))
    if workers == 1 or len(todo) == 1:
        for l, e in todo:
            fill_expert(cfg, l, e, view[l, e])
        return
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda le: fill_expert(cfg, le[0], le[1], view[le[0], le[1]]), todo))


def concept_directions(cfg: Config) -> np.ndarray:
    """E random unit vectors in R^d (fp32), one per concept."""
    u = _rng(cfg, TAG_DIR).standard_normal((cfg.experts, cfg.d_model))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    return u.astype(np.float32)


def zipf_probabilities(E: int, s: float) -> np.ndarray:
    r = np.arange(1, E + 1, dtype=np.float64)
    p = r ** (-s)
    return p / p.sum()


def concept_chain(cfg: Config, tokens: int) -> np.ndarray:
    """Concept per token: Zipf(s) over E concepts with Markov persistence p.

    Each token consumes two uniforms: the first decides persistence, the second
    drives the inverse-CDF Zipf draw (rank r -> concept r-1).
    """
    u = _rng(cfg, TAG_CHAIN).random((tokens, 2))
    cdf = np.cumsum(zipf_probabilities(cfg.experts, cfg.zipf_s))
    fresh = np.minimum(np.searchsorted(cdf, u[:, 1], side="right"), cfg.experts - 1)
    c = np.empty(tokens, dtype=np.int64)
    for t in range(tokens):
        c[t] = c[t - 1] if (t > 0 and u[t, 0] < cfg.markov_p) else fresh[t]
    return c


def hidden_states(cfg: Config, tokens: Optional[int] = None) -> np.ndarray:
    """Layer-0 hidden states [tokens][d] fp32: alpha * u_c + N(0, I).

    With a prefill, tokens 0..prefill_tokens-1 are the prefill batch and the
    decode tokens follow.
    """
    T = tokens if tokens is not None else cfg.prefill_tokens + cfg.tokens
    c = concept_chain(cfg, T)
    u = concept_directions(cfg)
    n = _rng(cfg, TAG_NOISE).standard_normal((T, cfg.d_model), dtype=np.float32)
    return (np.float32(cfg.alpha) * u[c] + n).astype(np.float32)


def scaled(cfg: Config, **kw) -> Config:
    """A copy with some fields changed (e.g. fewer tokens for a parity slice)."""
    return cfg.with_(**kw)
