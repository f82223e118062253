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

Group-quantised storage ("q2g16", the paper's expert setting of Sec. 5.1:
2-bit codes, groups of 16, compressed zero points): each matrix [rows x cols]
becomes three planes, back to back:
  codes  [rows][cols / 4] uint8, column c at bits 2 (c % 4) of byte c / 4;
  scales [rows][cols / 16] fp16, one per group of 16 consecutive columns;
  zeros  [rows][cols / 16] uint8, zero point = code / 64.
The stored weight is (q - zero) * scale.  The codes come from a plain
round-to-nearest min/max quantiser of the fp32 draw (HQQ's own optimiser needs
real weights and is not reproduced); the gate stays bf16.
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

# group-quantised storage: 16 weights per group, 2-bit codes, fp16 scale,
# 8-bit zero code (zero point = code / Q_ZERO_STEPS); 2 + 16/16 + 8/16 bits
# = 3.5 bits per weight, i.e. 7 bytes per 16 weights
Q_GROUP = 16
Q_ZERO_STEPS = 64
Q_BITS_PER_WEIGHT_X16 = 7


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    seed: int
    layers: int
    experts: int
    top_k: int
    d_model: int
    d_ff: int
    dtype: str            # "f32", "bf16" or "q2g16" (storage type of the experts)
    tokens: int           # batch-1 decode tokens
    slots: tuple          # cache slots per layer to run
    policies: tuple       # ("lru", "lfu") subset
    zipf_s: float
    markov_p: float
    prefetch_max: int = 0
    prefill_tokens: int = 0

    @property
    def gate_dtype(self) -> str:
        """Storage type of the gate: fp32 for the fp32 stack, bf16 otherwise."""
        return "f32" if self.dtype == "f32" else "bf16"

    @property
    def matrix_elems(self) -> int:
        return self.d_model * self.d_ff

    @property
    def expert_elems(self) -> int:
        return 3 * self.matrix_elems

    @property
    def matrix_bytes(self) -> int:
        """Stored bytes of one expert matrix."""
        if self.dtype == "q2g16":
            return self.matrix_elems * Q_BITS_PER_WEIGHT_X16 // 16
        return self.matrix_elems * (4 if self.dtype == "f32" else 2)

    @property
    def expert_bytes(self) -> int:
        return 3 * self.matrix_bytes

    @property
    def storage_dtype(self):
        """numpy type an expert is viewed as: fp32 values, bf16 bit patterns or bytes."""
        return {"f32": np.float32, "bf16": np.uint16, "q2g16": np.uint8}[self.dtype]

    @property
    def expert_storage_len(self) -> int:
        return self.expert_bytes // np.dtype(self.storage_dtype).itemsize

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
    # group-quantised experts (2-bit codes, groups of 16, compressed zeros)
    "tiny-q2": Config("tiny-q2", 251106, 2, 8, 2, 512, 1024, "q2g16", 64,
                      (4,), ("lru", "lfu"), 1.1, 0.6),
    "mixtral-layer-q2": Config("mixtral-layer-q2", 251107, 1, 8, 2, 4096, 14336, "q2g16",
                               256, (4,), ("lru", "lfu"), 1.1, 0.6),
    "mixtral-stack-q2": Config("mixtral-stack-q2", 251108, 32, 8, 2, 4096, 14336, "q2g16",
                               128, (4,), ("lfu",), 1.1, 0.6, prefetch_max=2),
}


def _rng(cfg: Config, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(cfg.seed, spawn_key=tuple(key)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _storage_dtype(cfg: Config):
    return cfg.storage_dtype


def _draw_into(rng: np.random.Generator, out: np.ndarray, dtype: str) -> None:
    """Fill flat `out` with N(0, 0.02^2) drawn in fp32, stored as `dtype`
    ('f32' values or 'bf16' bit patterns)."""
    n = out.size
    std = np.float32(WEIGHT_STD)
    for i in range(0, n, _CHUNK):
        m = min(_CHUNK, n - i)
        v = rng.standard_normal(m, dtype=np.float32)
        v *= std
        out[i:i + m] = v if dtype == "f32" else f32_to_bf16_bits(v)


def quantize_q2g16(w: np.ndarray):
    """Round-to-nearest 2-bit quantisation of fp32 rows in groups of 16
    consecutive columns: scale = (max - min) / 3 rounded to fp16, zero code =
    round(-min / scale * 64) clipped to [0, 255], code = round(w / scale +
    zero) clipped to [0, 3].  Returns (packed codes [rows][cols/4] uint8,
    scales [rows][cols/16] fp16, zero codes [rows][cols/16] uint8)."""
    rows, cols = w.shape
    g = np.asarray(w, np.float32).reshape(rows, cols // Q_GROUP, Q_GROUP)
    lo, hi = g.min(axis=2), g.max(axis=2)
    s = (hi - lo) / np.float32(3)
    s16 = np.where(s > 0, s, np.float32(1)).astype(np.float16)
    s16 = np.where(s16 > 0, s16, np.float16(2.0 ** -24))  # keep every scale positive
    sf = s16.astype(np.float32)
    zc = np.clip(np.rint(-lo / sf * np.float32(Q_ZERO_STEPS)), 0, 255).astype(np.uint8)
    z = zc.astype(np.float32) / np.float32(Q_ZERO_STEPS)
    q = np.clip(np.rint(g / sf[..., None] + z[..., None]), 0, 3).astype(np.uint8).reshape(rows, cols // 4, 4)
    packed = (q[..., 0] | (q[..., 1] << 2) | (q[..., 2] << 4) | (q[..., 3] << 6)).astype(np.uint8)
    return packed, s16, zc


def q2_planes(buf: np.ndarray, rows: int, cols: int):
    """Views (codes, scales, zeros) of one stored q2g16 matrix in byte buffer `buf`."""
    n = rows * cols
    codes = buf[:n // 4].reshape(rows, cols // 4)
    scales = buf[n // 4:n // 4 + n // 8].view(np.float16).reshape(rows, cols // Q_GROUP)
    zeros = buf[n // 4 + n // 8:n // 4 + n // 8 + n // 16].reshape(rows, cols // Q_GROUP)
    return codes, scales, zeros


def _draw_quantized(rng: np.random.Generator, out: np.ndarray, rows: int, cols: int) -> None:
    """Draw a [rows x cols] fp32 matrix (the same stream as the other storage
    types) and store it group-quantised into byte buffer `out`."""
    codes, scales, zeros = q2_planes(out, rows, cols)
    std = np.float32(WEIGHT_STD)
    step = max(1, _CHUNK // cols)
    for r in range(0, rows, step):
        m = min(step, rows - r)
        v = rng.standard_normal(m * cols, dtype=np.float32)
        v *= std
        codes[r:r + m], scales[r:r + m], zeros[r:r + m] = quantize_q2g16(v.reshape(m, cols))


def gate_weights(cfg: Config) -> np.ndarray:
    """Gate tensor [layers][experts][d_model] in the gate's storage dtype."""
    g = np.empty((cfg.layers, cfg.experts, cfg.d_model),
                 dtype=np.float32 if cfg.gate_dtype == "f32" else np.uint16)
    for l in range(cfg.layers):
        _draw_into(_rng(cfg, TAG_GATE, l), g[l].reshape(-1), cfg.gate_dtype)
    return g


def fill_expert(cfg: Config, layer: int, expert: int, out: np.ndarray) -> None:
    """Write expert (layer, expert) as W1 | W3 | W2 into flat `out` (storage dtype)."""
    assert out.size == cfg.expert_storage_len
    shapes = ((cfg.d_ff, cfg.d_model), (cfg.d_ff, cfg.d_model), (cfg.d_model, cfg.d_ff))
    n = out.size // 3
    for j, tag in enumerate((TAG_W1, TAG_W3, TAG_W2)):
        part = out[j * n:(j + 1) * n]
        if cfg.dtype == "q2g16":
            _draw_quantized(_rng(cfg, tag, layer, expert), part, *shapes[j])
        else:
            _draw_into(_rng(cfg, tag, layer, expert), part, cfg.dtype)


def expert_matrix(cfg: Config, layer: int, expert: int, j: int) -> np.ndarray:
    """Matrix j (0 W1, 1 W3, 2 W2) of expert (layer, expert), flat, in the
    storage dtype of a bf16 or fp32 model: the same values fill_expert writes."""
    if cfg.dtype == "q2g16":
        raise ValueError("quantised experts are drawn whole")
    out = np.empty(cfg.matrix_elems, dtype=_storage_dtype(cfg))
    _draw_into(_rng(cfg, (TAG_W1, TAG_W3, TAG_W2)[j], layer, expert), out, cfg.dtype)
    return out


def expert_weights(cfg: Config, layer: int, expert: int) -> np.ndarray:
    out = np.empty(cfg.expert_storage_len, dtype=_storage_dtype(cfg))
    fill_expert(cfg, layer, expert, out)
    return out


def fill_host_store(cfg: Config, out: np.ndarray, workers: Optional[int] = None,
                    layers: Optional[range] = None) -> None:
    """Fill a flat byte buffer laid out [layers][experts][W1|W3|W2].

    `out` may be a view of pinned host memory; it is written in place.
    `layers` restricts the fill to a subset of layers (offsets are unchanged).
    """
    view = out.view(_storage_dtype(cfg)).reshape(cfg.layers, cfg.experts, cfg.expert_storage_len)
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
