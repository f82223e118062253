"""Plain fp64 CPU oracle for MoE decode under expert offloading.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path (the HIP library and its
Python binding) never does, and nothing here imports the product path.  It
reads the same input bytes as the HIP path (produced by the seeded workload
generator) and recomputes everything by its plain definition:

* moe.py      rms pre-norm, gate logits, top-k, combine weights, SwiGLU FFN
              (Sec. 2.2 MoE layer; Sec. 4.3 gate = Linear[len_hidden, num_experts],
              softmax then top-K)
* cache.py    per-layer expert cache with LRU (Sec. 3.1) or LFU (Sec. 4.2)
              eviction, the next-layer speculative prefetch (Sec. 3.2, Sec. 4.3)
              and the batched-prefill residency rule
* belady.py   Belady's MIN bound and an exhaustive search for tiny traces
* metrics.py  hit rate, cache precision/recall (Sec. 4.2, Table 2) and
              speculative guess precision/recall (Sec. 5.4)
* stack.py    the residual MoE stack, free-running or teacher-forced

Parity status of every function is listed in its docstring; all functions are
pinned by tests/test_oracle_*.py unless a docstring says "parity unpinned".
"""
