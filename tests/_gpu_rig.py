"""Shared set-up for the GPU tests: host store, device gates and the oracle's
fp64 view of the same bytes for one configuration."""
import numpy as np

from oracle import stack
from paper_2511_05814_amd import workload as wl


def _say(*a):
    print("[gpu-test]", *a, flush=True)


# The layer-output bounds the specification states (relative L2 against the
# fp64 oracle): 2e-2 for bf16 experts, 1e-5 for fp32 experts.  Group-quantised
# experts dequantise to exact fp32 numbers on both sides, so they take 1e-5.
SPEC_TOL = {"bf16": 2e-2, "f32": 1e-5, "q2g16": 1e-5}
# What the kernels are held to, well inside that ceiling, so that a dropped or
# mis-weighted rank (a combine weight of 0.01 among eight is a 1e-2 error)
# cannot pass: decode keeps fp32 activations and accumulates in fp32 on
# weights that are exact in fp32 (measured about 1e-6); the batch path rounds
# its activations to bf16 for the matrix cores (measured about 3e-3).
DECODE_TOL = 1e-4
BATCH_TOL = 6e-3


def _tol(cfg):
    """Decode bound for this weight type (never above the stated ceiling)."""
    return min(SPEC_TOL[cfg.dtype], DECODE_TOL)


def _batch_tol(cfg):
    return min(SPEC_TOL[cfg.dtype], BATCH_TOL)


class Rig:
    """Host store + gates + oracle model for one configuration."""

    def __init__(self, cfg):
        from paper_2511_05814_amd import offload
        self.cfg = cfg
        self.store = offload.HostStore(cfg)
        self.gates = offload.DeviceGates(cfg)
        self.model = stack.Model(self.gates.host, lambda l, e: self.store.expert(l, e),
                                 cfg.d_model, cfg.d_ff, cfg.dtype)

    def cache(self, slots, policy, **kw):
        from paper_2511_05814_amd import offload
        return offload.OffloadedMoE(self.cfg, self.store, self.gates, slots, policy, **kw)

    def run(self, moe, tokens, flags=0, h0=None):
        cfg = self.cfg
        if h0 is None:
            h0 = wl.hidden_states(cfg, tokens)
        import torch
        H = torch.from_numpy(np.ascontiguousarray(h0[:tokens])).to("cuda")
        snaps = torch.empty((tokens, cfg.layers + 1, cfg.d_model), device="cuda")
        moe.decode(H, flags=flags, snapshots=snaps)
        moe.sync()
        recs, dropped = moe.trace_records()
        assert dropped == 0
        return snaps.cpu().numpy().astype(np.float64), recs, H.cpu().numpy()




class LazyRig(Rig):
    """Rig whose oracle model widens experts on demand and keeps none (the
    90 GB store would not fit in fp64)."""

    def __init__(self, cfg):
        super().__init__(cfg)
        self.model = stack.Model(self.gates.host, lambda l, e: self.store.expert(l, e),
                                 cfg.d_model, cfg.d_ff, cfg.dtype, keep=False)
