"""Shared set-up for the GPU tests: host store, device gates and the oracle's
fp64 view of the same bytes for one configuration."""
import numpy as np

from oracle import stack
from paper_2511_05814_amd import workload as wl


def _say(*a):
    print("[gpu-test]", *a, flush=True)


def _tol(cfg):
    # fp32 and group-quantised weights are exact fp32 numbers on both sides;
    # bf16 uses the bound stated for bf16 experts
    return 2e-2 if cfg.dtype == "bf16" else 1e-5


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
