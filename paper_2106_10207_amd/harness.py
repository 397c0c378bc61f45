"""Device-side set-up of one averaging round for a synthetic workload.

Builds, on one GPU, what a round needs: every peer's encoded message (each
peer's fp32 mean gradient encoded by the library, as that peer would before
sending), the sample counts, shard bounds, the optimizer state and the
workspace, and a pre-marshalled dedloc_round call.  Used by the benchmark
and the smoke check; the GPU tests use it to set up the same launch
configuration the benchmark times.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import dedloc as D
from . import workloads as W


def codec_id(wl: W.Workload) -> int:
    return D.DEDLOC_CODEC_FP16 if wl.codec == "fp16" else D.DEDLOC_CODEC_I8


class DeviceRound:
    """All buffers of one round of workload `wl` on `device`.

    sample_ranges: element ranges [a, b) whose fp32 peer gradients are kept
    on the host (for checking against a CPU evaluation of the same inputs).
    poison_zero: zero-sample peers get NaN-filled messages (they must never
    be read).  fresh: start from m = v = 0.  fused_local: the round itself
    encodes the local peer's fp32 gradient into its message (the local
    gradient is kept on the device)."""

    def __init__(self, wl: W.Workload, device="cuda", fresh: bool = False,
                 poison_zero: bool = True, step: Optional[int] = None,
                 sample_ranges: Sequence[Tuple[int, int]] = (), keep_local_grad: bool = False,
                 with_mean: bool = False, optimizer: str = "lamb", fused_local: bool = False):
        import torch
        self.wl = wl
        self.device = device
        self.codec = codec_id(wl)
        self.block = D.DEDLOC_I8_BLOCK if wl.codec == "i8" else 0
        P = wl.P
        self.counts = W.sample_counts(wl)
        self.bounds = D.dedloc_partition(P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
        self.offsets = wl.offsets()
        self.flags = wl.flags()
        self.local = int(np.flatnonzero(self.counts)[0])  # this GPU's own peer
        self.codes: List = []
        self.scales: List = []
        self.host_grads: Dict[int, List[np.ndarray]] = {p: [] for p in range(wl.n_peers)}
        self.local_grad = None
        cdt = torch.int16 if self.codec == D.DEDLOC_CODEC_FP16 else torch.int8
        nsc = (P + 1023) // 1024
        for p in range(wl.n_peers):
            g = W.peer_gradient(wl, p, device)
            for (a, b) in sample_ranges:
                self.host_grads[p].append(g[a:b].cpu().numpy())
            c = torch.empty(P, dtype=cdt, device=device)
            s = torch.empty(nsc, dtype=torch.float32, device=device) if self.codec == D.DEDLOC_CODEC_I8 else None
            if self.counts[p] == 0 and poison_zero:
                W.nan_poison(c)
                if s is not None:
                    W.nan_poison(s)
            else:
                D.dedloc_encode(g, self.codec, self.block or D.DEDLOC_I8_BLOCK, c, s)
            if p == self.local and (keep_local_grad or fused_local):
                self.local_grad = g
            del g
            self.codes.append(c)
            self.scales.append(s)
        self.x, self.m, self.v = W.optimizer_state(wl, device, fresh=fresh)
        self.out_codes = torch.empty(P, dtype=cdt, device=device)
        self.out_scales = (torch.empty(nsc, dtype=torch.float32, device=device)
                           if self.codec == D.DEDLOC_CODEC_I8 else None)
        self.trust = torch.empty(wl.n_tensors, dtype=torch.float32, device=device)
        self.mean = torch.empty(P, dtype=torch.float32, device=device) if with_mean else None
        self.ws = D.make_workspace(P, self.offsets, device)
        self.step = wl.step if step is None else step
        self.optimizer = optimizer
        if optimizer == "lamb":
            self.cfg = D.lamb_cfg(wl.lr, wl.beta1, wl.beta2, wl.eps, wl.weight_decay, step=self.step)
        elif optimizer == "lars":
            # LARS keeps one buffer: the momentum (held in m; v is unused)
            self.cfg = D.lars_cfg(wl.lars_lr, wl.lars_momentum, wl.lars_trust_coef, wl.lars_weight_decay)
            self.v = self.m
        else:
            raise ValueError(f"unknown optimizer {optimizer!r}")
        self.fused_local = fused_local
        args = (self.codes, self.counts, self.bounds, self.codec, self.out_codes,
                self.x, self.m, self.v, self.offsets, self.flags, self.cfg, self.ws)
        kw = dict(peer_scales=self.scales if self.codec == D.DEDLOC_CODEC_I8 else None,
                  out_scales=self.out_scales, trust_out=self.trust, out_mean=self.mean,
                  block=self.block or D.DEDLOC_I8_BLOCK)
        self.call = D.RoundCall(*args, **kw, local=(self.local, self.local_grad) if fused_local else None)
        # the round alone, over the messages as they stand (every peer's
        # message already encoded)
        self.call_round_only = D.RoundCall(*args, **kw) if fused_local else self.call
        torch.cuda.synchronize()

    def set_step(self, step: int):
        self.step = step
        self.cfg.step = step

    def encode_local(self):
        """The local peer encodes its own fresh gradient into its message
        slot (the sender side of the exchange)."""
        D.dedloc_encode(self.local_grad, self.codec, self.block or D.DEDLOC_I8_BLOCK,
                        self.codes[self.local], self.scales[self.local])

    def run(self):
        self.call()

    # byte accounting of one round (the algorithmic traffic)
    def bytes_peer_input(self) -> float:
        n_act = int(np.count_nonzero(self.counts))
        return n_act * self.wl.P * self.wl.wire_bytes_per_elem

    def bytes_round(self) -> float:
        """Compulsory bytes: peer messages, the gathered message, and the
        optimizer state read and written once (x, m, v for LAMB; x and the
        momentum for LARS)."""
        P = self.wl.P
        state = 24.0 if self.optimizer == "lamb" else 16.0
        return self.bytes_peer_input() + P * self.wl.wire_bytes_per_elem + state * P

    def bytes_encode_local(self) -> float:
        return self.wl.P * (4.0 + self.wl.wire_bytes_per_elem)

    def bytes_step(self) -> float:
        """Compulsory bytes of one step: the local peer's encode and the
        round.  With the encode inside the averaging pass, the local message
        is written but not read back."""
        b = self.bytes_round() + self.bytes_encode_local()
        return b - self.wl.P * self.wl.wire_bytes_per_elem if self.local_in_kernel else b

    @property
    def local_in_kernel(self) -> bool:
        """The local peer's encode runs inside the averaging pass (the fp16
        round; the int8 round encodes it in a launch of its own)."""
        return self.fused_local and self.codec == D.DEDLOC_CODEC_FP16
