"""Seeded synthetic workloads for the collaborative averaging round.

This module only describes shapes and draws random numbers: tensor tables,
peer sample counts, peer bandwidths, per-peer mean gradients and optimizer
state.  It holds none of the method's arithmetic (no weighting, no codec, no
optimizer), so both the GPU library's callers and the CPU checker can take
their inputs from it.

The shapes follow the paper's workloads:
  * ALBERT-large / ALBERT-xlarge parameter tables (Section 4.2 trains
    ALBERT-large; the appendix on sahajBERT-XL describes an ALBERT-xlarge-sized
    model with d_model 2048).
  * ResNet-50 (Section 4.1 trains SwAV with a ResNet-50 backbone).
The datasets behind those runs are not needed: only the parameter shapes
matter for the averaging round, and every value here is synthetic.

Gradient values are per-peer *mean* gradients (the global gradient is the
sample-weighted mean of the peers' means; appendix "Convergence analysis").
"""

from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Per-tensor flags handed to the LAMB step: bit 0 = apply weight decay,
# bit 1 = apply the layer-wise trust ratio.
FLAG_DECAY = 1
FLAG_ADAPT = 2

# kinds: 'w' weight matrix / conv kernel, 'g' normalisation gain, 'b' bias or
# normalisation shift, 'd' a tensor with weight decay but no trust ratio
# (its update is elementwise: r = 1).
_KIND_FLAGS = {"w": FLAG_DECAY | FLAG_ADAPT, "g": FLAG_ADAPT, "b": FLAG_ADAPT, "d": FLAG_DECAY}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cid: int                      # seed namespace: seeds are 1000*cid + k
    tensors: Tuple[Tuple[str, int, str], ...]   # (name, numel, kind)
    n_peers: int
    codec: str                    # "fp16" or "i8"
    sigma: float                  # std-dev of each peer's mean gradient
    count_range: Tuple[int, int]  # inclusive uniform range of sample counts
    n_zero_peers: int = 0         # peers forced to zero samples (weight 0)
    outlier_p: float = 0.0        # per-element probability of a heavy tail
    outlier_scale: float = 1.0
    bandwidth_range: Optional[Tuple[int, int]] = None  # Mbit/s, None = equal
    single_shard: bool = False
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-6
    weight_decay: float = 0.01
    step: int = 10
    # LARS (the SwAV runs' optimizer): lr, momentum, trust coefficient, decay
    lars_lr: float = 4.8
    lars_momentum: float = 0.9
    lars_trust_coef: float = 1e-3
    lars_weight_decay: float = 1e-6

    @property
    def P(self) -> int:
        return int(sum(t[1] for t in self.tensors))

    @property
    def n_tensors(self) -> int:
        return len(self.tensors)

    @property
    def block(self) -> int:
        return 1024 if self.codec == "i8" else 1

    @property
    def shard_align(self) -> int:
        # fp16 shards start on 64-element (128 B) rows; int8 shards on codec
        # blocks so that a block never straddles two reducers.
        return 1024 if self.codec == "i8" else 64

    @property
    def n_shards(self) -> int:
        return 1 if self.single_shard else self.n_peers

    @property
    def wire_bytes_per_elem(self) -> float:
        return 2.0 if self.codec == "fp16" else 1.0 + 4.0 / 1024.0

    def offsets(self) -> np.ndarray:
        off = np.zeros(self.n_tensors + 1, dtype=np.uint64)
        off[1:] = np.cumsum([t[1] for t in self.tensors], dtype=np.uint64)
        return off

    def flags(self) -> np.ndarray:
        return np.array([_KIND_FLAGS[t[2]] for t in self.tensors], dtype=np.uint8)


def _albert(H: int, F: int, V: int = 30000, E: int = 128, S: int = 512):
    t = [("word_emb", V * E, "w"), ("pos_emb", S * E, "w"),
         ("type_emb", 2 * E, "w"), ("emb_ln_g", E, "g"), ("emb_ln_b", E, "b"),
         ("emb_proj_w", E * H, "w"), ("emb_proj_b", H, "b")]
    for n in "qkvo":
        t += [(f"attn_{n}_w", H * H, "w"), (f"attn_{n}_b", H, "b")]
    t += [("attn_ln_g", H, "g"), ("attn_ln_b", H, "b"),
          ("ffn_in_w", H * F, "w"), ("ffn_in_b", F, "b"),
          ("ffn_out_w", F * H, "w"), ("ffn_out_b", H, "b"),
          ("ffn_ln_g", H, "g"), ("ffn_ln_b", H, "b"),
          ("pool_w", H * H, "w"), ("pool_b", H, "b")]
    return tuple(t)


def _resnet50():
    t = [("conv1", 7 * 7 * 3 * 64, "w"), ("bn1_g", 64, "g"), ("bn1_b", 64, "b")]
    cin = 64
    for si, (nblocks, w) in enumerate(zip([3, 4, 6, 3], [64, 128, 256, 512])):
        for bi in range(nblocks):
            p = f"l{si + 1}.{bi}"
            t += [(p + ".conv1", cin * w, "w"), (p + ".bn1_g", w, "g"), (p + ".bn1_b", w, "b"),
                  (p + ".conv2", 9 * w * w, "w"), (p + ".bn2_g", w, "g"), (p + ".bn2_b", w, "b"),
                  (p + ".conv3", w * 4 * w, "w"), (p + ".bn3_g", 4 * w, "g"), (p + ".bn3_b", 4 * w, "b")]
            if bi == 0:
                t += [(p + ".down", cin * 4 * w, "w"), (p + ".down_bn_g", 4 * w, "g"),
                      (p + ".down_bn_b", 4 * w, "b")]
            cin = 4 * w
    t += [("fc_w", 2048 * 1000, "w"), ("fc_b", 1000, "b")]
    return tuple(t)


TINY = Workload("tiny", 0, tuple((f"t{i}", 131072, "w") for i in range(8)),
                n_peers=4, codec="fp16", sigma=1e-3, count_range=(16, 64))
ALBERT_LARGE = Workload("albert_large", 1, _albert(1024, 4096), n_peers=16,
                        codec="fp16", sigma=1e-3, count_range=(8, 256),
                        outlier_p=0.01, outlier_scale=100.0)
RESNET50 = Workload("resnet50", 2, _resnet50(), n_peers=32, codec="fp16",
                    sigma=1e-3, count_range=(8, 256), bandwidth_range=(10, 1000))
ALBERT_XLARGE = Workload("albert_xlarge", 3, _albert(2048, 8192), n_peers=64,
                         codec="i8", sigma=1e-3, count_range=(1, 512),
                         n_zero_peers=4)
STRESS = Workload("stress", 4, tuple((f"s{i}", 1 << 20, "w") for i in range(1024)),
                  n_peers=8, codec="fp16", sigma=1e-2, count_range=(16, 64),
                  single_shard=True)

WORKLOADS = {w.name: w for w in (TINY, ALBERT_LARGE, RESNET50, ALBERT_XLARGE, STRESS)}


def scaled(wl: Workload, name: str, tensor_sizes: Sequence[int],
           kinds: Optional[Sequence[str]] = None, **over) -> Workload:
    """A copy of `wl` with another tensor table (for small parity cases)."""
    kinds = kinds or ["w"] * len(tensor_sizes)
    t = tuple((f"t{i}", int(n), k) for i, (n, k) in enumerate(zip(tensor_sizes, kinds)))
    return dataclasses.replace(wl, name=name, tensors=t, **over)


def _rng(wl: Workload, k: int) -> np.random.Generator:
    return np.random.default_rng(1000 * wl.cid + k)


def sample_counts(wl: Workload) -> np.ndarray:
    """Accumulated sample count of every peer (uint32); some may be zero."""
    r = _rng(wl, 900)
    lo, hi = wl.count_range
    c = r.integers(lo, hi + 1, size=wl.n_peers).astype(np.uint32)
    if wl.n_zero_peers:
        z = r.choice(wl.n_peers, size=wl.n_zero_peers, replace=False)
        c[z] = 0
    return c


def bandwidth_weights(wl: Workload) -> Optional[np.ndarray]:
    """Integer peer bandwidths (Mbit/s) that set shard sizes, or None (equal)."""
    if wl.bandwidth_range is None or wl.single_shard:
        return None
    lo, hi = wl.bandwidth_range
    return _rng(wl, 901).integers(lo, hi + 1, size=wl.n_shards).astype(np.uint64)


def _torch_gen(seed: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def peer_gradient(wl: Workload, p: int, device="cpu"):
    """Peer p's mean gradient over the whole flat vector, fp32 torch tensor.

    N(0, sigma^2) per element; with outlier_p > 0 each element is, with that
    probability, multiplied by outlier_scale (a heavy tail)."""
    import torch
    g = _torch_gen(1000 * wl.cid + p, device)
    x = torch.randn(wl.P, generator=g, device=device, dtype=torch.float32)
    x.mul_(wl.sigma)
    if wl.outlier_p > 0:
        mask = torch.rand(wl.P, generator=g, device=device) < wl.outlier_p
        x[mask] *= wl.outlier_scale
    return x


def optimizer_state(wl: Workload, device="cpu", fresh: bool = False):
    """(x, m, v) flat fp32 tensors.

    x: N(0, 0.02^2) for weight tensors, 1 for gains, 0 for biases.
    m: N(0, (1e-4)^2); v: square of N(0, (1e-3)^2).  fresh=True gives m = v = 0
    (the state before the first step)."""
    import torch
    g = _torch_gen(1000 * wl.cid + 950, device)
    P = wl.P
    x = torch.empty(P, device=device, dtype=torch.float32)
    off = wl.offsets()
    for i, (_, n, kind) in enumerate(wl.tensors):
        sl = x[int(off[i]):int(off[i + 1])]
        if kind == "w":
            sl.copy_(torch.randn(n, generator=g, device=device) * 0.02)
        elif kind == "g":
            sl.fill_(1.0)
        else:
            sl.zero_()
    if fresh:
        m = torch.zeros(P, device=device)
        v = torch.zeros(P, device=device)
    else:
        m = torch.randn(P, generator=g, device=device) * 1e-4
        v = torch.randn(P, generator=g, device=device).mul_(1e-3).square_()
    return x, m, v


def nan_poison(t):
    """Fill a buffer with NaN bit patterns (for zero-sample peers that must
    never be read)."""
    import torch
    if t.dtype == torch.float32:
        t.fill_(float("nan"))
    elif t.dtype in (torch.float16, torch.int16, torch.uint16):
        t.view(torch.int16).fill_(0x7E00)
    else:
        t.view(torch.uint8).fill_(0xFF)
    return t
