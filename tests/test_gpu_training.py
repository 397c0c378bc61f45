"""Many rounds in a row: the library as the optimizer of a small training
run, against the oracle running the same run (GPU, through the C ABI).

Eight peers (one without samples) minimise a separable quadratic
f(x) = 1/2 sum a_e (x_e - x*_e)^2 over a four-tensor parameter vector.  Each
step every peer computes its gradient a (x - x*) plus seeded noise, encodes
it for the wire (fp16 or int8), and the round averages the messages and
applies LAMB (bias correction follows the step count) or LARS.  The oracle
runs the same loop on the host from the same initial state and noise.

Checks: the loss falls well below its start (the round is a working
optimizer, not only a match of one step), and the two trajectories agree:
every step's loss within 1e-4 relative and the final parameters within
1e-4 of their scale.  Bit-identity is not expected after the first step: x'
is held to 1e-5 of its scale per step (the trust ratio's fp64 sums are added
in another order), so later gradients may differ in their last bits."""

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
F = np.float32


def _loss(a, x, xs):
    return 0.5 * float(np.sum(a.astype(np.float64) * (x.astype(np.float64) - xs) ** 2))


@pytest.mark.parametrize("codec", [D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8])
@pytest.mark.parametrize("opt", ["lamb", "lars"])
def test_training_run_matches_oracle(codec, opt):
    print(f"\n[training] codec={codec} opt={opt}", flush=True)
    rng = np.random.default_rng(3 + codec)
    sizes = [4096, 8000, 512, 24005]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    flags = np.array([3, 3, 2, 3], np.uint8)
    a = rng.uniform(0.5, 2.0, P).astype(F)
    xs = (rng.standard_normal(P) * 0.5).astype(F)
    x0 = (rng.standard_normal(P) * 0.5).astype(F)
    counts = np.array([5, 9, 0, 3, 12, 7, 1, 4], np.uint32)
    n = len(counts)
    align = 64 if codec == D.DEDLOC_CODEC_FP16 else 1024
    bounds = oracle.partition(P, 4, None, align)
    steps = 40

    xo, mo, vo = x0.copy(), np.zeros(P, F), np.zeros(P, F)
    xd = torch.from_numpy(x0.copy()).to(DEV)
    md, vd = torch.zeros(P, device=DEV), torch.zeros(P, device=DEV)
    ad, xsd = torch.from_numpy(a).to(DEV), torch.from_numpy(xs).to(DEV)
    ws = D.make_workspace(P, off, DEV)
    L0 = _loss(a, x0, xs)
    lo, ld = [], []
    for step in range(1, steps + 1):
        noise = (rng.standard_normal((n, P)) * 0.01).astype(F)
        # oracle side
        go = [(a * (xo - xs) + noise[p]).astype(F) for p in range(n)]
        if codec == D.DEDLOC_CODEC_FP16:
            oc, osc = [oracle.encode_fp16(g) for g in go], None
        else:
            enc = [oracle.encode_i8(g, 1024) for g in go]
            oc, osc = [e[0] for e in enc], [e[1] for e in enc]
        # library side: gradients, encodes and the round on the device
        nd = torch.from_numpy(noise).to(DEV)
        msgs = [D.dedloc_encode(ad * (xd - xsd) + nd[p], codec) for p in range(n)]
        dc = [c for c, _ in msgs]
        ds = None if codec == D.DEDLOC_CODEC_FP16 else [s for _, s in msgs]
        if opt == "lamb":
            cfg = dict(lr=0.05, weight_decay=0.0, step=step)
            r = oracle.round_(oc, counts, bounds, codec, xo, mo, vo, off, flags, oracle.lamb_cfg(**cfg), osc, 1024)
            xo, mo, vo = r["x"], r["m"], r["v"]
            D.dedloc_round(dc, counts, bounds, codec, xd, md, vd, off, flags, D.lamb_cfg(**cfg),
                           peer_scales=ds, ws=ws)
        else:
            cfg = dict(lr=0.5, momentum=0.9, trust_coef=0.02, weight_decay=0.0)
            r = oracle.round_lars(oc, counts, bounds, codec, xo, vo, off, flags, oracle.lars_cfg(**cfg), osc, 1024)
            xo, vo = r["x"], r["v"]
            D.dedloc_round_lars(dc, counts, bounds, codec, xd, vd, off, flags, D.lars_cfg(**cfg),
                                peer_scales=ds, ws=ws)
        torch.cuda.synchronize()
        lo.append(_loss(a, xo, xs))
        ld.append(_loss(a, xd.cpu().numpy(), xs))
    print(f"loss / start: oracle {lo[-1] / L0:.4f}, library {ld[-1] / L0:.4f}", flush=True)
    assert ld[-1] < 0.1 * L0 and lo[-1] < 0.1 * L0
    assert np.allclose(ld, lo, rtol=1e-4, atol=0), max(abs(p - q) / q for p, q in zip(ld, lo))
    xg = xd.cpu().numpy()
    assert float(np.max(np.abs(xg.astype(np.float64) - xo))) <= 1e-4 * float(np.max(np.abs(xo)))
