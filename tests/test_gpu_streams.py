"""Stream behaviour of the C ABI on the GPU.

* Delayed parameter updates (Section 3.2) run the next round's local
  accumulation beside the current round: both enqueued on two streams at
  once, each result still equals the oracle.
* A round captured into a HIP graph and replayed several times, with eager
  work and synchronisation between replays, gives the eager result every
  time (the library records only kernel launches), also when the replays
  are consecutive steps whose trust ratios differ."""

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import harness as H
from paper_2106_10207_amd import workloads as W
from tests.test_gpu_parity import DEV, SMALL, _bits, _np, _u16, _up

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def test_round_beside_accumulation_on_two_streams():
    wl = SMALL[1]
    dr = H.DeviceRound(wl, DEV, sample_ranges=[(0, wl.P)])
    x0, m0, v0 = (t.cpu().numpy() for t in (dr.x, dr.m, dr.v))
    rng = np.random.default_rng(5)
    acc_h = np.zeros(wl.P, np.float32)
    grads = [(rng.standard_normal(wl.P) * 1e-3).astype(np.float32) for _ in range(6)]
    acc = torch.zeros(wl.P, device=DEV)
    gdev = [_up(g) for g in grads]
    s_round, s_acc = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s_round):
        dr.call(stream=s_round)
    with torch.cuda.stream(s_acc):
        for b, g in enumerate(gdev):
            D.dedloc_accumulate(acc, g, float(b + 1), stream=s_acc)
    torch.cuda.synchronize()
    for b, g in enumerate(grads):
        acc_h = oracle.accumulate(acc_h, g, float(b + 1))
    assert np.array_equal(_bits(_np(acc)), _bits(acc_h))
    codes = [oracle.encode_fp16(dr.host_grads[p][0]) for p in range(wl.n_peers)]
    cfg = oracle.lamb_cfg(wl.lr, wl.beta1, wl.beta2, wl.eps, wl.weight_decay, step=dr.step)
    r = oracle.round_(codes, dr.counts, dr.bounds, oracle.CODEC_FP16, x0, m0, v0, wl.offsets(), wl.flags(), cfg)
    assert np.array_equal(_u16(dr.out_codes), r["codes"])
    assert np.array_equal(_bits(_np(dr.m)), _bits(r["m"]))


@pytest.mark.parametrize("idx", [0, 3])
def test_round_in_graph_replays(idx):
    wl = SMALL[idx]
    dr = H.DeviceRound(wl, DEV)
    state0 = [t.clone() for t in (dr.x, dr.m, dr.v)]

    def reset():
        for t, t0 in zip((dr.x, dr.m, dr.v), state0):
            t.copy_(t0)

    # eager reference
    reset()
    dr.run()
    ref = [_np(t).copy() for t in (dr.out_codes, dr.x, dr.m, dr.v, dr.trust)]
    # capture on a side stream, then replay three times
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        dr.call(stream=s)
    for _ in range(3):
        reset()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [_np(t).copy() for t in (dr.out_codes, dr.x, dr.m, dr.v, dr.trust)]
        for a, b in zip(got, ref):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
        _ = torch.ones(1024, device=DEV).sum().item()  # eager work between replays


@pytest.mark.parametrize("idx", [0, 3])
def test_round_in_graph_consecutive_steps(idx):
    """Replays of a captured round as consecutive optimizer steps (the state
    evolves, so every replay has other trust ratios): every replay equals
    the eager round run on the same state, bit for bit.  Each replay's
    ratios carry a tag of their own although the captured kernel arguments
    are the same."""
    print(f"\n[graph steps] {SMALL[idx].name}", flush=True)
    dr = H.DeviceRound(SMALL[idx], DEV)
    state0 = [t.clone() for t in (dr.x, dr.m, dr.v)]

    def reset():
        for t, t0 in zip((dr.x, dr.m, dr.v), state0):
            t.copy_(t0)

    def outs():
        return [_np(t).copy() for t in (dr.out_codes, dr.x, dr.m, dr.v, dr.trust)]

    reset()
    ref = []
    for _ in range(4):
        dr.run()
        ref.append(outs())
    assert not np.array_equal(ref[0][4], ref[1][4])  # the ratios change from step to step
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        dr.call(stream=s)
    reset()
    torch.cuda.synchronize()
    for step in range(4):
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), ref[step]):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), step
        _ = torch.ones(1024, device=DEV).sum().item()  # eager work between replays
