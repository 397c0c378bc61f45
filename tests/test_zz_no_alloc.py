"""The round without a workspace (dedloc_round_noalloc, for callers that
cannot allocate device memory) against dedloc_round on the same inputs,
through the C ABI: two calls in a row on the library's one static array, the
second over a smaller vector, each compared bit for bit (both run the same
kernels in the same order, so every output is identical: codes, scales, the
fp32 average, m', v', x' and the trust ratios)."""

import numpy as np
import pytest

from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import harness as H
from paper_2106_10207_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _bits(t):
    torch.cuda.synchronize()
    a = t.cpu().numpy()
    return a.view(np.uint8)


def _case(wl, local):
    """Both entry points on copies of one set of inputs; returns the two sets
    of outputs."""
    dr = H.DeviceRound(wl, DEV, with_mean=True, keep_local_grad=True)
    x0, m0, v0 = dr.x.clone(), dr.m.clone(), dr.v.clone()
    msg0 = dr.codes[dr.local].clone()
    loc = (dr.local, dr.local_grad) if local else None
    kw = dict(peer_scales=dr.scales if dr.codec == D.DEDLOC_CODEC_I8 else None, block=D.DEDLOC_I8_BLOCK)
    outs = []
    for noalloc in (False, True):
        dr.x.copy_(x0)
        dr.m.copy_(m0)
        dr.v.copy_(v0)
        dr.codes[dr.local].copy_(msg0)
        oc = torch.full_like(dr.out_codes, 0x55)
        osc = None if dr.out_scales is None else torch.full_like(dr.out_scales, 7.0)
        tr = torch.full((wl.n_tensors,), -1.0, device=DEV)
        mean = torch.full((wl.P,), 3.0, device=DEV)
        args = (dr.codes, dr.counts, dr.bounds, dr.codec, dr.x, dr.m, dr.v, dr.offsets, dr.flags, dr.cfg)
        if noalloc:
            D.dedloc_round_noalloc(*args, out_codes=oc, out_scales=osc, trust_out=tr, out_mean=mean,
                                   local=loc, **kw)
        else:
            D.dedloc_round(*args, out_codes=oc, out_scales=osc, trust_out=tr, out_mean=mean,
                           ws=dr.ws, local=loc, **kw)
        got = [oc, mean, dr.x, dr.m, dr.v, tr, dr.codes[dr.local]] + ([osc] if osc is not None else [])
        outs.append([_bits(t).copy() for t in got])
    return outs


def test_noalloc_matches_round_twice_smaller_second():
    first = W.scaled(W.ALBERT_LARGE, "noalloc_first", [30000 * 16, 4096, 1024 * 1024, 1024, 777 * 8 + 3 * 8],
                     ["w", "g", "w", "b", "w"], n_peers=16)
    second = W.scaled(W.ALBERT_XLARGE, "noalloc_second", [8192, 128, 10000, 2048, 7],
                      ["w", "g", "w", "b", "b"], n_peers=12, n_zero_peers=2)
    assert second.P < first.P
    for wl, local in ((first, True), (second, False)):
        print(f"\n[no-alloc] {wl.name}: P={wl.P} peers={wl.n_peers} codec={wl.codec} local={local}", flush=True)
        ref, got = _case(wl, local)
        names = ["out_codes", "out_mean", "x", "m", "v", "trust", "local message", "out_scales"]
        for name, a, b in zip(names, ref, got):
            assert np.array_equal(a, b), (wl.name, name)
