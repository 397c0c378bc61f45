"""GPU parity of the round with the local peer's encode fused in
(dedloc_local_peer).

Every peer encodes its own gradient before the exchange; the round can take
the local peer's fp32 gradient instead and write that peer's message itself
in the pass that averages it.  The contract: every output, the local
message included, is bit-identical to an encode followed by the round.
Checked against the oracle (its encode, then its round) on small tables with
the local peer first, in the middle and last among the peers with samples,
for both codecs and both optimizers, with more than 64 peers (the local
peer in an earlier launch of the chain and in the last), and at full size
against the library's own separate-encode path in the benchmark's launch
configuration."""

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import harness as H
from paper_2106_10207_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
FP16, I8 = D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8


def _up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


SIZES = [4096 * 3, 128, 128, 2048 + 8, 1024, 5]
KINDS = ["w", "g", "b", "w", "b", "b"]


def _case(codec, n_peers, n_zero=2):
    base = W.ALBERT_LARGE if codec == FP16 else W.ALBERT_XLARGE
    wl = W.scaled(base, f"{base.name}_local_{n_peers}", SIZES, KINDS, n_peers=n_peers, n_zero_peers=n_zero)
    counts = W.sample_counts(wl)
    grads = [W.peer_gradient(wl, p).numpy() for p in range(n_peers)]
    if codec == FP16:
        codes, scales = [oracle.encode_fp16(g) for g in grads], None
    else:
        enc = [oracle.encode_i8(g, 1024) for g in grads]
        codes, scales = [c for c, _ in enc], [s for _, s in enc]
    return wl, counts, grads, codes, scales


def _device(codec, counts, codes, scales, local):
    dc = [_up(c.view(np.int16) if codec == FP16 else c) for c in codes]
    ds = None if scales is None else [_up(s) for s in scales]
    for p in range(len(counts)):
        if counts[p] == 0 or p == local:  # unread, or written by the round
            W.nan_poison(dc[p])
            if ds is not None:
                W.nan_poison(ds[p])
    return dc, ds


def _check_local_msg(codec, dc, ds, codes, scales, local):
    if codec == FP16:
        assert np.array_equal(_np(dc[local]).view(np.uint16), codes[local])
    else:
        assert np.array_equal(_np(dc[local]).view(np.int8), codes[local])
        assert np.array_equal(_bits(_np(ds[local])), _bits(scales[local]))


def _run(wl, counts, grads, codes, scales, local, optimizer):
    codec = H.codec_id(wl)
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, m, v = (t.numpy() for t in W.optimizer_state(wl))
    dc, ds = _device(codec, counts, codes, scales, local)
    xd, md, vd = _up(x), _up(m), _up(v)
    ws = D.make_workspace(wl.P, wl.offsets(), DEV)
    mean = torch.empty(wl.P, dtype=torch.float32, device=DEV)
    tr = torch.empty(wl.n_tensors, dtype=torch.float32, device=DEV)
    g_local = _up(grads[local])
    if optimizer == "lamb":
        cfg = dict(lr=wl.lr, beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, weight_decay=wl.weight_decay,
                   step=wl.step)
        r = oracle.round_(codes, counts, bounds, codec, x, m, v, wl.offsets(), wl.flags(),
                          oracle.lamb_cfg(**cfg), scales, 1024)
        oc, osc = D.dedloc_round(dc, counts, bounds, codec, xd, md, vd, wl.offsets(), wl.flags(),
                                 D.lamb_cfg(**cfg), peer_scales=ds, trust_out=tr, out_mean=mean, ws=ws,
                                 local=(local, g_local))
        assert np.array_equal(_bits(_np(md)), _bits(r["m"]))
        assert np.array_equal(_bits(_np(vd)), _bits(r["v"]))
    else:
        cfg = dict(lr=wl.lars_lr, momentum=wl.lars_momentum, trust_coef=wl.lars_trust_coef,
                   weight_decay=wl.lars_weight_decay)
        r = oracle.round_lars(codes, counts, bounds, codec, x, m, wl.offsets(), wl.flags(),
                              oracle.lars_cfg(**cfg), scales, 1024)
        oc, osc = D.dedloc_round_lars(dc, counts, bounds, codec, xd, md, wl.offsets(), wl.flags(),
                                      D.lars_cfg(**cfg), peer_scales=ds, trust_out=tr, out_mean=mean, ws=ws,
                                      local=(local, g_local))
    _check_local_msg(codec, dc, ds, codes, scales, local)
    assert np.array_equal(_bits(_np(mean)), _bits(r["mean"]))
    if codec == FP16:
        assert np.array_equal(_np(oc).view(np.uint16), r["codes"])
    else:
        assert np.array_equal(_np(oc).view(np.int8), r["codes"])
        assert np.array_equal(_bits(_np(osc)), _bits(r["scales"]))
    assert np.allclose(_np(tr), r["trust"], rtol=1e-6, atol=0)
    tol = 1e-5 * float(np.max(np.abs(x)))
    assert np.max(np.abs(_np(xd).astype(np.float64) - r["x"])) <= tol


def _local_at(counts, where):
    act = np.flatnonzero(counts)
    return int({"first": act[0], "middle": act[len(act) // 2], "last": act[-1]}[where])


@pytest.mark.parametrize("optimizer", ["lamb", "lars"])
@pytest.mark.parametrize("where", ["first", "middle", "last"])
@pytest.mark.parametrize("codec,n_peers", [(FP16, 16), (I8, 12)])
def test_round_local_matches_oracle(codec, n_peers, where, optimizer):
    wl, counts, grads, codes, scales = _case(codec, n_peers)
    _run(wl, counts, grads, codes, scales, _local_at(counts, where), optimizer)


@pytest.mark.parametrize("where", ["first", "last"])
@pytest.mark.parametrize("codec,n_peers", [(FP16, 100), (I8, 130)])
def test_round_local_chained(codec, n_peers, where):
    # first: the local peer is averaged by an earlier launch of the chain;
    # last: by the final one (the fused optimizer pass for fp16)
    wl, counts, grads, codes, scales = _case(codec, n_peers, n_zero=5)
    _run(wl, counts, grads, codes, scales, _local_at(counts, where), "lamb")


@pytest.mark.parametrize("name", ["albert_large", "albert_xlarge"])
def test_full_size_fused_equals_separate(name):
    """The benchmark's configuration: the fused round and encode + round
    from the same state give the same bits everywhere."""
    wl = W.WORKLOADS[name]
    outs = []
    for fused in (False, True):
        dr = H.DeviceRound(wl, DEV, keep_local_grad=True, fused_local=fused, with_mean=True)
        W.nan_poison(dr.codes[dr.local])
        if dr.scales[dr.local] is not None:
            W.nan_poison(dr.scales[dr.local])
        if not fused:
            dr.encode_local()
        dr.run()
        ts = [dr.codes[dr.local], dr.out_codes, dr.mean, dr.x, dr.m, dr.v, dr.trust]
        if dr.codec == I8:
            ts += [dr.scales[dr.local], dr.out_scales]
        outs.append([_np(t).view(np.uint8).copy() for t in ts])
        del dr
        torch.cuda.empty_cache()
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
