"""GPU parity for collaborations larger than one launch's peer table.

Up to 64 peers with samples are averaged in one launch; more are averaged in
launches of 64 that carry the fp32 running sum through the caller's out_mean
buffer.  The sum is stored exactly between launches and each launch continues
the same per-peer fused multiply-add chain, so the codes, scales and average
must be bit-identical to the oracle's single pass over all peers.  The
volunteer run had 40 participants (Section 4.3) and the discussion of node
failures (Section 3.2) speaks of several hundred, so these cases cover the
boundary at 64 and go up to 1024 peers."""

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
F = np.float32
FP16, I8 = D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8


def _up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def _messages(codec, counts, length, seed):
    """Oracle-encoded messages of every peer and their device copies (the
    copies of zero-sample peers NaN-poisoned: they must never be read)."""
    rng = np.random.default_rng(seed)
    codes, scales, dc, ds = [], [], [], []
    for c in counts:
        g = (rng.standard_normal(length) * 1e-3).astype(F)
        g[rng.random(length) < 0.01] *= 100
        if codec == FP16:
            k, s = oracle.encode_fp16(g), None
        else:
            k, s = oracle.encode_i8(g, 1024)
        codes.append(k)
        scales.append(s)
        kd = _up(k.view(np.int16) if codec == FP16 else k)
        sd = None if s is None else _up(s)
        if c == 0:
            W.nan_poison(kd)
            if sd is not None:
                W.nan_poison(sd)
        dc.append(kd)
        ds.append(sd)
    return codes, (scales if codec == I8 else None), dc, (ds if codec == I8 else None)


def _counts(n, seed, zero_frac=0.1):
    rng = np.random.default_rng(seed)
    c = rng.integers(1, 300, n).astype(np.uint32)
    c[rng.random(n) < zero_frac] = 0
    c[0] = max(int(c[0]), 1)
    return c


@pytest.mark.parametrize("codec", [FP16, I8])
@pytest.mark.parametrize("n_peers,length", [(65, 5 * 2048 + 7), (100, 3 * 1024 + 100), (128, 2048 * 4),
                                            (129, 1024 * 3 + 1), (300, 20_000 + 3), (1024, 4096 + 9)])
def test_reduce_shard_chained(codec, n_peers, length):
    counts = _counts(n_peers, 7 * n_peers + codec, zero_frac=0.0 if n_peers == 65 else 0.1)
    codes, scales, dc, ds = _messages(codec, counts, length, n_peers + length)
    mean = torch.empty(length, dtype=torch.float32, device=DEV)
    oc, osc = D.dedloc_reduce_shard(dc, counts, length, codec, ds, out_mean=mean)
    rc, rs, rm = oracle.reduce(codes, counts, codec, scales, 1024)
    assert np.array_equal(_bits(_np(mean)), _bits(rm))
    if codec == FP16:
        assert np.array_equal(_np(oc).view(np.uint16), rc)
    else:
        assert np.array_equal(_np(oc).view(np.int8), rc)
        assert np.array_equal(_bits(_np(osc)), _bits(rs))


@pytest.mark.parametrize("codec", [FP16, I8])
def test_reduce_shard_65_peers_64_active_needs_no_mean(codec):
    # one peer without samples leaves 64 for a single launch
    counts = _counts(65, 11, zero_frac=0.0)
    counts[40] = 0
    length = 3 * 2048 + 5
    codes, scales, dc, ds = _messages(codec, counts, length, 12)
    oc, osc = D.dedloc_reduce_shard(dc, counts, length, codec, ds)
    rc, rs, _ = oracle.reduce(codes, counts, codec, scales, 1024)
    if codec == FP16:
        assert np.array_equal(_np(oc).view(np.uint16), rc)
    else:
        assert np.array_equal(_np(oc).view(np.int8), rc)
        assert np.array_equal(_bits(_np(osc)), _bits(rs))


def test_reduce_shard_chained_needs_mean():
    counts = _counts(70, 3, zero_frac=0.0)
    _, _, dc, _ = _messages(FP16, counts, 64, 4)
    with pytest.raises(D.DedlocError) as e:
        D.dedloc_reduce_shard(dc, counts, 64, FP16)
    assert e.value.code == D.DEDLOC_ERR_INVALID_ARG


SIZES = [3000 * 8, 128, 128, 4096, 1024, 5]
KINDS = ["w", "g", "b", "w", "b", "b"]


@pytest.mark.parametrize("codec,n_peers", [(FP16, 100), (FP16, 129), (I8, 100), (I8, 200)])
def test_round_chained_two_steps(codec, n_peers):
    base = W.ALBERT_LARGE if codec == FP16 else W.ALBERT_XLARGE
    wl = W.scaled(base, f"{base.name}_{n_peers}_peers", SIZES, KINDS, n_peers=n_peers, n_zero_peers=5)
    counts = W.sample_counts(wl)
    grads = [W.peer_gradient(wl, p).numpy() for p in range(n_peers)]
    if codec == FP16:
        codes, scales = [oracle.encode_fp16(g) for g in grads], None
    else:
        enc = [oracle.encode_i8(g, 1024) for g in grads]
        codes, scales = [c for c, _ in enc], [s for _, s in enc]
    dc = [_up(c.view(np.int16) if codec == FP16 else c) for c in codes]
    ds = None if scales is None else [_up(s) for s in scales]
    for p in np.flatnonzero(counts == 0):
        W.nan_poison(dc[p])
        if ds is not None:
            W.nan_poison(ds[p])
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, m, v = (t.numpy() for t in W.optimizer_state(wl, fresh=True))
    xd, md, vd = _up(x), _up(m), _up(v)
    ws = D.make_workspace(wl.P, wl.offsets(), DEV)
    mean = torch.empty(wl.P, dtype=torch.float32, device=DEV)
    tr = torch.empty(wl.n_tensors, dtype=torch.float32, device=DEV)
    for step in (1, 2):
        cfg = dict(lr=wl.lr, beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps,
                   weight_decay=wl.weight_decay, step=step)
        r = oracle.round_(codes, counts, bounds, codec, x, m, v, wl.offsets(), wl.flags(),
                          oracle.lamb_cfg(**cfg), scales, 1024)
        oc, osc = D.dedloc_round(dc, counts, bounds, codec, xd, md, vd, wl.offsets(), wl.flags(),
                                 D.lamb_cfg(**cfg), peer_scales=ds, trust_out=tr, out_mean=mean, ws=ws)
        assert np.array_equal(_bits(_np(mean)), _bits(r["mean"])), step
        if codec == FP16:
            assert np.array_equal(_np(oc).view(np.uint16), r["codes"]), step
        else:
            assert np.array_equal(_np(oc).view(np.int8), r["codes"]), step
            assert np.array_equal(_bits(_np(osc)), _bits(r["scales"])), step
        # each step starts from the oracle's state, so m' and v' are bit-identical
        assert np.array_equal(_bits(_np(md)), _bits(r["m"])), step
        assert np.array_equal(_bits(_np(vd)), _bits(r["v"])), step
        assert np.allclose(_np(tr), r["trust"], rtol=1e-6, atol=0), step
        tol = 1e-5 * float(np.max(np.abs(x)))
        assert np.max(np.abs(_np(xd).astype(np.float64) - r["x"])) <= tol, step
        x, m, v = r["x"], r["m"], r["v"]
        xd.copy_(_up(x))
        md.copy_(_up(m))
        vd.copy_(_up(v))


def test_round_lars_chained():
    wl = W.scaled(W.RESNET50, "resnet50_130_peers", SIZES, KINDS, n_peers=130, n_zero_peers=3)
    counts = W.sample_counts(wl)
    codes = [oracle.encode_fp16(W.peer_gradient(wl, p).numpy()) for p in range(wl.n_peers)]
    dc = [_up(c.view(np.int16)) for c in codes]
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, m, _ = (t.numpy() for t in W.optimizer_state(wl))
    cfg = dict(lr=wl.lars_lr, momentum=wl.lars_momentum, trust_coef=wl.lars_trust_coef,
               weight_decay=wl.lars_weight_decay)
    r = oracle.round_lars(codes, counts, bounds, FP16, x, m, wl.offsets(), wl.flags(), oracle.lars_cfg(**cfg))
    xd, vd = _up(x), _up(m)
    ws = D.make_workspace(wl.P, wl.offsets(), DEV)
    mean = torch.empty(wl.P, dtype=torch.float32, device=DEV)
    oc, _ = D.dedloc_round_lars(dc, counts, bounds, FP16, xd, vd, wl.offsets(), wl.flags(),
                                D.lars_cfg(**cfg), out_mean=mean, ws=ws)
    assert np.array_equal(_bits(_np(mean)), _bits(r["mean"]))
    assert np.array_equal(_np(oc).view(np.uint16), r["codes"])
    tol = 1e-5 * float(np.max(np.abs(x)))
    assert np.max(np.abs(_np(xd).astype(np.float64) - r["x"])) <= tol
