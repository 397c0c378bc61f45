"""GPU parity of the LARS entry points (dedloc_lars_step, dedloc_round_lars)
against the CPU oracle, through the C ABI.

Bars: codes, scales and the fp32 average bit-identical; the rate ratio
within 1e-6 relative (fp64 norms summed in another order); v' and x' within
1e-5 of their scale (they follow from the ratio)."""

import zlib

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import harness as H
from paper_2106_10207_amd import workloads as W
from tests.test_gpu_parity import (DEV, SMALL, TABLES, _bits, _device_msgs, _i8, _np, _oracle_inputs,
                                   _sample, _superset, _u16, _up)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
F = np.float32


def _close(got, ref, scale_ref, rel=1e-5):
    scale = max(float(np.max(np.abs(scale_ref))) if np.size(scale_ref) else 0.0, 1e-30)
    err = float(np.max(np.abs(got.astype(np.float64) - ref.astype(np.float64)))) if np.size(got) else 0.0
    assert err <= rel * scale, (err, rel * scale)


@pytest.mark.parametrize("src", ["f32", "fp16", "i8"])
@pytest.mark.parametrize("table", list(TABLES))
@pytest.mark.parametrize("unit", [False, True])
def test_lars_step(src, table, unit):
    rng = np.random.default_rng(zlib.crc32(f"lars/{src}/{table}".encode()) % 1000)
    sizes = TABLES[table]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    flags = rng.integers(0, 4, len(sizes)).astype(np.uint8)
    flags[0] = 3
    x = (rng.standard_normal(P) * 0.02).astype(F)
    if len(sizes) > 2:
        x[int(off[1]):int(off[2])] = 0.0
    v = (rng.standard_normal(P) * 1e-3).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    cfg = dict(lr=4.8, momentum=0.9, trust_coef=1e-3, weight_decay=1e-4, force_unit_trust=unit)
    if src == "f32":
        ghat, gdev, gsc, codec = g, _up(g), None, D.DEDLOC_CODEC_F32
    elif src == "fp16":
        c = oracle.encode_fp16(g)
        ghat, gdev, gsc, codec = oracle.decode_fp16(c), _up(c.view(np.int16)), None, D.DEDLOC_CODEC_FP16
    else:
        c, s = oracle.encode_i8(g, 1024)
        ghat, gdev, gsc, codec = oracle.decode_i8(c, s, 1024), _up(c), _up(s), D.DEDLOC_CODEC_I8
    xo, vo, to = oracle.lars(x, v, ghat, off, flags, oracle.lars_cfg(**cfg))
    xd, vd = _up(x), _up(v)
    tr = torch.full((len(flags),), -1.0, device=DEV)
    D.dedloc_lars_step(xd, vd, gdev, off, flags, D.lars_cfg(**cfg), grad_codec=codec, grad_scales=gsc,
                       trust_out=tr)
    assert np.allclose(_np(tr), to, rtol=1e-6, atol=0)
    _close(_np(vd), vo, vo)
    _close(_np(xd) - x, xo - x, xo - x)


@pytest.mark.parametrize("wl", [SMALL[2], SMALL[3]], ids=lambda w: w.name)
def test_round_lars_small_three_steps(wl):
    counts, codes, scales = _oracle_inputs(wl)
    codec = H.codec_id(wl)
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, _, _ = (t.numpy() for t in W.optimizer_state(wl, fresh=True))
    v = np.zeros(wl.P, F)
    dc, ds = _device_msgs(wl, codes, scales, counts)
    xd, vd = _up(x), _up(v)
    ws = D.make_workspace(wl.P, wl.offsets(), DEV)
    mean = torch.empty(wl.P, dtype=torch.float32, device=DEV)
    tr = torch.empty(wl.n_tensors, dtype=torch.float32, device=DEV)
    cfg = dict(lr=wl.lars_lr, momentum=wl.lars_momentum, trust_coef=wl.lars_trust_coef,
               weight_decay=wl.lars_weight_decay)
    for step in (1, 2, 3):
        r = oracle.round_lars(codes, counts, bounds, codec, x, v, wl.offsets(), wl.flags(),
                              oracle.lars_cfg(**cfg), scales, 1024)
        oc, osc = D.dedloc_round_lars(dc, counts, bounds, codec, xd, vd, wl.offsets(), wl.flags(),
                                      D.lars_cfg(**cfg), peer_scales=ds if scales else None,
                                      trust_out=tr, out_mean=mean, ws=ws)
        assert np.array_equal(_bits(_np(mean)), _bits(r["mean"])), step
        if codec == D.DEDLOC_CODEC_FP16:
            assert np.array_equal(_u16(oc), r["codes"]), step
        else:
            assert np.array_equal(_i8(oc), r["codes"]), step
            assert np.array_equal(_bits(_np(osc)), _bits(r["scales"])), step
        assert np.allclose(_np(tr), r["trust"], rtol=1e-6, atol=0), step
        _close(_np(vd), r["v"], r["v"])
        _close(_np(xd) - x, r["x"] - x, r["x"] - x)
        x, v = r["x"], r["v"]


@pytest.mark.parametrize("name", ["resnet50", "albert_xlarge"])
def test_round_lars_full_size_sampled(name):
    """The LARS round at full size in the benchmark's launch configuration,
    whole sampled tensors checked against the oracle."""
    wl = W.WORKLOADS[name]
    codec = H.codec_id(wl)
    tensors, _ = _sample(wl, n_blocks=0)
    off = wl.offsets()
    ranges = [_superset(int(off[t]), int(off[t + 1]), wl.P, codec) for t in tensors]
    print(f"\n[{name} lars] tensors={tensors}", flush=True)
    dr = H.DeviceRound(wl, DEV, sample_ranges=ranges, optimizer="lars")
    x0 = [dr.x[A:B].cpu().numpy() for A, B in ranges]
    v0 = [dr.v[A:B].cpu().numpy() for A, B in ranges]
    dr.run()
    torch.cuda.synchronize()
    cfg = oracle.lars_cfg(wl.lars_lr, wl.lars_momentum, wl.lars_trust_coef, wl.lars_weight_decay)
    trust = _np(dr.trust)
    for i, (A, B) in enumerate(ranges):
        g = [dr.host_grads[p][i] for p in range(wl.n_peers)]
        if codec == D.DEDLOC_CODEC_FP16:
            codes, scales = [oracle.encode_fp16(q) for q in g], None
        else:
            enc = [oracle.encode_i8(q, 1024) for q in g]
            codes, scales = [c for c, _ in enc], [s for _, s in enc]
        t = tensors[i]
        a, b = int(off[t]), int(off[t + 1])
        sub_off = np.array([0, a - A, b - A, B - A], np.uint64)
        sub_fl = np.array([0, wl.flags()[t], 0], np.uint8)
        r = oracle.round_lars(codes, dr.counts, np.array([0, B - A], np.uint64), codec, x0[i], v0[i],
                              sub_off, sub_fl, cfg, scales, 1024)
        s = slice(a - A, b - A)
        assert np.isclose(trust[t], r["trust"][1], rtol=1e-6, atol=0), (name, t)
        _close(_np(dr.v[a:b]), r["v"][s], r["v"][s])
        _close(_np(dr.x[a:b]) - x0[i][s], r["x"][s] - x0[i][s], r["x"][s] - x0[i][s])
    del dr
    torch.cuda.empty_cache()
