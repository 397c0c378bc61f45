"""GPU parity: every entry point of libdedloc against the CPU oracle on the
same seeded inputs, through the C ABI.

Bars (from the definitions in include/dedloc.h, which fix every rounding):
  * fp16 codes, int8 codes and scales, the fp32 average and the new moments
    m', v' must be bit-identical to the oracle;
  * x' within 1e-5 * max|x| (it also depends on the trust ratio, whose fp64
    norm sums are added in another order) and the trust ratio within 1e-6
    relative.
Sizes span several 2048-element tiles / 1024-element blocks and end in a
ragged tail; the full-size cases run the round in the configuration the
benchmark times and compare whole sampled tensors and sampled blocks."""

import zlib

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import harness as H
from paper_2106_10207_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
F = np.float32


def _up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _u16(t):
    return _np(t).view(np.uint16)


def _i8(t):
    return _np(t).view(np.int8)


def _bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def _assert_x(xg, xo, x0):
    tol = 1e-5 * max(float(np.max(np.abs(x0))), 1e-30)
    err = np.max(np.abs(xg.astype(np.float64) - xo.astype(np.float64))) if xg.size else 0.0
    assert err <= tol, (err, tol)


# ----------------------------------------------------------------- codecs

def _values(n, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(n) * 10.0 ** rng.uniform(-9, 4.9, n)).astype(F)
    special = np.array([0.0, -0.0, 65504, 65519.99, 65520, -65520, 1e30, 2.0 ** -24, 2.0 ** -25,
                        3 * 2.0 ** -26, 1e-40, np.inf, -np.inf], F)
    k = min(n, special.size)
    x[:k] = special[:k]
    return x


@pytest.mark.parametrize("n", [0, 1, 7, 8, 2047, 2048, 2049, 100003])
def test_encode_fp16(n):
    x = _values(n, n)
    codes, _ = D.dedloc_encode(_up(x), D.DEDLOC_CODEC_FP16)
    assert np.array_equal(_u16(codes), oracle.encode_fp16(x))


def test_encode_fp16_nan():
    """A NaN encodes to a NaN of the same sign (the payload is not part of
    the definition); the oracle's and the kernel's may differ in it."""
    x = np.array([np.nan, -np.nan, 1.0, np.float32(np.nan) * 0], F)
    x.view(np.uint32)[0] = 0x7fc01234  # a quiet NaN with a payload
    x.view(np.uint32)[3] = 0xff800001  # a signalling NaN
    g = _u16(D.dedloc_encode(_up(x), D.DEDLOC_CODEC_FP16)[0])
    o = oracle.encode_fp16(x)
    for i in (0, 1, 3):
        assert (g[i] & 0x7c00) == 0x7c00 and (g[i] & 0x3ff) != 0, hex(g[i])
        assert (g[i] & 0x8000) == (o[i] & 0x8000) and (o[i] & 0x7fff) > 0x7c00
    assert g[2] == o[2]


def _fp16_boundaries():
    """Every fp32 value at which binary16 rounding can go wrong: each finite
    fp16 value and its fp32 neighbours, each midpoint between consecutive
    fp16 values (a tie) and its fp32 neighbours, the overflow threshold
    65520 and its neighbours, both signs."""
    h = np.arange(0x7C00, dtype=np.uint16)
    v = h.view(np.float16).astype(F)
    mid = ((v[:-1].astype(np.float64) + v[1:].astype(np.float64)) / 2).astype(F)  # exact in fp32
    mid = np.concatenate([mid, [F(65520.0)]])
    base = np.concatenate([v, mid])
    up = np.nextafter(base, F(np.inf))
    dn = np.nextafter(base, F(-np.inf))
    pos = np.concatenate([base, up, dn])
    return np.concatenate([pos, -pos]).astype(F)


def test_encode_fp16_every_boundary():
    x = _fp16_boundaries()
    codes, _ = D.dedloc_encode(_up(x), D.DEDLOC_CODEC_FP16)
    assert np.array_equal(_u16(codes), oracle.encode_fp16(x))


def test_round_fp16_encodes_every_boundary():
    """The round's own fp16 encodes: the local peer's fp32 gradient (encoded
    inside the pass that averages it) holds every boundary value, and two
    peers of equal counts whose codes are consecutive fp16 values make every
    average an exact tie, which the re-encode must round to even."""
    x_all = _fp16_boundaries()
    x_all = x_all[np.abs(x_all) < 65504]  # keep the optimizer's state finite
    P = x_all.size
    h = np.arange(0x7BFF, dtype=np.uint16)
    lo = np.resize(np.concatenate([h, h | 0x8000]), P)
    hi = (lo + 1).astype(np.uint16)  # the next magnitude, same sign
    rng = np.random.default_rng(3)
    codes = [lo, hi, oracle.encode_fp16(x_all)]
    counts = np.array([4, 4, 0], np.uint32)
    off, flags = np.array([0, P], np.uint64), np.array([3], np.uint8)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    m, v = np.zeros(P, F), np.zeros(P, F)
    cfg = dict(lr=1e-3, weight_decay=0.01, step=1)
    bounds = oracle.partition(P, 2, None, 64)
    for local in (None, 2):
        cnt = counts.copy()
        if local is not None:
            cnt[2] = 1
        dc = [_up(c.view(np.int16)) for c in codes]
        if local is not None:
            W.nan_poison(dc[local])
        xd, md, vd = _up(x), _up(m), _up(v)
        mean = torch.empty(P, dtype=torch.float32, device=DEV)
        loc = None if local is None else (local, _up(x_all))
        oc, _ = D.dedloc_round(dc, cnt, bounds, D.DEDLOC_CODEC_FP16, xd, md, vd, off, flags,
                               D.lamb_cfg(**cfg), out_mean=mean, local=loc)
        r = oracle.round_(codes, cnt, bounds, oracle.CODEC_FP16, x, m, v, off, flags, oracle.lamb_cfg(**cfg))
        if local is None:  # the two peers' averages are exact ties
            assert np.array_equal(r["mean"].astype(np.float64),
                                  (lo.view(np.float16).astype(np.float64) + hi.view(np.float16)) / 2)
        else:
            assert np.array_equal(_u16(dc[local]), codes[local])
        assert np.array_equal(_bits(_np(mean)), _bits(r["mean"]))
        assert np.array_equal(_u16(oc), r["codes"])
        assert np.array_equal(_bits(_np(md)), _bits(r["m"]))
        _assert_x(_np(xd), r["x"], x)


def test_decode_fp16_all_patterns():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    out = D.dedloc_decode(_up(h.view(np.int16)), None, h.size, D.DEDLOC_CODEC_FP16)
    g, o = _np(out), oracle.decode_fp16(h)
    nan = np.isnan(o)
    assert np.array_equal(_bits(g[~nan]), _bits(o[~nan])) and np.isnan(g[nan]).all()


@pytest.mark.parametrize("n", [1, 15, 16, 1023, 1024, 1025, 3 * 4096 + 17, 200_000])
def test_encode_decode_i8(n):
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * 10.0 ** rng.uniform(-6, 2, n)).astype(F)
    if n > 3000:
        x[1024:2048] = 0.0  # an all-zero block
    codes, scales = D.dedloc_encode(_up(x), D.DEDLOC_CODEC_I8)
    oc, osc = oracle.encode_i8(x, 1024)
    assert np.array_equal(_i8(codes), oc)
    assert np.array_equal(_bits(_np(scales)), _bits(osc))
    dec = D.dedloc_decode(_up(oc), _up(osc), n, D.DEDLOC_CODEC_I8)
    assert np.array_equal(_bits(_np(dec)), _bits(oracle.decode_i8(oc, osc, 1024)))


def _near_ties(rng, n_blocks, log_scale):
    """Blocks whose quotients x / s sit on and within a few ulps of
    half-integers (where the rounded quotient decides the code), within 1e-3
    of them (across the distance at which the kernel stops trusting its
    reciprocal product), or between 2^-13 and 1e-3 from them (where it
    trusts it); each block keeps its maximum at 10**log_scale."""
    out = []
    for b in range(n_blocks):
        a = np.float32(10.0 ** log_scale[b % len(log_scale)])
        s = np.float32(a / np.float32(127))
        k = rng.integers(-127, 127, 1024).astype(np.float64) + 0.5
        if b % 3 == 1:
            k += rng.uniform(-1e-3, 1e-3, 1024)
        elif b % 3 == 2:
            k += rng.choice([-1.0, 1.0], 1024) * rng.uniform(2.0 ** -13, 1e-3, 1024)
        x = (k * np.float64(s)).astype(F)
        step = rng.integers(-3, 4, 1024)
        for _ in range(3):
            up, dn = step > 0, step < 0
            x[up] = np.nextafter(x[up], np.float32(np.inf))
            x[dn] = np.nextafter(x[dn], np.float32(-np.inf))
            step = step - np.sign(step)
        x[rng.integers(0, 1024)] = a if b % 4 < 2 else -a
        out.append(x)
    return np.concatenate(out)


@pytest.mark.parametrize("log_scale", [[-3.0, 0.0, 2.0], [-37.0, 37.0]], ids=["normal", "extreme"])
def test_encode_i8_near_ties(log_scale):
    # codes are rint of the correctly rounded quotient; the kernel takes them
    # from a reciprocal product only where that provably agrees.  "extreme"
    # scales (outside [2^-100, 2^100]) always divide.
    rng = np.random.default_rng(7)
    x = _near_ties(rng, 96, log_scale)
    codes, scales = D.dedloc_encode(_up(x), D.DEDLOC_CODEC_I8)
    oc, osc = oracle.encode_i8(x, 1024)
    assert np.array_equal(_bits(_np(scales)), _bits(osc))
    assert np.array_equal(_i8(codes), oc)


def test_encode_i8_tiny_blocks():
    """Blocks at the bottom of the fp32 range: max|x| <= 63 * 2^-149 makes
    max|x| / 127 underflow to 0 (every code 0), 64 * 2^-149 gives the smallest
    nonzero scale, and subnormal maxima give subnormal scales.  Also through
    the reducer and the encode of its average."""
    tiny = np.float32(2.0 ** -149)
    rng = np.random.default_rng(11)
    blocks = []
    for amax in [1, 2, 63, 64, 65, 127, 128, 1000, 2 ** 20, 2 ** 23, 2 ** 24, -150, -190, -300]:
        k = rng.integers(-abs(amax), abs(amax) + 1, 1024)
        k[rng.integers(0, 1024)] = amax  # a negative maximum: a / s >= 127.5 saturates at -127
        blocks.append(k.astype(F) * tiny)
    x = np.concatenate(blocks)
    codes, scales = D.dedloc_encode(_up(x), D.DEDLOC_CODEC_I8)
    oc, osc = oracle.encode_i8(x, 1024)
    assert np.array_equal(_bits(_np(scales)), _bits(osc))
    assert np.array_equal(_i8(codes), oc)
    assert osc[0] == 0 and osc[2] == 0 and osc[3] > 0 and not oc[:1024].any()
    # two peers whose average is that small
    c2, s2 = oracle.encode_i8(x[::-1].copy(), 1024)
    counts = np.array([3, 1], np.uint32)
    rc, rs = D.dedloc_reduce_shard([_up(oc), _up(c2)], counts, x.size, D.DEDLOC_CODEC_I8,
                                   peer_scales=[_up(osc), _up(s2)])
    orc, ors, _ = oracle.reduce([oc, c2], counts, oracle.CODEC_I8, [osc, s2], 1024)
    assert np.array_equal(_bits(_np(rs)), _bits(ors))
    assert np.array_equal(_i8(rc), orc)


# --------------------------------------------------------------- reducer

def _peer_messages(codec, n, length, seed, outliers=True):
    rng = np.random.default_rng(seed)
    grads = []
    for p in range(n):
        g = (rng.standard_normal(length) * 1e-3).astype(F)
        if outliers:
            g[rng.random(length) < 0.01] *= 100
        grads.append(g)
    if codec == D.DEDLOC_CODEC_FP16:
        return [oracle.encode_fp16(g) for g in grads], None
    enc = [oracle.encode_i8(g, 1024) for g in grads]
    return [c for c, _ in enc], [s for _, s in enc]


@pytest.mark.parametrize("codec", [D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8])
@pytest.mark.parametrize("n_peers,length", [(1, 1), (3, 2049 * 8 + 3), (16, 5 * 2048 + 7),
                                            (64, 3 * 1024 + 100), (5, 0), (7, 1024 * 9)])
def test_reduce_shard(codec, n_peers, length):
    rng = np.random.default_rng(1000 * codec + n_peers + length)
    counts = rng.integers(0, 300, n_peers).astype(np.uint32)
    counts[rng.integers(0, n_peers)] = 17
    codes, scales = _peer_messages(codec, n_peers, length, n_peers + length)
    dc, ds = [], []
    for p in range(n_peers):
        c = _up(codes[p].view(np.int16) if codec == D.DEDLOC_CODEC_FP16 else codes[p])
        s = None if scales is None else _up(scales[p])
        if counts[p] == 0:
            W.nan_poison(c)  # never read
            if s is not None:
                W.nan_poison(s)
            if p % 2:
                c = s = None  # a zero-count peer may pass NULL
        dc.append(c)
        ds.append(s)
    mean = torch.empty(max(length, 1), dtype=torch.float32, device=DEV)
    oc, osc = D.dedloc_reduce_shard(dc, counts, length, codec, ds if scales is not None else None,
                                    out_mean=mean)
    rc, rs, rm = oracle.reduce(codes, counts, codec, scales, 1024)
    if length == 0:
        return
    assert np.array_equal(_bits(_np(mean)[:length]), _bits(rm))
    if codec == D.DEDLOC_CODEC_FP16:
        assert np.array_equal(_u16(oc), rc)
    else:
        assert np.array_equal(_i8(oc), rc)
        assert np.array_equal(_bits(_np(osc)), _bits(rs))


def test_reduce_shards_of_a_vector():
    # per-shard pointers offset into full-vector messages, bandwidth-weighted bounds
    P, n = 300_000 + 24, 6
    codes, _ = _peer_messages(D.DEDLOC_CODEC_FP16, n, P, 77)
    counts = np.array([5, 9, 0, 1, 30, 2], np.uint32)
    dev = [_up(c.view(np.int16)) for c in codes]
    bounds = D.dedloc_partition(P, n, [100, 10, 500, 0, 250, 40], 64)
    out = torch.empty(P, dtype=torch.int16, device=DEV)
    for k in range(n):
        a, b = int(bounds[k]), int(bounds[k + 1])
        D.dedloc_reduce_shard([d[a:b] for d in dev], counts, b - a, D.DEDLOC_CODEC_FP16, out_codes=out[a:b])
    rc, _, _ = oracle.reduce(codes, counts, oracle.CODEC_FP16)
    assert np.array_equal(_u16(out), rc)


# ------------------------------------------------------------------ LAMB

TABLES = {
    "ragged": [8, 2048, 2056, 0, 64, 10000, 3],
    "single": [4097],
    "many_small": [64] * 100 + [128] * 30 + [2048 * 3 + 8] * 5 + [19],
    "empty_chunk": [4096] * 64 + [0] * 6,
    # 450 tensors: three launch chunks of at most 192 tensors, tensor sizes
    # 0 to 3 tiles, the last one ragged
    "chunks": [8 * ((i * 37) % 769) for i in range(449)] + [2048 * 3 + 5],
}


def _state(sizes, seed):
    rng = np.random.default_rng(seed)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    flags = rng.integers(0, 4, len(sizes)).astype(np.uint8)
    flags[0] = 3
    x = (rng.standard_normal(P) * 0.02).astype(F)
    if len(sizes) > 2:
        x[int(off[1]):int(off[2])] = 0.0  # a zero tensor
    m = (rng.standard_normal(P) * 1e-4).astype(F)
    v = ((rng.standard_normal(P) * 1e-3) ** 2).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    return off, flags, x, m, v, g


@pytest.mark.parametrize("src", ["f32", "fp16", "i8"])
@pytest.mark.parametrize("table", list(TABLES))
@pytest.mark.parametrize("unit", [False, True])
def test_lamb_step(src, table, unit):
    off, flags, x, m, v, g = _state(TABLES[table], zlib.crc32(f"{src}/{table}".encode()) % 1000)
    P = int(off[-1])
    cfg = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, step=7,
               force_unit_trust=unit)
    if src == "f32":
        ghat, gdev, gsc, codec = g, _up(g), None, D.DEDLOC_CODEC_F32
    elif src == "fp16":
        c = oracle.encode_fp16(g)
        ghat, gdev, gsc, codec = oracle.decode_fp16(c), _up(c.view(np.int16)), None, D.DEDLOC_CODEC_FP16
    else:
        c, s = oracle.encode_i8(g, 1024)
        ghat, gdev, gsc, codec = oracle.decode_i8(c, s, 1024), _up(c), _up(s), D.DEDLOC_CODEC_I8
    xo, mo, vo, to = oracle.lamb(x, m, v, ghat, off, flags, oracle.lamb_cfg(**cfg))
    xd, md, vd = _up(x), _up(m), _up(v)
    tr = torch.full((len(flags),), -1.0, device=DEV)
    D.dedloc_lamb_step(xd, md, vd, gdev, off, flags, D.lamb_cfg(**cfg), grad_codec=codec,
                       grad_scales=gsc, trust_out=tr)
    assert np.array_equal(_bits(_np(md)), _bits(mo))
    assert np.array_equal(_bits(_np(vd)), _bits(vo))
    assert np.allclose(_np(tr), to, rtol=1e-6, atol=0)
    _assert_x(_np(xd), xo, x)


# ----------------------------------------------------------------- round

def _small(base, sizes, kinds=None, **over):
    return W.scaled(base, base.name + "_small", sizes, kinds, **over)


SMALL = [
    _small(W.TINY, [4096, 4096, 2048, 8]),
    _small(W.ALBERT_LARGE, [3000 * 8, 128, 128, 4096, 1024, 5], ["w", "g", "b", "w", "b", "b"], n_peers=16),
    _small(W.RESNET50, [9408, 64, 64, 4096, 256, 256, 1000], ["w", "g", "b", "w", "g", "b", "b"], n_peers=32),
    _small(W.ALBERT_XLARGE, [8192, 128, 128, 10000, 2048, 7], ["w", "g", "b", "w", "b", "b"],
           n_peers=64, n_zero_peers=4),
    _small(W.STRESS, [2048 * 5] * 3, n_peers=8),
]


def _oracle_inputs(wl):
    counts = W.sample_counts(wl)
    grads = [W.peer_gradient(wl, p).numpy() for p in range(wl.n_peers)]
    if wl.codec == "fp16":
        codes, scales = [oracle.encode_fp16(g) for g in grads], None
    else:
        enc = [oracle.encode_i8(g, 1024) for g in grads]
        codes, scales = [c for c, _ in enc], [s for _, s in enc]
    return counts, codes, scales


def _device_msgs(wl, codes, scales, counts):
    dc, ds = [], []
    for p in range(wl.n_peers):
        c = _up(codes[p].view(np.int16) if wl.codec == "fp16" else codes[p])
        s = None if scales is None else _up(scales[p])
        if counts[p] == 0:
            W.nan_poison(c)
            if s is not None:
                W.nan_poison(s)
        dc.append(c)
        ds.append(s)
    return dc, ds


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_round_small_three_steps(wl):
    """Three consecutive rounds from m = v = 0 (steps 1, 2, 3)."""
    counts, codes, scales = _oracle_inputs(wl)
    codec = H.codec_id(wl)
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, m, v = (t.numpy() for t in W.optimizer_state(wl, fresh=True))
    dc, ds = _device_msgs(wl, codes, scales, counts)
    xd, md, vd = _up(x), _up(m), _up(v)
    ws = D.make_workspace(wl.P, wl.offsets(), DEV)
    mean = torch.empty(wl.P, dtype=torch.float32, device=DEV)
    tr = torch.empty(wl.n_tensors, dtype=torch.float32, device=DEV)
    for step in (1, 2, 3):
        cfg = dict(lr=wl.lr, beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps,
                   weight_decay=wl.weight_decay, step=step)
        r = oracle.round_(codes, counts, bounds, codec, x, m, v, wl.offsets(), wl.flags(),
                          oracle.lamb_cfg(**cfg), scales, 1024)
        oc, osc = D.dedloc_round(dc, counts, bounds, codec, xd, md, vd, wl.offsets(), wl.flags(),
                                 D.lamb_cfg(**cfg), peer_scales=ds if scales else None,
                                 trust_out=tr, out_mean=mean, ws=ws)
        assert np.array_equal(_bits(_np(mean)), _bits(r["mean"])), step
        if codec == D.DEDLOC_CODEC_FP16:
            assert np.array_equal(_u16(oc), r["codes"]), step
        else:
            assert np.array_equal(_i8(oc), r["codes"]), step
            assert np.array_equal(_bits(_np(osc)), _bits(r["scales"])), step
        # m' and v' do not depend on x: from bit-identical moments and the same
        # gathered gradient they stay bit-identical at every step
        assert np.array_equal(_bits(_np(md)), _bits(r["m"])), step
        assert np.array_equal(_bits(_np(vd)), _bits(r["v"])), step
        assert np.allclose(_np(tr), r["trust"], rtol=1e-6, atol=0), step
        _assert_x(_np(xd), r["x"], x)
        x, m, v = r["x"], r["m"], r["v"]


def test_round_is_deterministic():
    wl = SMALL[2]
    dr = H.DeviceRound(wl, DEV)
    x0, m0, v0 = dr.x.clone(), dr.m.clone(), dr.v.clone()
    outs = []
    for _ in range(2):
        dr.x.copy_(x0)
        dr.m.copy_(m0)
        dr.v.copy_(v0)
        dr.run()
        outs.append([_np(t).copy() for t in (dr.out_codes, dr.x, dr.m, dr.v, dr.trust)])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


# ------------------------------------------------- full-size, sampled

def _sample(wl, n_tensors=3, n_blocks=8, max_len=17_000_000):
    rng = np.random.default_rng(4242 + wl.cid)
    off = wl.offsets()
    sizes = np.diff(off.astype(np.int64))
    cand = [t for t in range(wl.n_tensors) if 0 < sizes[t] <= max_len]
    pick = {min(cand, key=lambda t: sizes[t]), max(cand, key=lambda t: sizes[t])}
    while len(pick) < min(n_tensors, len(cand)):
        pick.add(int(rng.choice(cand)))
    nblk = (wl.P + 1023) // 1024
    blocks = sorted(set(int(b) for b in rng.integers(0, nblk, n_blocks)) | {nblk - 1}) if n_blocks else []
    return sorted(pick), blocks


def _superset(a, b, P, codec):
    if codec == D.DEDLOC_CODEC_FP16:
        return a, b
    return a // 1024 * 1024, min((b + 1023) // 1024 * 1024, P)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_round_full_size_sampled(name):
    _full_size_sampled(W.WORKLOADS[name])


# Vectors past 2^31 elements: the largest tensor alone has more than 2^31
# elements, so element indices, tile numbers, chunk offsets and grid sizes
# all leave the 32-bit signed range (the stress workload stops at 2^30).  It
# takes weight decay without the trust ratio (r = 1), so its update is
# elementwise and the sampled blocks inside it check x' as well as m', v'.
BEYOND_2P31 = [W.Workload(name=f"beyond_2p31_{c}", cid=20 + i,
                          tensors=(("big_d", 2 ** 31 + 2 ** 20, "d"), ("mid_w", 2 ** 20, "w"),
                                   ("tail_g", 2 ** 20 + 13, "g")),
                          n_peers=3, codec=c, sigma=1e-3, count_range=(1, 64))
               for i, c in enumerate(("fp16", "i8"))]


@pytest.mark.parametrize("wl", BEYOND_2P31, ids=lambda w: w.name)
def test_round_beyond_2p31_elements(wl):
    _full_size_sampled(wl)


def _full_size_sampled(wl):
    name = wl.name
    codec = H.codec_id(wl)
    tensors, blocks = _sample(wl)
    off = wl.offsets()
    ranges = []
    for t in tensors:
        ranges.append(_superset(int(off[t]), int(off[t + 1]), wl.P, codec))
    for b in blocks:
        ranges.append((b * 1024, min((b + 1) * 1024, wl.P)))
    print(f"\n[{name}] P={wl.P} peers={wl.n_peers} tensors={tensors} blocks={blocks}", flush=True)
    dr = H.DeviceRound(wl, DEV, sample_ranges=ranges)
    x0 = [dr.x[A:B].cpu().numpy() for A, B in ranges]
    m0 = [dr.m[A:B].cpu().numpy() for A, B in ranges]
    v0 = [dr.v[A:B].cpu().numpy() for A, B in ranges]
    dr.run()
    torch.cuda.synchronize()
    cfg = oracle.lamb_cfg(wl.lr, wl.beta1, wl.beta2, wl.eps, wl.weight_decay, step=dr.step)
    trust = _np(dr.trust)
    for i, (A, B) in enumerate(ranges):
        g = [dr.host_grads[p][i] for p in range(wl.n_peers)]
        if codec == D.DEDLOC_CODEC_FP16:
            codes, scales = [oracle.encode_fp16(x) for x in g], None
        else:
            enc = [oracle.encode_i8(x, 1024) for x in g]
            codes, scales = [c for c, _ in enc], [s for _, s in enc]
        for p in np.flatnonzero(dr.counts == 0):  # never read
            codes[p] = np.full_like(codes[p], 0x7E)
            if scales is not None:
                scales[p] = np.full_like(scales[p], np.nan)
        if i < len(tensors):
            t = tensors[i]
            a, b = int(off[t]), int(off[t + 1])
            sub_off = np.array([0, a - A, b - A, B - A], np.uint64)
            sub_fl = np.array([0, wl.flags()[t], 0], np.uint8)
            elementwise = []
        else:
            # a block: the pieces of the tensors it overlaps, with the trust
            # ratio left out (only a whole tensor gives its norms); pieces of
            # tensors without the trust ratio have r = 1 on both sides
            a, b, t = A, B, None
            ts = [k for k in range(wl.n_tensors) if int(off[k]) < B and int(off[k + 1]) > A]
            cuts = [A] + [int(off[k]) for k in ts[1:]] + [B]
            sub_off = np.array([c - A for c in cuts], np.uint64)
            sub_fl = np.array([int(wl.flags()[k]) & ~W.FLAG_ADAPT for k in ts], np.uint8)
            elementwise = [(cuts[j] - A, cuts[j + 1] - A) for j, k in enumerate(ts)
                           if not int(wl.flags()[k]) & W.FLAG_ADAPT]
        r = oracle.round_(codes, dr.counts, np.array([0, B - A], np.uint64), codec, x0[i], m0[i], v0[i],
                          sub_off, sub_fl, cfg, scales, 1024)
        if codec == D.DEDLOC_CODEC_FP16:
            assert np.array_equal(_u16(dr.out_codes[A:B]), r["codes"]), (name, A, B)
        else:
            assert np.array_equal(_i8(dr.out_codes[A:B]), r["codes"]), (name, A, B)
            assert np.array_equal(_bits(_np(dr.out_scales[A // 1024:(B + 1023) // 1024])),
                                  _bits(r["scales"])), (name, A, B)
        # m' and v' are elementwise: bit-exact over the whole sampled range
        assert np.array_equal(_bits(_np(dr.m[A:B])), _bits(r["m"])), (name, A, B)
        assert np.array_equal(_bits(_np(dr.v[A:B])), _bits(r["v"])), (name, A, B)
        if t is not None:
            s = slice(a - A, b - A)
            assert np.isclose(trust[t], r["trust"][1], rtol=1e-6, atol=0), (name, t, trust[t], r["trust"][1])
            _assert_x(_np(dr.x[a:b]), r["x"][s], x0[i][s])
        for lo, hi in elementwise:
            _assert_x(_np(dr.x[A + lo:A + hi]), r["x"][lo:hi], x0[i][lo:hi])
    assert np.isfinite(trust).all() and (trust > 0).all()
    del dr
    torch.cuda.empty_cache()


def test_pending_hip_error_is_not_reported():
    """A launch reports its own status: an error left pending by an earlier,
    unrelated HIP call of the caller's (here hipSetDevice on a device that
    does not exist) does not make a library call fail."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    x = _up(np.linspace(-1, 1, 4096).astype(F))
    torch.cuda.synchronize()
    assert hip.hipSetDevice(ctypes.c_int(4096)) != 0  # leaves hipErrorInvalidDevice pending
    try:
        codes, _ = D.dedloc_encode(x, D.DEDLOC_CODEC_FP16)
    finally:
        hip.hipGetLastError()  # clear it for the rest of the process
        torch.cuda.set_device(0)
    assert np.array_equal(_u16(codes), oracle.encode_fp16(_np(x)))


def test_binding_rejects_bad_buffers():
    """The library reads and writes raw memory, so the Python binding refuses
    a tensor the call would overrun or misread before anything is launched:
    non-contiguous or broadcast views, the wrong dtype, too few elements.  A
    peer without samples is never read, so its buffer is not checked."""
    n = 4096
    x = _up(np.linspace(-1, 1, n).astype(F))
    with pytest.raises(ValueError, match="contiguous"):
        D.dedloc_encode(torch.zeros(n, 2, device=DEV)[:, 0], D.DEDLOC_CODEC_FP16)
    with pytest.raises(ValueError, match="contiguous"):
        D.dedloc_encode(torch.zeros(1, device=DEV).expand(n), D.DEDLOC_CODEC_FP16)
    with pytest.raises(ValueError, match="float32"):
        D.dedloc_encode(x.half(), D.DEDLOC_CODEC_FP16)
    with pytest.raises(ValueError, match="codes"):
        D.dedloc_encode(x, D.DEDLOC_CODEC_FP16, codes=torch.empty(n - 1, dtype=torch.int16, device=DEV))
    off, flags = np.array([0, n], np.uint64), np.array([3], np.uint8)
    with pytest.raises(ValueError, match="m:"):
        D.dedloc_lamb_step(x.clone(), torch.zeros(n - 8, device=DEV), torch.zeros(n, device=DEV), x, off, flags,
                           D.lamb_cfg())
    codes, _ = D.dedloc_encode(x, D.DEDLOC_CODEC_FP16)
    short = codes[: n // 2]
    with pytest.raises(ValueError, match=r"peer_codes\[1\]"):
        D.dedloc_reduce_shard([codes, short], [1, 1], n, D.DEDLOC_CODEC_FP16)
    out, _ = D.dedloc_reduce_shard([codes, short], [1, 0], n, D.DEDLOC_CODEC_FP16)  # peer 1 is never read
    assert np.array_equal(_u16(out), _u16(codes))
