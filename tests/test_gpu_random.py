"""Randomised GPU parity of the whole round (dedloc_round, dedloc_round_lars)
against the CPU oracle, through the C ABI.

Each seed draws one configuration: a tensor table mixing empty tensors,
tensors shorter than a vector, sub-tile, whole-tile and ragged tensors and a
scalar tail at the end of the vector; 1 to 12 peers (some seeds 65 to 70,
which chains reduce launches) with zero-sample peers whose buffers hold NaN;
shard bounds from random bandwidth weights; either wire codec; LAMB or LARS
with random step, learning rate, weight decay and tensor flags; and, on half
of the seeds, a local peer whose fp32 gradient the round encodes itself.

Bars as in test_gpu_parity: codes, scales, the fp32 average, the local
peer's message and LAMB's m', v' bit-identical; trust ratios within 1e-6
relative; x' (and LARS's v') within 1e-5 of their scale."""

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
    return np.ascontiguousarray(a, F).view(np.uint32)


def _close(got, ref, scale_ref, rel=1e-5):
    scale = max(float(np.max(np.abs(scale_ref))) if np.size(scale_ref) else 0.0, 1e-30)
    err = float(np.max(np.abs(got.astype(np.float64) - ref.astype(np.float64)))) if np.size(got) else 0.0
    assert err <= rel * scale, (err, rel * scale)


def _table(rng):
    sizes = []
    for _ in range(int(rng.integers(1, 10))):
        kind = int(rng.integers(0, 6))
        if kind == 0:
            n = 0
        elif kind == 1:
            n = 8 * int(rng.integers(1, 8))
        elif kind == 2:
            n = 8 * int(rng.integers(1, 300))
        elif kind == 3:
            n = 2048 * int(rng.integers(1, 4))
        elif kind == 4:
            n = 2048 * int(rng.integers(1, 4)) + 8 * int(rng.integers(1, 255))
        else:
            n = 1024 * int(rng.integers(1, 6)) + 8 * int(rng.integers(0, 128))
        sizes.append(n)
    sizes[-1] += int(rng.integers(0, 8))  # only the vector's end may fall inside a vector
    if sum(sizes) == 0:
        sizes[-1] = 8 + int(rng.integers(0, 8))
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    return off, rng.integers(0, 4, len(sizes)).astype(np.uint8)


def _case(seed):
    rng = np.random.default_rng(7000 + seed)
    codec = FP16 if seed % 2 == 0 else I8
    opt = "lamb" if seed % 4 < 2 else "lars"
    off, flags = _table(rng)
    P = int(off[-1])
    n = int(rng.integers(65, 71)) if seed % 10 == 9 else int(rng.integers(1, 13))
    counts = rng.integers(0, 300, n).astype(np.uint32)
    counts[rng.random(n) < 0.25] = 0
    if counts.sum() == 0:
        counts[int(rng.integers(0, n))] = int(rng.integers(1, 300))
    active = np.flatnonzero(counts)
    local = int(rng.choice(active)) if seed % 3 != 0 else None
    grads = []
    for _ in range(n):
        g = (rng.standard_normal(P) * 10.0 ** rng.uniform(-4, -2)).astype(F)
        g[rng.random(P) < 0.01] *= 100.0
        grads.append(g)
    n_shards = int(rng.integers(1, n + 1))
    align = 64 if codec == FP16 else 1024
    bounds = oracle.partition(P, n_shards, rng.integers(1, 1000, n_shards), align)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    T = len(flags)
    zt = int(rng.integers(0, T))
    x[int(off[zt]):int(off[zt + 1])] = 0.0  # a tensor with ||x|| = 0
    if rng.random() < 0.5:
        m = (rng.standard_normal(P) * 1e-4).astype(F)
        v = np.square(rng.standard_normal(P) * 1e-3).astype(F)
    else:
        m = np.zeros(P, F)
        v = np.zeros(P, F)
    if opt == "lamb":
        cfg = dict(lr=float(10.0 ** rng.uniform(-4, -2)), beta1=0.9, beta2=0.999, eps=1e-6,
                   weight_decay=float(rng.choice([0.0, 0.01, 0.1])), step=int(rng.integers(1, 6)))
    else:
        cfg = dict(lr=float(rng.uniform(0.1, 5.0)), momentum=0.9, trust_coef=1e-3,
                   weight_decay=float(rng.choice([0.0, 1e-6, 1e-4])))
    return dict(codec=codec, opt=opt, off=off, flags=flags, P=P, counts=counts, local=local, grads=grads,
                bounds=bounds, x=x, m=m, v=v, cfg=cfg)


@pytest.mark.parametrize("seed", range(300))
def test_random_round(seed):
    c = _case(seed)
    print(f"\n[seed {seed}] codec={c['codec']} opt={c['opt']} P={c['P']} tensors={len(c['flags'])} "
          f"peers={len(c['counts'])} active={int(np.count_nonzero(c['counts']))} "
          f"shards={len(c['bounds']) - 1} local={c['local']}", flush=True)
    _check_round(c)


@pytest.mark.parametrize("seed", range(0, 300, 6))
def test_random_round_without_published_ratios(seed):
    """The same rounds with every workgroup of the update pass computing its
    tensor's trust ratio itself (no polling for the published one)."""
    c = _case(seed)
    print(f"\n[seed {seed}, no polls] codec={c['codec']} opt={c['opt']} P={c['P']} tensors={len(c['flags'])}",
          flush=True)
    old = D.dedloc_test_trust_polls(0)
    try:
        _check_round(c)
    finally:
        D.dedloc_test_trust_polls(old)


def _degenerate(name, codec, opt):
    """Edge cases of the round: an empty vector, a vector shorter than one
    lane's vector, one peer, an empty shard, all-zero gradients (int8 scale
    0; with m = v = 0 and no weight decay ||u|| = 0, so r = 1), and a lone
    peer with samples among many without."""
    rng = np.random.default_rng(len(name) * 7 + codec)
    sizes, n, counts, local, zero_g, n_shards = [2048], 3, None, None, False, 1
    if name == "empty":
        sizes = [0]
    elif name == "short":
        sizes, n, local = [5], 1, 0
    elif name == "empty_shard":
        sizes, n_shards = [1024 + 3], 4
    elif name == "zero_grads":
        sizes, zero_g = [8, 1024, 2048 + 16], True
    elif name == "lone_peer":
        n = 40
        counts = np.zeros(n, np.uint32)
        counts[17] = 5
        local = 17
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    flags = np.full(len(sizes), 2 if zero_g else 3, np.uint8)  # zero_grads: adapt, no decay
    if counts is None:
        counts = rng.integers(1, 100, n).astype(np.uint32)
    grads = [np.zeros(P, F) if zero_g else (rng.standard_normal(P) * 1e-3).astype(F) for _ in range(n)]
    align = 64 if codec == FP16 else 1024
    bounds = oracle.partition(P, n_shards, None, align)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    m = np.zeros(P, F)
    v = np.zeros(P, F)
    if opt == "lamb":
        cfg = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.0 if zero_g else 0.01, step=1)
    else:
        cfg = dict(lr=4.8, momentum=0.9, trust_coef=1e-3, weight_decay=0.0 if zero_g else 1e-6)
    return dict(codec=codec, opt=opt, off=off, flags=flags, P=P, counts=counts, local=local, grads=grads,
                bounds=bounds, x=x, m=m, v=v, cfg=cfg)


@pytest.mark.parametrize("name", ["empty", "short", "empty_shard", "zero_grads", "lone_peer"])
@pytest.mark.parametrize("codec", [FP16, I8])
@pytest.mark.parametrize("opt", ["lamb", "lars"])
def test_degenerate_round(name, codec, opt):
    print(f"\n[{name}] codec={codec} opt={opt}", flush=True)
    _check_round(_degenerate(name, codec, opt))


@pytest.mark.parametrize("codec", [FP16, I8])
@pytest.mark.parametrize("opt", ["lamb", "lars"])
def test_round_many_chunks(codec, opt):
    """450 tensors: the optimizer passes run in three launch chunks of at
    most 192 tensors; with the fp16 codec every chunk's pass A also averages
    its own range of the messages (and encodes the local peer's)."""
    print(f"\n[many chunks] codec={codec} opt={opt}", flush=True)
    rng = np.random.default_rng(4500 + codec)
    sizes = [8 * int(k) for k in rng.integers(0, 700, 449)] + [2048 * 3 + 5]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    n = 6
    counts = np.array([5, 0, 9, 1, 30, 2], np.uint32)
    grads = [(rng.standard_normal(P) * 1e-3).astype(F) for _ in range(n)]
    align = 64 if codec == FP16 else 1024
    bounds = oracle.partition(P, 4, rng.integers(1, 1000, 4), align)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    m = (rng.standard_normal(P) * 1e-4).astype(F)
    v = np.square(rng.standard_normal(P) * 1e-3).astype(F)
    if opt == "lamb":
        cfg = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, step=4)
    else:
        cfg = dict(lr=4.8, momentum=0.9, trust_coef=1e-3, weight_decay=1e-5)
    _check_round(dict(codec=codec, opt=opt, off=off, flags=rng.integers(0, 4, len(sizes)).astype(np.uint8), P=P,
                      counts=counts, local=2, grads=grads, bounds=bounds, x=x, m=m, v=v, cfg=cfg))


@pytest.mark.parametrize("n_peers", [3, 9, 70])
def test_round_i8_tensor_pieces(n_peers):
    """int8 LAMB round whose tensors start inside codec blocks and inside
    LAMB tiles: several tensors in one block (8-element and empty ones among
    them), tensors over many blocks, a ragged end; 3 active peers (small
    peer batch), 9 (full batch) and 70 (two launches chained through the
    fp32 running sum)."""
    print(f"\n[i8 pieces] peers={n_peers}", flush=True)
    rng = np.random.default_rng(8100 + n_peers)
    sizes = [8, 0, 8, 16, 1000, 0, 4096 + 8, 24, 3 * 4096, 8, 2040, 2 * 4096 + 512, 0, 4088, 8, 5]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    P = int(off[-1])
    counts = rng.integers(1, 300, n_peers).astype(np.uint32)
    grads = [(rng.standard_normal(P) * 1e-3).astype(F) for _ in range(n_peers)]
    bounds = oracle.partition(P, 3, rng.integers(1, 1000, 3), 1024)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    m = (rng.standard_normal(P) * 1e-4).astype(F)
    v = np.square(rng.standard_normal(P) * 1e-3).astype(F)
    cfg = dict(lr=2e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, step=3)
    flags = rng.integers(0, 4, len(sizes)).astype(np.uint8)
    flags[6] = 3
    flags[8] = 3
    _check_round(dict(codec=I8, opt="lamb", off=off, flags=flags, P=P, counts=counts, local=1, grads=grads,
                      bounds=bounds, x=x, m=m, v=v, cfg=cfg))


def _check_round(c):
    codec, P, counts, local = c["codec"], c["P"], c["counts"], c["local"]
    n = len(counts)
    if codec == FP16:
        codes, scales = [oracle.encode_fp16(g) for g in c["grads"]], None
    else:
        enc = [oracle.encode_i8(g, 1024) for g in c["grads"]]
        codes, scales = [e[0] for e in enc], [e[1] for e in enc]
    # oracle side: zero-sample peers' messages are garbage it must not read
    ocodes = [np.full_like(codes[p], 0x7E) if counts[p] == 0 else codes[p] for p in range(n)]
    oscales = None if scales is None else [
        np.full_like(scales[p], np.nan) if counts[p] == 0 else scales[p] for p in range(n)]
    dc = [_up(cd.view(np.int16) if codec == FP16 else cd) for cd in codes]
    ds = None if scales is None else [_up(s) for s in scales]
    for p in range(n):
        if counts[p] == 0 or p == local:  # never read, or written by the round
            W.nan_poison(dc[p])
            if ds is not None:
                W.nan_poison(ds[p])
    T = len(c["flags"])
    xd, md, vd = _up(c["x"]), _up(c["m"]), _up(c["v"])
    mean = torch.empty(P, dtype=torch.float32, device=DEV)
    tr = torch.full((T,), -1.0, dtype=torch.float32, device=DEV)
    ws = D.make_workspace(P, c["off"], DEV)
    loc = None if local is None else (local, _up(c["grads"][local]))
    if c["opt"] == "lamb":
        r = oracle.round_(ocodes, counts, c["bounds"], codec, c["x"], c["m"], c["v"], c["off"], c["flags"],
                          oracle.lamb_cfg(**c["cfg"]), oscales, 1024)
        oc, osc = D.dedloc_round(dc, counts, c["bounds"], codec, xd, md, vd, c["off"], c["flags"],
                                 D.lamb_cfg(**c["cfg"]), peer_scales=ds, trust_out=tr, out_mean=mean,
                                 ws=ws, local=loc)
        assert np.array_equal(_bits(_np(md)), _bits(r["m"]))
        assert np.array_equal(_bits(_np(vd)), _bits(r["v"]))
    else:
        r = oracle.round_lars(ocodes, counts, c["bounds"], codec, c["x"], c["v"], c["off"], c["flags"],
                              oracle.lars_cfg(**c["cfg"]), oscales, 1024)
        oc, osc = D.dedloc_round_lars(dc, counts, c["bounds"], codec, xd, vd, c["off"], c["flags"],
                                      D.lars_cfg(**c["cfg"]), peer_scales=ds, trust_out=tr, out_mean=mean,
                                      ws=ws, local=loc)
        _close(_np(vd), r["v"], r["v"])
    assert np.array_equal(_bits(_np(mean)), _bits(r["mean"]))
    if codec == FP16:
        assert np.array_equal(_np(oc).view(np.uint16), r["codes"])
    else:
        assert np.array_equal(_np(oc).view(np.int8), r["codes"])
        assert np.array_equal(_bits(_np(osc)), _bits(r["scales"]))
    if local is not None:
        if codec == FP16:
            assert np.array_equal(_np(dc[local]).view(np.uint16), codes[local])
        else:
            assert np.array_equal(_np(dc[local]).view(np.int8), codes[local])
            assert np.array_equal(_bits(_np(ds[local])), _bits(scales[local]))
    assert np.allclose(_np(tr), r["trust"], rtol=1e-6, atol=0)
    _close(_np(xd), r["x"], c["x"])
