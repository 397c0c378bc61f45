"""Pins for the oracle on non-finite inputs.  Nothing is skipped or
clamped, so IEEE arithmetic alone fixes what comes out, and each pin states
a consequence that can be checked without the oracle's own formulas:

* reduce (fp16): an infinity from one peer with samples makes that element
  that infinity, +inf meeting -inf or a NaN code makes it NaN; a peer with
  zero samples is not read, so its infinities change nothing; every other
  element equals the reduce of the same messages with each non-finite code
  replaced by 0.
* LAMB: an infinite gradient element makes m' and v' infinite there and
  u = inf/inf = NaN, so ||u|| is NaN and the trust ratio falls back to 1;
  every other element of that tensor then equals the unit-trust step of the
  same state with that gradient element set to 0.
* LARS: an infinite gradient element makes ||g|| infinite, so the trust
  ratio is eta*||x|| / inf = 0; every other element of the tensor gets the
  pure momentum decay v' = mu*v (one fp32 product) and x' = x - v'.  A NaN
  gradient element makes ||g|| NaN and the trust ratio 1, as for LAMB."""

import numpy as np

import oracle

F = np.float32
FP16 = oracle.CODEC_FP16


def test_reduce_fp16_nonfinite():
    rng = np.random.default_rng(5)
    n, L = 4, 300
    codes = [oracle.encode_fp16((rng.standard_normal(L) * 0.1).astype(F)) for _ in range(n)]
    counts = np.array([2, 0, 7, 1], np.uint32)
    codes[0][10] = 0x7C00                       # +inf
    codes[2][20] = 0xFC00                       # -inf
    codes[2][30], codes[3][30] = 0x7C00, 0xFC00  # cancel
    codes[3][40] = 0x7E00                       # NaN
    codes[1][50] = 0x7C00                       # zero-sample peer: not read
    _, _, mean = oracle.reduce(codes, counts, FP16)
    assert np.isposinf(mean[10]) and np.isneginf(mean[20])
    assert np.isnan(mean[30]) and np.isnan(mean[40]) and np.isfinite(mean[50])
    clean = [c.copy() for c in codes]
    for c in clean:
        c[(c & 0x7C00) == 0x7C00] = 0  # the non-finite codes only
    _, _, ref = oracle.reduce(clean, counts, FP16)
    keep = np.setdiff1d(np.arange(L), [10, 20, 30, 40])  # 50 included: peer 1 is not read
    assert np.array_equal(mean[keep].view(np.uint32), ref[keep].view(np.uint32))


def test_lamb_infinite_gradient_gives_unit_trust():
    rng = np.random.default_rng(6)
    P = 512
    off = np.array([0, 256, P], np.uint64)
    flags = np.array([3, 3], np.uint8)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    m = (rng.standard_normal(P) * 1e-4).astype(F)
    v = np.square(rng.standard_normal(P) * 1e-3).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    g[300] = np.inf
    cfg = dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, step=4)
    xo, mo, vo, tr = oracle.lamb(x, m, v, g, off, flags, oracle.lamb_cfg(**cfg))
    assert np.isposinf(mo[300]) and np.isposinf(vo[300]) and np.isnan(xo[300])
    assert tr[1] == 1.0 and np.isfinite(tr[0]) and tr[0] != 1.0
    g0 = g.copy()
    g0[300] = 0.0
    xu, mu, vu, _ = oracle.lamb(x, m, v, g0, off, flags, oracle.lamb_cfg(**cfg, force_unit_trust=True))
    rest = np.setdiff1d(np.arange(256, P), [300])
    assert np.array_equal(xo[rest], xu[rest])
    assert np.array_equal(mo[rest], mu[rest]) and np.array_equal(vo[rest], vu[rest])


def test_lamb_nan_gradient_gives_unit_trust():
    P = 64
    x = np.linspace(-1, 1, P).astype(F)
    g = np.full(P, 1e-3, F)
    g[7] = np.nan
    xo, _, _, tr = oracle.lamb(x, np.zeros(P, F), np.zeros(P, F), g, np.array([0, P], np.uint64),
                               np.array([3], np.uint8), oracle.lamb_cfg(lr=1e-2, weight_decay=0.0, step=1))
    assert tr[0] == 1.0 and np.isnan(xo[7]) and np.isfinite(np.delete(xo, 7)).all()


def test_lars_infinite_gradient_gives_zero_trust():
    rng = np.random.default_rng(7)
    P = 256
    x = (rng.standard_normal(P) * 0.02).astype(F)
    v = (rng.standard_normal(P) * 1e-3).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    g[9] = -np.inf
    mu = 0.9
    xo, vo, tr = oracle.lars(x, v, g, np.array([0, P], np.uint64), np.array([3], np.uint8),
                             oracle.lars_cfg(lr=4.8, momentum=mu, trust_coef=1e-3, weight_decay=1e-5))
    assert tr[0] == 0.0 and np.isnan(vo[9]) and np.isnan(xo[9])
    rest = np.delete(np.arange(P), 9)
    v_ref = F(mu) * v[rest]
    assert np.array_equal(vo[rest], v_ref)
    assert np.array_equal(xo[rest], x[rest] - v_ref)


def test_lars_nan_gradient_gives_unit_trust():
    """A NaN gradient element makes ||g|| NaN, so r = 1; every other element
    equals the unit-trust step with that element's gradient set to 0."""
    rng = np.random.default_rng(8)
    P = 256
    x = (rng.standard_normal(P) * 0.02).astype(F)
    v = (rng.standard_normal(P) * 1e-3).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    g[200] = np.nan
    cfg = dict(lr=0.5, momentum=0.9, trust_coef=1e-3, weight_decay=1e-5)
    off, flags = np.array([0, P], np.uint64), np.array([3], np.uint8)
    xo, vo, tr = oracle.lars(x, v, g, off, flags, oracle.lars_cfg(**cfg))
    assert tr[0] == 1.0 and np.isnan(xo[200])
    g0 = g.copy()
    g0[200] = 0.0
    xu, vu, _ = oracle.lars(x, v, g0, off, flags, oracle.lars_cfg(**cfg, force_unit_trust=True))
    rest = np.delete(np.arange(P), 200)
    assert np.array_equal(xo[rest], xu[rest]) and np.array_equal(vo[rest], vu[rest])
