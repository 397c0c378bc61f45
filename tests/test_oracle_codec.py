"""Pins for the oracle's wire codecs.

fp16: IEEE binary16 round-to-nearest-even; numpy's float16 conversion is an
independent library implementation of the same standard, so encode must match
it bit for bit on every finite input and decode on all 2^16 patterns.
int8 absmax: hand-derived fixture, an independent numpy fp32 implementation,
and the half-step error bound."""

import json
import os

import numpy as np
import pytest

import oracle


def test_fp16_decode_all_patterns():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    d = oracle.decode_fp16(h)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(d[~nan].view(np.uint32), ref[~nan].view(np.uint32))
    assert np.isnan(d[nan]).all()


def _np_f16(x):
    with np.errstate(over="ignore"):
        return x.astype(np.float16).view(np.uint16)


@pytest.mark.parametrize("scale", [1e-9, 1e-6, 1e-3, 1.0, 1e3, 7e4])
def test_fp16_encode_random(scale):
    rng = np.random.default_rng(int(scale * 1e9) % 97)
    x = (rng.standard_normal(200_000) * scale).astype(np.float32)
    assert np.array_equal(oracle.encode_fp16(x), _np_f16(x))


def test_fp16_encode_boundaries():
    # every fp16 value, the midpoints between neighbours and one fp32 ulp
    # either side of each midpoint: exercises ties-to-even, subnormals and the
    # overflow threshold
    h = np.arange(0, 0x7c00, dtype=np.uint16)
    f = h.view(np.float16).astype(np.float64)
    mids = (f[:-1] + f[1:]) / 2
    mid32 = mids.astype(np.float32)
    cand = np.concatenate([f.astype(np.float32), mid32,
                           np.nextafter(mid32, np.float32(np.inf)),
                           np.nextafter(mid32, np.float32(0)),
                           np.float32([65504, 65519.996, 65520, 65536, 1e30, np.inf,
                                       1e-45, 1e-38, 2.0 ** -25, 2.0 ** -24])])
    cand = np.concatenate([cand, -cand])
    assert np.array_equal(oracle.encode_fp16(cand), _np_f16(cand))


def test_fp16_encode_nan():
    x = np.array([np.nan, -np.nan], dtype=np.float32)
    d = oracle.decode_fp16(oracle.encode_fp16(x))
    assert np.isnan(d).all()


def test_fp16_golden(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "codec_examples.json")))
    for c in d["fp16_cases"]:
        x = np.array(c["x"], dtype=np.float32)
        assert oracle.encode_fp16(x).tolist() == c["codes"], c["derivation"]


def test_i8_golden(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "codec_examples.json")))
    for c in d["int8_cases"]:
        codes, scales = oracle.encode_i8(np.array(c["x"], np.float32), c["block"])
        assert codes.tolist() == c["codes"], c["derivation"]
        assert scales.tolist() == c["scales"]


def _np_i8(x, block):
    """Independent numpy fp32 statement of the int8 absmax codec."""
    n = x.size
    nb = (n + block - 1) // block
    codes = np.zeros(n, np.int8)
    scales = np.zeros(nb, np.float32)
    for b in range(nb):
        blk = x[b * block:(b + 1) * block]
        a = np.max(np.abs(blk))
        if a == 0:
            continue
        s = np.float32(a) / np.float32(127.0)
        scales[b] = s
        q = np.rint(blk / s)          # fp32 division, ties-to-even rint
        codes[b * block:(b + 1) * block] = np.clip(q, -127, 127).astype(np.int8)
    return codes, scales


@pytest.mark.parametrize("n,block", [(1, 1024), (1023, 1024), (5000, 1024), (777, 64), (4096, 1024)])
def test_i8_matches_numpy(n, block):
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    x[rng.random(n) < 0.01] *= 100
    if n > 2000:
        x[1024:2048] = 0  # an all-zero block
    c, s = oracle.encode_i8(x, block)
    rc, rs = _np_i8(x, block)
    assert np.array_equal(c, rc)
    assert np.array_equal(s.view(np.uint32), rs.view(np.uint32))


def test_i8_error_bound_and_extremes():
    rng = np.random.default_rng(7)
    block = 1024
    x = (rng.standard_normal(64 * block) * np.repeat(10.0 ** rng.uniform(-8, 3, 64), block)).astype(np.float32)
    c, s = oracle.encode_i8(x, block)
    d = oracle.decode_i8(c, s, block)
    srep = np.repeat(s, block)
    # |x - dec| <= s/2 plus the roundings of x/s and q*s (a few fp32 ulps of x)
    err = np.abs(x.astype(np.float64) - d.astype(np.float64))
    bound = srep.astype(np.float64) / 2 + 4 * np.spacing(np.abs(x)).astype(np.float64)
    assert np.all(err <= bound)
    # the element of largest magnitude in every block maps to +-127
    for b in range(64):
        blk = x[b * block:(b + 1) * block]
        i = int(np.argmax(np.abs(blk)))
        assert abs(int(c[b * block + i])) == 127
    assert c.min() >= -127


def test_i8_zero_block():
    c, s = oracle.encode_i8(np.zeros(2500, np.float32), 1024)
    assert not c.any() and not s.any()
    assert not oracle.decode_i8(c, s, 1024).any()
