"""Pins for the oracle's reducer (Section 3.2: the owner of a share
averages every sender's copy of it; weighting by accumulated samples per the
appendix 'Convergence analysis').

* hand-derived dyadic fixtures (exact);
* equal counts over a power-of-two peer count give the arithmetic mean;
* an exact-rational replay of the fused multiply-add chain (one rounding per
  peer, ascending peer order) must reproduce the mean bit for bit;
* float64 brute force within the recursive-summation bound;
* zero-sample peers are never read (their buffers hold NaN)."""

import json
import os

import numpy as np
import pytest

import oracle
from tests.exact import fma_f32


def _enc16(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def test_reduce_golden(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "reduce_examples.json")))
    for c in d["cases"]:
        grads = [np.array([np.nan if v is None else v for v in g], np.float32) for g in c["grads"]]
        codes = [_enc16(g) for g in grads]
        out, _, mean = oracle.reduce(codes, c["counts"], oracle.CODEC_FP16)
        assert mean.tolist() == c["mean"], c["derivation"]
        assert out.tolist() == c["fp16_codes"]


@pytest.mark.parametrize("n_peers", [1, 2, 4, 8, 16])
def test_equal_weights_arithmetic_mean(n_peers):
    rng = np.random.default_rng(n_peers)
    # dyadic values with few significant bits: every partial sum is exact
    g = [(rng.integers(-512, 512, 4096) / 1024.0).astype(np.float32) for _ in range(n_peers)]
    codes = [_enc16(x) for x in g]
    _, _, mean = oracle.reduce(codes, [5] * n_peers, oracle.CODEC_FP16)
    ref = np.mean(np.stack(g).astype(np.float64), axis=0)
    assert np.array_equal(mean.astype(np.float64), ref)


@pytest.mark.parametrize("seed", range(6))
def test_fma_chain_exact_replay(seed):
    rng = np.random.default_rng(200 + seed)
    n = int(rng.integers(1, 9))
    L = 48
    counts = rng.integers(0, 50, n)
    counts[rng.integers(0, n)] = 7
    g = [(rng.standard_normal(L) * 10.0 ** rng.uniform(-5, 1)).astype(np.float32) for _ in range(n)]
    codes = [_enc16(x) for x in g]
    dec = [c.view(np.float16).astype(np.float32) for c in codes]
    w = oracle.weights(counts)
    _, _, mean = oracle.reduce(codes, counts, oracle.CODEC_FP16)
    for e in range(L):
        acc = np.float32(0.0)
        for p in range(n):
            if counts[p]:
                acc = fma_f32(w[p], dec[p][e], acc)
        assert mean[e].view(np.uint32) == np.float32(acc).view(np.uint32), (e, mean[e], acc)


@pytest.mark.parametrize("codec", [oracle.CODEC_FP16, oracle.CODEC_I8])
def test_brute_force_float64_bound(codec):
    rng = np.random.default_rng(31 + codec)
    n, L, block = 13, 3000, 1024
    counts = rng.integers(1, 300, n)
    g = [(rng.standard_normal(L) * 1e-3).astype(np.float32) for _ in range(n)]
    if codec == oracle.CODEC_FP16:
        codes = [_enc16(x) for x in g]
        scales = None
        dec = [c.view(np.float16).astype(np.float64) for c in codes]
    else:
        enc = [oracle.encode_i8(x, block) for x in g]
        codes = [c for c, _ in enc]
        scales = [s for _, s in enc]
        dec = [oracle.decode_i8(c, s, block).astype(np.float64) for c, s in enc]
    out, osc, mean = oracle.reduce(codes, counts, codec, scales, block)
    W = counts.sum()
    exact = sum((counts[p] / W) * dec[p] for p in range(n))
    absw = sum((counts[p] / W) * np.abs(dec[p]) for p in range(n))
    # one weight rounding (2^-24 rel) plus n fma roundings of the running sum
    gamma = (n + 1) * 2.0 ** -24 / (1 - (n + 1) * 2.0 ** -24)
    assert np.all(np.abs(mean - exact) <= gamma * absw + 1e-45)
    # the re-encoded mean is the codec applied to the fp32 mean
    if codec == oracle.CODEC_FP16:
        assert np.array_equal(out, oracle.encode_fp16(mean))
    else:
        c2, s2 = oracle.encode_i8(mean, block)
        assert np.array_equal(out, c2) and np.array_equal(osc, s2)


def test_zero_count_peers_not_read():
    rng = np.random.default_rng(9)
    L = 2048
    g = [(rng.standard_normal(L) * 1e-3).astype(np.float32) for _ in range(5)]
    enc = [oracle.encode_i8(x, 1024) for x in g]
    codes = [c.copy() for c, _ in enc]
    scales = [s.copy() for _, s in enc]
    counts = [10, 0, 20, 0, 30]
    for p in (1, 3):
        codes[p][:] = 99
        scales[p][:] = np.nan
    out, osc, mean = oracle.reduce(codes, counts, oracle.CODEC_I8, scales)
    keep = [0, 2, 4]
    o2, s2, m2 = oracle.reduce([codes[p] for p in keep], [counts[p] for p in keep],
                               oracle.CODEC_I8, [scales[p] for p in keep])
    assert np.isfinite(mean).all()
    assert np.array_equal(mean, m2) and np.array_equal(out, o2) and np.array_equal(osc, s2)


def test_all_zero_counts_error():
    c = [_enc16(np.ones(8)), _enc16(np.ones(8))]
    with pytest.raises(oracle.OracleError) as e:
        oracle.reduce(c, [0, 0], oracle.CODEC_FP16)
    assert e.value.code == oracle.EZERO


def test_empty_shard():
    c = [np.zeros(0, np.uint16)] * 3
    out, _, mean = oracle.reduce(c, [1, 2, 3], oracle.CODEC_FP16)
    assert out.size == 0 and mean.size == 0
