"""Pins for the oracle's shard partition and peer weights.

Partition: Section 3.2 / Appendix B (share proportional to throughput), with
the integer reading B_k = align*floor(P*C_k/(C_n*align)).  Checked against
hand-derived fixtures, exact rational brute force and tiling invariants.
Weights: appendix "Convergence analysis" (global mean over all samples),
checked to be the correctly rounded fp32 value of n_p / sum(n)."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.exact import round_f32


def test_partition_golden(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "partition_examples.json")))
    for c in d["cases"]:
        n = len(c["bounds"]) - 1
        b = oracle.partition(c["P"], n, c["beta"], c["align"])
        assert b.tolist() == c["bounds"], c["derivation"]


def _brute(P, beta, align):
    n = len(beta)
    tot = sum(beta)
    out = [0]
    cum = 0
    for k in range(1, n):
        cum += beta[k - 1]
        share = Fraction(P * cum, tot)          # exact cumulative share
        out.append(align * int(share / align))  # floor to the alignment
    out.append(P)
    return out


@pytest.mark.parametrize("seed", range(40))
def test_partition_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    P = int(rng.integers(0, 10 ** 7))
    align = int(rng.choice([1, 8, 64, 1024]))
    beta = rng.integers(0, 1000, size=n)
    if beta.sum() == 0:
        beta[0] = 1
    b = oracle.partition(P, n, beta, align)
    assert b.tolist() == _brute(P, beta.tolist(), align)
    # invariants: tiles [0, P), monotone, interior bounds aligned,
    # each share within align of its exact value
    assert b[0] == 0 and b[-1] == P
    assert np.all(np.diff(b.astype(np.int64)) >= 0)
    assert all(int(x) % align == 0 for x in b[1:-1])
    cum = np.concatenate([[0], np.cumsum(beta)])
    for k in range(1, n):
        exact = Fraction(P * int(cum[k]), int(beta.sum()))
        assert 0 <= exact - int(b[k]) < align


def test_partition_equal_split_large():
    # the 1.07e9-element single-vector case and a product above 2^64
    b = oracle.partition(1 << 30, 8, None, 64)
    assert np.all(np.diff(b.astype(np.int64)) == (1 << 27))
    beta = [2 ** 40] * 4
    b = oracle.partition(2 ** 40, 4, beta, 64)
    assert np.all(np.diff(b.astype(np.int64)) == 2 ** 38)


def test_partition_rejects():
    for args in [(100, 0, None, 8), (100, 3, [0, 0, 0], 8), (100, 2, None, 0)]:
        with pytest.raises(oracle.OracleError):
            oracle.partition(*args)


@pytest.mark.parametrize("seed", range(20))
def test_weights_correctly_rounded(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 80))
    counts = rng.integers(0, 600, size=n)
    if counts.sum() == 0:
        counts[0] = 3
    w = oracle.weights(counts)
    W = int(counts.sum())
    for p in range(n):
        assert w[p] == round_f32(Fraction(int(counts[p]), W))
        if counts[p] == 0:
            assert w[p] == 0


def test_weights_equal_counts_power_of_two():
    w = oracle.weights([7, 7, 7, 7])
    assert np.all(w == np.float32(0.25))


def test_weights_all_zero():
    with pytest.raises(oracle.OracleError) as e:
        oracle.weights([0, 0, 0])
    assert e.value.code == oracle.EZERO
