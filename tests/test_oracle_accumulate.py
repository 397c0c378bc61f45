"""Pins for the oracle's local accumulation and finalize (Section 3.1:
peers accumulate gradients until the collaboration reaches the target
batch; the peer's mean gradient is then sent).

* accumulate replays exactly as one correctly rounded fma per element and
  batch (exact-rational replay);
* dyadic batches sum exactly; float64 within the summation bound;
* finalize = the pinned codec applied to acc / count (correctly rounded
  division), and resets the accumulator."""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.exact import fma_f32, round_f32

F = np.float32


def test_accumulate_exact_replay():
    rng = np.random.default_rng(1)
    acc = np.zeros(40, F)
    ref = np.zeros(40, F)
    for b in (3, 17, 1, 250):
        g = (rng.standard_normal(40) * 10.0 ** rng.uniform(-4, 1)).astype(F)
        acc = oracle.accumulate(acc, g, b)
        ref = np.array([fma_f32(F(b), g[i], ref[i]) for i in range(40)], F)
        assert np.array_equal(acc.view(np.uint32), ref.view(np.uint32))


def test_accumulate_fp16_and_dyadic_exact():
    rng = np.random.default_rng(2)
    gs = [(rng.integers(-512, 512, 4096) / 256.0).astype(F) for _ in range(6)]
    bs = [1, 2, 4, 8, 16, 32]
    acc = np.zeros(4096, F)
    for g, b in zip(gs, bs):
        acc = oracle.accumulate(acc, g.astype(np.float16).view(np.uint16), b)
    ref = sum(b * g.astype(np.float64) for g, b in zip(gs, bs))
    assert np.array_equal(acc.astype(np.float64), ref)


@pytest.mark.parametrize("codec", [oracle.CODEC_FP16, oracle.CODEC_I8])
def test_finalize_is_codec_of_mean(codec):
    rng = np.random.default_rng(3)
    acc = (rng.standard_normal(5000) * 0.3).astype(F)
    count = 37
    codes, scales, after = oracle.finalize(acc, count, codec)
    mean = np.array([round_f32(Fraction(float(a)) / count) for a in acc], F)
    assert np.array_equal(mean, (acc / F(count)).astype(F))  # numpy's fp32 division is correctly rounded
    if codec == oracle.CODEC_FP16:
        assert np.array_equal(codes, oracle.encode_fp16(mean))
    else:
        c, s = oracle.encode_i8(mean, 1024)
        assert np.array_equal(codes, c) and np.array_equal(scales, s)
    assert not after.any()
    _, _, kept = oracle.finalize(acc, count, codec, reset=False)
    assert np.array_equal(kept, acc)


def test_finalize_errors():
    with pytest.raises(oracle.OracleError):
        oracle.finalize(np.ones(4, F), 0, oracle.CODEC_FP16)
