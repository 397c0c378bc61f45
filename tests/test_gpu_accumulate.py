"""GPU parity of the sender side: dedloc_accumulate (micro-batch gradients
summed until the target batch, Section 3.1) and dedloc_finalize (the peer's
mean gradient encoded for the exchange) against the oracle, bit for bit."""

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from tests.test_gpu_parity import DEV, _bits, _i8, _np, _u16, _up

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
F = np.float32


@pytest.mark.parametrize("n", [1, 8, 2049, 100_003])
@pytest.mark.parametrize("fp16", [False, True])
def test_accumulate(n, fp16):
    rng = np.random.default_rng(n + fp16)
    acc_h = (rng.standard_normal(n) * 1e-2).astype(F)
    acc_d = _up(acc_h)
    for b in (7, 1, 32, 250):
        g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-4, 0)).astype(F)
        gh = oracle.encode_fp16(g) if fp16 else g
        acc_h = oracle.accumulate(acc_h, gh, b)
        D.dedloc_accumulate(acc_d, _up(gh.view(np.int16)) if fp16 else _up(gh), b)
    assert np.array_equal(_bits(_np(acc_d)), _bits(acc_h))


@pytest.mark.parametrize("n", [1, 1023, 1025, 4096 * 3 + 9, 300_000])
@pytest.mark.parametrize("codec", [D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8])
@pytest.mark.parametrize("reset", [True, False])
def test_finalize(n, codec, reset):
    rng = np.random.default_rng(n * 3 + codec)
    acc = (rng.standard_normal(n) * 0.5).astype(F)
    if n > 5000:
        acc[2048:3072] = 0.0
    count = 1237
    oc, osc, after = oracle.finalize(acc, count, codec, reset=reset)
    acc_d = _up(acc)
    codes, scales = D.dedloc_finalize(acc_d, count, codec, reset=reset)
    if codec == D.DEDLOC_CODEC_FP16:
        assert np.array_equal(_u16(codes), oc)
    else:
        assert np.array_equal(_i8(codes), oc)
        assert np.array_equal(_bits(_np(scales)), _bits(osc))
    assert np.array_equal(_bits(_np(acc_d)), _bits(after))


def test_finalize_errors():
    acc = torch.zeros(16, device=DEV)
    with pytest.raises(D.DedlocError) as e:
        D.dedloc_finalize(acc, 0, D.DEDLOC_CODEC_FP16)
    assert e.value.code == D.DEDLOC_ERR_ZERO_WEIGHT
