"""Property-based pins of the oracle (hypothesis): the same facts the
fixture and seeded-sample pins check, on inputs that hypothesis draws and
shrinks towards the edges (lengths around block and vector boundaries,
extreme magnitudes, ties, zero and repeated values).

* fp16 encode is IEEE binary16 round-to-nearest-even: numpy's float16
  conversion, an independent implementation, agrees bit for bit.
* int8 absmax, per block of 1024: s = fl(max|x| / 127); the element that
  attains the maximum codes to +-127; |x - q*s| <= s/2 plus the rounding of
  the quotient and of the product while s is a normal number; a block with
  s = 0 (all zero, or max|x| / 127 underflowing) has codes 0.
* Shard bounds: the closed form with exact integers (Python's unbounded
  ints), which tile [0, P) in order, each interior bound a multiple of the
  alignment.
* Peer weights: the correctly rounded fp32 value of the exact rational
  n_p / sum n (fractions.Fraction, rounded half to even by hand).
* The reduce of dyadic inputs is exact: with weights 1/2^k and fp16 codes of
  few significant bits, every fma is exact, so the result equals the exact
  rational sum."""

from fractions import Fraction

import numpy as np
from hypothesis import HealthCheck, example, given, settings
from hypothesis import strategies as st
from hypothesis.extra import numpy as hnp

import oracle

SETTINGS = settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])

finite32 = st.floats(width=32, allow_nan=False, allow_infinity=False)


@SETTINGS
@given(hnp.arrays(np.float32, st.integers(0, 3000), elements=finite32))
def test_fp16_encode_is_ieee_rne(x):
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.encode_fp16(x), ref)


def _f32_rne(fr: Fraction) -> np.float32:
    """fp32 nearest to the positive rational fr (ties to even), normal range."""
    assert fr > 0
    e = fr.numerator.bit_length() - fr.denominator.bit_length()
    if Fraction(2) ** e > fr:
        e -= 1
    # fr in [2^e, 2^(e+1)): 24 significant bits -> unit 2^(e-23)
    unit = Fraction(2) ** (e - 23)
    q, r = divmod(fr / unit, 1)
    q = int(q)
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and q % 2 == 1):
        q += 1
    return np.float32(Fraction(q) * unit)  # q * unit has at most 25 bits: exact in fp32


@SETTINGS
@given(st.lists(st.integers(0, 512), min_size=1, max_size=70).filter(lambda c: sum(c) > 0))
def test_weights_correctly_rounded(counts):
    W = sum(counts)
    w = oracle.weights(np.array(counts, np.uint32))
    for n, got in zip(counts, w):
        want = np.float32(0.0) if n == 0 else _f32_rne(Fraction(n, W))
        assert got.view(np.uint32) == want.view(np.uint32), (n, W, got, want)


@SETTINGS
@given(st.integers(0, 2 ** 40), st.integers(1, 80), st.sampled_from([1, 8, 64, 1024]), st.data())
def test_partition_closed_form(P, n, align, data):
    beta = data.draw(st.one_of(st.none(), st.lists(st.integers(0, 10 ** 6), min_size=n, max_size=n)
                               .filter(lambda b: sum(b) > 0)))
    b = oracle.partition(P, n, None if beta is None else np.array(beta, np.uint64), align)
    w = [1] * n if beta is None else beta
    total = sum(w)
    want = [0] + [align * ((P * sum(w[:k])) // (total * align)) for k in range(1, n)] + [P]
    assert [int(v) for v in b] == want
    assert all(want[k] <= want[k + 1] for k in range(n))
    assert all(v % align == 0 for v in want[1:-1])


block_values = hnp.arrays(np.float32, st.integers(1, 2600),
                          elements=st.floats(-2.0 ** 100, 2.0 ** 100, width=32, allow_nan=False))


TINY = 2.0 ** -149  # the smallest fp32 subnormal


@SETTINGS
@given(block_values)
@example(np.array([TINY], np.float32))                          # a / 127 underflows: s = 0
@example(np.array([63 * TINY, -TINY, 0.0], np.float32))         # the largest block with s = 0
@example(np.array([64 * TINY, 3 * TINY, -64 * TINY], np.float32))  # the smallest nonzero scale
@example(np.array([1e-40, -3e-41, 2e-42], np.float32))          # subnormal scale
@example(np.array([-150 * TINY, 3 * TINY], np.float32))         # a / s = 150: the clamp at -127 decides
def test_int8_codec_properties(x):
    codes, scales = oracle.encode_i8(x, 1024)
    dec = oracle.decode_i8(codes, scales, 1024)
    assert scales.size == (x.size + 1023) // 1024
    for b in range(scales.size):
        blk = x[b * 1024:(b + 1) * 1024].astype(np.float64)
        q = codes[b * 1024:(b + 1) * 1024].astype(np.int64)
        a = float(np.max(np.abs(blk)))
        s = float(scales[b])
        assert s == float(np.float32(np.float32(a) / np.float32(127.0)))
        if s == 0.0:  # all zero, or a / 127 below half the smallest subnormal
            assert a <= 63 * TINY and not q.any()
            continue
        assert np.all(np.abs(q) <= 127)
        i = int(np.argmax(np.abs(blk)))
        assert q[i] != 0 and np.sign(q[i]) == np.sign(blk[i])
        err = np.abs(blk - dec[b * 1024:(b + 1) * 1024].astype(np.float64))
        if s >= 2.0 ** -126:
            assert abs(int(q[i])) == 127  # a / s rounds to 127 when s is normal
            # half a step, plus the rounding of x/s (half an ulp below 128 ->
            # 2^-17 of a step) and of q*s (half an fp32 ulp of the value)
            bound = s / 2 * (1 + 2.0 ** -16) + np.abs(blk) * 2.0 ** -23 + TINY
        else:
            # a subnormal scale carries few significant bits, so a / s may
            # exceed 127 and the clamp may cost more than half a step
            bound = np.full(blk.shape, a + s)
        assert np.all(err <= bound)


@SETTINGS
@given(st.integers(1, 8), st.integers(1, 700), st.data())
def test_reduce_dyadic_is_exact(k_log, n_elem, data):
    """2^k_log peers with equal counts (weights 2^-k exactly) and fp16 codes
    that are small integers times 2^-6: every product and partial sum is
    exactly representable, so the fp32 mean is the exact rational mean."""
    n = 2 ** min(k_log, 6)
    ints = data.draw(hnp.arrays(np.int64, (n, n_elem), elements=st.integers(-64, 64)))
    vals = (ints.astype(np.float64) / 64.0).astype(np.float32)
    codes = [oracle.encode_fp16(v) for v in vals]
    out, _, mean = oracle.reduce(codes, np.full(n, 3, np.uint32), oracle.CODEC_FP16)
    exact = [Fraction(int(ints[:, e].sum()), 64 * n) for e in range(n_elem)]
    assert [Fraction(float(m)) for m in mean] == exact
