"""Pins for the oracle's group (Moshpit) all-reduce (Section 3.2 "Node
failures"; Appendix C: groups of m, the global average after
ceil(log_m n) iterations).

* one group (m >= n) is exactly the plain reducer;
* after ceil(log_m n) iterations every peer holds the global sample-weighted
  mean, up to the wire codec's rounding per iteration (float64 reference);
* one iteration fewer does not reach it (peers in different groups still
  disagree by far more than the rounding);
* peers of the same final group hold the same message; zero-sample peers
  and the empty slots of an incomplete grid change nothing;
* groups of m = 2 (Section 3.2's decentralized-SGD case): every iteration
  averages disjoint pairs of peers, and after the first one each pair holds
  exactly what the plain reducer makes of the two messages."""

import numpy as np
import pytest

import oracle

F = np.float32


def _msgs(n, L, seed, codec, scale=1e-3, spread=False):
    rng = np.random.default_rng(seed)
    g = []
    for p in range(n):
        mu = (p - n / 2) * 1e-3 if spread else 0.0   # peers differ systematically
        g.append((mu + rng.standard_normal(L) * scale).astype(F))
    if codec == oracle.CODEC_FP16:
        return g, [oracle.encode_fp16(x) for x in g], None
    enc = [oracle.encode_i8(x, 1024) for x in g]
    return g, [c for c, _ in enc], [s for _, s in enc]


def _dec(codec, codes, scales):
    return oracle.decode_fp16(codes) if codec == oracle.CODEC_FP16 else oracle.decode_i8(codes, scales, 1024)


@pytest.mark.parametrize("codec", [oracle.CODEC_FP16, oracle.CODEC_I8])
def test_single_group_is_plain_reduce(codec):
    n, L = 7, 3000
    _, codes, scales = _msgs(n, L, 1, codec)
    counts = np.array([5, 0, 9, 1, 30, 2, 7], np.uint32)
    out, osc, peer_out = oracle.group_allreduce(codes, counts, 8, codec, scales)
    rc, rs, _ = oracle.reduce(codes, counts, codec, scales)
    assert out.shape[0] == 1 and np.array_equal(out[0], rc)
    if codec == oracle.CODEC_I8:
        assert np.array_equal(osc[0], rs)
    assert np.all(peer_out == 0)


@pytest.mark.parametrize("codec", [oracle.CODEC_FP16, oracle.CODEC_I8])
@pytest.mark.parametrize("n,m", [(8, 2), (9, 3), (64, 8), (10, 3), (64, 4), (5, 2), (30, 4)])
def test_reaches_global_weighted_mean(codec, n, m):
    L = 2048 + 77
    g, codes, scales = _msgs(n, L, 100 + n * m, codec, spread=True)
    rng = np.random.default_rng(n + m)
    counts = rng.integers(0, 200, n).astype(np.uint32)
    counts[0] = 50
    out, osc, peer_out = oracle.group_allreduce(codes, counts, m, codec, scales)
    d = oracle.group_iterations(n, m)
    assert m ** (d - 1) < n <= m ** d or (d == 1 and n <= m)
    dec = [_dec(codec, codes[p], None if scales is None else scales[p]).astype(np.float64) for p in range(n)]
    W = counts.sum()
    ref = sum(counts[p] / W * dec[p] for p in range(n))
    amax = max(np.max(np.abs(x)) for x in dec)
    # each iteration re-encodes: half a wire step of the largest value, plus
    # the fp32 accumulation; int8's step is max/127 per 1024-block
    step = 2.0 ** -11 if codec == oracle.CODEC_FP16 else 1.0 / 127
    tol = d * (step * amax) + 1e-6 * amax
    for p in range(n):
        got = _dec(codec, out[peer_out[p]], None if osc is None else osc[peer_out[p]])
        assert np.max(np.abs(got - ref)) <= tol, (p, np.max(np.abs(got - ref)), tol)


@pytest.mark.parametrize("n,m", [(8, 2), (27, 3), (64, 8)])
def test_one_iteration_fewer_is_not_global(n, m):
    L = 1024
    g, codes, _ = _msgs(n, L, 7, oracle.CODEC_FP16, scale=1e-5, spread=True)
    counts = np.full(n, 10, np.uint32)
    d = oracle.group_iterations(n, m)
    out, _, peer_out = oracle.group_allreduce(codes, counts, m, oracle.CODEC_FP16, iters=d - 1) if d > 1 else (None, None, None)
    if d == 1:
        return
    vals = np.array([oracle.decode_fp16(out[peer_out[p]]).mean() for p in range(n)])
    # the systematic per-peer offsets are still visible: not yet the global mean
    assert vals.max() - vals.min() > 1e-3
    out, _, peer_out = oracle.group_allreduce(codes, counts, m, oracle.CODEC_FP16)
    vals = np.array([oracle.decode_fp16(out[peer_out[p]]).mean() for p in range(n)])
    assert vals.max() - vals.min() < 1e-5


def test_same_final_group_same_message_and_zero_peers():
    n, m, L = 16, 2, 512
    _, codes, _ = _msgs(n, L, 9, oracle.CODEC_FP16)
    counts = np.arange(n, dtype=np.uint32) % 5
    counts[3] = 0
    out, _, peer_out = oracle.group_allreduce(codes, counts, m, oracle.CODEC_FP16)
    # zero-sample peers are never read: poisoning them changes nothing
    poisoned = [c.copy() for c in codes]
    for p in np.flatnonzero(counts == 0):
        poisoned[p][:] = 0x7E00
    out2, _, peer_out2 = oracle.group_allreduce(poisoned, counts, m, oracle.CODEC_FP16)
    assert np.array_equal(out, out2) and np.array_equal(peer_out, peer_out2)
    assert out.shape[0] == m ** (oracle.group_iterations(n, m) - 1)
    for a in range(n):
        for b in range(n):
            if peer_out[a] == peer_out[b]:
                assert np.array_equal(out[peer_out[a]], out[peer_out[b]])


def test_errors():
    codes = [np.zeros(8, np.uint16)] * 3
    with pytest.raises(oracle.OracleError):
        oracle.group_allreduce(codes, [0, 0, 0], 2, oracle.CODEC_FP16)
    with pytest.raises(oracle.OracleError):
        oracle.group_allreduce(codes, [1, 1, 1], 1, oracle.CODEC_FP16)


@pytest.mark.parametrize("codec", [oracle.CODEC_FP16, oracle.CODEC_I8])
def test_group_size_two_is_pairwise_gossip(codec):
    """Section 3.2: with m = 2 all communication happens between pairs of
    nodes, as in D-PSGD.  Iteration 1 groups the slots that differ in the
    lowest base-2 digit: peers 2g and 2g+1 both end with the pair's
    sample-weighted average, which is the plain reducer on those two
    messages (a peer without samples contributes nothing)."""
    n, L = 8, 3000
    _, codes, scales = _msgs(n, L, 5, codec, spread=True)
    counts = np.array([3, 9, 1, 1, 0, 4, 7, 2], np.uint32)
    out, osc, peer_out = oracle.group_allreduce(codes, counts, 2, codec, scales, iters=1)
    assert out.shape[0] == n // 2
    for g in range(n // 2):
        pair = [2 * g, 2 * g + 1]
        rc, rs, _ = oracle.reduce([codes[i] for i in pair], counts[pair], codec,
                                  None if scales is None else [scales[i] for i in pair])
        assert np.array_equal(out[g], rc), g
        if codec == oracle.CODEC_I8:
            assert np.array_equal(osc[g], rs), g
        assert peer_out[2 * g] == peer_out[2 * g + 1] == g
    # pairs are still far apart after one iteration: gossip, not yet the average
    dec = [_dec(codec, out[g], None if osc is None else osc[g]) for g in range(n // 2)]
    assert np.max(np.abs(dec[0] - dec[3])) > 1e-3
