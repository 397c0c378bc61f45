"""Host-side checks of the C-ABI library (no GPU needed).

* the shared library loads and exports every entry point include/dedloc.h
  declares (and the binding knows each of them);
* the host-only integer entry points (shard bounds, peer weights) agree bit
  for bit with the oracle;
* argument validation rejects bad calls before anything reaches the GPU."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2106_10207_amd import dedloc as D
from paper_2106_10207_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in os.listdir(inc):
        if f.endswith(".h"):
            src = open(os.path.join(inc, f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(dedloc_\w+)\s*\(", src))
    return names


def test_exports_every_declared_symbol():
    names = _declared()
    assert {"dedloc_reduce_shard", "dedloc_encode", "dedloc_decode", "dedloc_lamb_step",
            "dedloc_round"} <= names
    lib = D.load()
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.check_output(["nm", "-D", "--defined-only", D.LIB_PATH]).decode()
    exported = set(re.findall(r"\bT (dedloc_\w+)$", out, flags=re.M))
    assert names <= exported
    assert names == set(D.EXPORTS)


def test_library_is_gfx950():
    # the offload bundle of our own build names its target triple
    data = open(D.LIB_PATH, "rb").read()
    assert b"amdgcn-amd-amdhsa--gfx950" in data


@pytest.mark.parametrize("seed", range(30))
def test_partition_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 70))
    P = int(rng.integers(0, 2 ** 34))
    align = int(rng.choice([1, 8, 64, 1024]))
    beta = None if seed % 3 == 0 else rng.integers(0, 1000, n)
    if beta is not None and beta.sum() == 0:
        beta[0] = 1
    assert np.array_equal(D.dedloc_partition(P, n, beta, align), oracle.partition(P, n, beta, align))


def test_partition_workloads():
    for wl in W.WORKLOADS.values():
        bw = W.bandwidth_weights(wl)
        assert np.array_equal(D.dedloc_partition(wl.P, wl.n_shards, bw, wl.shard_align),
                              oracle.partition(wl.P, wl.n_shards, bw, wl.shard_align))


@pytest.mark.parametrize("seed", range(30))
def test_weights_match_oracle(seed):
    rng = np.random.default_rng(50 + seed)
    c = rng.integers(0, 513, int(rng.integers(1, 65)))
    if c.sum() == 0:
        c[0] = 1
    assert np.array_equal(D.dedloc_weights(c).view(np.uint32), oracle.weights(c).view(np.uint32))


def test_host_errors():
    with pytest.raises(D.DedlocError) as e:
        D.dedloc_weights([0, 0])
    assert e.value.code == D.DEDLOC_ERR_ZERO_WEIGHT
    with pytest.raises(D.DedlocError):
        D.dedloc_weights([1 << 24, 1])
    with pytest.raises(D.DedlocError):
        D.dedloc_partition(10, 0)
    with pytest.raises(D.DedlocError):
        D.dedloc_partition(10, 3, [0, 0, 0])


def test_encoded_bytes():
    assert D.dedloc_encoded_bytes(D.DEDLOC_CODEC_FP16, 0, 1000) == (2000, 0)
    assert D.dedloc_encoded_bytes(D.DEDLOC_CODEC_I8, 1024, 2049) == (2049, 3)
    assert D.dedloc_encoded_bytes(99, 0, 10)[0] == 0


def _call_reduce(codes, scales, counts, n, length, codec, block, out, osc, mean):
    lib = D.load()
    arr = (ctypes.c_void_p * n)(*codes)
    sarr = None if scales is None else (ctypes.c_void_p * n)(*scales)
    cnt = np.asarray(counts, np.uint32)
    return lib.dedloc_reduce_shard(arr, sarr, cnt.ctypes.data, n, length, codec, block, out, osc, mean, None)


def test_reduce_validation_before_launch():
    A = 1 << 20  # fake, 16-byte aligned addresses: never dereferenced on the host
    F = D.DEDLOC_CODEC_FP16
    assert _call_reduce([A, A], None, [0, 0], 2, 64, F, 0, A, None, None) == D.DEDLOC_ERR_ZERO_WEIGHT
    assert _call_reduce([A + 2, A], None, [1, 1], 2, 64, F, 0, A, None, None) == D.DEDLOC_ERR_ALIGN
    assert _call_reduce([A, A], None, [1, 1], 2, 64, F, 0, A + 8, None, None) == D.DEDLOC_ERR_ALIGN
    # too many peers; more than one launch's worth of peers with samples and
    # no fp32 buffer to carry the running sum
    assert _call_reduce([A] * 1025, None, [1] * 1025, 1025, 64, F, 0, A, None, A) == D.DEDLOC_ERR_INVALID_ARG
    assert _call_reduce([A] * 65, None, [1] * 65, 65, 64, F, 0, A, None, None) == D.DEDLOC_ERR_INVALID_ARG
    assert "out_mean" in D.load().dedloc_last_error().decode()
    assert _call_reduce([A, None], None, [1, 1], 2, 64, F, 0, A, None, None) == D.DEDLOC_ERR_INVALID_ARG
    assert _call_reduce([A, A], None, [1, 1], 2, 64, 7, 0, A, None, None) == D.DEDLOC_ERR_INVALID_ARG
    # int8 needs scales and block 1024
    assert _call_reduce([A, A], None, [1, 1], 2, 64, D.DEDLOC_CODEC_I8, 1024, A, A, None) == D.DEDLOC_ERR_INVALID_ARG
    assert _call_reduce([A, A], [A, A], [1, 1], 2, 64, D.DEDLOC_CODEC_I8, 512, A, A, None) == D.DEDLOC_ERR_INVALID_ARG
    # a zero-count peer may be NULL; empty shard is a no-op after validation
    assert _call_reduce([A, None], None, [1, 0], 2, 0, F, 0, A, None, None) == D.DEDLOC_OK
    assert "aligned" in D.load().dedloc_last_error().decode() or True


def test_lamb_validation_before_launch():
    lib = D.load()
    A = 1 << 20
    cfg = D.lamb_cfg(step=1)
    off = np.array([0, 64, 128], np.uint64)
    fl = np.array([3, 3], np.uint8)
    need = D.dedloc_lamb_workspace_bytes(128, off)
    assert need > 0

    def call(P=128, off=off, fl=fl, x=A, ws=A, wsb=need, cfg=cfg, grad=A, codec=0):
        return lib.dedloc_lamb_step(x, A, A, grad, None, codec, 0, P, off.ctypes.data,
                                    None if fl is None else fl.ctypes.data, len(off) - 1,
                                    ctypes.byref(cfg), None, ws, wsb, None)
    assert call(P=129) == D.DEDLOC_ERR_INVALID_ARG                         # offsets do not end at P
    assert call(off=np.array([0, 60, 128], np.uint64)) == D.DEDLOC_ERR_ALIGN  # interior offset % 8
    assert call(off=np.array([0, 100, 64, 128], np.uint64), fl=np.array([3, 3, 3], np.uint8)) == D.DEDLOC_ERR_INVALID_ARG
    assert call(x=A + 4) == D.DEDLOC_ERR_ALIGN
    assert call(wsb=need - 1) == D.DEDLOC_ERR_WORKSPACE
    assert call(ws=A + 128) == D.DEDLOC_ERR_ALIGN
    assert call(cfg=D.lamb_cfg(step=0)) == D.DEDLOC_ERR_INVALID_ARG
    assert call(fl=None) == D.DEDLOC_ERR_INVALID_ARG
    assert call(grad=A + 2) == D.DEDLOC_ERR_ALIGN
    assert call(codec=D.DEDLOC_CODEC_I8) == D.DEDLOC_ERR_INVALID_ARG     # block 0 / no scales


def test_round_validation_before_launch():
    lib = D.load()
    A = 1 << 20
    cfg = D.lamb_cfg(step=1)
    P = 4096
    off = np.array([0, 2048, P], np.uint64)
    fl = np.array([3, 3], np.uint8)
    need = D.dedloc_lamb_workspace_bytes(P, off)
    pc = (ctypes.c_void_p * 2)(A, A)
    cnt = np.array([1, 1], np.uint32)

    def call(bounds, codec=D.DEDLOC_CODEC_FP16, block=0, ps=None, osc=None, local=None):
        b = np.asarray(bounds, np.uint64)
        return lib.dedloc_round(pc, ps, cnt.ctypes.data, 2, b.ctypes.data, len(b) - 1, codec, block,
                                A, osc, A, A, A, P, off.ctypes.data, fl.ctypes.data, 2,
                                ctypes.byref(cfg), None, None, local, A, need, None)
    assert call([0, 100, P - 1]) == D.DEDLOC_ERR_INVALID_ARG          # does not end at P
    assert call([0, 3000, 1000, P]) == D.DEDLOC_ERR_INVALID_ARG       # decreasing
    ps = (ctypes.c_void_p * 2)(A, A)
    assert call([0, 1000, P], D.DEDLOC_CODEC_I8, 1024, ps, A) == D.DEDLOC_ERR_INVALID_ARG  # not on a block
    # 65 peers with samples need out_mean
    pc65 = (ctypes.c_void_p * 65)(*([A] * 65))
    c65 = np.ones(65, np.uint32)
    b = np.array([0, P], np.uint64)
    assert lib.dedloc_round(pc65, None, c65.ctypes.data, 65, b.ctypes.data, 1, D.DEDLOC_CODEC_FP16, 0,
                            A, None, A, A, A, P, off.ctypes.data, fl.ctypes.data, 2,
                            ctypes.byref(cfg), None, None, None, A, need, None) == D.DEDLOC_ERR_INVALID_ARG
    assert "out_mean" in lib.dedloc_last_error().decode()
    # the local peer must be a peer with samples and bring an aligned gradient
    lp = lambda i, g=A: ctypes.byref(D.dedloc_local_peer(i, g))
    assert call([0, P], local=lp(2)) == D.DEDLOC_ERR_INVALID_ARG
    assert call([0, P], local=lp(1, A + 4)) == D.DEDLOC_ERR_ALIGN
    assert call([0, P], local=lp(1, 0)) == D.DEDLOC_ERR_ALIGN
    cnt[1] = 0
    assert call([0, P], local=lp(1)) == D.DEDLOC_ERR_INVALID_ARG
    assert "local" in lib.dedloc_last_error().decode()
    cnt[1] = 1


def test_round_noalloc_validation_before_launch():
    """The no-allocation round validates like dedloc_round and refuses a
    tensor table whose workspace exceeds its static array, before it looks
    the array up on the device or launches anything (no GPU here)."""
    lib = D.load()
    A = 1 << 20
    cfg = D.lamb_cfg(step=1)
    pc = (ctypes.c_void_p * 2)(A, A)
    cnt = np.array([1, 1], np.uint32)

    def call(P, off, bounds=None):
        off = np.asarray(off, np.uint64)
        fl = np.full(len(off) - 1, 3, np.uint8)
        b = np.asarray([0, P] if bounds is None else bounds, np.uint64)
        return lib.dedloc_round_noalloc(pc, None, cnt.ctypes.data, 2, b.ctypes.data, len(b) - 1,
                                        D.DEDLOC_CODEC_FP16, 0, A, None, A, A, A, P, off.ctypes.data,
                                        fl.ctypes.data, len(fl), ctypes.byref(cfg), None, None, None, None)
    assert call(4096, [0, 2048, 4096], [0, 100, 4095]) == D.DEDLOC_ERR_INVALID_ARG
    assert call(4096, [0, 2047, 4096]) == D.DEDLOC_ERR_ALIGN
    # 2^31 + 2^30 elements in two tensors: 3 * 2^20 tiles, 48 MiB of partials
    big = 3 << 30
    assert _ws_expected([big // 2, big // 2]) > D.DEDLOC_NOALLOC_SCRATCH_BYTES
    assert call(big, [0, big // 2, big]) == D.DEDLOC_ERR_WORKSPACE
    assert "static scratch" in lib.dedloc_last_error().decode()
    # the largest vector it takes: partials of 2^20 tiles and the ratios
    assert _ws_expected([(1 << 31) - 2048 * 256]) <= D.DEDLOC_NOALLOC_SCRATCH_BYTES


def _ws_expected(sizes, tile=2048):
    tiles = sum((n + tile - 1) // tile for n in sizes)
    r = lambda v: (v + 255) // 256 * 256
    # two fp64 sums per tile, one tagged 8-byte ratio per tensor, the tag counter
    return r(tiles * 16) + r(len(sizes) * 8) + 256


@pytest.mark.parametrize("sizes", [
    [3_000_000_000, 3_000_000_000, 8],       # launches split where a chunk would span 2^32 elements
    [64] * 500 + [100],                      # more tensors than one launch describes
    [0, 0, 8, 0],                            # empty tensors own no tiles
])
def test_workspace_bytes_large_tables(sizes):
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    assert D.dedloc_lamb_workspace_bytes(int(off[-1]), off) == _ws_expected(sizes)


def test_workspace_rejects_huge_tensor():
    off = np.array([0, 1 << 32], np.uint64)
    with pytest.raises(D.DedlocError):
        D.dedloc_lamb_workspace_bytes(1 << 32, off)


def test_accumulate_finalize_validation():
    lib = D.load()
    A = 1 << 20
    assert lib.dedloc_accumulate(A, A, 7, 64, 1.0, None) == D.DEDLOC_ERR_INVALID_ARG      # codec
    assert lib.dedloc_accumulate(A + 4, A, 0, 64, 1.0, None) == D.DEDLOC_ERR_ALIGN
    assert lib.dedloc_accumulate(A, A, 0, 0, 1.0, None) == D.DEDLOC_OK                    # empty
    assert lib.dedloc_finalize(A, 64, 0, 1, 0, A, None, 1, None) == D.DEDLOC_ERR_ZERO_WEIGHT
    assert lib.dedloc_finalize(A, 64, (1 << 24) + 1, 1, 0, A, None, 1, None) == D.DEDLOC_ERR_INVALID_ARG
    assert lib.dedloc_finalize(A, 64, 5, 2, 1024, A, None, 1, None) == D.DEDLOC_ERR_INVALID_ARG  # no scales
    assert lib.dedloc_finalize(A, 64, 5, 1, 0, A + 2, None, 1, None) == D.DEDLOC_ERR_ALIGN


def test_group_allreduce_validation():
    lib = D.load()
    A = 1 << 20
    pc = (ctypes.c_void_p * 3)(A, A, A)
    cnt = np.array([1, 2, 3], np.uint32)
    po = np.zeros(3, np.uint32)
    nout = ctypes.c_uint32(0)
    call = lambda m, ws=A, wsb=1 << 30, out=A: lib.dedloc_group_allreduce(
        pc, None, cnt.ctypes.data, 3, m, 64, D.DEDLOC_CODEC_FP16, 0, out, None, po.ctypes.data,
        ctypes.byref(nout), ws, wsb, None)
    assert call(1) == D.DEDLOC_ERR_INVALID_ARG             # group size < 2
    assert call(2, out=A + 16) == D.DEDLOC_ERR_ALIGN       # outputs on 256-byte boundaries
    assert call(2, wsb=0) == D.DEDLOC_ERR_WORKSPACE
    assert lib.dedloc_group_allreduce_workspace_bytes(3, 2, 64, D.DEDLOC_CODEC_FP16, 0) == 2 * 2 * 256
    assert lib.dedloc_group_allreduce_workspace_bytes(1025, 2, 64, D.DEDLOC_CODEC_FP16, 0) == 0
    assert lib.dedloc_group_allreduce_workspace_bytes(8, 65, 64, D.DEDLOC_CODEC_FP16, 0) == 0
    assert lib.dedloc_group_allreduce_workspace_bytes(1024, 32, 64, D.DEDLOC_CODEC_FP16, 0) == 2 * 32 * 256


def test_workspace_clear_validation():
    lib = D.load()
    A = 1 << 20
    assert lib.dedloc_workspace_clear(None, 256, None) == D.DEDLOC_ERR_INVALID_ARG
    assert lib.dedloc_workspace_clear(A + 2, 256, None) == D.DEDLOC_ERR_INVALID_ARG   # alignment
    assert lib.dedloc_workspace_clear(A, 255, None) == D.DEDLOC_ERR_INVALID_ARG       # not whole words
    assert lib.dedloc_workspace_clear(A, 0, None) == D.DEDLOC_OK                      # nothing to clear


def test_codec_and_weights_validation():
    lib = D.load()
    A = 1 << 20
    F, I8 = D.DEDLOC_CODEC_FP16, D.DEDLOC_CODEC_I8
    assert lib.dedloc_encode(A, 64, 7, 0, A, None, None) == D.DEDLOC_ERR_INVALID_ARG        # codec
    assert lib.dedloc_encode(A, 64, I8, 512, A, A, None) == D.DEDLOC_ERR_INVALID_ARG       # block
    assert lib.dedloc_encode(None, 64, F, 0, A, None, None) == D.DEDLOC_ERR_INVALID_ARG
    assert lib.dedloc_encode(A, 64, I8, 1024, A, None, None) == D.DEDLOC_ERR_INVALID_ARG   # no scales
    assert lib.dedloc_encode(A + 4, 64, F, 0, A, None, None) == D.DEDLOC_ERR_ALIGN
    assert lib.dedloc_encode(A, 64, I8, 1024, A, A + 2, None) == D.DEDLOC_ERR_ALIGN
    assert lib.dedloc_encode(None, 0, F, 0, None, None, None) == D.DEDLOC_OK               # empty
    assert lib.dedloc_decode(A, None, 64, F, 0, None, None) == D.DEDLOC_ERR_INVALID_ARG
    assert lib.dedloc_decode(A + 8, None, 64, F, 0, A, None) == D.DEDLOC_ERR_ALIGN
    assert lib.dedloc_decode(A, None, 64, I8, 1024, A, None) == D.DEDLOC_ERR_INVALID_ARG   # no scales
    w = np.zeros(2, np.float32)
    c = np.array([1, 2], np.uint32)
    assert lib.dedloc_weights(None, 2, w.ctypes.data) == D.DEDLOC_ERR_INVALID_ARG
    assert lib.dedloc_weights(c.ctypes.data, 0, w.ctypes.data) == D.DEDLOC_ERR_INVALID_ARG
    big = np.array([1 << 24, 1], np.uint32)
    assert lib.dedloc_weights(big.ctypes.data, 2, w.ctypes.data) == D.DEDLOC_ERR_INVALID_ARG
