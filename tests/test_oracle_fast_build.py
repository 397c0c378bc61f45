"""The CPU baseline's build of the oracle (-O3 -march=native, OpenMP element
loops on) computes the same bits as the plain build, single-threaded and on
several threads: whole fp16 and int8 rounds, LAMB and LARS (CPU only)."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_RUN = r"""
import sys, numpy as np, oracle
from paper_2106_10207_amd import workloads as W
lib, nthreads, out = sys.argv[1], int(sys.argv[2]), sys.argv[3]
oracle.use_library(lib)
if nthreads:
    assert oracle.threads(nthreads) == nthreads
res = {}
base = W.scaled(W.ALBERT_LARGE, "fast_build", [30000 * 8, 128, 4096 * 3 + 8, 1024, 77 * 8],
                ["w", "g", "w", "b", "w"], n_peers=6)
for wl in (base, W.scaled(W.ALBERT_XLARGE, "fast_build_i8", [8192 * 3, 128, 10000, 7], ["w", "g", "w", "b"],
                          n_peers=9, n_zero_peers=2)):
    grads = [W.peer_gradient(wl, p).numpy() for p in range(wl.n_peers)]
    counts = W.sample_counts(wl)
    if wl.codec == "fp16":
        codes, scales, codec = [oracle.encode_fp16(g) for g in grads], None, oracle.CODEC_FP16
    else:
        enc = [oracle.encode_i8(g, 1024) for g in grads]
        codes, scales, codec = [c for c, _ in enc], [s for _, s in enc], oracle.CODEC_I8
    bounds = oracle.partition(wl.P, wl.n_shards, W.bandwidth_weights(wl), wl.shard_align)
    x, m, v = (t.numpy() for t in W.optimizer_state(wl))
    cfg = oracle.lamb_cfg(wl.lr, wl.beta1, wl.beta2, wl.eps, wl.weight_decay, step=wl.step)
    r = oracle.round_(codes, counts, bounds, codec, x, m, v, wl.offsets(), wl.flags(), cfg, scales, 1024)
    for k, a in r.items():
        if a is not None:
            res[f"{wl.name}_lamb_{k}"] = np.asarray(a)
    lc = oracle.lars_cfg(wl.lars_lr, wl.lars_momentum, wl.lars_trust_coef, wl.lars_weight_decay)
    r = oracle.round_lars(codes, counts, bounds, codec, x, m, wl.offsets(), wl.flags(), lc, scales, 1024)
    for k, a in r.items():
        if a is not None:
            res[f"{wl.name}_lars_{k}"] = np.asarray(a)
    for p, c in enumerate(codes):
        res[f"{wl.name}_codes_{p}"] = np.asarray(c)
np.savez(out, **res)
"""


def _run(lib, nthreads, out):
    subprocess.check_call([sys.executable, "-c", _RUN, lib, str(nthreads), out], cwd=ROOT,
                          env=dict(os.environ, PYTHONPATH=ROOT))


def test_fast_build_is_bit_identical(tmp_path):
    import numpy as np
    import oracle
    plain = os.path.join(ROOT, "oracle", "liboracle.so")
    fast = oracle.build_fast(str(tmp_path / "liboracle_fast.so"))
    outs = []
    for lib, nt in ((plain, 0), (fast, 1), (fast, 7)):
        out = str(tmp_path / f"r_{os.path.basename(lib)}_{nt}.npz")
        _run(lib, nt, out)
        outs.append(np.load(out))
    ref = outs[0]
    for other in outs[1:]:
        assert set(other.files) == set(ref.files)
        for k in ref.files:
            assert np.array_equal(ref[k].view(np.uint8), other[k].view(np.uint8)), k


if __name__ == "__main__":
    pytest.main([__file__, "-q"])
