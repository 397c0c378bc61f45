"""CPU oracle for the DeDLOC averaging round: TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It wraps `dedloc_oracle.c` (plain sequential C, no fused
multiply-add except where the definition asks for one) with numpy arrays.
Nothing here touches the GPU library or shares code with it.

Functions and the passages they follow:
  partition  - Section 3.2 / Appendix B (shares proportional to throughput)
  weights    - appendix "Convergence analysis" (mean over all samples)
  encode_*/decode_* - the build's wire codecs (fp16 RNE; int8 absmax/127)
  reduce     - Section 3.2 (the owner of a share averages every sender's copy of it)
  lamb       - Section 3.1 and the XL appendix (LAMB, layer-wise trust ratio)
  lars       - Section 4.1 (SwAV trains with LARS: layer-wise rate scaling)
  round      - Sections 3.1-3.2 (reduce-scatter, gather, one optimizer step)
  round_lars - the same round with the LARS step
  group_allreduce - Section 3.2 "Node failures" / Appendix C (group averaging)
  accumulate/finalize - Section 3.1 (local accumulation to the target batch)
  lp (module)     - Appendix B (the load-balancing LP, solved by HiGHS)
  groups (module) - Appendix C (the group size of the group all-reduce)
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dedloc_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, EZERO = 0, -1, -3
CODEC_FP16, CODEC_I8 = 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                               "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-Wextra", "-Werror",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def build_fast(path: Optional[str] = None) -> str:
    """The CPU baseline's build of the same source: -O3 for this host's CPU
    (-march=native) with the OpenMP element loops on.  Still no contraction
    and no fast-math, so every result is the same bits as the plain build,
    for any thread count."""
    path = path or os.path.join(_HERE, "liboracle_fast.so")
    tmp = path + ".tmp"
    subprocess.check_call(["gcc", "-O3", "-march=native", "-fopenmp", "-std=c11", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fno-fast-math",
                           "-Wall", "-Wextra", "-Werror",
                           _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, path)
    return path


def use_library(path: str) -> None:
    """Call a given build of the oracle (for example build_fast()'s) from now on."""
    global _LIB, _lib
    _LIB, _lib = path, None


def threads(n: int = 0) -> int:
    """Threads of the OpenMP element loops (n > 0 sets them); 1 for the plain build."""
    return int(_L().oracle_threads(n))


class _LambCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("step", ctypes.c_uint64),
                ("bias_correction", ctypes.c_int32),
                ("force_unit_trust", ctypes.c_int32)]


class _LarsCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("trust_coef", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("force_unit_trust", ctypes.c_int32)]


_lib = None


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = ctypes.CDLL(_LIB)
        vp, sz = ctypes.c_void_p, ctypes.c_size_t
        u32, u64 = ctypes.c_uint32, ctypes.c_uint64
        _lib.oracle_threads.argtypes = [ctypes.c_int]
        _lib.oracle_partition.argtypes = [u64, u32, vp, u32, vp]
        _lib.oracle_weights.argtypes = [vp, u32, vp]
        _lib.oracle_encode_fp16.argtypes = [vp, sz, vp]
        _lib.oracle_decode_fp16.argtypes = [vp, sz, vp]
        _lib.oracle_encode_i8.argtypes = [vp, sz, u32, vp, vp]
        _lib.oracle_decode_i8.argtypes = [vp, vp, sz, u32, vp]
        _lib.oracle_reduce.argtypes = [vp, vp, vp, u32, sz, ctypes.c_int, u32,
                                       vp, vp, vp, vp]
        _lib.oracle_lamb.argtypes = [vp, vp, vp, vp, u64, vp, vp, u32,
                                     ctypes.POINTER(_LambCfg), vp, vp]
        _lib.oracle_round.argtypes = [vp, vp, vp, u32, vp, u32, ctypes.c_int, u32,
                                      vp, vp, vp, vp, vp, u64, vp, vp, u32,
                                      ctypes.POINTER(_LambCfg), vp, vp, vp]
        _lib.oracle_lars.argtypes = [vp, vp, vp, u64, vp, vp, u32, ctypes.POINTER(_LarsCfg), vp]
        _lib.oracle_round_lars.argtypes = [vp, vp, vp, u32, vp, u32, ctypes.c_int, u32,
                                           vp, vp, vp, vp, u64, vp, vp, u32,
                                           ctypes.POINTER(_LarsCfg), vp, vp, vp]
        _lib.oracle_accumulate.argtypes = [vp, vp, ctypes.c_int, sz, ctypes.c_float]
        _lib.oracle_finalize.argtypes = [vp, sz, u32, ctypes.c_int, u32, vp, vp, ctypes.c_int, vp]
        _lib.oracle_group_allreduce.argtypes = [vp, vp, vp, u32, u32, sz, ctypes.c_int, u32, u32,
                                                vp, vp, vp, vp, vp, vp, vp]
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle returned status {code}")
        self.code = code


def _check(rc):
    if rc != OK:
        raise OracleError(rc)


def partition(P: int, n: int, beta: Optional[Sequence[int]] = None, align: int = 64) -> np.ndarray:
    b = None if beta is None else _c(beta, np.uint64)
    out = np.zeros(n + 1, dtype=np.uint64)
    _check(_L().oracle_partition(P, n, _p(b), align, _p(out)))
    return out


def weights(counts) -> np.ndarray:
    c = _c(counts, np.uint32)
    w = np.zeros(len(c), dtype=np.float32)
    _check(_L().oracle_weights(_p(c), len(c), _p(w)))
    return w


def encode_fp16(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.size, dtype=np.uint16)
    _L().oracle_encode_fp16(_p(x), x.size, _p(out))
    return out


def decode_fp16(codes) -> np.ndarray:
    c = _c(codes, np.uint16)
    out = np.empty(c.size, dtype=np.float32)
    _L().oracle_decode_fp16(_p(c), c.size, _p(out))
    return out


def encode_i8(x, block: int = 1024):
    x = _c(x, np.float32)
    codes = np.empty(x.size, dtype=np.int8)
    scales = np.empty((x.size + block - 1) // block, dtype=np.float32)
    _L().oracle_encode_i8(_p(x), x.size, block, _p(codes), _p(scales))
    return codes, scales


def decode_i8(codes, scales, block: int = 1024) -> np.ndarray:
    c = _c(codes, np.int8)
    s = _c(scales, np.float32)
    out = np.empty(c.size, dtype=np.float32)
    _L().oracle_decode_i8(_p(c), _p(s), c.size, block, _p(out))
    return out


def _ptr_array(arrs):
    return (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])


def reduce(peer_codes: Sequence[np.ndarray], counts, codec: int,
           peer_scales: Optional[Sequence[np.ndarray]] = None, block: int = 1024):
    """Weighted mean of one shard from N peer messages, re-encoded.

    Returns (codes, scales or None, mean_f32)."""
    n = len(peer_codes)
    ln = peer_codes[0].size
    cnt = _c(counts, np.uint32)
    pc = [np.ascontiguousarray(a) for a in peer_codes]
    ps = None if peer_scales is None else [_c(s, np.float32) for s in peer_scales]
    if codec == CODEC_FP16:
        out = np.empty(ln, dtype=np.uint16)
        osc = None
    else:
        out = np.empty(ln, dtype=np.int8)
        osc = np.empty((ln + block - 1) // block, dtype=np.float32)
    mean = np.empty(ln, dtype=np.float32)
    scratch = np.empty(2 * max(ln, 1), dtype=np.float32)
    rc = _L().oracle_reduce(_ptr_array(pc), None if ps is None else _ptr_array(ps),
                            _p(cnt), n, ln, codec, block, _p(out), _p(osc), _p(mean),
                            _p(scratch))
    _check(rc)
    return out, osc, mean


def lamb_cfg(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01,
             step=1, bias_correction=True, force_unit_trust=False) -> _LambCfg:
    return _LambCfg(lr, beta1, beta2, eps, weight_decay, step,
                    int(bias_correction), int(force_unit_trust))


def lamb(x, m, v, g, offsets, flags, cfg: _LambCfg):
    """One LAMB step; returns new (x, m, v, trust)."""
    x = _c(x, np.float32).copy()
    m = _c(m, np.float32).copy()
    v = _c(v, np.float32).copy()
    g = _c(g, np.float32)
    off = _c(offsets, np.uint64)
    fl = _c(flags, np.uint8)
    T = len(fl)
    trust = np.empty(T, dtype=np.float32)
    u = np.empty(max(x.size, 1), dtype=np.float32)
    _check(_L().oracle_lamb(_p(x), _p(m), _p(v), _p(g), x.size, _p(off), _p(fl), T,
                            ctypes.byref(cfg), _p(trust), _p(u)))
    return x, m, v, trust


def round_(peer_codes, counts, bounds, codec, x, m, v, offsets, flags, cfg,
           peer_scales=None, block=1024):
    """One averaging round over full-vector peer messages.

    Returns dict(codes, scales, mean, x, m, v, trust)."""
    n = len(peer_codes)
    P = x.size
    pc = [np.ascontiguousarray(a) for a in peer_codes]
    ps = None if peer_scales is None else [_c(s, np.float32) for s in peer_scales]
    cnt = _c(counts, np.uint32)
    bnd = _c(bounds, np.uint64)
    x = _c(x, np.float32).copy()
    m = _c(m, np.float32).copy()
    v = _c(v, np.float32).copy()
    off = _c(offsets, np.uint64)
    fl = _c(flags, np.uint8)
    T = len(fl)
    if codec == CODEC_FP16:
        out = np.empty(P, dtype=np.uint16)
        osc = None
    else:
        out = np.empty(P, dtype=np.int8)
        osc = np.empty((P + block - 1) // block, dtype=np.float32)
    trust = np.empty(T, dtype=np.float32)
    mean = np.empty(P, dtype=np.float32)
    scratch = np.empty(3 * max(P, 1), dtype=np.float32)
    rc = _L().oracle_round(_ptr_array(pc), None if ps is None else _ptr_array(ps),
                           _p(cnt), n, _p(bnd), len(bnd) - 1, codec, block,
                           _p(out), _p(osc), _p(x), _p(m), _p(v), P, _p(off), _p(fl),
                           T, ctypes.byref(cfg), _p(trust), _p(mean), _p(scratch))
    _check(rc)
    return dict(codes=out, scales=osc, mean=mean, x=x, m=m, v=v, trust=trust)


def lars_cfg(lr=4.8, momentum=0.9, trust_coef=1e-3, weight_decay=1e-6,
             force_unit_trust=False) -> _LarsCfg:
    return _LarsCfg(lr, momentum, trust_coef, weight_decay, int(force_unit_trust))


def lars(x, v, g, offsets, flags, cfg: _LarsCfg):
    """One LARS step; returns new (x, v, trust)."""
    x = _c(x, np.float32).copy()
    v = _c(v, np.float32).copy()
    g = _c(g, np.float32)
    off = _c(offsets, np.uint64)
    fl = _c(flags, np.uint8)
    T = len(fl)
    trust = np.empty(T, dtype=np.float32)
    _check(_L().oracle_lars(_p(x), _p(v), _p(g), x.size, _p(off), _p(fl), T,
                            ctypes.byref(cfg), _p(trust)))
    return x, v, trust


def round_lars(peer_codes, counts, bounds, codec, x, v, offsets, flags, cfg: _LarsCfg,
               peer_scales=None, block=1024):
    """One averaging round followed by a LARS step.

    Returns dict(codes, scales, mean, x, v, trust)."""
    n = len(peer_codes)
    P = x.size
    pc = [np.ascontiguousarray(a) for a in peer_codes]
    ps = None if peer_scales is None else [_c(s, np.float32) for s in peer_scales]
    cnt = _c(counts, np.uint32)
    bnd = _c(bounds, np.uint64)
    x = _c(x, np.float32).copy()
    v = _c(v, np.float32).copy()
    off = _c(offsets, np.uint64)
    fl = _c(flags, np.uint8)
    T = len(fl)
    if codec == CODEC_FP16:
        out = np.empty(P, dtype=np.uint16)
        osc = None
    else:
        out = np.empty(P, dtype=np.int8)
        osc = np.empty((P + block - 1) // block, dtype=np.float32)
    trust = np.empty(T, dtype=np.float32)
    mean = np.empty(P, dtype=np.float32)
    scratch = np.empty(3 * max(P, 1), dtype=np.float32)
    rc = _L().oracle_round_lars(_ptr_array(pc), None if ps is None else _ptr_array(ps),
                                _p(cnt), n, _p(bnd), len(bnd) - 1, codec, block,
                                _p(out), _p(osc), _p(x), _p(v), P, _p(off), _p(fl), T,
                                ctypes.byref(cfg), _p(trust), _p(mean), _p(scratch))
    _check(rc)
    return dict(codes=out, scales=osc, mean=mean, x=x, v=v, trust=trust)


def group_iterations(n: int, m: int) -> int:
    """ceil(log_m n), at least 1 (m < 2 has no grid: 1, and the C call fails)."""
    d = 1
    while m >= 2 and m ** d < n:
        d += 1
    return d


def group_allreduce(peer_codes, counts, m: int, codec: int, peer_scales=None, block: int = 1024,
                    iters: int = 0):
    """Group (Moshpit) all-reduce of n peer messages in groups of m.

    Returns (codes [n_out, len], scales [n_out, nblk] or None, peer_out [n])."""
    n = len(peer_codes)
    ln = peer_codes[0].size
    d = group_iterations(n, m)
    groups = m ** d // m
    cnt = _c(counts, np.uint32)
    pc = [np.ascontiguousarray(a) for a in peer_codes]
    ps = None if peer_scales is None else [_c(s, np.float32) for s in peer_scales]
    nsc = 0 if codec == CODEC_FP16 else (ln + block - 1) // block
    cdt = np.uint16 if codec == CODEC_FP16 else np.int8
    out = np.zeros((groups, ln), dtype=cdt)
    osc = np.zeros((groups, max(nsc, 1)), dtype=np.float32)
    work = np.zeros((2, groups, ln), dtype=cdt)
    wsc = np.zeros((2, groups, max(nsc, 1)), dtype=np.float32)
    if nsc == 0:
        osc = np.zeros((groups, 0), np.float32)
        wsc = np.zeros((2, groups, 0), np.float32)
    peer_out = np.zeros(n, dtype=np.uint32)
    n_out = ctypes.c_uint32(0)
    scratch = np.empty(2 * max(ln, 1), dtype=np.float32)
    rc = _L().oracle_group_allreduce(_ptr_array(pc), None if ps is None else _ptr_array(ps), _p(cnt), n, m,
                                     ln, codec, block, iters, _p(out), _p(osc) if nsc else None, _p(peer_out),
                                     ctypes.byref(n_out), _p(work), _p(wsc) if nsc else None, _p(scratch))
    _check(rc)
    return out, (osc if nsc else None), peer_out


def accumulate(acc, g, b: float):
    """acc + b*g (fma per element); g fp32 or fp16 codes (uint16)."""
    acc = _c(acc, np.float32).copy()
    if g.dtype == np.uint16:
        gc, code = _c(g, np.uint16), 1
    else:
        gc, code = _c(g, np.float32), 0
    _L().oracle_accumulate(_p(acc), _p(gc), code, acc.size, b)
    return acc


def finalize(acc, count: int, codec: int, block: int = 1024, reset: bool = True):
    """Encode acc / count; returns (codes, scales or None, acc after)."""
    acc = _c(acc, np.float32).copy()
    n = acc.size
    if codec == CODEC_FP16:
        codes, scales = np.empty(n, np.uint16), None
    else:
        codes, scales = np.empty(n, np.int8), np.empty((n + block - 1) // block, np.float32)
    scratch = np.empty(max(n, 1), np.float32)
    _check(_L().oracle_finalize(_p(acc), n, count, codec, block, _p(codes), _p(scales), int(reset),
                                _p(scratch)))
    return codes, scales, acc
