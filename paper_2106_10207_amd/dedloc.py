"""Thin ctypes binding over libdedloc's C ABI (include/dedloc.h).

Each function has the name of the C entry point it calls and only marshals
arguments: device tensors become raw pointers, the current torch stream
becomes the HIP stream, host tables become numpy arrays.  Every step of the
computation runs in the library's HIP kernels; there is no fallback, and a
missing or unloadable library raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdedloc.so")

DEDLOC_OK = 0
DEDLOC_ERR_INVALID_ARG = -1
DEDLOC_ERR_ALIGN = -2
DEDLOC_ERR_ZERO_WEIGHT = -3
DEDLOC_ERR_WORKSPACE = -4
DEDLOC_ERR_HIP = -5

DEDLOC_CODEC_F32 = 0
DEDLOC_CODEC_FP16 = 1
DEDLOC_CODEC_I8 = 2
DEDLOC_I8_BLOCK = 1024
DEDLOC_NOALLOC_SCRATCH_BYTES = 16 << 20  # static workspace of dedloc_round_noalloc
DEDLOC_BALANCE_MAX_PEERS = 128
DEDLOC_MAX_PEERS = 1024
DEDLOC_MAX_GROUP_PEERS = 1024
DEDLOC_MAX_GROUP_SIZE = 64
DEDLOC_LAUNCH_PEERS = 64  # peers with samples reduced per launch
DEDLOC_TENSOR_DECAY = 1
DEDLOC_TENSOR_ADAPT = 2

CODECS = {"f32": DEDLOC_CODEC_F32, "fp16": DEDLOC_CODEC_FP16, "i8": DEDLOC_CODEC_I8}


class DedlocError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libdedloc error {code}: {msg}")
        self.code = code


class dedloc_lamb_cfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("step", ctypes.c_uint64),
                ("bias_correction", ctypes.c_int32),
                ("force_unit_trust", ctypes.c_int32)]


def lamb_cfg(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, step=1,
             bias_correction=True, force_unit_trust=False) -> dedloc_lamb_cfg:
    return dedloc_lamb_cfg(lr, beta1, beta2, eps, weight_decay, step,
                           int(bias_correction), int(force_unit_trust))


class dedloc_lars_cfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("trust_coef", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("force_unit_trust", ctypes.c_int32)]


def lars_cfg(lr=4.8, momentum=0.9, trust_coef=1e-3, weight_decay=1e-6,
             force_unit_trust=False) -> dedloc_lars_cfg:
    return dedloc_lars_cfg(lr, momentum, trust_coef, weight_decay, int(force_unit_trust))


class dedloc_local_peer(ctypes.Structure):
    _fields_ = [("index", ctypes.c_uint32), ("grad", ctypes.c_void_p)]


class dedloc_balance_problem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint32), ("s", ctypes.c_void_p), ("d", ctypes.c_void_p),
                ("u", ctypes.c_void_p), ("t", ctypes.c_void_p), ("can_aggregate", ctypes.c_void_p),
                ("B", ctypes.c_double), ("P", ctypes.c_double), ("c_fixed", ctypes.c_void_p)]


_lib = None

_SIGS = {
    "dedloc_version": ([], ctypes.c_int),
    "dedloc_last_error": ([], ctypes.c_char_p),
    "dedloc_encoded_bytes": ([ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p], ctypes.c_size_t),
    "dedloc_partition": ([ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p], ctypes.c_int),
    "dedloc_weights": ([ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p], ctypes.c_int),
    "dedloc_encode": ([ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p,
                       ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dedloc_decode": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_uint32,
                       ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dedloc_reduce_shard": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64,
                             ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_void_p], ctypes.c_int),
    "dedloc_lamb_workspace_bytes": ([ctypes.c_uint64, ctypes.c_void_p, ctypes.c_uint32], ctypes.c_size_t),
    "dedloc_workspace_clear": ([ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p], ctypes.c_int),
    "dedloc_lamb_step": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_uint32, ctypes.POINTER(dedloc_lamb_cfg), ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_size_t, ctypes.c_void_p], ctypes.c_int),
    "dedloc_round": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
                      ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                      ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(dedloc_lamb_cfg), ctypes.c_void_p,
                      ctypes.c_void_p, ctypes.POINTER(dedloc_local_peer), ctypes.c_void_p, ctypes.c_size_t,
                      ctypes.c_void_p], ctypes.c_int),
    "dedloc_round_noalloc": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
                              ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(dedloc_lamb_cfg), ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.POINTER(dedloc_local_peer), ctypes.c_void_p], ctypes.c_int),
    "dedloc_lars_step": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                          ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32,
                          ctypes.POINTER(dedloc_lars_cfg), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                          ctypes.c_void_p], ctypes.c_int),
    "dedloc_round_lars": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
                           ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(dedloc_lars_cfg), ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.POINTER(dedloc_local_peer), ctypes.c_void_p, ctypes.c_size_t,
                           ctypes.c_void_p], ctypes.c_int),
    "dedloc_group_allreduce_workspace_bytes": ([ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32,
                                                ctypes.c_uint32], ctypes.c_size_t),
    "dedloc_group_allreduce": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32,
                                ctypes.c_uint64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p],
                               ctypes.c_int),
    "dedloc_accumulate": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_float,
                           ctypes.c_void_p], ctypes.c_int),
    "dedloc_finalize": ([ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint32,
                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p], ctypes.c_int),
    "dedloc_balance": ([ctypes.POINTER(dedloc_balance_problem), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dedloc_group_size": ([ctypes.c_uint32, ctypes.c_double, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p],
                          ctypes.c_int),
    "dedloc_profile_begin": ([ctypes.c_uint32], ctypes.c_int),
    "dedloc_profile_end": ([ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dedloc_kernel_kinds": ([], ctypes.c_int),
    "dedloc_test_trust_polls": ([ctypes.c_uint32], ctypes.c_uint32),
    "dedloc_kernel_name": ([ctypes.c_int], ctypes.c_char_p),
}

EXPORTS = tuple(_SIGS)


def load():
    """Load libdedloc.so (building it first only if it is absent)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build
            build.build()
        lib = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(lib, name)
            f.argtypes = args
            f.restype = res
        _lib = lib
    return _lib


def _check(rc: int):
    if rc != DEDLOC_OK:
        raise DedlocError(rc, load().dedloc_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _dev(t, nbytes: Optional[int] = None, name: str = "buffer", f32: bool = False):
    """Device address of a tensor for the C ABI (None passes as NULL).  The
    library reads and writes raw memory, so the tensor must be a contiguous
    device tensor holding at least the `nbytes` the call touches; `f32`:
    it must also be float32 (a buffer the library reads as fp32)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name}: expected a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    if f32 and str(t.dtype) != "torch.float32":
        raise ValueError(f"{name}: expected float32, got {t.dtype}")
    if nbytes is not None and t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name}: holds {t.numel() * t.element_size()} bytes, the call touches {nbytes}")
    return t.data_ptr()


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _code_bytes(codec: int, n: int) -> int:
    return n * (4 if codec == DEDLOC_CODEC_F32 else 2 if codec == DEDLOC_CODEC_FP16 else 1)


def _scale_bytes(codec: int, n: int, block: int) -> int:
    return 4 * ((n + block - 1) // block) if codec == DEDLOC_CODEC_I8 and block > 0 else 0


def _peer_ptrs(ts: Sequence, counts, nbytes: int, name: str) -> ctypes.Array:
    """Pointer table of the peers' buffers: a peer with samples must hold
    `nbytes`; a peer without samples is never read (any buffer, or None)."""
    out = []
    for p, t in enumerate(ts):
        if t is None or counts[p] == 0:
            out.append(None if t is None else t.data_ptr())
        else:
            out.append(_dev(t, nbytes, f"{name}[{p}]"))
    return (ctypes.c_void_p * len(ts))(*out)


def _stream(stream=None) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _host(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


# ------------------------------------------------------------- host helpers

def dedloc_version() -> int:
    return load().dedloc_version()


def dedloc_encoded_bytes(codec: int, block: int, n: int):
    ns = ctypes.c_uint64(0)
    nb = load().dedloc_encoded_bytes(codec, block, n, ctypes.byref(ns))
    return nb, ns.value


def dedloc_partition(P: int, n_shards: int, weights=None, align: int = 64) -> np.ndarray:
    w = None if weights is None else _host(weights, np.uint64)
    out = np.zeros(n_shards + 1, dtype=np.uint64)
    _check(load().dedloc_partition(P, n_shards, _ptr(w), align, _ptr(out)))
    return out


def dedloc_weights(counts) -> np.ndarray:
    c = _host(counts, np.uint32)
    w = np.zeros(len(c), dtype=np.float32)
    _check(load().dedloc_weights(_ptr(c), len(c), _ptr(w)))
    return w


# ------------------------------------------------------------- device calls

def dedloc_encode(x, codec: int, block: int = DEDLOC_I8_BLOCK, codes=None, scales=None, stream=None):
    import torch
    n = x.numel()
    if codes is None:
        codes = torch.empty(n, dtype=torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8, device=x.device)
    if scales is None and codec == DEDLOC_CODEC_I8:
        scales = torch.empty((n + block - 1) // block, dtype=torch.float32, device=x.device)
    _check(load().dedloc_encode(_dev(x, 4 * n, "x", f32=True), n, codec, block,
                                _dev(codes, _code_bytes(codec, n), "codes"),
                                _dev(scales, _scale_bytes(codec, n, block), "scales"), _stream(stream)))
    return codes, scales


def dedloc_decode(codes, scales, n: int, codec: int, block: int = DEDLOC_I8_BLOCK, out=None, stream=None):
    import torch
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=codes.device)
    _check(load().dedloc_decode(_dev(codes, _code_bytes(codec, n), "codes"),
                                _dev(scales, _scale_bytes(codec, n, block), "scales"), n, codec, block,
                                _dev(out, 4 * n, "out", f32=True), _stream(stream)))
    return out


def dedloc_reduce_shard(peer_codes: Sequence, counts, shard_len: int, codec: int, peer_scales=None,
                        block: int = DEDLOC_I8_BLOCK, out_codes=None, out_scales=None, out_mean=None,
                        stream=None):
    """Average one shard from the peers' messages (None for zero-count peers)."""
    import torch
    dev = next(t.device for t in peer_codes if t is not None)
    if out_codes is None:
        out_codes = torch.empty(shard_len, dtype=torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8,
                                device=dev)
    if out_scales is None and codec == DEDLOC_CODEC_I8:
        out_scales = torch.empty((shard_len + block - 1) // block, dtype=torch.float32, device=dev)
    cnt = _host(counts, np.uint32)
    if len(cnt) != len(peer_codes):
        raise ValueError("counts and peer_codes differ in length")
    pc = _peer_ptrs(peer_codes, cnt, _code_bytes(codec, shard_len), "peer_codes")
    ps = None if peer_scales is None else _peer_ptrs(peer_scales, cnt, _scale_bytes(codec, shard_len, block),
                                                     "peer_scales")
    _check(load().dedloc_reduce_shard(pc, ps, _ptr(cnt), len(peer_codes), shard_len, codec, block,
                                      _dev(out_codes, _code_bytes(codec, shard_len), "out_codes"),
                                      _dev(out_scales, _scale_bytes(codec, shard_len, block), "out_scales"),
                                      _dev(out_mean, 4 * shard_len, "out_mean", f32=True), _stream(stream)))
    return out_codes, out_scales


def dedloc_lamb_workspace_bytes(P: int, offsets) -> int:
    off = _host(offsets, np.uint64)
    n = load().dedloc_lamb_workspace_bytes(P, _ptr(off), len(off) - 1)
    if n == 0:
        raise DedlocError(DEDLOC_ERR_INVALID_ARG, load().dedloc_last_error().decode())
    return n


def dedloc_workspace_clear(ws, stream=None):
    _check(load().dedloc_workspace_clear(_dev(ws, name="ws"), _nbytes(ws), _stream(stream)))


def make_workspace(P: int, offsets, device="cuda"):
    """A zero-filled workspace for dedloc_lamb_step / dedloc_round."""
    import torch
    nb = dedloc_lamb_workspace_bytes(P, offsets)
    ws = torch.empty(nb, dtype=torch.uint8, device=device)
    dedloc_workspace_clear(ws)
    return ws


def dedloc_lamb_step(x, m, v, grad, offsets, flags, cfg: dedloc_lamb_cfg, grad_codec: int = DEDLOC_CODEC_F32,
                     grad_scales=None, block: int = DEDLOC_I8_BLOCK, trust_out=None, ws=None, stream=None):
    off = _host(offsets, np.uint64)
    fl = _host(flags, np.uint8)
    P = x.numel()
    if ws is None:
        ws = make_workspace(P, off, x.device)
    _check(load().dedloc_lamb_step(_dev(x, 4 * P, "x", f32=True), _dev(m, 4 * P, "m", f32=True),
                                   _dev(v, 4 * P, "v", f32=True), _dev(grad, _code_bytes(grad_codec, P), "grad"),
                                   _dev(grad_scales, _scale_bytes(grad_codec, P, block), "grad_scales"),
                                   grad_codec, block, P, _ptr(off), _ptr(fl), len(fl), ctypes.byref(cfg),
                                   _dev(trust_out, 4 * len(fl), "trust_out", f32=True), _dev(ws, name="ws"),
                                   _nbytes(ws), _stream(stream)))
    return ws


def dedloc_lars_step(x, v, grad, offsets, flags, cfg: dedloc_lars_cfg, grad_codec: int = DEDLOC_CODEC_F32,
                     grad_scales=None, block: int = DEDLOC_I8_BLOCK, trust_out=None, ws=None, stream=None):
    off = _host(offsets, np.uint64)
    fl = _host(flags, np.uint8)
    P = x.numel()
    if ws is None:
        ws = make_workspace(P, off, x.device)
    _check(load().dedloc_lars_step(_dev(x, 4 * P, "x", f32=True), _dev(v, 4 * P, "v", f32=True),
                                   _dev(grad, _code_bytes(grad_codec, P), "grad"),
                                   _dev(grad_scales, _scale_bytes(grad_codec, P, block), "grad_scales"),
                                   grad_codec, block, P, _ptr(off), _ptr(fl), len(fl), ctypes.byref(cfg),
                                   _dev(trust_out, 4 * len(fl), "trust_out", f32=True), _dev(ws, name="ws"),
                                   _nbytes(ws), _stream(stream)))
    return ws


class RoundCall:
    """Pre-marshalled arguments of one dedloc_round call (dedloc_round_lars
    when `cfg` is a dedloc_lars_cfg; then `m` is unused and `v` is the
    momentum buffer): building the pointer arrays once keeps per-call host
    overhead to the C call itself."""

    def __init__(self, peer_codes, counts, bounds, codec, out_codes, x, m, v, offsets, flags,
                 cfg, ws, peer_scales=None, out_scales=None, trust_out=None,
                 out_mean=None, block: int = DEDLOC_I8_BLOCK, local=None):
        """local: optional (index, fp32 gradient tensor): that peer's message
        buffers are written by the round (dedloc_local_peer).  ws None with a
        LAMB cfg: the call is dedloc_round_noalloc (the library's static
        workspace)."""
        self._keep = (peer_codes, peer_scales, out_codes, out_scales, x, m, v, ws, trust_out, out_mean, local)
        P = x.numel()
        self.local = None if local is None else ctypes.byref(
            dedloc_local_peer(int(local[0]), _dev(local[1], 4 * P, "local gradient", f32=True)))
        self.cnt = _host(counts, np.uint32)
        if len(self.cnt) != len(peer_codes):
            raise ValueError("counts and peer_codes differ in length")
        self.pc = _peer_ptrs(peer_codes, self.cnt, _code_bytes(codec, P), "peer_codes")
        self.ps = None if peer_scales is None else _peer_ptrs(peer_scales, self.cnt, _scale_bytes(codec, P, block),
                                                              "peer_scales")
        self.bnd = _host(bounds, np.uint64)
        self.off = _host(offsets, np.uint64)
        self.fl = _host(flags, np.uint8)
        self.cfg = cfg
        self.args = None
        self.codec, self.block = codec, block
        self.lars = isinstance(cfg, dedloc_lars_cfg)
        self.out = (_dev(out_codes, _code_bytes(codec, P), "out_codes"),
                    _dev(out_scales, _scale_bytes(codec, P, block), "out_scales"), _dev(x, 4 * P, "x", f32=True),
                    None if self.lars else _dev(m, 4 * P, "m", f32=True), _dev(v, 4 * P, "v", f32=True), P,
                    _dev(trust_out, 4 * len(self.fl), "trust_out", f32=True),
                    _dev(out_mean, 4 * P, "out_mean", f32=True), _dev(ws, name="ws"),
                    0 if ws is None else _nbytes(ws))

    def __call__(self, stream=None):
        oc, osc, x, m, v, P, tr, om, ws, wsb = self.out
        lib = load()
        if self.lars:
            rc = lib.dedloc_round_lars(self.pc, self.ps, _ptr(self.cnt), len(self.cnt), _ptr(self.bnd),
                                       len(self.bnd) - 1, self.codec, self.block, oc, osc, x, v, P,
                                       _ptr(self.off), _ptr(self.fl), len(self.fl), ctypes.byref(self.cfg),
                                       tr, om, self.local, ws, wsb, _stream(stream))
        elif ws is None:
            rc = lib.dedloc_round_noalloc(self.pc, self.ps, _ptr(self.cnt), len(self.cnt), _ptr(self.bnd),
                                          len(self.bnd) - 1, self.codec, self.block, oc, osc, x, m, v, P,
                                          _ptr(self.off), _ptr(self.fl), len(self.fl), ctypes.byref(self.cfg),
                                          tr, om, self.local, _stream(stream))
        else:
            rc = lib.dedloc_round(self.pc, self.ps, _ptr(self.cnt), len(self.cnt), _ptr(self.bnd),
                                  len(self.bnd) - 1, self.codec, self.block, oc, osc, x, m, v, P,
                                  _ptr(self.off), _ptr(self.fl), len(self.fl), ctypes.byref(self.cfg),
                                  tr, om, self.local, ws, wsb, _stream(stream))
        _check(rc)


def dedloc_round(peer_codes, counts, bounds, codec: int, x, m, v, offsets, flags, cfg: dedloc_lamb_cfg,
                 peer_scales=None, block: int = DEDLOC_I8_BLOCK, out_codes=None, out_scales=None,
                 trust_out=None, out_mean=None, ws=None, stream=None, local=None):
    """One averaging round; returns (out_codes, out_scales).  local: optional
    (peer index, fp32 gradient) encoded by the round into that peer's
    message."""
    import torch
    P = x.numel()
    if out_codes is None:
        out_codes = torch.empty(P, dtype=torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8, device=x.device)
    if out_scales is None and codec == DEDLOC_CODEC_I8:
        out_scales = torch.empty((P + block - 1) // block, dtype=torch.float32, device=x.device)
    if ws is None:
        ws = make_workspace(P, offsets, x.device)
    RoundCall(peer_codes, counts, bounds, codec, out_codes, x, m, v, offsets, flags, cfg, ws, peer_scales,
              out_scales, trust_out, out_mean, block, local)(stream)
    return out_codes, out_scales


def dedloc_round_noalloc(peer_codes, counts, bounds, codec: int, x, m, v, offsets, flags,
                         cfg: dedloc_lamb_cfg, out_codes, out_scales=None, peer_scales=None,
                         block: int = DEDLOC_I8_BLOCK, trust_out=None, out_mean=None, stream=None, local=None):
    """dedloc_round without a workspace (the library's static array) and
    with caller-provided outputs: nothing is allocated."""
    if isinstance(cfg, dedloc_lars_cfg):
        raise ValueError("dedloc_round_noalloc takes a LAMB cfg")
    RoundCall(peer_codes, counts, bounds, codec, out_codes, x, m, v, offsets, flags, cfg, None, peer_scales,
              out_scales, trust_out, out_mean, block, local)(stream)
    return out_codes, out_scales


# ------------------------------------------------------------- profiling

def dedloc_profile_begin(max_launches: int = 1 << 16):
    _check(load().dedloc_profile_begin(max_launches))


def dedloc_test_trust_polls(polls: int) -> int:
    """Test hook: how often a workgroup polls for a tensor's published trust
    ratio before computing it itself (0: always itself); returns the
    previous value.  Results do not depend on it."""
    return int(load().dedloc_test_trust_polls(int(polls)))


def dedloc_profile_end():
    """{kernel name: (total ms, launches)} for the kernels enqueued since
    dedloc_profile_begin (waits for them)."""
    lib = load()
    n = lib.dedloc_kernel_kinds()
    ms = np.zeros(n, np.float64)
    cnt = np.zeros(n, np.uint64)
    _check(lib.dedloc_profile_end(n, _ptr(ms), _ptr(cnt)))
    return {lib.dedloc_kernel_name(k).decode(): (float(ms[k]), int(cnt[k])) for k in range(n) if cnt[k]}


def dedloc_round_lars(peer_codes, counts, bounds, codec: int, x, v, offsets, flags, cfg: dedloc_lars_cfg,
                      peer_scales=None, block: int = DEDLOC_I8_BLOCK, out_codes=None, out_scales=None,
                      trust_out=None, out_mean=None, ws=None, stream=None, local=None):
    """One averaging round followed by a LARS step; returns (out_codes, out_scales)."""
    import torch
    P = x.numel()
    if out_codes is None:
        out_codes = torch.empty(P, dtype=torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8, device=x.device)
    if out_scales is None and codec == DEDLOC_CODEC_I8:
        out_scales = torch.empty((P + block - 1) // block, dtype=torch.float32, device=x.device)
    if ws is None:
        ws = make_workspace(P, offsets, x.device)
    RoundCall(peer_codes, counts, bounds, codec, out_codes, x, None, v, offsets, flags, cfg, ws, peer_scales,
              out_scales, trust_out, out_mean, block, local)(stream)
    return out_codes, out_scales


def dedloc_group_size(n_peers: int, failure_rate: float, max_group: int = 0):
    """(m, expected iterations) of the group size minimising the expected
    iterations to the global average (dedloc.h)."""
    m = ctypes.c_uint32(0)
    e = ctypes.c_double(0.0)
    lib = load()
    rc = lib.dedloc_group_size(n_peers, failure_rate, max_group, ctypes.byref(m), ctypes.byref(e))
    if rc != DEDLOC_OK:
        raise DedlocError(rc, "dedloc_group_size: n_peers in [2, 1024], 0 <= failure_rate < 1, max_group 0 or >= 2")
    return m.value, e.value


def group_iterations(n_peers: int, group_size: int) -> int:
    d = 1
    while group_size >= 2 and group_size ** d < n_peers:
        d += 1
    return d


class GroupAllreduce:
    """Pre-allocated buffers and marshalled arguments of dedloc_group_allreduce
    for fixed peers, counts and group size.  After a call, messages[g] (and
    scales[g] for int8) is group g's output and peer_out[i] the output peer i
    holds."""

    def __init__(self, peer_codes, counts, group_size: int, length: int, codec: int, peer_scales=None,
                 block: int = DEDLOC_I8_BLOCK, device="cuda"):
        import torch
        n = len(peer_codes)
        d = group_iterations(n, group_size)
        self.n_out = group_size ** d // group_size
        cb = 2 if codec == DEDLOC_CODEC_FP16 else 1
        self.stride = (length * cb + 255) // 256 * 256
        nsc = (length + block - 1) // block if codec == DEDLOC_CODEC_I8 else 0
        self.out = torch.empty(max(self.n_out * self.stride, 256), dtype=torch.uint8, device=device)
        self.out_scales = (torch.empty(self.n_out * nsc, dtype=torch.float32, device=device)
                           if codec == DEDLOC_CODEC_I8 else None)
        nb = load().dedloc_group_allreduce_workspace_bytes(n, group_size, length, codec, block)
        if nb == 0:
            raise DedlocError(DEDLOC_ERR_INVALID_ARG, load().dedloc_last_error().decode())
        self.ws = torch.empty(nb, dtype=torch.uint8, device=device)
        dt = torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8
        self.messages = [self.out[g * self.stride: g * self.stride + length * cb].view(dt)
                         for g in range(self.n_out)]
        self.scales = ([self.out_scales[g * nsc:(g + 1) * nsc] for g in range(self.n_out)]
                       if codec == DEDLOC_CODEC_I8 else None)
        self.peer_out = np.zeros(n, dtype=np.uint32)
        self._n_out = ctypes.c_uint32(0)
        self._keep = (peer_codes, peer_scales)
        self.cnt = _host(counts, np.uint32)
        if len(self.cnt) != n:
            raise ValueError("counts and peer_codes differ in length")
        self.pc = _peer_ptrs(peer_codes, self.cnt, _code_bytes(codec, length), "peer_codes")
        self.ps = None if peer_scales is None else _peer_ptrs(peer_scales, self.cnt,
                                                              _scale_bytes(codec, length, block), "peer_scales")
        self.args = (n, group_size, length, codec, block)

    def __call__(self, stream=None):
        n, m, length, codec, block = self.args
        _check(load().dedloc_group_allreduce(self.pc, self.ps, _ptr(self.cnt), n, m, length, codec, block,
                                             _dev(self.out), _dev(self.out_scales), _ptr(self.peer_out),
                                             ctypes.byref(self._n_out), _dev(self.ws), _nbytes(self.ws),
                                             _stream(stream)))
        return self


def dedloc_group_allreduce(peer_codes, counts, group_size: int, length: int, codec: int, peer_scales=None,
                           block: int = DEDLOC_I8_BLOCK, stream=None) -> GroupAllreduce:
    dev = next(t.device for t in peer_codes if t is not None)
    return GroupAllreduce(peer_codes, counts, group_size, length, codec, peer_scales, block, dev)(stream)


def dedloc_accumulate(acc, grad, batch_samples: float, stream=None):
    """acc += batch_samples * grad (fp32 grad, or fp16 codes as int16)."""
    import torch
    codec = DEDLOC_CODEC_FP16 if grad.dtype in (torch.int16, torch.float16) else DEDLOC_CODEC_F32
    n = acc.numel()
    _check(load().dedloc_accumulate(_dev(acc, 4 * n, "acc", f32=True), _dev(grad, _code_bytes(codec, n), "grad"),
                                    codec, n, batch_samples, _stream(stream)))


def dedloc_finalize(acc, count: int, codec: int, block: int = DEDLOC_I8_BLOCK, codes=None, scales=None,
                    reset: bool = True, stream=None):
    import torch
    n = acc.numel()
    if codes is None:
        codes = torch.empty(n, dtype=torch.int16 if codec == DEDLOC_CODEC_FP16 else torch.int8, device=acc.device)
    if scales is None and codec == DEDLOC_CODEC_I8:
        scales = torch.empty((n + block - 1) // block, dtype=torch.float32, device=acc.device)
    _check(load().dedloc_finalize(_dev(acc, 4 * n, "acc", f32=True), n, count, codec, block,
                                  _dev(codes, _code_bytes(codec, n), "codes"),
                                  _dev(scales, _scale_bytes(codec, n, block), "scales"), int(reset),
                                  _stream(stream)))
    return codes, scales


def dedloc_balance(s, d, u, B: float, P: float, t=None, can_aggregate=None, c_fixed=None):
    """Solve the load-balancing LP on the host.  Returns dict(xi, c, frac,
    weights, a, g) (rates in parameters/s).  c_fixed: optional per-peer
    compute indicators (NaN = free)."""
    s, d, u = (_host(v, np.float64) for v in (s, d, u))
    n = s.size
    for name, v in (("d", d), ("u", u)):
        if v.size != n:
            raise ValueError(f"{name} has {v.size} entries, s has {n}")
    tt = None if t is None else _host(t, np.float64).reshape(n * n)
    ca = None if can_aggregate is None else _host(can_aggregate, np.uint8)
    cf = None if c_fixed is None else _host(c_fixed, np.float64)
    if ca is not None and ca.size != n or cf is not None and cf.size != n:
        raise ValueError("can_aggregate and c_fixed need one entry per peer")
    pr = dedloc_balance_problem(n, _ptr(s), _ptr(d), _ptr(u), _ptr(tt), _ptr(ca), B, P, _ptr(cf))
    xi = ctypes.c_double(0.0)
    c = np.zeros(n)
    frac = np.zeros(n)
    w = np.zeros(n, np.uint64)
    a = np.zeros(n * n)
    g = np.zeros(n * n)
    rc = load().dedloc_balance(ctypes.byref(pr), ctypes.byref(xi), _ptr(c), _ptr(frac), _ptr(w), _ptr(a), _ptr(g))
    if rc != DEDLOC_OK:
        raise DedlocError(rc, "load-balancing LP failed (invalid problem or no convergence)")
    return dict(xi=xi.value, c=c, frac=frac, weights=w, a=a.reshape(n, n), g=g.reshape(n, n))
