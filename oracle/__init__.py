"""Reference oracle for the NEURON-Fabric bucket reducer (ctypes over libnfo.so).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke entry point and the
benchmark's CPU-baseline leg may import this package; the GPU library and its
binding never do.  Every function takes and returns plain numpy arrays on the
host and calls the single-threaded C++ code in nfo.cpp.
"""
import ctypes
import os

import numpy as np

from . import build as _build

ROUTE_L, ROUTE_F, ROUTE_P = 0, 1, 2
R_NOT_ADMITTED, R_NO_ELIGIBLE, R_VETO, R_GUARD = 1, 2, 4, 8
R_NONFINITE, R_ZERO_WORKER, R_NORM_SPIKE, R_FORCED = 16, 32, 64, 128
DECODE_SOFT, DECODE_MAJORITY = 0, 1
OP_SUM, OP_MEAN = 0, 1


class Stats(ctypes.Structure):
    _fields_ = [("nonfinite", ctypes.c_uint64), ("sum_abs_elig", ctypes.c_double),
                ("sum_sq", ctypes.c_double)]


class Policy(ctypes.Structure):
    _fields_ = [("admitted", ctypes.c_int), ("veto", ctypes.c_int),
                ("guard_ok", ctypes.c_int), ("force_lowbit", ctypes.c_int),
                ("decode_mode", ctypes.c_int), ("fp32_op", ctypes.c_int),
                ("kappa", ctypes.c_double), ("format", ctypes.c_int), ("tau", ctypes.c_float)]


class Decision(ctypes.Structure):
    _fields_ = [("route", ctypes.c_int32), ("reasons", ctypes.c_uint32),
                ("scale", ctypes.c_float), ("n_eligible", ctypes.c_int64),
                ("bytes_route", ctypes.c_double), ("bytes_fp32", ctypes.c_double)]


STATS_DTYPE = np.dtype([("nonfinite", "<u8"), ("sum_abs_elig", "<f8"), ("sum_sq", "<f8")])

_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32


def load(path=None):
    """Load (building first if absent) the oracle library; returns the CDLL."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or _build.LIB
    if not os.path.exists(path):
        _build.build(path)
    lib = ctypes.CDLL(path)
    sig = {
        "nfo_mask_from_segments": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _P]),
        "nfo_count_eligible": (_I64, [_P, _I64]),
        "nfo_health": (None, [_P, _I64, _I32, _I64, _P, _P]),
        "nfo_scale": (ctypes.c_float, [_P, _I32, _I64]),
        "nfo_decide": (None, [_P, _I32, _I64, _I64, _P, _P]),
        "nfo_pack": (None, [_P, _I64, _I32, _I64, _P, _P, _I64]),
        "nfo_counts": (None, [_P, _I64, _I32, _I64, _P]),
        "nfo_fp32_path": (None, [_P, _I64, _I32, _I64, _I32, _P]),
        "nfo_decode_table": (None, [_I32, _I32, _P]),
        "nfo_output": (None, [_P, _I64, _P, _P, _P, ctypes.c_float, _I32, _P]),
        "nfo_reduce_bucket": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _I64,
                                             _P, _P, _P, _P]),
        "nfo_ternary_threshold": (ctypes.c_float, [_P, _I64, ctypes.c_float]),
        "nfo_pack_ternary": (None, [_P, _I64, _I32, _I64, _P, _P, _P, _P, _I64]),
        "nfo_ternary_decode_table": (None, [_I32, _I32, _P]),
        "nfo_ternary_output": (None, [_P, _I64, _P, _P, _P, _P, ctypes.c_float, _I32, _I32, _P]),
        "nfo_pack_compact": (None, [_P, _I64, _I32, _I64, _P, _P, _I64]),
        "nfo_slice_scales": (None, [_P, _I64, _I32, _P, _P, _I64, _P, _P]),
        "nfo_sliced_output": (None, [_P, _I64, _P, _P, _P, _P, _P, _I64, _P, _I32, _P]),
        "nfo_reduce_bucket_ternary": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _P, _I64,
                                                     _P, _P, _P, _P, _P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    if path == _build.LIB:
        _lib = lib
    return lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None and a.size else ctypes.c_void_p(0)


def _grads(g):
    g = np.asarray(g)
    assert g.dtype == np.float32 and g.ndim == 2 and g.strides[1] == 4
    return g, g.strides[0] // 4


def policy(admitted=1, veto=0, guard_ok=1, force_lowbit=0, decode_mode=DECODE_SOFT,
           fp32_op=OP_SUM, kappa=4.0, format=0, tau=0.5):
    return Policy(admitted, veto, guard_ok, force_lowbit, decode_mode, fp32_op, kappa, format, tau)


def mask_from_segments(off, length, eligible, n, lib=None):
    lib = lib or load()
    off = np.ascontiguousarray(off, dtype=np.int64)
    length = np.ascontiguousarray(length, dtype=np.int64)
    eligible = np.ascontiguousarray(eligible, dtype=np.uint8)
    mask = np.zeros(max((n + 63) // 64, 1), dtype=np.uint64)
    rc = lib.nfo_mask_from_segments(_ptr(off), _ptr(length), _ptr(eligible),
                                    len(off), n, _ptr(mask))
    if rc != 0:
        raise ValueError("segment outside the bucket")
    return mask[: (n + 63) // 64]


def count_eligible(mask, n, lib=None):
    lib = lib or load()
    mask = np.ascontiguousarray(mask, dtype=np.uint64)
    return int(lib.nfo_count_eligible(_ptr(mask), n))


def health(g, mask, lib=None):
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    st = np.zeros(W, dtype=STATS_DTYPE)
    lib.nfo_health(_ptr(g), stride, W, n, _ptr(np.ascontiguousarray(mask, np.uint64)), _ptr(st))
    return st


def scale(stats, n_eligible, lib=None):
    lib = lib or load()
    st = np.ascontiguousarray(stats, dtype=STATS_DTYPE)
    return np.float32(lib.nfo_scale(_ptr(st), len(st), n_eligible))


def decide(stats, n, n_eligible, pol=None, lib=None):
    lib = lib or load()
    st = np.ascontiguousarray(stats, dtype=STATS_DTYPE)
    d = Decision()
    pol = pol or policy()
    lib.nfo_decide(_ptr(st), len(st), n, n_eligible, ctypes.byref(pol), ctypes.byref(d))
    return d


def pack(g, mask, lib=None):
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    nw = (n + 63) // 64
    bits = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    lib.nfo_pack(_ptr(g), stride, W, n, _ptr(np.ascontiguousarray(mask, np.uint64)),
                 _ptr(bits), bits.shape[1])
    return bits[:, :nw]


def counts(bits, n, lib=None):
    lib = lib or load()
    bits = np.ascontiguousarray(bits, dtype=np.uint64)
    W = bits.shape[0]
    c = np.zeros(n, dtype=np.uint8)
    lib.nfo_counts(_ptr(bits), bits.shape[1], W, n, _ptr(c))
    return c


def fp32_path(g, op=OP_SUM, lib=None):
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    y = np.zeros(n, dtype=np.float32)
    lib.nfo_fp32_path(_ptr(g), stride, W, n, op, _ptr(y))
    return y


def decode_table(W, mode=DECODE_SOFT, lib=None):
    lib = lib or load()
    q = np.zeros(W + 1, dtype=np.float32)
    lib.nfo_decode_table(W, mode, _ptr(q))
    return q


def output(mask, n, counts, y, q, scale, route, lib=None):
    """Step 10 on its own: decoded values at mask = 1 under route L, the FP32
    path elsewhere (and everywhere under F and P)."""
    lib = lib or load()
    out = np.zeros(max(n, 1), dtype=np.float32)
    m = np.ascontiguousarray(mask, np.uint64)
    lib.nfo_output(_ptr(m if m.size else np.zeros(1, np.uint64)), n, _ptr(np.ascontiguousarray(counts, np.uint8)),
                   _ptr(np.ascontiguousarray(y, np.float32)), _ptr(np.ascontiguousarray(q, np.float32)),
                   ctypes.c_float(scale), route, _ptr(out))
    return out[:n]


def reduce_bucket(g, mask, pol=None, lib=None):
    """Whole bucket.  Returns dict(bits, counts, out, stats, decision)."""
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    nw = (n + 63) // 64
    bits = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    c = np.zeros(max(n, 1), dtype=np.uint8)
    out = np.zeros(max(n, 1), dtype=np.float32)
    st = np.zeros(W, dtype=STATS_DTYPE)
    d = Decision()
    pol = pol or policy()
    m = np.ascontiguousarray(mask, np.uint64)
    if m.size == 0:
        m = np.zeros(1, np.uint64)
    rc = lib.nfo_reduce_bucket(_ptr(g), stride, W, n, _ptr(m), ctypes.byref(pol),
                               _ptr(bits), bits.shape[1], _ptr(c), _ptr(out), _ptr(st),
                               ctypes.byref(d))
    if rc != 0:
        raise ValueError("invalid arguments")
    return dict(bits=bits[:, :nw], counts=c[:n], out=out[:n], stats=st, decision=d)


# ---------------------------------------------------------- G-Ternary

FORMAT_BINARY, FORMAT_TERNARY = 0, 1


def ternary_threshold(stats_w, n_eligible, tau, lib=None):
    """theta for one worker's stats record (STATS_DTYPE scalar or 1-array)."""
    lib = lib or load()
    st = np.ascontiguousarray(np.atleast_1d(stats_w)[:1], dtype=STATS_DTYPE)
    return np.float32(lib.nfo_ternary_threshold(_ptr(st), n_eligible, ctypes.c_float(tau)))


def pack_ternary(g, mask, theta, lib=None):
    """(pos, neg) planes [W, ceil(n/64)] with per-worker thresholds theta."""
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    nw = (n + 63) // 64
    pos = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    neg = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    th = np.ascontiguousarray(theta, dtype=np.float32)
    lib.nfo_pack_ternary(_ptr(g), stride, W, n, _ptr(np.ascontiguousarray(mask, np.uint64)), _ptr(th),
                         _ptr(pos), _ptr(neg), pos.shape[1])
    return pos[:, :nw], neg[:, :nw]


def ternary_decode_table(W, mode=DECODE_SOFT, lib=None):
    """q[d + W] for d in [-W, W]."""
    lib = lib or load()
    q = np.zeros(2 * W + 1, dtype=np.float32)
    lib.nfo_ternary_decode_table(W, mode, _ptr(q))
    return q


def ternary_output(mask, n, cpos, cneg, y, q, scale, W, route, lib=None):
    """The G-Ternary output step on its own (R20): fl32(scale * q[c+ - c-])
    at mask = 1 under route L, the FP32 path elsewhere."""
    lib = lib or load()
    out = np.zeros(max(n, 1), dtype=np.float32)
    m = np.ascontiguousarray(mask, np.uint64)
    lib.nfo_ternary_output(_ptr(m if m.size else np.zeros(1, np.uint64)), n,
                           _ptr(np.ascontiguousarray(cpos, np.uint8)), _ptr(np.ascontiguousarray(cneg, np.uint8)),
                           _ptr(np.ascontiguousarray(y, np.float32)), _ptr(np.ascontiguousarray(q, np.float32)),
                           ctypes.c_float(scale), W, route, _ptr(out))
    return out[:n]


def reduce_bucket_ternary(g, mask, pol, lib=None):
    """Whole bucket, G-Ternary payload.  Returns dict(pos, neg, cpos, cneg,
    out, stats, decision)."""
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    nw = (n + 63) // 64
    pos = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    neg = np.zeros((W, max(nw, 1)), dtype=np.uint64)
    cp = np.zeros(max(n, 1), dtype=np.uint8)
    cn = np.zeros(max(n, 1), dtype=np.uint8)
    out = np.zeros(max(n, 1), dtype=np.float32)
    st = np.zeros(W, dtype=STATS_DTYPE)
    d = Decision()
    m = np.ascontiguousarray(mask, np.uint64)
    if m.size == 0:
        m = np.zeros(1, np.uint64)
    rc = lib.nfo_reduce_bucket_ternary(_ptr(g), stride, W, n, _ptr(m), ctypes.byref(pol), _ptr(pos),
                                       _ptr(neg), pos.shape[1], _ptr(cp), _ptr(cn), _ptr(out), _ptr(st),
                                       ctypes.byref(d))
    if rc != 0:
        raise ValueError("invalid arguments")
    return dict(pos=pos[:, :nw], neg=neg[:, :nw], cpos=cp[:n], cneg=cn[:n], out=out[:n], stats=st,
                decision=d)


def pack_compact(g, mask, lib=None):
    """Compacted sign payload [W, ceil(n_E/64)] (R30)."""
    lib = lib or load()
    g, stride = _grads(g)
    W, n = g.shape
    m = np.ascontiguousarray(mask, np.uint64)
    ne = count_eligible(m, n, lib=lib) if n else 0
    cw = (ne + 63) // 64
    cb = np.zeros((W, max(cw, 1)), dtype=np.uint64)
    lib.nfo_pack_compact(_ptr(g), stride, W, n, _ptr(m if m.size else np.zeros(1, np.uint64)), _ptr(cb),
                         cb.shape[1])
    return cb[:, :cw]


def slice_scales(g, off, length, lib=None):
    """(sums [S, W] float64, scales [S] float32) of the slices (R31)."""
    lib = lib or load()
    g, stride = _grads(g)
    W = g.shape[0]
    off = np.ascontiguousarray(off, dtype=np.int64)
    length = np.ascontiguousarray(length, dtype=np.int64)
    S = len(off)
    sums = np.zeros((max(S, 1), W), dtype=np.float64)
    sc = np.zeros(max(S, 1), dtype=np.float32)
    lib.nfo_slice_scales(_ptr(g), stride, W, _ptr(off), _ptr(length), S, _ptr(sums), _ptr(sc))
    return sums[:S], sc[:S]


def sliced_output(mask, counts, y, q, off, length, scales, route=ROUTE_L, lib=None):
    """Positional output with per-slice scales (R32)."""
    lib = lib or load()
    n = len(y)
    out = np.zeros(max(n, 1), dtype=np.float32)
    m = np.ascontiguousarray(mask, np.uint64)
    lib.nfo_sliced_output(_ptr(m if m.size else np.zeros(1, np.uint64)), n,
                          _ptr(np.ascontiguousarray(counts, np.uint8)), _ptr(np.ascontiguousarray(y, np.float32)),
                          _ptr(np.ascontiguousarray(q, np.float32)), _ptr(np.ascontiguousarray(off, np.int64)),
                          _ptr(np.ascontiguousarray(length, np.int64)), len(off),
                          _ptr(np.ascontiguousarray(scales, np.float32)), route, _ptr(out))
    return out[:n]
