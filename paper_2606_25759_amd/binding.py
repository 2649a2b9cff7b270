"""ctypes binding of libnf.so (the C ABI of include/nf.h), same function names.

Argument marshalling only: every wrapper checks dtypes and devices, turns
torch tensors into device pointers and the current torch stream into a
hipStream_t, calls the library, and raises NFError on a non-zero status.  No
step of the reducer runs here, and there is no fallback: if libnf.so is
missing, loading fails loudly.
"""
import ctypes
import os

import numpy as np

try:  # torch first: its HIP runtime is the one the library then binds to
    import torch
except ImportError:  # pragma: no cover - the library itself needs no torch
    torch = None

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnf.so")

NF_OK, NF_ERR_INVALID_ARG, NF_ERR_ALIGNMENT, NF_ERR_UNSUPPORTED, NF_ERR_HIP, NF_ERR_WORKSPACE = range(6)
NF_ROUTE_LOWBIT, NF_ROUTE_FALLBACK, NF_ROUTE_PLAIN = 0, 1, 2
NF_REASON_NOT_ADMITTED, NF_REASON_NO_ELIGIBLE, NF_REASON_VETO, NF_REASON_GUARD = 1, 2, 4, 8
NF_REASON_NONFINITE, NF_REASON_ZERO_WORKER, NF_REASON_NORM_SPIKE, NF_REASON_FORCED = 16, 32, 64, 128
NF_DECODE_SOFT, NF_DECODE_MAJORITY = 0, 1
NF_FP32_SUM, NF_FP32_MEAN = 0, 1
NF_SEL_ROUTED, NF_SEL_ELIGIBLE, NF_SEL_ALL = 0, 1, 2
NF_FORMAT_BINARY, NF_FORMAT_TERNARY = 0, 1

# Exported names, in the order include/nf.h declares them.
EXPORTS = ["nf_abi_version", "nf_last_error", "nf_mask_from_segments", "nf_workspace_bytes",
           "nf_bucket_health", "nf_pack_signs", "nf_fp32_reduce", "nf_signcount_reduce",
           "nf_route_decide", "nf_route_bucket", "nf_workspace_bytes_buckets", "nf_route_buckets",
           "nf_route_buckets_noalloc", "nf_bucket_table_bytes", "nf_bucket_table_init",
           "nf_workspace_bytes_table", "nf_pass1_launches_table", "nf_route_bucket_table",
           "nf_set_phase_events", "nf_pass1_launches", "nf_pass1_chunk_elems", "nf_slice_scales_from_pass1", "nf_ternary_threshold", "nf_pack_ternary",
           "nf_ternary_reduce", "nf_partial_counts", "nf_partial_count_reduce", "nf_stock_signcount",
           "nf_supervisor_init", "nf_supervisor_policy", "nf_supervisor_update", "nf_endpoint_guard",
           "nf_sliced_layout_sizes", "nf_sliced_layout", "nf_compact_signs", "nf_slice_workspace_bytes",
           "nf_slice_scales", "nf_compact_signcount_reduce"]
NF_SUP_WARMUP, NF_SUP_LOWBIT, NF_SUP_COOLDOWN, NF_SUP_GUARD = 0, 1, 2, 3


class nf_worker_stats(ctypes.Structure):
    _fields_ = [("nonfinite", ctypes.c_uint64), ("sum_abs_elig", ctypes.c_double),
                ("sum_sq", ctypes.c_double)]


class nf_route_policy(ctypes.Structure):
    _fields_ = [("admitted", ctypes.c_int32), ("veto", ctypes.c_int32),
                ("guard_ok", ctypes.c_int32), ("force_lowbit", ctypes.c_int32),
                ("decode_mode", ctypes.c_int32), ("fp32_op", ctypes.c_int32),
                ("kappa", ctypes.c_double), ("format", ctypes.c_int32), ("tau", ctypes.c_float)]


class nf_route_decision(ctypes.Structure):
    _fields_ = [("route", ctypes.c_int32), ("reasons", ctypes.c_uint32),
                ("scale", ctypes.c_float), ("resummed", ctypes.c_uint32),
                ("n_eligible", ctypes.c_int64), ("bytes_route", ctypes.c_double),
                ("bytes_fp32", ctypes.c_double)]


class nf_supervisor_profile(ctypes.Structure):
    _fields_ = [("admit_step", ctypes.c_int32), ("cooldown_steps", ctypes.c_int32),
                ("guard_steps", ctypes.c_int32), ("short_cooldown_steps", ctypes.c_int32),
                ("ema_alpha", ctypes.c_double), ("slack", ctypes.c_double), ("threshold", ctypes.c_double),
                ("guard_scale", ctypes.c_double), ("near_band", ctypes.c_double),
                ("small_move", ctypes.c_double), ("target_share", ctypes.c_double),
                ("share_margin", ctypes.c_double)]


class nf_supervisor_state(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int64), ("state", ctypes.c_int32), ("has_prev", ctypes.c_int32),
                ("cooldown_left", ctypes.c_int32), ("guard_left", ctypes.c_int32),
                ("smoothed", ctypes.c_double), ("cusum", ctypes.c_double), ("prev_loss", ctypes.c_double),
                ("alarms", ctypes.c_int64), ("short_recoveries", ctypes.c_int64),
                ("readmissions", ctypes.c_int64), ("budget_vetoes", ctypes.c_int64),
                ("events_l", ctypes.c_int64), ("events_f", ctypes.c_int64), ("events_p", ctypes.c_int64),
                ("bytes_route", ctypes.c_double), ("bytes_fp32", ctypes.c_double)]


class nf_endpoint_model(ctypes.Structure):
    _fields_ = [("nodes", ctypes.c_int32), ("gpus_per_node", ctypes.c_int32),
                ("bits_per_element", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("net_bytes_per_s", ctypes.c_double), ("endpoint_bytes_per_s", ctypes.c_double),
                ("latency_fp32_s", ctypes.c_double), ("latency_lowbit_s", ctypes.c_double)]


STATS_DTYPE = np.dtype([("nonfinite", "<u8"), ("sum_abs_elig", "<f8"), ("sum_sq", "<f8")])
DECISION_DTYPE = np.dtype([("route", "<i4"), ("reasons", "<u4"), ("scale", "<f4"),
                           ("resummed", "<u4"), ("n_eligible", "<i8"),
                           ("bytes_route", "<f8"), ("bytes_fp32", "<f8")])
STATS_BYTES = ctypes.sizeof(nf_worker_stats)        # 24
DECISION_BYTES = ctypes.sizeof(nf_route_decision)   # 40


class NFError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"nf status {status}: {message}")
        self.status = status


_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t


def load(path=None):
    """Load libnf.so (built by paper_2606_25759_amd/build.py); raises if absent."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise OSError(f"{path} is missing: build it with python -c "
                      "'import __graft_entry__; __graft_entry__.build()'")
    lib = ctypes.CDLL(path)
    sigs = {
        "nf_abi_version": (ctypes.c_int, []),
        "nf_last_error": (ctypes.c_char_p, []),
        "nf_mask_from_segments": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _P]),
        "nf_workspace_bytes": (_SZ, [_I32, _I64]),
        "nf_workspace_bytes_buckets": (_SZ, [_I32, _I64, _I64]),
        "nf_bucket_health": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _SZ, _P]),
        "nf_pack_signs": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _I64, _P, _P, _SZ, _P]),
        "nf_fp32_reduce": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _I32, _I32, _P, _P]),
        "nf_signcount_reduce": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _I32, _P, _P, _P]),
        "nf_route_decide": (ctypes.c_int, [_P, _I32, _I64, _I64, _P, _P]),
        "nf_route_bucket": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _I64, _P, _P, _P, _P,
                                           _P, _SZ, _P]),
        "nf_route_buckets": (ctypes.c_int, [_P, _I64, _I32, _I64, _I64, _P, _P, _P, _I64, _P, _P,
                                            _P, _P, _P, _SZ, _P]),
        "nf_route_buckets_noalloc": (ctypes.c_int, [_P, _I64, _I32, _I64, _I64, _P, _P, _P, _I64, _P,
                                                    _P, _P, _P, _P]),
        "nf_bucket_table_bytes": (_SZ, [_I32, _P, _I32]),
        "nf_bucket_table_init": (ctypes.c_int, [_I32, _P, _I32, _P, _SZ, _P]),
        "nf_workspace_bytes_table": (_SZ, [_I32, _P, _I32]),
        "nf_pass1_launches_table": (_I64, [_I32, _P, _I32, _I32]),
        "nf_route_bucket_table": (ctypes.c_int, [_P, _I64, _I32, _P, _I32, _P, _P, _P, _P, _I64, _P, _P,
                                                 _P, _P, _P, _SZ, _P]),
        "nf_set_phase_events": (ctypes.c_int, [_P, _P, _P, _P]),
        "nf_slice_scales_from_pass1": (_I32, [_P, _I64, _I32, _I64, _P, _P, _I64, _P, _P, _P, _SZ, _P]),
        "nf_pass1_launches": (_I64, [_I32, _I64, _I64, _I32]),
        "nf_pass1_chunk_elems": (_I64, [_I32, _I64, _I64, _P]),
        "nf_ternary_threshold": (ctypes.c_int, [_P, _I32, _I64, ctypes.c_float, _P]),
        "nf_pack_ternary": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _I64, _P]),
        "nf_ternary_reduce": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _I32, _P, _P, _P]),
        "nf_partial_counts": (ctypes.c_int, [_P, _I64, _I32, _I32, _I64, _P, _I64, _P]),
        "nf_partial_count_reduce": (ctypes.c_int, [_P, _I64, _I32, _I32, _I64, _P, _P, _I32, _P, _P, _P]),
        "nf_stock_signcount": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _I32, _I32, _P, _P, _I64, _P]),
        "nf_supervisor_init": (ctypes.c_int, [_P, _P]),
        "nf_supervisor_policy": (ctypes.c_int, [_P, _P, _P]),
        "nf_supervisor_update": (ctypes.c_int, [_P, _P, _P, _I64, ctypes.c_double]),
        "nf_endpoint_guard": (ctypes.c_int, [_P, _I64, _I64, _P, _P, _P]),
        "nf_sliced_layout_sizes": (ctypes.c_int, [_P, _I64, _P, _P]),
        "nf_sliced_layout": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P]),
        "nf_compact_signs": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _I64, _P, _I64, _P]),
        "nf_slice_workspace_bytes": (_SZ, [_I32, _I64]),
        "nf_slice_scales": (ctypes.c_int, [_P, _I64, _I32, _P, _P, _P, _I64, _I64, _P, _P, _P, _SZ, _P]),
        "nf_compact_signcount_reduce": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _P, _P, _P, _I64, _I64, _P,
                                                        _I32, _P, _P, _P]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        _lib = lib
    return lib


def _check(status):
    if status != NF_OK:
        raise NFError(status, load().nf_last_error().decode())


def _dev_ptr(t, dtype=None, name="tensor"):
    """Device pointer of a CUDA/HIP tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _rows(grads):
    """(pointer, worker_stride, W) of a [W, >= n] float32 device tensor."""
    if grads.dim() != 2 or grads.stride(1) != 1:
        raise ValueError("grads must be a [W, stride] tensor with unit element stride")
    return _dev_ptr(grads, torch.float32, "grads"), grads.stride(0), grads.shape[0]


def _bits_rows(bits):
    if bits is None:
        return None, 0
    if bits.dim() != 2 or bits.stride(1) != 1:
        raise ValueError("bits must be a [W, words] int64/uint64 tensor")
    if bits.dtype not in (torch.int64, torch.uint64):
        raise ValueError("bits must be 64-bit")
    return _dev_ptr(bits, None, "bits"), bits.stride(0)


def _words(mask):
    if mask is None:
        return None
    if mask.dtype not in (torch.int64, torch.uint64):
        raise ValueError("mask must be 64-bit words")
    return _dev_ptr(mask, None, "mask")


# --------------------------------------------------------------- host calls

def nf_abi_version():
    return load().nf_abi_version()


def nf_last_error():
    return load().nf_last_error().decode()


def nf_mask_from_segments(off, length, eligible, n):
    """Host segments -> host uint64 mask words (numpy)."""
    off = np.ascontiguousarray(off, dtype=np.int64)
    length = np.ascontiguousarray(length, dtype=np.int64)
    eligible = np.ascontiguousarray(eligible, dtype=np.uint8)
    mask = np.zeros(max((n + 63) // 64, 1), dtype=np.uint64)
    _check(load().nf_mask_from_segments(off.ctypes.data, length.ctypes.data, eligible.ctypes.data,
                                        len(off), n, mask.ctypes.data))
    return mask[: (n + 63) // 64]


def nf_workspace_bytes(W, n):
    return int(load().nf_workspace_bytes(W, n))


def nf_workspace_bytes_buckets(W, n_total, bucket_n):
    return int(load().nf_workspace_bytes_buckets(W, n_total, bucket_n))


def policy(admitted=1, veto=0, guard_ok=1, force_lowbit=0, decode_mode=NF_DECODE_SOFT,
           fp32_op=NF_FP32_SUM, kappa=4.0, format=NF_FORMAT_BINARY, tau=0.5):
    return nf_route_policy(admitted, veto, guard_ok, force_lowbit, decode_mode, fp32_op, kappa, format,
                           tau)


def nf_route_decide(stats, n, n_eligible, pol=None):
    """Host decision from a numpy STATS_DTYPE array; returns nf_route_decision."""
    st = np.ascontiguousarray(stats, dtype=STATS_DTYPE)
    d = nf_route_decision()
    pol = pol or policy()
    _check(load().nf_route_decide(st.ctypes.data, len(st), n, n_eligible, ctypes.byref(pol),
                                  ctypes.byref(d)))
    return d


# ------------------------------------------------------- controller (host)

def supervisor_profile(admit_step=0, cooldown_steps=10, guard_steps=0, short_cooldown_steps=0, ema_alpha=0.1,
                       slack=0.0, threshold=1.0, guard_scale=1.0, near_band=0.0, small_move=0.0,
                       target_share=1.0, share_margin=0.0):
    return nf_supervisor_profile(admit_step, cooldown_steps, guard_steps, short_cooldown_steps, ema_alpha, slack,
                                 threshold, guard_scale, near_band, small_move, target_share, share_margin)


def nf_supervisor_init(profile):
    st = nf_supervisor_state()
    _check(load().nf_supervisor_init(ctypes.byref(profile), ctypes.byref(st)))
    return st


def nf_supervisor_policy(profile, state, pol=None):
    """Sets admitted and veto of pol (a new default policy if None); returns it."""
    pol = pol if pol is not None else policy()
    _check(load().nf_supervisor_policy(ctypes.byref(profile), ctypes.byref(state), ctypes.byref(pol)))
    return pol


def nf_supervisor_update(profile, state, decisions, loss):
    """decisions: numpy DECISION_DTYPE array of the step's buckets (host)."""
    d = np.ascontiguousarray(decisions, dtype=DECISION_DTYPE)
    _check(load().nf_supervisor_update(ctypes.byref(profile), ctypes.byref(state),
                                       d.ctypes.data if len(d) else None, len(d), float(loss)))
    return state


def nf_endpoint_guard(model, n, n_eligible):
    """Returns (t_fp32, t_lowbit, guard_ok)."""
    tf, tl, ok = ctypes.c_double(), ctypes.c_double(), ctypes.c_int32()
    _check(load().nf_endpoint_guard(ctypes.byref(model), n, n_eligible, ctypes.byref(tf), ctypes.byref(tl),
                                    ctypes.byref(ok)))
    return tf.value, tl.value, bool(ok.value)


# ------------------------------------------------------------- device calls

def empty_workspace(nbytes, device="cuda"):
    """Caller-owned workspace (the torch allocator aligns to 512 bytes)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def nf_bucket_health(grads, n, mask, stats, ws, stream=None):
    g, stride, W = _rows(grads)
    _check(load().nf_bucket_health(g, stride, W, n, _words(mask), _dev_ptr(stats, torch.uint8, "stats"),
                                   _dev_ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)))


def nf_pack_signs(grads, n, mask, bits, stats, ws, stream=None):
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    _check(load().nf_pack_signs(g, stride, W, n, _words(mask), b, bstride,
                                _dev_ptr(stats, torch.uint8, "stats"), _dev_ptr(ws, torch.uint8, "ws"),
                                ws.numel(), _stream(stream)))


def nf_fp32_reduce(grads, n, mask, select, fp32_op, out, stream=None):
    g, stride, W = _rows(grads)
    _check(load().nf_fp32_reduce(g, stride, W, n, _words(mask), select, fp32_op,
                                 _dev_ptr(out, torch.float32, "out"), _stream(stream)))


def nf_signcount_reduce(bits, W, n, mask, scale, decode_mode, counts, out, stream=None):
    b, bstride = _bits_rows(bits)
    _check(load().nf_signcount_reduce(b, bstride, W, n, _words(mask),
                                      _dev_ptr(scale, torch.float32, "scale"), decode_mode,
                                      _dev_ptr(counts, torch.uint8, "counts"),
                                      _dev_ptr(out, torch.float32, "out"), _stream(stream)))


def nf_partial_counts(bits, W, P, n, partial, stream=None):
    """Node-local counts: partial is a uint8 device tensor [W // P, stride >= n]."""
    b, bstride = _bits_rows(bits)
    if partial is not None and (partial.dim() != 2 or partial.stride(1) != 1):
        raise ValueError("partial must be a 2-D row-major uint8 tensor")
    _check(load().nf_partial_counts(b, bstride, W, P, n, _dev_ptr(partial, torch.uint8, "partial"),
                                    partial.stride(0) if partial is not None else 0, _stream(stream)))


def nf_partial_count_reduce(partial, W, n, mask, scale, decode_mode, counts, out, stream=None):
    """Sum of the G partial-count rows of partial ([G, stride] uint8) and decode."""
    if partial.dim() != 2 or partial.stride(1) != 1:
        raise ValueError("partial must be a 2-D row-major uint8 tensor")
    _check(load().nf_partial_count_reduce(_dev_ptr(partial, torch.uint8, "partial"), partial.stride(0),
                                          partial.shape[0], W, n, _words(mask),
                                          _dev_ptr(scale, torch.float32, "scale"), decode_mode,
                                          _dev_ptr(counts, torch.uint8, "counts"),
                                          _dev_ptr(out, torch.float32, "out"), _stream(stream)))


def nf_stock_signcount(bits, W, n, mask, scale, decode_mode, replicas, counts, out, replica_stride,
                       stream=None):
    """Replicated count and decode: replica r at counts/out + r * replica_stride."""
    b, bstride = _bits_rows(bits)
    _check(load().nf_stock_signcount(b, bstride, W, n, _words(mask), _dev_ptr(scale, torch.float32, "scale"),
                                     decode_mode, replicas, _dev_ptr(counts, torch.uint8, "counts"),
                                     _dev_ptr(out, torch.float32, "out"), replica_stride, _stream(stream)))


class SlicedLayout:
    """Host layout tables of a slice table (nf_sliced_layout) and their device copies."""

    def __init__(self, off, length, n, device=None):
        self.off = np.ascontiguousarray(off, dtype=np.int64)
        self.len = np.ascontiguousarray(length, dtype=np.int64)
        self.S, self.n = len(self.off), int(n)
        ne, seg = ctypes.c_int64(), ctypes.c_int64()
        _check(load().nf_sliced_layout_sizes(self.len.ctypes.data if self.S else None, self.S, ctypes.byref(ne),
                                             ctypes.byref(seg)))
        self.n_eligible, self.segments = ne.value, seg.value
        nw = (self.n + 63) // 64
        self.mask = np.zeros(max(nw, 1), np.uint64)
        self.prefix = np.zeros(nw + 1, np.uint64)
        self.start = np.zeros(max((self.n_eligible + 63) // 64, 1), np.int64)
        self.wslice = np.zeros(max(nw, 1), np.int32)
        self.rstart = np.zeros(self.S + 1, np.int64)
        self.segp = np.zeros(self.S + 1, np.int64)
        _check(load().nf_sliced_layout(self.off.ctypes.data if self.S else None,
                                       self.len.ctypes.data if self.S else None, self.S, self.n,
                                       self.mask.ctypes.data, self.prefix.ctypes.data, self.start.ctypes.data,
                                       self.wslice.ctypes.data, self.rstart.ctypes.data, self.segp.ctypes.data))
        self.mask = self.mask[:nw]
        if device is not None:
            self.to(device)

    def to(self, device):
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.d_mask = t(self.mask.view(np.int64)) if len(self.mask) else torch.zeros(1, dtype=torch.int64, device=device)
        self.d_prefix = t(self.prefix.view(np.int64))
        self.d_start = t(self.start)
        self.d_wslice = t(self.wslice)
        self.d_rstart = t(self.rstart)
        self.d_segp = t(self.segp)
        self.d_off = t(self.off) if self.S else torch.zeros(1, dtype=torch.int64, device=device)
        self.d_len = t(self.len) if self.S else torch.zeros(1, dtype=torch.int64, device=device)
        return self


def nf_compact_signs(bits, W, n, lay, cbits, stream=None):
    b, bstride = _bits_rows(bits)
    c, cstride = _bits_rows(cbits)
    _check(load().nf_compact_signs(b, bstride, W, n, _words(lay.d_mask), lay.d_prefix.data_ptr(),
                                   lay.d_start.data_ptr(), lay.n_eligible, c, cstride, _stream(stream)))


def nf_slice_workspace_bytes(W, segments):
    return int(load().nf_slice_workspace_bytes(W, segments))


def nf_slice_scales(grads, lay, sums, scales, ws, stream=None):
    g, stride, W = _rows(grads)
    _check(load().nf_slice_scales(g, stride, W, lay.d_off.data_ptr(), lay.d_len.data_ptr(), lay.d_segp.data_ptr(),
                                  lay.S, lay.segments, _dev_ptr(sums, torch.float64, "sums"),
                                  _dev_ptr(scales, torch.float32, "scales"), _dev_ptr(ws, torch.uint8, "ws"),
                                  ws.numel(), _stream(stream)))


def nf_slice_scales_from_pass1(grads, n, lay, sums, scales, ws, stream=None):
    """Per-slice sums and scales from the partials a pass 1 over (grads, n,
    lay's mask) left in ws."""
    g, stride, W = _rows(grads)
    _check(load().nf_slice_scales_from_pass1(g, stride, W, n, lay.d_off.data_ptr(), lay.d_len.data_ptr(), lay.S,
                                             _dev_ptr(sums, torch.float64, "sums"),
                                             _dev_ptr(scales, torch.float32, "scales"),
                                             _dev_ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)))


def nf_compact_signcount_reduce(cbits, W, lay, scales, decode_mode, counts_c, out, stream=None):
    c, cstride = _bits_rows(cbits)
    _check(load().nf_compact_signcount_reduce(c, cstride, W, lay.n, _words(lay.d_mask), lay.d_prefix.data_ptr(),
                                              lay.d_wslice.data_ptr(), lay.d_rstart.data_ptr(), lay.S,
                                              lay.n_eligible, _dev_ptr(scales, torch.float32, "scales"),
                                              decode_mode, _dev_ptr(counts_c, torch.uint8, "counts_c"),
                                              _dev_ptr(out, torch.float32, "out"), _stream(stream)))


def nf_ternary_threshold(stats, n_eligible, tau):
    """Host thresholds from a numpy STATS_DTYPE array; returns float32 [W]."""
    st = np.ascontiguousarray(stats, dtype=STATS_DTYPE)
    theta = np.zeros(len(st), dtype=np.float32)
    _check(load().nf_ternary_threshold(st.ctypes.data, len(st), n_eligible, tau, theta.ctypes.data))
    return theta


def nf_pack_ternary(grads, n, mask, theta, bits, stream=None):
    """bits: int64 device tensor of 2W rows (positive planes, then negative)."""
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    if bits.shape[0] < 2 * W:
        raise ValueError("bits needs 2W rows")
    _check(load().nf_pack_ternary(g, stride, W, n, _words(mask), _dev_ptr(theta, torch.float32, "theta"), b,
                                  bstride, _stream(stream)))


def nf_ternary_reduce(bits, W, n, mask, scale, decode_mode, counts, out, stream=None):
    """counts (nullable): 2n uint8 (c+ then c-); out (nullable): n float32."""
    b, bstride = _bits_rows(bits)
    _check(load().nf_ternary_reduce(b, bstride, W, n, _words(mask), _dev_ptr(scale, torch.float32, "scale"),
                                    decode_mode, _dev_ptr(counts, torch.uint8, "counts"),
                                    _dev_ptr(out, torch.float32, "out"), _stream(stream)))


def nf_route_bucket(grads, n, mask, pol, bits, counts, out, stats, decision, ws, stream=None):
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    _check(load().nf_route_bucket(g, stride, W, n, _words(mask), ctypes.byref(pol), b, bstride,
                                  _dev_ptr(counts, torch.uint8, "counts"),
                                  _dev_ptr(out, torch.float32, "out"),
                                  _dev_ptr(stats, torch.uint8, "stats"),
                                  _dev_ptr(decision, torch.uint8, "decision"),
                                  _dev_ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)))


def nf_route_buckets(grads, n_total, bucket_n, mask, pol, bits, counts, out, stats, decisions, ws,
                     stream=None):
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    _check(load().nf_route_buckets(g, stride, W, n_total, bucket_n, _words(mask), ctypes.byref(pol),
                                   b, bstride, _dev_ptr(counts, torch.uint8, "counts"),
                                   _dev_ptr(out, torch.float32, "out"),
                                   _dev_ptr(stats, torch.uint8, "stats"),
                                   _dev_ptr(decisions, torch.uint8, "decisions"),
                                   _dev_ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)))


NF_STATIC_SCRATCH_BYTES = 64 << 20
NF_MAX_BUCKETS = 65535  # buckets per driver call at most


def nf_route_buckets_noalloc(grads, n_total, bucket_n, mask, pol, bits, counts, out, stats, decisions,
                             stream=None):
    """nf_route_buckets with the library's static device scratch instead of a
    caller workspace (no allocation by the call)."""
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    _check(load().nf_route_buckets_noalloc(g, stride, W, n_total, bucket_n, _words(mask), ctypes.byref(pol),
                                           b, bstride, _dev_ptr(counts, torch.uint8, "counts"),
                                           _dev_ptr(out, torch.float32, "out"),
                                           _dev_ptr(stats, torch.uint8, "stats"),
                                           _dev_ptr(decisions, torch.uint8, "decisions"), _stream(stream)))


def _offsets(offsets):
    """(int64 host array, its pointer, nb) of bucket offsets (nb + 1 values)."""
    o = np.ascontiguousarray(offsets, dtype=np.int64)
    if o.ndim != 1 or o.size < 1:
        raise ValueError("bucket offsets: a 1-D sequence of nb + 1 values")
    return o, o.ctypes.data_as(ctypes.c_void_p), int(o.size) - 1


def nf_bucket_table_bytes(W, offsets):
    o, p, nb = _offsets(offsets)
    return int(load().nf_bucket_table_bytes(W, p, nb))


def nf_bucket_table_init(W, offsets, table, stream=None):
    """Builds the device bucket table of these offsets into `table` (a uint8
    device tensor of at least nf_bucket_table_bytes); synchronises the stream."""
    o, p, nb = _offsets(offsets)
    _check(load().nf_bucket_table_init(W, p, nb, _dev_ptr(table, torch.uint8, "table"), table.numel(),
                                       _stream(stream)))


def nf_workspace_bytes_table(W, offsets):
    o, p, nb = _offsets(offsets)
    return int(load().nf_workspace_bytes_table(W, p, nb))


def nf_pass1_launches_table(W, offsets, sign_words=True):
    o, p, nb = _offsets(offsets)
    return int(load().nf_pass1_launches_table(W, p, nb, int(bool(sign_words))))


def nf_route_bucket_table(grads, offsets, table, mask, pol, bits, counts, out, stats, decisions, ws,
                          stream=None):
    g, stride, W = _rows(grads)
    b, bstride = _bits_rows(bits)
    o, p, nb = _offsets(offsets)
    _check(load().nf_route_bucket_table(g, stride, W, p, nb, _dev_ptr(table, torch.uint8, "table"),
                                        _words(mask), ctypes.byref(pol), b, bstride,
                                        _dev_ptr(counts, torch.uint8, "counts"),
                                        _dev_ptr(out, torch.float32, "out"),
                                        _dev_ptr(stats, torch.uint8, "stats"),
                                        _dev_ptr(decisions, torch.uint8, "decisions"),
                                        _dev_ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)))


def nf_set_phase_events(before_pass1=None, after_pass1=None, after_decide=None, after_pass2=None):
    """Raw hipEvent_t handles (ints) or None; all None turns recording off."""
    _check(load().nf_set_phase_events(before_pass1, after_pass1, after_decide, after_pass2))


def nf_pass1_launches(W, n_total, bucket_n, sign_words=True):
    """Pass-1 kernel launches of one nf_route_buckets call (profiling); pass
    sign_words=False for a pass 1 without sign words (G-Ternary, health)."""
    return int(load().nf_pass1_launches(W, n_total, bucket_n, int(bool(sign_words))))


def nf_pass1_chunk_elems(W, n_total, bucket_n):
    """(elements per pass-1 chunk, chunks of a full bucket) for these sizes
    (geometry query); (0, 0) for invalid sizes."""
    cpb = ctypes.c_int64(0)
    e = int(load().nf_pass1_chunk_elems(W, n_total, bucket_n, ctypes.byref(cpb)))
    return e, int(cpb.value)


# ------------------------------------------------------- result decoding

def stats_host(stats_dev, W, nb=1):
    """Device stats buffer (uint8) -> numpy STATS_DTYPE array [nb, W]."""
    raw = stats_dev[: nb * W * STATS_BYTES].cpu().numpy()
    return raw.view(STATS_DTYPE).reshape(nb, W)


def decisions_host(dec_dev, nb=1):
    raw = dec_dev[: nb * DECISION_BYTES].cpu().numpy()
    return raw.view(DECISION_DTYPE).reshape(nb)
