"""Helpers of the GPU parity tests: run the HIP path through the C ABI and
compare it with the oracle on the same seeded inputs.

Bars: bit-exact for bits, counts, masks, n_E, routes, reasons, modeled
bytes and FP32 sums; within 1e-6 relative for the FP64 statistics, the FP32
scale and the decoded values where the GPU adds its FP64 sums in another
order than the exact sum the oracle rounds once (with sign words: the scale
may then land one FP32 ulp away; decoded values are checked to be exactly
fl32(scale_gpu * q[c])).  Where the library rounds the exact |g| sum too (no
sign words: the G-Ternary route, nf_bucket_health, routes fixed before
reading), that sum, the scale and the decoded values are bit-exact.  NaN
equals NaN.
"""
import numpy as np
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth

REL_TOL = 1e-6
POOL = 16  # host threads for oracle work: the CPU share of one GPU on the test box


def oracle_masks(lay):
    """(the mask the GPU reads, from the library's host builder; the oracle's
    own mask from the same segments), checked equal word for word."""
    segs = synth.mask_segments(lay)
    m_dev = nf.nf_mask_from_segments(*segs, lay.n_total)
    m_o = nfo.mask_from_segments(*segs, lay.n_total)
    assert np.array_equal(m_dev, m_o), f"{lay.name}: mask builders disagree"
    return m_dev, m_o


def dev():
    return torch.device("cuda:0")


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.to(dev())


def mask_bool(mask_words, n):
    return np.unpackbits(np.ascontiguousarray(mask_words, np.uint64).view(np.uint8),
                         bitorder="little")[:n].astype(bool)


def same_f32(a, b):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    if a.shape != b.shape:
        return False
    na, nb_ = np.isnan(a), np.isnan(b)
    return np.array_equal(na, nb_) and np.array_equal(a[~na].view(np.uint32), b[~nb_].view(np.uint32))


def rel_close(a, b, tol=REL_TOL):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    with np.errstate(invalid="ignore"):  # inf - inf where both are infinite: covered by same_inf
        ok = both_nan | same_inf | (np.abs(a - b) <= tol * np.abs(b)) | (a == b)
        return bool(np.all(ok)), (float(np.max(np.abs(a - b)[~(both_nan | same_inf)] /
                                              np.maximum(np.abs(b[~(both_nan | same_inf)]), 1e-300)))
                                  if np.any(~(both_nan | same_inf)) else 0.0)


def same_f64(a, b):
    """Bitwise equality of FP64 arrays, any NaN equal to any NaN."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    na, nb_ = np.isnan(a), np.isnan(b)
    return np.array_equal(na, nb_) and np.array_equal(a[~na].view(np.uint64), b[~nb_].view(np.uint64))


def check_stats(gpu_st, ref_st, what="", exact_abs=False):
    """Non-finite counts exact; sums within 1e-6; with exact_abs the |g| sums
    bit for bit."""
    assert np.array_equal(gpu_st["nonfinite"], ref_st["nonfinite"]), f"{what} nonfinite"
    for f in ("sum_abs_elig", "sum_sq"):
        ok, err = rel_close(gpu_st[f], ref_st[f])
        assert ok, f"{what} {f}: max rel err {err}"
    if exact_abs:
        bad = np.nonzero(~((gpu_st["sum_abs_elig"] == ref_st["sum_abs_elig"]) |
                           (np.isnan(gpu_st["sum_abs_elig"]) & np.isnan(ref_st["sum_abs_elig"]))))[0]
        assert bad.size == 0, (f"{what} exact |g| sums differ for workers {bad[:8]}: "
                               f"{gpu_st['sum_abs_elig'][bad[:4]]} vs {ref_st['sum_abs_elig'][bad[:4]]}")


def check_decision(d, rd, what="", exact_scale=False):
    assert int(d["route"]) == rd.route, f"{what} route {int(d['route'])} != {rd.route}"
    assert int(d["reasons"]) == rd.reasons, f"{what} reasons {int(d['reasons'])} != {rd.reasons}"
    assert int(d["n_eligible"]) == rd.n_eligible, f"{what} n_E"
    assert float(d["bytes_route"]) == rd.bytes_route and float(d["bytes_fp32"]) == rd.bytes_fp32, \
        f"{what} modeled bytes"
    s, rs = np.float32(d["scale"]), np.float32(rd.scale)
    if exact_scale:
        assert same_f32(s, rs), f"{what} scale {s!r} != {rs!r} (bit-exact)"
    assert s == rs or (np.isnan(s) and np.isnan(rs)) or abs(float(s) - float(rs)) <= REL_TOL * abs(float(rs)), \
        f"{what} scale {s} {rs}"


def check_output(out, ref, mask_words, n, W, decision, decode_mode, what=""):
    """out against the oracle: bit-exact off the low-bit positions; on them,
    exactly fl32(scale_gpu * q[c]) and within 1e-6 of the oracle."""
    m = mask_bool(mask_words, n)
    route = int(decision["route"])
    if route != nfo.ROUTE_L:
        assert same_f32(out, ref["out"]), f"{what} FP32 output (route {route})"
        return
    assert same_f32(out[~m], ref["out"][~m]), f"{what} routed positions"
    q = nfo.decode_table(W, decode_mode)
    want = (np.float32(decision["scale"]) * q[ref["counts"][m]]).astype(np.float32)
    assert same_f32(out[m], want), f"{what} decoded values vs fl32(scale*q[c])"
    ok, err = rel_close(out[m], ref["out"][m])
    assert ok, f"{what} decoded values vs oracle: max rel err {err}"


class Bucket:
    """Device buffers of one flat buffer of buckets, and one call of the path."""

    def __init__(self, g_host, mask_words, n_total, bucket_n=None):
        self.g_host = g_host
        self.W = g_host.shape[0]
        self.n = n_total
        self.bucket_n = bucket_n or max(n_total, 1)
        self.nb = max(1, -(-n_total // self.bucket_n))
        self.mask = np.ascontiguousarray(mask_words, np.uint64)
        self.nw = (n_total + 63) // 64
        self.g = to_dev(g_host)
        self.m = to_dev(self.mask if self.mask.size else np.zeros(1, np.uint64), torch.int64)

    def alloc(self, bits_pad=3):
        d = dev()
        self.bits = torch.full((self.W, self.nw + bits_pad), -1, dtype=torch.int64, device=d)
        self.counts = torch.full((max(self.n, 1),), 0xAB, dtype=torch.uint8, device=d)
        self.out = torch.full((max(self.n, 1),), float("nan"), dtype=torch.float32, device=d)
        self.stats = torch.zeros(self.nb * self.W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        self.dec = torch.zeros(self.nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        if self.nb == 1:
            ws = nf.nf_workspace_bytes(self.W, self.n)
        else:
            ws = nf.nf_workspace_bytes_buckets(self.W, self.n, self.bucket_n)
        self.ws = nf.empty_workspace(ws, d)

    def route(self, pol, with_counts=True):
        self.alloc()
        if self.nb == 1 and self.bucket_n >= self.n:
            nf.nf_route_bucket(self.g, self.n, self.m, pol, self.bits,
                               self.counts if with_counts else None, self.out, self.stats, self.dec,
                               self.ws)
        else:
            nf.nf_route_buckets(self.g, self.n, self.bucket_n, self.m, pol, self.bits,
                                self.counts if with_counts else None, self.out, self.stats, self.dec,
                                self.ws)
        torch.cuda.synchronize()
        return dict(bits=self.bits.cpu().numpy().view(np.uint64),
                    counts=self.counts.cpu().numpy()[: self.n],
                    out=self.out.cpu().numpy()[: self.n],
                    stats=nf.stats_host(self.stats, self.W, self.nb),
                    dec=nf.decisions_host(self.dec, self.nb))


def oracle_bucket(g_host, mask_words, n, pol, b=0, bucket_n=None):
    """Oracle on bucket b of a flat buffer."""
    bucket_n = bucket_n or max(n, 1)
    a = b * bucket_n
    e = min(a + bucket_n, n)
    gm = np.ascontiguousarray(g_host[:, a:e])
    mw = np.ascontiguousarray(mask_words[a // 64: (e + 63) // 64])
    return nfo.reduce_bucket(gm, mw, pol), a, e


def oracle_policy(pol):
    return nfo.policy(admitted=pol.admitted, veto=pol.veto, guard_ok=pol.guard_ok,
                      force_lowbit=pol.force_lowbit, decode_mode=pol.decode_mode,
                      fp32_op=pol.fp32_op, kappa=pol.kappa, format=pol.format, tau=pol.tau)


def check_route(res, g_host, mask_words, n, pol, bucket_n=None, with_counts=True, what="",
                buckets=None):
    """Every output of a route call against the oracle, bucket by bucket."""
    bucket_n = bucket_n or max(n, 1)
    nb = max(1, -(-n // bucket_n))
    W = g_host.shape[0]
    opol = oracle_policy(pol)
    predecided = (not pol.admitted) or (not pol.force_lowbit and (pol.veto or not pol.guard_ok))
    for b in (range(nb) if buckets is None else buckets):
        ref, a, e = oracle_bucket(g_host, mask_words, n, opol, b, bucket_n)
        tag = f"{what} bucket {b}"
        d = res["dec"][b]
        check_decision(d, ref["decision"], tag, exact_scale=predecided)
        check_stats(res["stats"][b], ref["stats"], tag, exact_abs=predecided)
        ka, ke = a // 64, (e + 63) // 64
        if not predecided:
            assert np.array_equal(res["bits"][:, ka:ke], ref["bits"]), f"{tag} bits"
        if with_counts and int(d["route"]) == nfo.ROUTE_L:
            assert np.array_equal(res["counts"][a:e], ref["counts"]), f"{tag} counts"
        check_output(res["out"][a:e], ref, mask_words[ka:ke], e - a, W, d, pol.decode_mode, tag)
