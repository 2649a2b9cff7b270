"""GPU parity: every C-ABI entry point against the oracle, element by element.

Small cases span several pass-1 tiles and a ragged tail; the edge grid
covers n in {0, 1, 63, 64, 65, 4095, 1,000,013}, W in {1, 2, 3, 4, 8, 16, 31,
64, 255}, masks all-FP32, all-eligible, alternating words and random
unaligned runs, every policy combination, non-finite values, a zero worker
and norm spikes on both sides of kappa.  Bars are stated in nfgpu.py.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests import nfgpu as H

pytestmark = pytest.mark.gpu


def _mask(kind, n, seed):
    rng = np.random.default_rng(seed)
    nw = (n + 63) // 64
    if kind == "zeros":
        m = np.zeros(nw, np.uint64)
    elif kind == "ones":
        m = np.full(nw, np.uint64(0xFFFFFFFFFFFFFFFF))
    elif kind == "alt":
        m = np.where(np.arange(nw) % 2 == 0, np.uint64(0xFFFFFFFFFFFFFFFF), np.uint64(0)).astype(np.uint64)
    else:  # random unaligned runs
        lay = synth.small(1, n, seed, elig_frac=0.7, nruns=9)
        m = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    # bits past n are set on purpose: the library must ignore them
    if n % 64 and nw:
        m = m.copy()
        m[-1] |= np.uint64(0xFFFFFFFFFFFFFFFF) << np.uint64(n % 64)
    return m


def _grads(W, n, seed, sigma=(1e-6, 1e-2)):
    lay = synth.small(W, n, seed, sigma=sigma)
    return synth.generate_host(lay)


def _clean_mask(m, n):
    """The oracle's view: bits past n cleared."""
    m = np.array(m, np.uint64, copy=True)
    if n % 64 and len(m):
        m[-1] &= (np.uint64(1) << np.uint64(n % 64)) - np.uint64(1)
    return m


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available()
    nf.load()


# ------------------------------------------------------------- nf_fp32_reduce

@pytest.mark.parametrize("W", [1, 3, 16, 64, 255])
@pytest.mark.parametrize("n", [1, 65, 4095, 100_003])
def test_fp32_reduce(W, n):
    g = _grads(W, n, 100 + W + n)
    m = _mask("rand", n, W * 7 + n)
    gd, md = H.to_dev(g), H.to_dev(m, torch.int64)
    mb = H.mask_bool(_clean_mask(m, n), n)
    for op in (nf.NF_FP32_SUM, nf.NF_FP32_MEAN):
        y = nfo.fp32_path(np.ascontiguousarray(g[:, :n]), op)
        for sel, where in ((nf.NF_SEL_ROUTED, ~mb), (nf.NF_SEL_ELIGIBLE, mb), (nf.NF_SEL_ALL, np.ones(n, bool))):
            out = torch.full((n,), 7.0, dtype=torch.float32, device=H.dev())
            nf.nf_fp32_reduce(gd, n, md, sel, op, out)
            o = out.cpu().numpy()
            assert H.same_f32(o[where], y[where]), f"sel={sel} op={op}"
            assert np.all(o[~where] == 7.0), "unselected positions written"


# ----------------------------------------------------------- nf_bucket_health

@pytest.mark.parametrize("W", [1, 2, 3, 8, 16, 31, 64, 255])
@pytest.mark.parametrize("n", [0, 1, 64, 65, 4095, 200_001])
def test_bucket_health(W, n):
    g = _grads(W, n, 200 + W + n)
    if n > 10:
        g[W // 2, n // 3] = np.nan
        g[0, n - 1] = -np.inf
    m = _mask("rand", n, W + n)
    stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=H.dev())
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n))
    nf.nf_bucket_health(H.to_dev(g), n, H.to_dev(m if len(m) else np.zeros(1, np.uint64), torch.int64),
                        stats, ws)
    ref = nfo.health(np.ascontiguousarray(g[:, :n]), _clean_mask(m, n))
    # without sign words the |g| sums are the exact sums rounded once
    H.check_stats(nf.stats_host(stats, W)[0], ref, exact_abs=True)


# -------------------------------------------------------------- nf_pack_signs

@pytest.mark.parametrize("W", [1, 4, 16, 31, 64, 255])
@pytest.mark.parametrize("n", [1, 63, 64, 65, 4095, 150_017])
@pytest.mark.parametrize("mkind", ["zeros", "ones", "alt", "rand"])
def test_pack_signs(W, n, mkind):
    g = _grads(W, n, 300 + W + n)
    g[:, : min(n, 13)] = np.array([0.0, -0.0, 1e-45, -1e-45, np.nan, np.inf, -np.inf, 1.0, -1.0,
                                   3e38, -3e38, 1e-40, -1e-40], np.float32)[: min(n, 13)]
    m = _mask(mkind, n, W + 3 * n)
    nw = (n + 63) // 64
    bits = torch.full((W, nw + 2), -1, dtype=torch.int64, device=H.dev())
    stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=H.dev())
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n))
    nf.nf_pack_signs(H.to_dev(g), n, H.to_dev(m, torch.int64), bits, stats, ws)
    cm = _clean_mask(m, n)
    ref = nfo.pack(np.ascontiguousarray(g[:, :n]), cm)
    b = bits.cpu().numpy().view(np.uint64)
    assert np.array_equal(b[:, :nw], ref), "bits"
    assert np.all(b[:, nw:] == np.uint64(0xFFFFFFFFFFFFFFFF)), "bits written past the row"
    H.check_stats(nf.stats_host(stats, W)[0], nfo.health(np.ascontiguousarray(g[:, :n]), cm))
    # without statistics
    bits2 = torch.zeros((W, nw), dtype=torch.int64, device=H.dev())
    nf.nf_pack_signs(H.to_dev(g), n, H.to_dev(m, torch.int64), bits2, None, ws)
    assert np.array_equal(bits2.cpu().numpy().view(np.uint64), ref), "bits without stats"


# -------------------------------------------------------- nf_signcount_reduce

@pytest.mark.parametrize("W", [1, 2, 3, 8, 16, 64, 255])
@pytest.mark.parametrize("n", [1, 64, 65, 4095, 123_457])
@pytest.mark.parametrize("mode", [nf.NF_DECODE_SOFT, nf.NF_DECODE_MAJORITY])
def test_signcount_reduce(W, n, mode):
    rng = np.random.default_rng(W * 1000 + n)
    nw = (n + 63) // 64
    m = _mask("rand", n, n + W)
    cm = _clean_mask(m, n)
    g = _grads(W, n, 400 + W + n)
    bits = nfo.pack(np.ascontiguousarray(g[:, :n]), cm)
    c = nfo.counts(bits, n)
    scale = np.float32(rng.uniform(1e-5, 1e-1))
    q = nfo.decode_table(W, mode)
    want = np.where(H.mask_bool(cm, n), (scale * q[c]).astype(np.float32), np.float32(-5.0))
    bd = H.to_dev(np.concatenate([bits, np.zeros((W, 1), np.uint64)], axis=1), torch.int64)
    counts = torch.zeros(n, dtype=torch.uint8, device=H.dev())
    out = torch.full((n,), -5.0, dtype=torch.float32, device=H.dev())
    sd = torch.tensor([scale], dtype=torch.float32, device=H.dev())
    nf.nf_signcount_reduce(bd, W, n, H.to_dev(m, torch.int64), sd, mode, counts, out)
    assert np.array_equal(counts.cpu().numpy(), c), "counts"
    assert H.same_f32(out.cpu().numpy(), want), "decoded values"
    # counts only
    counts2 = torch.zeros(n, dtype=torch.uint8, device=H.dev())
    nf.nf_signcount_reduce(bd, W, n, None, None, mode, counts2, None)
    assert np.array_equal(counts2.cpu().numpy(), c), "counts only"


# ------------------------------------------------------------ nf_route_bucket

EDGE_W = [1, 2, 3, 4, 8, 16, 31, 64, 255]
EDGE_N = [0, 1, 63, 64, 65, 4095, 65_537]


@pytest.mark.parametrize("W", EDGE_W)
@pytest.mark.parametrize("n", EDGE_N)
@pytest.mark.parametrize("mkind", ["zeros", "ones", "alt", "rand"])
def test_route_bucket_edges(W, n, mkind):
    g = _grads(W, n, 500 + W + n)
    m = _mask(mkind, n, 3 * W + n)
    run = H.Bucket(g, m, n)
    pol = nf.policy()
    res = run.route(pol)
    H.check_route(res, g, _clean_mask(m, n), n, pol, what=f"W={W} n={n} {mkind}")


@pytest.mark.parametrize("W", [4, 16, 64])
def test_route_bucket_large(W):
    n = 1_000_013
    g = _grads(W, n, 600 + W)
    m = _mask("rand", n, W)
    run = H.Bucket(g, m, n)
    pol = nf.policy()
    res = run.route(pol)
    H.check_route(res, g, _clean_mask(m, n), n, pol, what=f"W={W} n={n}")


@pytest.mark.parametrize("W", [65, 128, 129, 200])
@pytest.mark.parametrize("kind", ["default", "veto_mean", "forced_mean"])
def test_route_row_groups(W, kind):
    """Above 64 workers pass 1 reads the worker rows in groups of up to 64, the
    FP32 sums at routed positions carried from one group to the next in the
    output.  Two buckets: the first clean, the second with a NaN and an
    infinity at routed positions in different groups and a routed position
    whose FP32 sum overflows only after the first group (every worker
    3e38).  Policies: the fused route, a vetoed route (FP32 sums over every
    element, no sign words, exact |g| sums) and forced low-bit, the last two
    with the FP32 mean (divided once, after the last group)."""
    n, bn = 300_007, 150_016
    g = _grads(W, n, 800 + W)
    el = np.random.default_rng(801 + W).random(n) < 0.8  # element-wise: routed positions in every chunk
    m = np.packbits(np.concatenate([el, np.zeros((-n) % 64, bool)]), bitorder="little").view(np.uint64).copy()
    routed = np.nonzero(~el)[0]
    routed = routed[routed >= bn]
    g[70 % W, routed[10]] = np.nan
    g[W - 1, routed[20]] = np.inf
    g[:, routed[30]] = np.float32(3e38)
    pol = {"default": nf.policy(),
           "veto_mean": nf.policy(veto=1, fp32_op=nf.NF_FP32_MEAN),
           "forced_mean": nf.policy(force_lowbit=1, fp32_op=nf.NF_FP32_MEAN)}[kind]
    run = H.Bucket(g, m, n, bucket_n=bn)
    res = run.route(pol)
    H.check_route(res, g, m, n, pol, bucket_n=bn, what=f"W={W} {kind}")
    if kind == "default":
        assert int(res["dec"][0]["route"]) == nfo.ROUTE_L
    assert np.isinf(res["out"][routed[30]])


@pytest.mark.parametrize("admitted,veto,guard_ok,force", [(a, v, gk, f) for a in (0, 1) for v in (0, 1)
                                                          for gk in (0, 1) for f in (0, 1)])
@pytest.mark.parametrize("mode,op", [(nf.NF_DECODE_SOFT, nf.NF_FP32_SUM),
                                     (nf.NF_DECODE_MAJORITY, nf.NF_FP32_MEAN)])
def test_route_policy_table(admitted, veto, guard_ok, force, mode, op):
    W, n = 6, 50_001
    g = _grads(W, n, 700)
    m = _clean_mask(_mask("rand", n, 701), n)
    pol = nf.policy(admitted=admitted, veto=veto, guard_ok=guard_ok, force_lowbit=force,
                    decode_mode=mode, fp32_op=op)
    run = H.Bucket(g, m, n)
    res = run.route(pol)
    H.check_route(res, g, m, n, pol, what=f"policy {admitted}{veto}{guard_ok}{force}")


def _fault_cases():
    W, n = 8, 40_000
    cases = {}
    rng = np.random.default_rng(9)
    base = (rng.standard_normal((W, n)) * 1e-3).astype(np.float32)
    g = base.copy(); g[3, 17] = np.nan; cases["nan"] = g
    g = base.copy(); g[5, 39_999] = np.inf; cases["posinf"] = g
    g = base.copy(); g[0, 0] = -np.inf; cases["neginf"] = g
    g = base.copy(); g[6, :] = 0.0; cases["zero_worker"] = g
    g = base.copy(); g[2] = base[0] * np.float32(3.9); g[1] = base[0]; g[3] = base[0]; g[4] = base[0]
    cases["x3.9"] = g
    g = g.copy(); g[2] = base[0] * np.float32(4.1); cases["x4.1"] = g
    g = g.copy(); g[2] = base[0] * np.float32(4.0); cases["x4.0"] = g
    g = base.copy(); g[1] *= 10; cases["x10"] = g
    return cases


@pytest.mark.parametrize("W", [3, 16, 64])
def test_route_fp32_overflow(W):
    """Finite inputs whose FP32 sums overflow: +Inf and -Inf at routed
    positions (added in worker order, as the oracle does), NaN where
    opposite overflows meet; the statistics stay finite in FP64."""
    n = 70_001
    g = _grads(W, n, 1200 + W)
    m = _clean_mask(_mask("rand", n, 1201), n)
    routed = np.flatnonzero(~H.mask_bool(m, n))
    g[:, routed[:50]] = np.float32(3e38)
    g[:, routed[50:100]] = np.float32(-3e38)
    g[: W // 2 + 1, routed[100:150]] = np.float32(3e38)
    g[W // 2 + 1:, routed[100:150]] = np.float32(-3e38)
    for pol in (nf.policy(), nf.policy(fp32_op=nf.NF_FP32_MEAN), nf.policy(veto=1)):
        run = H.Bucket(g, m, n)
        res = run.route(pol)
        H.check_route(res, g, m, n, pol, what=f"overflow W={W}")


@pytest.mark.parametrize("case", list(_fault_cases().keys()))
@pytest.mark.parametrize("force", [0, 1])
def test_route_faults(case, force):
    g = _fault_cases()[case]
    W, n = g.shape
    m = _clean_mask(_mask("rand", n, 11), n)
    pol = nf.policy(force_lowbit=force)
    run = H.Bucket(g, m, n)
    res = run.route(pol)
    H.check_route(res, g, m, n, pol, what=case)
    d = res["dec"][0]
    expect_f = case not in ("x3.9", "x4.0")
    assert int(d["route"]) == (nf.NF_ROUTE_LOWBIT if (force or not expect_f) else nf.NF_ROUTE_FALLBACK)


# ----------------------------------------------------------- nf_route_buckets

@pytest.mark.parametrize("W", [3, 16, 64])
def test_route_buckets_flat(W):
    # buckets of 4096 * 5 elements; the last one ragged; one all-FP32 bucket
    bucket_n = 4096 * 5
    n = bucket_n * 6 + 1_234
    g = _grads(W, n, 800 + W)
    m = _clean_mask(_mask("rand", n, 801), n)
    m[(2 * bucket_n) // 64: (3 * bucket_n) // 64] = 0
    for pol in (nf.policy(), nf.policy(fp32_op=nf.NF_FP32_MEAN, decode_mode=nf.NF_DECODE_MAJORITY),
                nf.policy(veto=1)):
        run = H.Bucket(g, m, n, bucket_n)
        res = run.route(pol)
        H.check_route(res, g, m, n, pol, bucket_n=bucket_n, what=f"flat W={W}")
        assert int(res["dec"][2]["route"]) == nf.NF_ROUTE_PLAIN


def test_route_without_counts():
    W, n = 16, 70_000
    g = _grads(W, n, 900)
    m = _clean_mask(_mask("rand", n, 901), n)
    run = H.Bucket(g, m, n)
    res = run.route(nf.policy(), with_counts=False)
    H.check_route(res, g, m, n, nf.policy(), with_counts=False)
    assert np.all(run.counts.cpu().numpy() == 0xAB), "counts written although NULL"


def test_determinism():
    W, n = 16, 300_001
    g = _grads(W, n, 1000)
    g[4, 1000] = np.nan
    m = _clean_mask(_mask("rand", n, 1001), n)
    run = H.Bucket(g, m, n)
    for pol in (nf.policy(), nf.policy(force_lowbit=1)):
        a = run.route(pol)
        b = run.route(pol)
        for k in ("bits", "counts"):
            assert np.array_equal(a[k], b[k]), k
        assert a["out"].view(np.uint32).tobytes() == b["out"].view(np.uint32).tobytes()
        assert a["stats"].tobytes() == b["stats"].tobytes()
        assert a["dec"].tobytes() == b["dec"].tobytes()


def test_non_default_streams_concurrent():
    W, n = 8, 200_000
    g1, g2 = _grads(W, n, 1100), _grads(W, n, 1101)
    m = _clean_mask(_mask("rand", n, 1102), n)
    r1, r2 = H.Bucket(g1, m, n), H.Bucket(g2, m, n)
    r1.alloc()
    r2.alloc()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for r, s in ((r1, s1), (r2, s2)):
        with torch.cuda.stream(s):
            nf.nf_route_bucket(r.g, n, r.m, nf.policy(), r.bits, r.counts, r.out, r.stats, r.dec, r.ws,
                               stream=s)
    torch.cuda.synchronize()
    for r, g in ((r1, g1), (r2, g2)):
        res = dict(bits=r.bits.cpu().numpy().view(np.uint64), counts=r.counts.cpu().numpy()[:n],
                   out=r.out.cpu().numpy()[:n], stats=nf.stats_host(r.stats, W),
                   dec=nf.decisions_host(r.dec))
        H.check_route(res, g, m, n, nf.policy())
