"""GPU parity of the compacted payload, per-slice scales and the sliced
decode against the oracle, through the C ABI.

Bars: compacted rows and compacted-order counts bit-exact; per-slice FP64
sums within 1e-12 relative (different fixed summation order); scales within
1e-6 relative (the FP32 bar of every parity test), and equal in the usual case; decoded values
exactly fl32(scale_gpu[s] * q[c]) and within 1e-6 of the oracle.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
from tests.nfgpu import same_f32, to_dev
from tests.test_sliced_layout import random_slices

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def case(W, n, count, max_len, seed):
    rng = np.random.default_rng(seed)
    off, ln = random_slices(n, rng, count, max_len)
    lay = nf.SlicedLayout(off, ln, n, device=DEV)
    g = rng.normal(0, 1e-3, (W, n)).astype(np.float32)
    g[rng.random((W, n)) < 0.02] = 0.0
    scale_w = np.float32(10.0) ** rng.uniform(-2, 1, W).astype(np.float32)
    g *= scale_w[:, None]
    return lay, g


CASES = [(1, 1000, 4, 300), (3, 4097, 9, 900), (16, 65_537, 12, 20_000), (8, 131_072, 2, 131_072),
         (64, 50_000, 30, 5000), (255, 6000, 7, 2000), (16, 300_000, 5, 200_000), (5, 10_000, 400, 40)]


@pytest.mark.parametrize("W,n,count,max_len", CASES)
def test_compact_signs_match_oracle(W, n, count, max_len):
    lay, g = case(W, n, count, max_len, W * 1000 + n)
    bits = nfo.pack(g, lay.mask)
    nwc = max((lay.n_eligible + 63) // 64, 1)
    cbits = torch.full((W, nwc + 2), -1, dtype=torch.int64, device=DEV)
    nf.nf_compact_signs(to_dev(bits.view(np.int64)), W, n, lay, cbits)
    torch.cuda.synchronize()
    got = cbits.cpu().numpy().view(np.uint64)
    want = nfo.pack_compact(g, lay.mask)
    assert np.array_equal(got[:, :want.shape[1]], want), "compacted rows"
    assert np.all(got[:, nwc:] == np.uint64(0xFFFFFFFFFFFFFFFF)), "words past the end untouched"


@pytest.mark.parametrize("W,n,count,max_len", CASES)
def test_slice_scales_match_oracle(W, n, count, max_len):
    lay, g = case(W, n, count, max_len, 7 * W + n)
    sums = torch.zeros((max(lay.S, 1), W), dtype=torch.float64, device=DEV)
    scales = torch.zeros(max(lay.S, 1), dtype=torch.float32, device=DEV)
    ws = nf.empty_workspace(nf.nf_slice_workspace_bytes(W, lay.segments), DEV)
    nf.nf_slice_scales(to_dev(g), lay, sums, scales, ws)
    torch.cuda.synchronize()
    ref_sums, ref_sc = nfo.slice_scales(g, lay.off, lay.len)
    s = sums.cpu().numpy()[:lay.S]
    sc = scales.cpu().numpy()[:lay.S]
    assert np.allclose(s, ref_sums, rtol=1e-12, atol=0), "slice sums"
    assert np.all(np.abs(sc - ref_sc) <= 1e-6 * np.abs(ref_sc)), "slice scales"
    assert np.mean(sc == ref_sc) >= 0.9, "scales equal in the usual case"


# (W, n, slice count, longest slice): tiny slices that share pass-1 chunks,
# slices across many chunks, a slice inside one chunk, many slices
FROM_PASS1 = CASES + [(16, 3_000_000, 40, 400_000), (16, 2_000_000, 3000, 600), (64, 700_000, 6, 300_000),
                      (4, 5_000_000, 25, 1_000_000), (255, 100_000, 50, 5000)]


@pytest.mark.parametrize("W,n,count,max_len", FROM_PASS1)
@pytest.mark.parametrize("first", ["pack", "pack_stats", "health", "route"])
def test_slice_scales_from_pass1(W, n, count, max_len, first):
    lay, g = case(W, n, count, max_len, 11 * W + n)
    gp = np.zeros((W, -(-n // 64) * 64), np.float32)  # pass 1 takes rows of 16-byte multiples
    gp[:, :n] = g
    gd = to_dev(gp)
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), DEV)
    nw = (n + 63) // 64
    stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=DEV)
    bits = torch.zeros((W, nw), dtype=torch.int64, device=DEV)
    if first == "pack":
        nf.nf_pack_signs(gd, n, lay.d_mask, bits, None, ws)
    elif first == "pack_stats":
        nf.nf_pack_signs(gd, n, lay.d_mask, bits, stats, ws)
    elif first == "health":
        nf.nf_bucket_health(gd, n, lay.d_mask, stats, ws)
    else:
        counts = torch.zeros(n, dtype=torch.uint8, device=DEV)
        out = torch.zeros(n, dtype=torch.float32, device=DEV)
        dec = torch.zeros(nf.DECISION_BYTES, dtype=torch.uint8, device=DEV)
        nf.nf_route_bucket(gd, n, lay.d_mask, nf.policy(), bits, counts, out, stats, dec, ws)
    S = max(lay.S, 1)
    sums = torch.full((S, W), float("nan"), dtype=torch.float64, device=DEV)
    scales = torch.full((S,), float("nan"), dtype=torch.float32, device=DEV)
    nf.nf_slice_scales_from_pass1(gd, n, lay, sums, scales, ws)
    # the two-pass statistics on the GPU, for comparison
    sums2 = torch.zeros((S, W), dtype=torch.float64, device=DEV)
    scales2 = torch.zeros(S, dtype=torch.float32, device=DEV)
    ws2 = nf.empty_workspace(nf.nf_slice_workspace_bytes(W, lay.segments), DEV)
    nf.nf_slice_scales(gd, lay, sums2, scales2, ws2)
    torch.cuda.synchronize()
    ref_sums, ref_sc = nfo.slice_scales(g, lay.off, lay.len)
    s1 = sums.cpu().numpy()[:lay.S]
    sc = scales.cpu().numpy()[:lay.S]
    assert np.allclose(s1, ref_sums, rtol=1e-12, atol=0), "slice sums"
    assert np.all(np.abs(sc - ref_sc) <= 1e-6 * np.abs(ref_sc)), "slice scales"
    assert np.mean(sc == ref_sc) >= 0.9, "scales equal in the usual case"
    assert np.allclose(s1, sums2.cpu().numpy()[:lay.S], rtol=1e-12, atol=0), "same sums as the two-pass statistics"
    if first == "pack_stats":
        # every slice's sums add up to the bucket's eligible |g| sums of pass 1
        st = nf.stats_host(stats, W)[0]
        assert np.allclose(s1.sum(axis=0), st["sum_abs_elig"], rtol=1e-12, atol=0)


@pytest.mark.parametrize("W,n,count,max_len", CASES)
@pytest.mark.parametrize("mode", [nfo.DECODE_SOFT, nfo.DECODE_MAJORITY])
def test_sliced_reduce_matches_oracle(W, n, count, max_len, mode):
    lay, g = case(W, n, count, max_len, 3 * W + n + mode)
    nE = lay.n_eligible
    cb = nfo.pack_compact(g, lay.mask)
    _, ref_sc = nfo.slice_scales(g, lay.off, lay.len)
    scales = to_dev(ref_sc)
    counts_c = torch.full((nE + 5,), 0xAB, dtype=torch.uint8, device=DEV)
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
    nf.nf_compact_signcount_reduce(to_dev(cb.view(np.int64)), W, lay, scales, mode, counts_c, out)
    torch.cuda.synchronize()
    c_c = counts_c.cpu().numpy()
    want_c = nfo.counts(cb, nE)
    assert np.array_equal(c_c[:nE], want_c), "compacted-order counts"
    assert np.all(c_c[nE:] == 0xAB)
    # the compacted counts are the positional counts at the eligible positions
    pos_c = nfo.counts(nfo.pack(g, lay.mask), n)
    elig = np.unpackbits(lay.mask.view(np.uint8), bitorder="little")[:n].astype(bool)
    assert np.array_equal(pos_c[elig], want_c), "compacted counts = positional counts"
    q = nfo.decode_table(W, mode)
    y = nfo.fp32_path(g)
    ref = nfo.sliced_output(lay.mask, pos_c, y, q, lay.off, lay.len, ref_sc)
    o = out.cpu().numpy()
    assert same_f32(o[elig], ref[elig]), "decoded values"
    assert np.all(np.isnan(o[~elig])), "positions outside the slices untouched"


def test_whole_sliced_path_against_oracle():
    """Pack (positional, G-Binary pass 1), compact, slice scales from the GPU, reduce: every output
    within the bar of the oracle's sliced bucket, decoded values exactly fl32(scale_gpu * q[c])."""
    W, n = 16, 400_000
    lay, g = case(W, n, 9, 120_000, 99)
    gd = to_dev(g)
    bits = torch.zeros((W, (n + 63) // 64), dtype=torch.int64, device=DEV)
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), DEV)
    nf.nf_pack_signs(gd, n, lay.d_mask, bits, None, ws)
    cbits = torch.zeros((W, (lay.n_eligible + 63) // 64), dtype=torch.int64, device=DEV)
    nf.nf_compact_signs(bits, W, n, lay, cbits)
    sums = torch.zeros((lay.S, W), dtype=torch.float64, device=DEV)
    scales = torch.zeros(lay.S, dtype=torch.float32, device=DEV)
    ws2 = nf.empty_workspace(nf.nf_slice_workspace_bytes(W, lay.segments), DEV)
    nf.nf_slice_scales(gd, lay, sums, scales, ws2)
    counts_c = torch.zeros(lay.n_eligible, dtype=torch.uint8, device=DEV)
    out = torch.zeros(n, dtype=torch.float32, device=DEV)
    nf.nf_compact_signcount_reduce(cbits, W, lay, scales, nfo.DECODE_SOFT, counts_c, out)
    torch.cuda.synchronize()
    assert np.array_equal(cbits.cpu().numpy().view(np.uint64), nfo.pack_compact(g, lay.mask))
    sc = scales.cpu().numpy()
    _, ref_sc = nfo.slice_scales(g, lay.off, lay.len)
    assert np.all(np.abs(sc - ref_sc) <= 1e-6 * np.abs(ref_sc))
    c = nfo.counts(nfo.pack(g, lay.mask), n)
    q = nfo.decode_table(W)
    elig = np.unpackbits(lay.mask.view(np.uint8), bitorder="little")[:n].astype(bool)
    o = out.cpu().numpy()
    exact = nfo.sliced_output(lay.mask, c, np.zeros(n, np.float32), q, lay.off, lay.len, sc)
    assert same_f32(o[elig], exact[elig]), "fl32(scale_gpu * q[c])"
    ref = nfo.sliced_output(lay.mask, c, np.zeros(n, np.float32), q, lay.off, lay.len, ref_sc)
    rel = np.abs(o[elig] - ref[elig]) / np.maximum(np.abs(ref[elig]), 1e-30)
    assert rel.max() <= 1e-6


def test_no_eligible_is_a_no_op():
    lay = nf.SlicedLayout([], [], 1000, device=DEV)
    bits = torch.zeros((4, 16), dtype=torch.int64, device=DEV)
    cbits = torch.zeros((4, 1), dtype=torch.int64, device=DEV)
    nf.nf_compact_signs(bits, 4, 1000, lay, cbits)
    torch.cuda.synchronize()
