"""Worker rows longer than 2^31 elements (8.6 GB of FP32 each), which one
MI355X holds many of: every element index, bucket offset and count of the
path must be 64-bit.

Two rows of 2^31 + 4,161 elements (a ragged last word; 72% eligible, the
last FP32-routed run crossing 2^31) are routed twice in each format (G-Binary
and G-Ternary): as one bucket longer than 2^31 elements (nf_route_buckets),
and through the bucket-table driver as two buckets whose second one crosses
the 2^31 offset.  Nothing is sampled: each bucket's statistics come from the oracle
per worker row over the whole bucket, its decision from the oracle's
decision on them, and its bits, counts and outputs from the oracle's
element-wise steps over consecutive 64-aligned ranges covering it, in a
pool of host threads.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import (POOL, check_decision, check_output, check_stats, mask_bool, oracle_masks, oracle_policy,
                         same_f32)

pytestmark = pytest.mark.gpu

W = 2
N = (1 << 31) + 4_161
SPLIT = 1_610_612_736  # 1.5 * 2^30: the table's second bucket runs from here past 2^31
RANGE = 1 << 22        # elements per oracle range (a multiple of 64)


def check_bucket(gh, mask_o, a, e, st, d, bits, counts, out, pol, tag):
    """Bucket [a, e) of one call against the oracle, in full."""
    ka, ke = a // 64, (e + 63) // 64
    mw = np.ascontiguousarray(mask_o[ka:ke])
    n_b = e - a
    with ThreadPoolExecutor(POOL) as ex:
        ref_st = np.array(list(ex.map(lambda w: nfo.health(gh[w:w + 1, a:e], mw)[0], range(W))),
                          dtype=nfo.STATS_DTYPE)
    check_stats(st, ref_st, tag)
    rd = nfo.decide(ref_st, n_b, nfo.count_eligible(mw, n_b), oracle_policy(pol))
    check_decision(d, rd, tag)
    assert int(d["route"]) == nfo.ROUTE_L, (tag, int(d["route"]))
    q = nfo.decode_table(W, pol.decode_mode)

    def check_range(r0):
        r1 = min(r0 + RANGE, e)
        k0, k1 = r0 // 64, (r1 + 63) // 64
        g = gh[:, r0:r1]
        m = np.ascontiguousarray(mask_o[k0:k1])
        ref_bits = nfo.pack(g, m)
        where = f"{tag} [{r0}, {r1})"
        assert np.array_equal(bits[:, k0:k1].cpu().numpy().view(np.uint64), ref_bits), f"{where} bits"
        c = nfo.counts(ref_bits, r1 - r0)
        assert np.array_equal(counts[r0:r1].cpu().numpy(), c), f"{where} counts"
        y = nfo.fp32_path(g, pol.fp32_op)
        ref_out = nfo.output(m, r1 - r0, c, y, q, rd.scale, rd.route)
        check_output(out[r0:r1].cpu().numpy(), {"out": ref_out, "counts": c}, m, r1 - r0, W, d,
                     pol.decode_mode, where)
        return r1 - r0

    with ThreadPoolExecutor(POOL) as ex:
        assert sum(ex.map(check_range, range(a, e, RANGE))) == n_b


def check_bucket_ternary(gh, mask_o, a, e, st, d, bits, counts, out, pol, tag):
    """G-Ternary bucket [a, e) against the oracle, in full: the exact |g|
    sums make thresholds, planes, scale and decoded values bit-exact."""
    ka, ke = a // 64, (e + 63) // 64
    mw = np.ascontiguousarray(mask_o[ka:ke])
    n_b = e - a
    n_e = nfo.count_eligible(mw, n_b)
    with ThreadPoolExecutor(POOL) as ex:
        ref_st = np.array(list(ex.map(lambda w: nfo.health(gh[w:w + 1, a:e], mw)[0], range(W))),
                          dtype=nfo.STATS_DTYPE)
    check_stats(st, ref_st, tag, exact_abs=True)
    rd = nfo.decide(ref_st, n_b, n_e, oracle_policy(pol))
    check_decision(d, rd, tag, exact_scale=True)
    assert int(d["route"]) == nfo.ROUTE_L, (tag, int(d["route"]))
    th_gpu = nf.nf_ternary_threshold(st, n_e, pol.tau)
    th_ref = np.array([nfo.ternary_threshold(ref_st[w], n_e, pol.tau) for w in range(W)], np.float32)
    assert np.array_equal(th_gpu.view(np.uint32), th_ref.view(np.uint32)), f"{tag} thresholds"
    q = nfo.ternary_decode_table(W, pol.decode_mode)

    def check_range(r0):
        r1 = min(r0 + RANGE, e)
        k0, k1 = r0 // 64, (r1 + 63) // 64
        g = gh[:, r0:r1]
        m = np.ascontiguousarray(mask_o[k0:k1])
        where = f"{tag} [{r0}, {r1})"
        pos, neg = nfo.pack_ternary(g, m, th_ref)
        b = bits[:, k0:k1].cpu().numpy().view(np.uint64)
        assert np.array_equal(b[:W], pos) and np.array_equal(b[W:], neg), f"{where} planes"
        cp, cn = nfo.counts(pos, r1 - r0), nfo.counts(neg, r1 - r0)
        assert np.array_equal(counts[r0:r1].cpu().numpy(), cp), f"{where} c+"
        assert np.array_equal(counts[N + r0:N + r1].cpu().numpy(), cn), f"{where} c-"
        y = nfo.fp32_path(g, pol.fp32_op)
        ref = nfo.ternary_output(m, r1 - r0, cp, cn, y, q, rd.scale, W, rd.route)
        got = out[r0:r1].cpu().numpy()
        sel = mask_bool(m, r1 - r0)
        assert same_f32(got[~sel], ref[~sel]), f"{where} routed positions"
        assert same_f32(got[sel], ref[sel]), f"{where} decoded values"
        return r1 - r0

    with ThreadPoolExecutor(POOL) as ex:
        assert sum(ex.map(check_range, range(a, e, RANGE))) == n_b


@pytest.fixture(scope="module")
def rows():
    """The two rows on the device and their host copy (17.2 GB each)."""
    lay = synth.small(W, N, 2033, elig_frac=0.7, nruns=40)
    # 15 FP32-routed runs; the last one crosses 2^31, so routed sums are written beyond it
    assert int((lay.eligible == 0).sum()) == 15 and not lay.eligible[-1] and lay.starts[-1] < 1 << 31
    d = torch.device("cuda:0")
    print(f"[large rows] W={W} n={N:,} stride={lay.stride:,}", flush=True)
    g = torch.empty((W, lay.stride), dtype=torch.float32, device=d)
    synth.generate_device(lay, g)
    mask_dev, mask_o = oracle_masks(lay)
    mask = torch.from_numpy(mask_dev.view(np.int64)).to(d)
    gh = g[:, :N].cpu().numpy()
    yield g, mask, mask_o, gh
    del g, mask, gh
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fmt", [nf.NF_FORMAT_BINARY, nf.NF_FORMAT_TERNARY])
def test_rows_longer_than_2_31_elements(rows, fmt):
    g, mask, mask_o, gh = rows
    d = torch.device("cuda:0")
    planes = 2 if fmt == nf.NF_FORMAT_TERNARY else 1
    nw = (N + 63) // 64
    bits = torch.empty((planes * W, nw), dtype=torch.int64, device=d)
    counts = torch.empty((planes * N,), dtype=torch.uint8, device=d)
    out = torch.empty((N,), dtype=torch.float32, device=d)
    pol = nf.policy(format=fmt, tau=0.5)
    check = check_bucket_ternary if planes == 2 else check_bucket
    try:
        for kind, off in (("one bucket", np.array([0, N], np.int64)),
                          ("bucket table", np.array([0, SPLIT, N], np.int64))):
            nb = len(off) - 1
            bits.fill_(-1)
            counts.fill_(0xAB)
            out.fill_(float("nan"))
            stats = torch.zeros(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
            dec = torch.zeros(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
            if nb == 1:
                ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, N, N), d)
                nf.nf_route_buckets(g, N, N, mask, pol, bits, counts, out, stats, dec, ws)
            else:
                table = torch.empty(nf.nf_bucket_table_bytes(W, off), dtype=torch.uint8, device=d)
                nf.nf_bucket_table_init(W, off, table)
                ws = nf.empty_workspace(nf.nf_workspace_bytes_table(W, off), d)
                nf.nf_route_bucket_table(g, off, table, mask, pol, bits, counts, out, stats, dec, ws)
            torch.cuda.synchronize()
            st, dc = nf.stats_host(stats, W, nb), nf.decisions_host(dec, nb)
            for b in range(nb):
                tag = f"fmt {fmt}, {kind}, bucket {b} [{int(off[b])}, {int(off[b + 1])})"
                print(f"[large rows] checking {tag}", flush=True)
                check(gh, mask_o, int(off[b]), int(off[b + 1]), st[b], dc[b], bits, counts, out, pol, tag)
            del ws, stats, dec
    finally:
        del bits, counts, out
        torch.cuda.empty_cache()
