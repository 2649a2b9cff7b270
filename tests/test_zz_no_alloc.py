"""The allocation-free driver nf_route_buckets_noalloc against
nf_route_buckets with a caller workspace, through the C ABI.

Both run the same kernels in the same order, so every output must be equal
bit for bit: sign words (or G-Ternary planes), counts, outputs, statistics
and decisions.  Two calls in a row on the library's one static scratch, the
second with a smaller input, check that nothing the first call left in the
scratch reaches the second's results.  A size beyond the scratch is
rejected before anything runs.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_route, to_dev

pytestmark = pytest.mark.gpu


def run_both(g_host, mask, n, bucket_n, pol, planes=1):
    W = g_host.shape[0]
    nb = max(1, -(-n // bucket_n))
    nw = (n + 63) // 64
    d = torch.device("cuda:0")
    gd, md = to_dev(g_host), to_dev(mask, torch.int64)
    res = []
    for noalloc in (False, True):
        bits = torch.full((planes * W, nw + 1), -1, dtype=torch.int64, device=d)
        counts = torch.full((planes * n,), 0xAB, dtype=torch.uint8, device=d)
        out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.full((nb * W * nf.STATS_BYTES,), 0x5A, dtype=torch.uint8, device=d)
        dec = torch.full((nb * nf.DECISION_BYTES,), 0x5A, dtype=torch.uint8, device=d)
        if noalloc:
            nf.nf_route_buckets_noalloc(gd, n, bucket_n, md, pol, bits, counts, out, stats, dec)
        else:
            ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bucket_n), d)
            ws.fill_(0xC3)  # stale contents must not matter either
            nf.nf_route_buckets(gd, n, bucket_n, md, pol, bits, counts, out, stats, dec, ws)
        torch.cuda.synchronize()
        res.append({k: v.cpu().numpy() for k, v in
                    dict(bits=bits, counts=counts, out=out, stats=stats, dec=dec).items()})
    a, b = res
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), f"{k} differs"
    return dict(bits=a["bits"].view(np.uint64), counts=a["counts"], out=a["out"],
                stats=nf.stats_host(torch.from_numpy(a["stats"]), W, nb),
                dec=nf.decisions_host(torch.from_numpy(a["dec"]), nb))


def test_noalloc_two_calls_second_smaller():
    # first call: a GPT-layout workload of 201 buckets x 16 workers, G-Binary
    lay = synth.scaled(synth.gpt1p3b, 256)
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), lay.n_total)
    pol = nf.policy()
    res = run_both(g, mask, lay.n_total, lay.bucket_n, pol)
    check_route(res, g, mask, lay.n_total, pol, bucket_n=lay.bucket_n, what="noalloc gpt/256",
                buckets=[0, 1, lay.nb // 2, lay.nb - 1])
    # second call, smaller: 7 workers, non-finite values, G-Ternary format
    lay2 = synth.small(7, 100_003, 42, bucket_n=16_384, elig_frac=0.8)
    g2 = synth.generate_host(lay2)
    g2[3, 777] = np.inf
    mask2 = nfo.mask_from_segments(*synth.mask_segments(lay2), lay2.n_total)
    pol2 = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=1)
    run_both(g2, mask2, lay2.n_total, lay2.bucket_n, pol2, planes=2)
    # third, smaller again, G-Binary route F on the non-finite bucket
    res3 = run_both(g2[:, :50_000].copy(), mask2[: (50_000 + 63) // 64], 50_000, 16_384, nf.policy())
    assert int(res3["dec"]["route"][0]) == nf.NF_ROUTE_FALLBACK


def test_noalloc_rejects_sizes_beyond_the_scratch():
    d = torch.device("cuda:0")
    W, n = 255, 100_000_000
    assert nf.nf_workspace_bytes(W, n) > nf.NF_STATIC_SCRATCH_BYTES
    g = torch.zeros((W, 64), dtype=torch.float32, device=d)  # only pointers: rejected before any launch
    m = torch.zeros(1, dtype=torch.int64, device=d)
    bits = torch.zeros((W, 1), dtype=torch.int64, device=d)
    out = torch.zeros(64, dtype=torch.float32, device=d)
    st = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    dec = torch.zeros(nf.DECISION_BYTES, dtype=torch.uint8, device=d)
    lib = nf.load()
    rc = lib.nf_route_buckets_noalloc(g.data_ptr(), n, W, n, n, m.data_ptr(), None, bits.data_ptr(), 1,
                                      None, out.data_ptr(), st.data_ptr(), dec.data_ptr(), None)
    assert rc == nf.NF_ERR_WORKSPACE, rc
    assert b"static" in lib.nf_last_error()
