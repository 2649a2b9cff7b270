"""Pass-1 launch shapes against the oracle: problems of at most 4,096
chunks in one launch, larger ones in launches of 256 chunks (1,024 without
sign words) that may overlap, buckets of more than 512 chunks (64 above 32
workers: their per-chunk partials are summed in groups before the
decision), and flat buffers of several buckets.  Every output of every
bucket is checked (G-Binary and G-Ternary)."""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_decision, check_output, check_stats, oracle_policy
from tests.test_gpu_ternary import check_ternary_bucket, ternary_route

pytestmark = pytest.mark.gpu


def run_binary(W, n, bucket_n, seed):
    lay = synth.small(W, n, seed, elig_frac=0.9, nruns=11)
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    d = torch.device("cuda:0")
    nb = -(-n // bucket_n)
    nw = (n + 63) // 64
    bits = torch.full((W, nw), -1, dtype=torch.int64, device=d)
    counts = torch.full((n,), 0xAB, dtype=torch.uint8, device=d)
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
    stats = torch.zeros(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    dec = torch.zeros(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bucket_n), d)
    pol = nf.policy()
    nf.nf_route_buckets(torch.from_numpy(g).to(d), n, bucket_n, torch.from_numpy(mask.view(np.int64)).to(d), pol,
                        bits, counts, out, stats, dec, ws)
    torch.cuda.synchronize()
    st, dc = nf.stats_host(stats, W, nb), nf.decisions_host(dec, nb)
    b_h, c_h, o_h = bits.cpu().numpy().view(np.uint64), counts.cpu().numpy(), out.cpu().numpy()
    for b in range(nb):
        a, e = b * bucket_n, min((b + 1) * bucket_n, n)
        ka, ke = a // 64, (e + 63) // 64
        mw = np.ascontiguousarray(mask[ka:ke])
        ref = nfo.reduce_bucket(np.ascontiguousarray(g[:, a:e]), mw, oracle_policy(pol))
        tag = f"W={W} n={n} bucket {b}"
        check_decision(dc[b], ref["decision"], tag)
        check_stats(st[b], ref["stats"], tag)
        assert np.array_equal(b_h[:, ka:ke], ref["bits"]), f"{tag} bits"
        assert np.array_equal(c_h[a:e], ref["counts"]), f"{tag} counts"
        check_output(o_h[a:e], ref, mw, e - a, W, dc[b], pol.decode_mode, tag)


@pytest.mark.parametrize("W,n,bucket_n,launches,launches_nosigns", [
    (16, 8_300_000, 8_300_000, 1, 1),      # a small problem: 1,014 chunks of 16 tiles, groups of 2 partials
    (16, 9_000_000, 9_000_000, 1, 1),      # 977 chunks of 18 tiles
    (16, 20_000_000, 20_000_000, 1, 1),    # 1,221 chunks of 32 tiles in one launch, groups of 3
    (16, 20_000_000, 9_000_000, 1, 1),     # three buckets, the last of 123 chunks
    (16, 70_000_000, 30_000_000, 17, 5),   # 4,275 chunks in three buckets: launches of 256 that may
                                           # overlap (1,024 without sign words), groups of 4
    (64, 3_000_000, 3_000_000, 2, 2),      # 977 chunks, two row groups of 32 (a launch each)
    (255, 600_000, 600_000, 4, 4),         # 782 chunks, one launch per group of 64 worker rows;
                                           # partials summed in groups of 13 (at most 64 per worker)
    (16, 1_000_000, 1_000_000, 1, 1),      # 977 chunks of 2 tiles
    (8, 6_000_000, 1_310_720, 1, 1),       # five buckets of at most 214 chunks: partials read directly
])
def test_pass1_launch_shapes(W, n, bucket_n, launches, launches_nosigns):
    assert nf.nf_pass1_launches(W, n, bucket_n) == launches
    assert nf.nf_pass1_launches(W, n, bucket_n, sign_words=False) == launches_nosigns
    run_binary(W, n, bucket_n, 31 + W)


def test_ternary_single_launch_flat():
    W, n, bn = 8, 3_000_000, 655_360
    lay = synth.small(W, n, 5, elig_frac=0.85, nruns=9)
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5)
    res = ternary_route(g, mask, n, pol, bucket_n=bn)
    for b in range(-(-n // bn)):
        check_ternary_bucket(res, g, mask, n, pol, b, bn, f"ternary flat bucket {b}")


def test_ternary_multi_launch():
    # 4,273 chunks: pass 1 without sign words in five launches (1,024 chunks
    # each at most), the plane pack in seventeen (256 at most)
    W, n = 16, 70_000_000
    assert nf.nf_pass1_launches(W, n, n, sign_words=False) == 5
    assert nf.nf_pass1_launches(W, n, n) == 17
    lay = synth.small(W, n, 77, elig_frac=0.85, nruns=9)
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5)
    res = ternary_route(g, mask, n, pol, bucket_n=n)
    check_ternary_bucket(res, g, mask, n, pol, 0, n, "ternary 4,273 chunks")
