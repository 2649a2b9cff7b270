"""GPU parity of the bucket-table driver (buckets of different sizes in one
flat buffer, §2.1, §2.3) through the C ABI.

Checked: on equal buckets the table driver gives the bits, counts, outputs,
statistics and decisions of nf_route_buckets byte for byte; on ragged
buckets (1 element to 25M, interior lengths multiples of 64 as the bitmap
words require) every bucket equals the oracle on that bucket, in both
formats and under the fused, forced low-bit and vetoed routes, with a
non-finite value sending one bucket to the fallback; 1,500 small buckets
(a chunk-to-bucket map of 1,500 entries); buckets of more than 512 chunks
(more than 64 above 32 workers), whose partials are summed in groups first.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests import nfgpu as H
from tests.test_gpu_ternary import check_ternary_bucket

pytestmark = pytest.mark.gpu


def layout_for(W, n, seed, elig_frac=0.85):
    lay = synth.small(W, n, seed, elig_frac=elig_frac, nruns=17)
    g = synth.generate_host(lay)
    m = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    return g, m


def table_route(g, mask, off, pol):
    """One nf_route_bucket_table call; host copies of every output."""
    W = g.shape[0]
    off = np.asarray(off, np.int64)
    n, nb = int(off[-1]), len(off) - 1
    d = H.dev()
    planes = 2 if pol.format == nf.NF_FORMAT_TERNARY else 1
    table = torch.empty(nf.nf_bucket_table_bytes(W, off), dtype=torch.uint8, device=d)
    nf.nf_bucket_table_init(W, off, table)
    nw = (n + 63) // 64
    bits = torch.full((planes * W, nw + 2), -1, dtype=torch.int64, device=d)
    counts = torch.full((planes * n,), 0xAB, dtype=torch.uint8, device=d)
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
    stats = torch.zeros(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    dec = torch.zeros(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_table(W, off), d)
    nf.nf_route_bucket_table(H.to_dev(g), off, table, H.to_dev(mask, torch.int64), pol, bits, counts, out, stats,
                             dec, ws)
    torch.cuda.synchronize()
    return dict(bits=bits.cpu().numpy().view(np.uint64), counts=counts.cpu().numpy(), out=out.cpu().numpy(),
                stats=nf.stats_host(stats, W, nb), dec=nf.decisions_host(dec, nb),
                raw_stats=stats.cpu().numpy(), raw_dec=dec.cpu().numpy())


def flat_route(g, mask, n, bucket_n, pol):
    W = g.shape[0]
    d = H.dev()
    nb = -(-n // bucket_n)
    planes = 2 if pol.format == nf.NF_FORMAT_TERNARY else 1
    nw = (n + 63) // 64
    bits = torch.full((planes * W, nw + 2), -1, dtype=torch.int64, device=d)
    counts = torch.full((planes * n,), 0xAB, dtype=torch.uint8, device=d)
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
    stats = torch.zeros(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    dec = torch.zeros(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bucket_n), d)
    nf.nf_route_buckets(H.to_dev(g), n, bucket_n, H.to_dev(mask, torch.int64), pol, bits, counts, out, stats, dec,
                        ws)
    torch.cuda.synchronize()
    return dict(bits=bits.cpu().numpy().view(np.uint64), counts=counts.cpu().numpy(), out=out.cpu().numpy(),
                raw_stats=stats.cpu().numpy(), raw_dec=dec.cpu().numpy())


def check_table_bucket(res, g, mask, off, b, pol, tag):
    """Bucket b of a table call against the oracle on that bucket."""
    a, e = int(off[b]), int(off[b + 1])
    n = int(off[-1])
    W = g.shape[0]
    ka, ke = a // 64, (e + 63) // 64
    mw = np.ascontiguousarray(mask[ka:ke])
    gs = np.ascontiguousarray(g[:, a:e])
    if pol.format == nf.NF_FORMAT_TERNARY:
        sub = dict(bits=res["bits"][:, ka:ke], counts=np.concatenate([res["counts"][a:e], res["counts"][n + a:n + e]]),
                   out=res["out"][a:e], stats=res["stats"][b:b + 1], dec=res["dec"][b:b + 1])
        return check_ternary_bucket(sub, gs, mw, e - a, pol, 0, e - a, tag)
    sub = dict(bits=res["bits"][:W, ka:ke], counts=res["counts"][a:e], out=res["out"][a:e],
               stats=res["stats"][b:b + 1], dec=res["dec"][b:b + 1])
    H.check_route(sub, gs, mw, e - a, pol, what=tag)
    return int(res["dec"][b]["route"])


@pytest.mark.parametrize("fmt", [nf.NF_FORMAT_BINARY, nf.NF_FORMAT_TERNARY])
@pytest.mark.parametrize("W", [3, 16, 64, 200])
def test_table_of_equal_buckets_equals_flat_driver(W, fmt):
    n, bn = 2_000_077, 262_144
    g, m = layout_for(W, n, 300 + W)
    pol = nf.policy(format=fmt, tau=0.5)
    off = list(range(0, n, bn)) + [n]
    t = table_route(g, m, off, pol)
    f = flat_route(g, m, n, bn, pol)
    for k in ("bits", "counts", "raw_stats", "raw_dec"):
        assert np.array_equal(t[k], f[k]), f"W={W} fmt={fmt}: {k} differ"
    assert H.same_f32(t["out"], f["out"]), f"W={W} fmt={fmt}: out differs"


RAGGED = [64, 1_000_000 // 64 * 64, 4096, 2_000_064, 128, 640, 1_311_744, 777_777]


@pytest.mark.parametrize("kind", ["default", "forced", "veto_mean", "ternary", "ternary_forced"])
@pytest.mark.parametrize("W", [4, 16, 65])
def test_table_ragged_buckets_match_oracle(W, kind):
    off = np.concatenate([[0], np.cumsum(RAGGED)]).astype(np.int64)
    n = int(off[-1])
    g, m = layout_for(W, n, 400 + W)
    # a NaN in bucket 3 sends it to the fallback (or is carried by the forced route)
    g[W - 1, off[3] + 1000] = np.nan
    pol = {"default": nf.policy(), "forced": nf.policy(force_lowbit=1),
           "veto_mean": nf.policy(veto=1, fp32_op=nf.NF_FP32_MEAN),
           "ternary": nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5),
           "ternary_forced": nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=1)}[kind]
    res = table_route(g, m, off, pol)
    routes = [check_table_bucket(res, g, m, off, b, pol, f"W={W} {kind} bucket {b}") for b in range(len(RAGGED))]
    if kind in ("default", "ternary"):
        assert routes[3] == nfo.ROUTE_F and routes[0] == nfo.ROUTE_L, routes


def test_table_many_small_buckets():
    rng = np.random.default_rng(5)
    sizes = rng.integers(1, 129, size=1500) * 64
    sizes[-1] += 17
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    W = 8
    g, m = layout_for(W, int(off[-1]), 77)
    pol = nf.policy()
    res = table_route(g, m, off, pol)
    for b in range(len(sizes)):
        check_table_bucket(res, g, m, off, b, pol, f"small bucket {b}")


@pytest.mark.parametrize("W,big", [(16, 25_000_000), (100, 3_000_000)])
def test_table_buckets_above_the_slot_threshold(W, big):
    """Buckets of more than 512 chunks (64 above 32 workers) next to small
    ones: the second-level group sums of each bucket cover its own slots."""
    sizes = [64 * 1000, big // 64 * 64, 4096, 777]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    _, chunks = nf.nf_pass1_chunk_elems(W, int(off[-1]), big)
    assert chunks > (512 if W <= 32 else 64), chunks
    g, m = layout_for(W, int(off[-1]), 500 + W)
    for pol in (nf.policy(), nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5)):
        res = table_route(g, m, off, pol)
        for b in range(len(sizes)):
            check_table_bucket(res, g, m, off, b, pol, f"W={W} fmt={pol.format} bucket {b}")
