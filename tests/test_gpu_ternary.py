"""GPU parity of the G-Ternary payload (pack, count and decode, and the route
drivers with the ternary format) against the oracle, through the C ABI.

Bars: planes, counts, routes, reasons and modeled bytes bit-exact; FP32 sums
bit-exact.  The thresholds fl32(tau * fl32(S_w / n_E)) come on both sides
from S_w, the exact sum of |g| over the eligible elements rounded once to
FP64, so S_w, the thresholds, the scale and every decoded value are
bit-exact as well; sums of squares within 1e-6.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_decision, check_stats, mask_bool, oracle_policy, same_f32, to_dev

pytestmark = pytest.mark.gpu

SPECIAL = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1e-45, -1e-45], dtype=np.float32)


def layout(W, n, seed, elig=0.85, special=False):
    lay = synth.small(W, n, seed, elig_frac=elig, nruns=9)
    g = synth.generate_host(lay)
    if special and n > 0:
        rng = np.random.default_rng(seed)
        idx = rng.integers(0, n, size=min(n, 40))
        g[rng.integers(0, W, size=len(idx)), idx] = rng.choice(SPECIAL, size=len(idx))
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    return g, mask


def unpack(words, n):
    return np.unpackbits(np.ascontiguousarray(words, np.uint64).view(np.uint8), bitorder="little",
                         axis=-1)[..., :n]


@pytest.mark.parametrize("W", [1, 2, 3, 8, 16, 64, 65, 255])
@pytest.mark.parametrize("n", [1, 63, 64, 65, 4095, 65537])
def test_pack_ternary_matches_oracle(W, n):
    g, mask = layout(W, n, 1000 * W + n, special=True)
    rng = np.random.default_rng(W + n)
    theta = (np.abs(rng.normal(0, 1e-3, W)) * rng.choice([0.0, 0.5, 1.0, 3.0], W)).astype(np.float32)
    theta[0] = 0.0
    pos, neg = nfo.pack_ternary(g, mask, theta)
    nw = (n + 63) // 64
    bits = torch.full((2 * W, nw + 3), -1, dtype=torch.int64, device="cuda:0")
    nf.nf_pack_ternary(to_dev(g), n, to_dev(mask, torch.int64), to_dev(theta), bits)
    torch.cuda.synchronize()
    b = bits.cpu().numpy().view(np.uint64)
    assert np.array_equal(b[:W, :nw], pos), "positive planes"
    assert np.array_equal(b[W:, :nw], neg), "negative planes"
    assert np.all(b[:, nw:] == np.uint64(0xFFFFFFFFFFFFFFFF)), "words past the end untouched"


@pytest.mark.parametrize("W", [1, 3, 16, 64, 129, 255])
@pytest.mark.parametrize("n", [1, 65, 4097, 100_003])
@pytest.mark.parametrize("mode", [nfo.DECODE_SOFT, nfo.DECODE_MAJORITY])
def test_ternary_reduce_matches_oracle(W, n, mode):
    g, mask = layout(W, n, 7 * W + n)
    rng = np.random.default_rng(n)
    theta = (np.abs(rng.normal(0, 1e-3, W)) * 0.7).astype(np.float32)
    pos, neg = nfo.pack_ternary(g, mask, theta)
    cp, cn = nfo.counts(pos, n), nfo.counts(neg, n)
    scale = np.float32(3.7e-4)
    q = nfo.ternary_decode_table(W, mode)
    nw = (n + 63) // 64
    bits = to_dev(np.concatenate([pos, neg]).view(np.int64))
    counts = torch.full((2 * n,), 0xAB, dtype=torch.uint8, device="cuda:0")
    out = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda:0")
    nf.nf_ternary_reduce(bits, W, n, to_dev(mask, torch.int64), to_dev(np.array([scale])), mode, counts, out)
    torch.cuda.synchronize()
    c = counts.cpu().numpy()
    assert np.array_equal(c[:n], cp) and np.array_equal(c[n:], cn), "counts"
    m = mask_bool(mask, n)
    o = out.cpu().numpy()
    want = (scale * q[cp.astype(int) - cn.astype(int) + W]).astype(np.float32)
    assert same_f32(o[m], want[m]), "decoded values"
    assert np.all(np.isnan(o[~m])), "routed positions untouched"
    assert nw == bits.shape[1]


def ternary_route(g, mask, n, pol, bucket_n=None):
    """One driver call with the ternary format; returns host copies."""
    W = g.shape[0]
    d = torch.device("cuda:0")
    bucket_n = bucket_n or max(n, 1)
    nb = max(1, -(-n // bucket_n))
    nw = (n + 63) // 64
    bits = torch.full((2 * W, nw + 2), -1, dtype=torch.int64, device=d)
    counts = torch.full((max(2 * n, 1),), 0xAB, dtype=torch.uint8, device=d)
    out = torch.full((max(n, 1),), float("nan"), dtype=torch.float32, device=d)
    stats = torch.zeros(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    dec = torch.zeros(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
    gd, md = to_dev(g), to_dev(mask if mask.size else np.zeros(1, np.uint64), torch.int64)
    if nb == 1 and bucket_n >= n:
        ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), d)
        nf.nf_route_bucket(gd, n, md, pol, bits, counts, out, stats, dec, ws)
    else:
        ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bucket_n), d)
        nf.nf_route_buckets(gd, n, bucket_n, md, pol, bits, counts, out, stats, dec, ws)
    torch.cuda.synchronize()
    return dict(bits=bits.cpu().numpy().view(np.uint64), counts=counts.cpu().numpy(), out=out.cpu().numpy(),
                stats=nf.stats_host(stats, W, nb), dec=nf.decisions_host(dec, nb))


def check_ternary_bucket(res, g, mask, n, pol, b, bucket_n, tag):
    """Every output of bucket b against the oracle's ternary whole bucket, bit
    for bit (sums of squares within 1e-6)."""
    W = g.shape[0]
    a, e = b * bucket_n, min((b + 1) * bucket_n, n)
    ka, ke = a // 64, (e + 63) // 64
    mw = np.ascontiguousarray(mask[ka:ke])
    ref = nfo.reduce_bucket_ternary(np.ascontiguousarray(g[:, a:e]), mw, oracle_policy(pol))
    d = res["dec"][b]
    check_decision(d, ref["decision"], tag, exact_scale=True)
    check_stats(res["stats"][b], ref["stats"], tag, exact_abs=True)
    route = int(d["route"])
    out = res["out"][a:e]
    if route != nfo.ROUTE_L:
        assert same_f32(out, ref["out"]), f"{tag} FP32 output (route {route})"
        return route
    ne = int(d["n_eligible"])
    th_gpu = nf.nf_ternary_threshold(res["stats"][b], ne, pol.tau)
    th_ref = np.array([nfo.ternary_threshold(ref["stats"][w], ne, pol.tau) for w in range(W)], np.float32)
    assert same_f32(th_gpu, th_ref), \
        f"{tag} thresholds differ for workers {np.nonzero(th_gpu.view(np.uint32) != th_ref.view(np.uint32))[0]}"
    pos, neg = res["bits"][:W, ka:ke], res["bits"][W:2 * W, ka:ke]
    assert np.array_equal(pos, ref["pos"]) and np.array_equal(neg, ref["neg"]), f"{tag} planes"
    assert np.array_equal(res["counts"][a:e], ref["cpos"]), f"{tag} c+"
    assert np.array_equal(res["counts"][n + a:n + e], ref["cneg"]), f"{tag} c-"
    assert same_f32(out, ref["out"]), f"{tag} outputs"
    return route


@pytest.mark.parametrize("W", [1, 3, 16, 64])
@pytest.mark.parametrize("n", [1000, 65537])
@pytest.mark.parametrize("tau", [0.0, 0.5, 1.5])
def test_route_bucket_ternary(W, n, tau):
    g, mask = layout(W, n, 11 * W + n + int(tau * 10))
    mode = nf.NF_DECODE_MAJORITY if W == 3 else nf.NF_DECODE_SOFT
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=tau, decode_mode=mode)
    res = ternary_route(g, mask, n, pol)
    route = check_ternary_bucket(res, g, mask, n, pol, 0, max(n, 1), f"W={W} n={n} tau={tau}")
    assert route == nfo.ROUTE_L


@pytest.mark.parametrize("W", [2, 16, 64])
def test_route_ternary_everything_gated(W):
    """A gate above every |g|: both planes empty, every eligible element
    decodes from d = 0; routed elements keep their FP32 sums."""
    n = 65_537
    g, mask = layout(W, n, 21 * W)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=1e30)
    res = ternary_route(g, mask, n, pol)
    assert check_ternary_bucket(res, g, mask, n, pol, 0, n, f"gated W={W}") == nfo.ROUTE_L
    assert not res["bits"][:, :(n + 63) // 64].any(), "every plane word zero"


def test_route_buckets_ternary_flat():
    W, n, bn = 16, 1_000_000, 131_072
    g, mask = layout(W, n, 99)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, fp32_op=nf.NF_FP32_MEAN)
    res = ternary_route(g, mask, n, pol, bucket_n=bn)
    for b in range(-(-n // bn)):
        check_ternary_bucket(res, g, mask, n, pol, b, bn, f"flat bucket {b}")


@pytest.mark.parametrize("force", [0, 1])
def test_route_ternary_faults(force):
    W, n = 8, 70_001
    g, mask = layout(W, n, 5)
    g[3, 17] = np.nan
    g[6] *= 10
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=force)
    res = ternary_route(g, mask, n, pol)
    route = check_ternary_bucket(res, g, mask, n, pol, 0, n, f"faults force={force}")
    assert route == (nfo.ROUTE_L if force else nfo.ROUTE_F)


def test_route_ternary_no_counts_and_policy_predecided():
    W, n = 4, 5000
    g, mask = layout(W, n, 6)
    d = torch.device("cuda:0")
    gd, md = to_dev(g), to_dev(mask, torch.int64)
    nw = (n + 63) // 64
    for pol, route in ((nf.policy(format=1, veto=1), nfo.ROUTE_F), (nf.policy(format=1, admitted=0), nfo.ROUTE_P)):
        bits = torch.full((2 * W, nw), -1, dtype=torch.int64, device=d)
        out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        dec = torch.zeros(nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), d)
        nf.nf_route_bucket(gd, n, md, pol, bits, None, out, stats, dec, ws)
        torch.cuda.synchronize()
        assert int(nf.decisions_host(dec, 1)[0]["route"]) == route
        ref = nfo.reduce_bucket_ternary(np.ascontiguousarray(g[:, :n]), mask, oracle_policy(pol))
        assert same_f32(out.cpu().numpy(), ref["out"]), "predecided output"
        assert np.all(bits.cpu().numpy() == -1), "predecided: no payload written"
    res = ternary_route(g, mask, n, nf.policy(format=1, tau=0.5))
    assert int(res["dec"][0]["route"]) == nfo.ROUTE_L
