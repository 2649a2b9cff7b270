"""GPU parity of the exactly rounded |g| sums (no sign words: the G-Ternary
route, nf_bucket_health, routes fixed before reading) through the C ABI.

Each worker's sum of |g| over the eligible elements must equal, bit for bit,
the oracle's exact sum rounded once to FP64.  The library carries the sum as
a TwoSum pair with an error bound and, where the bound cannot prove the
rounding, sums the worker again exactly; the decision's `resummed` field
counts those workers.  Sums built to land on or next to a rounding midpoint
must take that path and still round correctly; ordinary gradients, and
sums exactly on a midpoint, must not.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_stats, oracle_policy, same_f64, to_dev
from tests.test_gpu_ternary import check_ternary_bucket, ternary_route

pytestmark = pytest.mark.gpu


def padded(g):
    """g in rows of a stride rounded up to a multiple of 4 (the library's
    alignment rule), as a view of the first n columns."""
    W, n = g.shape
    p = np.zeros((W, max(4, -(-n // 4) * 4)), np.float32)
    p[:, :n] = g
    return p[:, :n]


def health_gpu(g, mask, n):
    W = g.shape[0]
    stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device="cuda:0")
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n))
    nf.nf_bucket_health(to_dev(g.base if g.base is not None else g), n, to_dev(mask if mask.size else np.zeros(1, np.uint64), torch.int64),
                        stats, ws)
    torch.cuda.synchronize()
    return nf.stats_host(stats, W)[0]


def rand_mask(n, seed, frac=0.8):
    m = (np.random.default_rng(seed).random(n) < frac).astype(np.uint8)
    return np.packbits(np.concatenate([m, np.zeros((-n) % 64, np.uint8)]),
                       bitorder="little").view(np.uint64).copy()


@pytest.mark.parametrize("W", [1, 3, 16, 64, 255])
@pytest.mark.parametrize("n", [1, 64, 4097, 300_001])
def test_health_exact_wide_range(W, n):
    """|g| spread over 2^-60 .. 2^60 (and subnormals): any order-dependent
    FP64 sum would differ from the exact one in the last bits."""
    rng = np.random.default_rng(W * 7919 + n)
    g = (rng.standard_normal((W, n)) * np.exp2(rng.uniform(-60, 60, (W, n)))).astype(np.float32)
    g[:, ::97] = np.float32(1e-45) * rng.integers(1, 9, size=g[:, ::97].shape).astype(np.float32)
    g = padded(g)
    mask = rand_mask(n, n + W)
    st = health_gpu(g, mask, n)
    ref = nfo.health(g, mask)
    check_stats(st, ref, f"W={W} n={n}", exact_abs=True)


def test_health_exact_nonfinite():
    """A NaN term makes the sum NaN, an infinity +Inf; off the mask neither counts."""
    W, n = 5, 70_000
    rng = np.random.default_rng(3)
    g = (rng.standard_normal((W, n)) * 1e-3).astype(np.float32)
    m = np.ones(n, np.uint8)
    m[100] = 0
    mask = np.packbits(np.concatenate([m, np.zeros((-n) % 64, np.uint8)]), bitorder="little").view(np.uint64).copy()
    g[0, 5] = np.nan
    g[1, 6] = np.inf
    g[2, 7], g[2, 9000] = -np.inf, np.nan
    g[3, 100] = np.nan  # off the mask
    st = health_gpu(g, mask, n)
    ref = nfo.health(g, mask)
    check_stats(st, ref, "nonfinite", exact_abs=True)
    assert np.isnan(st["sum_abs_elig"][0]) and st["sum_abs_elig"][1] == np.inf and np.isnan(st["sum_abs_elig"][2])
    assert np.isfinite(st["sum_abs_elig"][3])


def midpoint_rows(W, n, seed, above, bucket_n):
    """Rows whose eligible |g| are 1, 2^-53 and (above) 2^-140, the rest 0,
    at random positions of bucket w % nb for worker w: that bucket's exact sum
    1 + 2^-53 (+ 2^-140) lies on (or just above) the midpoint between 1 and
    1 + 2^-52."""
    rng = np.random.default_rng(seed)
    g = np.zeros((W, n), np.float32)
    vals = [1.0, 2.0 ** -53] + ([2.0 ** -140] if above else [])
    nb = -(-n // bucket_n)
    for w in range(W):
        a = (w % nb) * bucket_n
        pos = a + rng.choice(min(bucket_n, n - a), size=len(vals), replace=False)
        g[w, pos] = np.array(vals, np.float32) * rng.choice([-1.0, 1.0], size=len(vals)).astype(np.float32)
    return g


@pytest.mark.parametrize("above", [False, True])
@pytest.mark.parametrize("W,n,bucket_n", [(1, 5000, None), (4, 3_000_000, None), (16, 2_000_000, 655_360),
                                          (64, 1_500_000, None)])
def test_route_ternary_midpoint_sums_resummed(W, n, bucket_n, above):
    """A sum exactly on a rounding midpoint (1 + 2^-53) is carried exactly (its
    error part needs few bits), so one FP64 rounding gives it, ties to even,
    without a re-summation.  Just above the midpoint (+ 2^-140) the error part
    needs 88 bits: the carried bound cannot place the total on one side of
    the midpoint, and every worker is re-summed exactly.  Either way the route
    matches the oracle bit for bit."""
    bn = bucket_n or n
    g = midpoint_rows(W, n, 17 * W + n + above, above, bn)
    mask = np.full((n + 63) // 64, np.uint64(0xFFFFFFFFFFFFFFFF))
    if n % 64:
        mask[-1] = np.uint64((1 << (n % 64)) - 1)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=1)
    res = ternary_route(g, mask, n, pol, bucket_n=bn)
    nb = -(-n // bn)
    for b in range(nb):
        check_ternary_bucket(res, g, mask, n, pol, b, bn, f"midpoint W={W} n={n} bucket {b}")
    want = 1.0 + 2.0 ** -52 if above else 1.0
    for w in range(W):
        assert res["stats"][w % nb]["sum_abs_elig"][w] == want, (w, res["stats"][w % nb]["sum_abs_elig"][w])
    # above the midpoint every worker is re-summed once, in the bucket holding
    # its values; the others' all-zero rows there are exact (0)
    want_re = [len(range(b, W, nb)) if above else 0 for b in range(nb)]
    assert [int(d["resummed"]) for d in res["dec"]] == want_re


@pytest.mark.parametrize("name", ["small", "scaled"])
@pytest.mark.parametrize("W", [4, 16, 64])
def test_route_ternary_ordinary_data_certified(name, W):
    """Gradient-like data: every sum is certified by the carried bound (no
    worker re-summed) and equals the oracle's exact sum."""
    bn = 655_360
    lay = synth.small(W, 2_500_000, 40 + W, elig_frac=0.9, nruns=11) if name == "small" else \
        synth.scaled(synth.vitb16, 32, W=W, bucket_n=bn)
    n = lay.n_total
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5)
    res = ternary_route(g, mask, n, pol, bucket_n=bn)
    for b in range(-(-n // bn)):
        check_ternary_bucket(res, g, mask, n, pol, b, bn, f"{name} W={W} bucket {b}")
    assert all(int(d["resummed"]) == 0 for d in res["dec"]), [int(d["resummed"]) for d in res["dec"]]


def test_predecided_binary_route_exact():
    """A route the policy fixes before reading (veto) builds no sign words, so
    its |g| sums are exact as well."""
    W, n = 8, 777_777
    rng = np.random.default_rng(8)
    g = padded((rng.standard_normal((W, n)) * np.exp2(rng.uniform(-30, 10, (W, n)))).astype(np.float32))
    mask = rand_mask(n, 9, 0.7)
    pol = nf.policy(veto=1)
    res = ternary_route(g.base, mask, n, pol)  # the binary format through the same driver
    ref = nfo.reduce_bucket(g, mask, oracle_policy(pol))
    assert same_f64(res["stats"][0]["sum_abs_elig"], ref["stats"]["sum_abs_elig"])
    assert int(res["dec"][0]["route"]) == nfo.ROUTE_F
