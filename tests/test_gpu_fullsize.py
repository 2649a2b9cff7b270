"""Parity at the full workload sizes, in the launch configuration that
bench.py times: one nf_route_buckets call over the whole stacked buffer of
a workload, inputs generated on the device.

Buckets are checked in full against the oracle (every output of the bucket:
bits, counts, decoded and FP32 values, statistics, decision) on all buckets
of the small workloads and on sampled buckets of the GPT-1.3B-scale one.
The stress workload is one 100M-element bucket of 64 workers: its health
statistics are checked over every element (the oracle run per worker row),
its decision against the oracle's decision on those statistics, and its
bits and outputs on sampled 64-element word blocks.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_decision, check_output, check_stats, mask_bool, oracle_policy

pytestmark = pytest.mark.gpu


class Full:
    """A full-size workload on the device and one route call over it."""

    def __init__(self, name, pol):
        self.lay = lay = synth.CONFIGS[name]()
        d = torch.device("cuda:0")
        self.W, self.n, self.bn, self.nb = lay.W, lay.n_total, lay.bucket_n, lay.nb
        nw = (self.n + 63) // 64
        print(f"[fullsize] {name}: W={self.W} n={self.n:,} buckets={self.nb}", flush=True)
        self.g = torch.empty((self.W, lay.stride), dtype=torch.float32, device=d)
        synth.generate_device(lay, self.g)
        self.mask_h = nf.nf_mask_from_segments(*synth.mask_segments(lay), self.n)
        mask = torch.from_numpy(self.mask_h.view(np.int64)).to(d)
        self.bits = torch.full((self.W, nw), -1, dtype=torch.int64, device=d)
        self.counts = torch.full((self.n,), 0xAB, dtype=torch.uint8, device=d)
        self.out = torch.full((self.n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.zeros(self.nb * self.W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        dec = torch.zeros(self.nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(self.W, self.n, self.bn), d)
        self.pol = pol
        nf.nf_route_buckets(self.g, self.n, self.bn, mask, pol, self.bits, self.counts, self.out,
                            stats, dec, ws)
        torch.cuda.synchronize()
        self.stats = nf.stats_host(stats, self.W, self.nb)
        self.dec = nf.decisions_host(dec, self.nb)
        del mask, ws

    def release(self):
        del self.g, self.bits, self.counts, self.out
        torch.cuda.empty_cache()

    def check_bucket(self, b):
        """Every output of bucket b against the oracle on that bucket."""
        a, e = b * self.bn, min((b + 1) * self.bn, self.n)
        ka, ke = a // 64, (e + 63) // 64
        gh = self.g[:, a:e].contiguous().cpu().numpy()
        mw = np.ascontiguousarray(self.mask_h[ka:ke])
        ref = nfo.reduce_bucket(gh, mw, oracle_policy(self.pol))
        tag = f"{self.lay.name} bucket {b}"
        d = self.dec[b]
        check_decision(d, ref["decision"], tag)
        check_stats(self.stats[b], ref["stats"], tag)
        assert np.array_equal(self.bits[:, ka:ke].cpu().numpy().view(np.uint64), ref["bits"]), f"{tag} bits"
        if int(d["route"]) == nfo.ROUTE_L:
            assert np.array_equal(self.counts[a:e].cpu().numpy(), ref["counts"]), f"{tag} counts"
        check_output(self.out[a:e].cpu().numpy(), ref, mw, e - a, self.W, d, self.pol.decode_mode, tag)
        return int(d["route"])


@pytest.mark.parametrize("name", ["tiny", "resnet50", "vitb16"])
def test_fullsize_every_bucket(name):
    f = Full(name, nf.policy())
    try:
        routes = [f.check_bucket(b) for b in range(f.nb)]
        assert all(r == nfo.ROUTE_L for r in routes), routes
    finally:
        f.release()


def test_fullsize_gpt1p3b_sampled_buckets():
    f = Full("gpt1p3b", nf.policy())
    try:
        # buckets 185..200 hold only FP32-routed tensors (embeddings): route P
        routes = f.dec["route"].astype(int)
        assert (routes[:185] == nfo.ROUTE_L).all() and (routes[185:] == nfo.ROUTE_P).all()
        for b in (0, 1, 100, 183, 184, 185, 199, 200):
            f.check_bucket(b)
    finally:
        f.release()


def _stress_checks(f, expect_route):
    W, n = f.W, f.n
    mask = f.mask_h
    n_e = nfo.count_eligible(mask, n)
    # health over every element, one oracle call per worker row
    def row_stats(w):
        return nfo.health(f.g[w:w + 1, :n].cpu().numpy(), mask)[0]
    with ThreadPoolExecutor(8) as ex:
        ref_st = np.array(list(ex.map(row_stats, range(W))), dtype=nfo.STATS_DTYPE)
    check_stats(f.stats[0], ref_st, "stress")
    rd = nfo.decide(ref_st, n, n_e, oracle_policy(f.pol))
    d = f.dec[0]
    check_decision(d, rd, "stress")
    assert int(d["route"]) == expect_route
    assert int(d["reasons"]) & (nfo.R_NONFINITE | nfo.R_ZERO_WORKER | nfo.R_NORM_SPIKE) == \
        (nfo.R_NONFINITE | nfo.R_ZERO_WORKER | nfo.R_NORM_SPIKE)
    # sampled 64-element word blocks, including the injected non-finite values
    rng = np.random.default_rng(11)
    nw = (n + 63) // 64
    words = set(rng.integers(0, nw, 48).tolist()) | {0, nw - 1}
    words |= {int(i) // 64 for i in f.lay.inject_i[:24]}
    scale = np.float32(d["scale"])
    q = nfo.decode_table(W, f.pol.decode_mode)
    for k in sorted(words):
        a, e = 64 * k, min(64 * k + 64, n)
        gh = f.g[:, a:e].contiguous().cpu().numpy()
        mw = np.ascontiguousarray(mask[k:k + 1])
        ref_bits = nfo.pack(gh, mw)
        assert np.array_equal(f.bits[:, k:k + 1].cpu().numpy().view(np.uint64), ref_bits), f"bits word {k}"
        fp32 = nfo.fp32_path(gh, f.pol.fp32_op)
        c = nfo.counts(ref_bits, e - a)
        m = mask_bool(mw, e - a)
        if int(d["route"]) == nfo.ROUTE_L:
            assert np.array_equal(f.counts[a:e].cpu().numpy(), c), f"counts word {k}"
            out_ref = np.where(m, (np.float32(rd.scale) * q[c]).astype(np.float32), fp32)
        else:
            out_ref = fp32
        check_output(f.out[a:e].cpu().numpy(), {"out": out_ref, "counts": c}, mw, e - a, W, d,
                     f.pol.decode_mode, f"stress word {k}")


def test_fullsize_stress_fallback():
    f = Full("stress", nf.policy())
    try:
        _stress_checks(f, nfo.ROUTE_F)
    finally:
        f.release()


def test_fullsize_stress_forced_lowbit():
    f = Full("stress", nf.policy(force_lowbit=1))
    try:
        _stress_checks(f, nfo.ROUTE_L)
    finally:
        f.release()
