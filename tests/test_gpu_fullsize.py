"""Parity at the full workload sizes, in the launch configuration that
bench.py times: one nf_route_buckets call over the whole stacked buffer of
a workload, inputs generated on the device.

Nothing is sampled.  Every bucket of every workload is checked against the
oracle: bits, counts, decoded and FP32 values, statistics and the decision.
The oracle builds its own mask from the layout's segments; the mask the GPU
reads comes from the library's host builder, and the two are compared word
for word first.

The GPT-1.3B-scale buckets (201 x 16 x 6,553,600) are copied to the host one
at a time and reduced by the oracle in a pool of threads (its calls release
the interpreter lock).  The stress workload is one bucket of 64 x 100M: the
oracle takes its statistics per worker row over all 100M elements, decides
on them, then runs its element-wise steps (pack, counts, FP32 path, output)
over consecutive 64-aligned ranges that together cover the bucket, and every
word and value is compared.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import (POOL, check_decision, check_output, check_stats, oracle_masks, oracle_policy)

pytestmark = pytest.mark.gpu

RANGE = 1 << 20  # elements per oracle range of the one-bucket stress workload (a multiple of 64)


class Full:
    """A full-size workload on the device and one route call over it."""

    def __init__(self, name, pol, ddp=False):
        """ddp: buckets cut at tensor boundaries (synth.ddp_offsets) and
        routed through the bucket-table driver; else equal buckets."""
        self.lay = lay = synth.CONFIGS[name]()
        d = torch.device("cuda:0")
        self.W, self.n = lay.W, lay.n_total
        self.off = synth.ddp_offsets(lay) if ddp else \
            np.array(list(range(0, self.n, lay.bucket_n)) + [self.n], np.int64)
        self.nb = len(self.off) - 1
        nw = (self.n + 63) // 64
        print(f"[fullsize] {name}: W={self.W} n={self.n:,} buckets={self.nb} ({'DDP' if ddp else 'equal'})",
              flush=True)
        self.g = torch.empty((self.W, lay.stride), dtype=torch.float32, device=d)
        synth.generate_device(lay, self.g)
        mask_dev, self.mask_o = oracle_masks(lay)
        mask = torch.from_numpy(mask_dev.view(np.int64)).to(d)
        self.bits = torch.full((self.W, nw), -1, dtype=torch.int64, device=d)
        self.counts = torch.full((self.n,), 0xAB, dtype=torch.uint8, device=d)
        self.out = torch.full((self.n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.zeros(self.nb * self.W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        dec = torch.zeros(self.nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        self.pol = pol
        if ddp:
            table = torch.empty(nf.nf_bucket_table_bytes(self.W, self.off), dtype=torch.uint8, device=d)
            nf.nf_bucket_table_init(self.W, self.off, table)
            ws = nf.empty_workspace(nf.nf_workspace_bytes_table(self.W, self.off), d)
            nf.nf_route_bucket_table(self.g, self.off, table, mask, pol, self.bits, self.counts, self.out,
                                     stats, dec, ws)
        else:
            ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(self.W, self.n, lay.bucket_n), d)
            nf.nf_route_buckets(self.g, self.n, lay.bucket_n, mask, pol, self.bits, self.counts, self.out,
                                stats, dec, ws)
        torch.cuda.synchronize()
        self.stats = nf.stats_host(stats, self.W, self.nb)
        self.dec = nf.decisions_host(dec, self.nb)
        del mask, ws

    def release(self):
        del self.g, self.bits, self.counts, self.out
        torch.cuda.empty_cache()

    def check_bucket(self, b):
        """Every output of bucket b against the oracle on that bucket.  A
        route the policy fixes before reading writes no sign words, and its
        |g| sums and scale are the exact ones rounded once."""
        a, e = int(self.off[b]), int(self.off[b + 1])
        ka, ke = a // 64, (e + 63) // 64
        gh = self.g[:, a:e].cpu().numpy()
        mw = np.ascontiguousarray(self.mask_o[ka:ke])
        ref = nfo.reduce_bucket(gh, mw, oracle_policy(self.pol))
        del gh
        tag = f"{self.lay.name} bucket {b}"
        d = self.dec[b]
        predecided = bool(self.pol.veto) and not self.pol.force_lowbit
        check_decision(d, ref["decision"], tag, exact_scale=predecided)
        check_stats(self.stats[b], ref["stats"], tag, exact_abs=predecided)
        if not predecided:
            assert np.array_equal(self.bits[:, ka:ke].cpu().numpy().view(np.uint64), ref["bits"]), f"{tag} bits"
        if int(d["route"]) == nfo.ROUTE_L:
            assert np.array_equal(self.counts[a:e].cpu().numpy(), ref["counts"]), f"{tag} counts"
        check_output(self.out[a:e].cpu().numpy(), ref, mw, e - a, self.W, d, self.pol.decode_mode, tag)
        return int(d["route"])

    def check_every_bucket(self):
        with ThreadPoolExecutor(POOL) as ex:
            return list(ex.map(self.check_bucket, range(self.nb)))


@pytest.mark.parametrize("name", ["tiny", "resnet50", "vitb16", "fanin255"])
def test_fullsize_every_bucket(name):
    f = Full(name, nf.policy())
    try:
        routes = f.check_every_bucket()
        assert all(r == nfo.ROUTE_L for r in routes), routes
    finally:
        f.release()


def test_fullsize_fanin255_vetoed_mean():
    """W = 255 with the low-bit route vetoed and the FP32 mean: pass 1 adds
    every element's FP32 sum in four groups of 64 worker rows, divided once
    after the last."""
    f = Full("fanin255", nf.policy(veto=1, fp32_op=nf.NF_FP32_MEAN))
    try:
        routes = f.check_every_bucket()
        assert all(r == nfo.ROUTE_F for r in routes), routes
    finally:
        f.release()


@pytest.mark.parametrize("name", ["vitb16", "gpt1p3b"])
def test_fullsize_ddp_buckets_every_bucket(name):
    """Buckets as DDP cuts the model (25 MiB capacity, closed at tensor
    boundaries, the first of 1 MiB; GPT scale: 73 buckets of 16.8M to 107M
    elements) through the bucket-table driver, every bucket in full."""
    f = Full(name, nf.policy(), ddp=True)
    try:
        routes = f.check_every_bucket()
        assert set(routes) <= {nfo.ROUTE_L, nfo.ROUTE_P} and nfo.ROUTE_L in routes, routes
        print(f"[fullsize] {name} DDP buckets: {f.nb} checked, routes {routes}", flush=True)
    finally:
        f.release()


def test_fullsize_gpt1p3b_every_bucket():
    f = Full("gpt1p3b", nf.policy())
    try:
        routes = np.array(f.check_every_bucket())
        # buckets 185..200 hold only FP32-routed tensors (embeddings): route P
        assert (routes[:185] == nfo.ROUTE_L).all() and (routes[185:] == nfo.ROUTE_P).all(), routes
        print(f"[fullsize] gpt1p3b: {f.nb} buckets checked", flush=True)
    finally:
        f.release()


def _stress_checks(f, expect_route):
    W, n = f.W, f.n
    mask = f.mask_o
    n_e = nfo.count_eligible(mask, n)
    gh = f.g[:, :n].cpu().numpy()  # 25.6 GB of host memory, released at the end
    try:
        # statistics over every element: the oracle per worker row
        with ThreadPoolExecutor(POOL) as ex:
            ref_st = np.array(list(ex.map(lambda w: nfo.health(gh[w:w + 1], mask)[0], range(W))),
                              dtype=nfo.STATS_DTYPE)
        check_stats(f.stats[0], ref_st, "stress")
        rd = nfo.decide(ref_st, n, n_e, oracle_policy(f.pol))
        d = f.dec[0]
        check_decision(d, rd, "stress")
        assert int(d["route"]) == expect_route
        assert int(d["reasons"]) & (nfo.R_NONFINITE | nfo.R_ZERO_WORKER | nfo.R_NORM_SPIKE) == \
            (nfo.R_NONFINITE | nfo.R_ZERO_WORKER | nfo.R_NORM_SPIKE)
        q = nfo.decode_table(W, f.pol.decode_mode)
        route_l = int(d["route"]) == nfo.ROUTE_L

        # the element-wise steps over consecutive ranges covering the bucket
        def check_range(a):
            e = min(a + RANGE, n)
            ka, ke = a // 64, (e + 63) // 64
            g = gh[:, a:e]
            mw = np.ascontiguousarray(mask[ka:ke])
            bits = nfo.pack(g, mw)
            tag = f"stress [{a}, {e})"
            assert np.array_equal(f.bits[:, ka:ke].cpu().numpy().view(np.uint64), bits), f"{tag} bits"
            c = nfo.counts(bits, e - a)
            if route_l:
                assert np.array_equal(f.counts[a:e].cpu().numpy(), c), f"{tag} counts"
            y = nfo.fp32_path(g, f.pol.fp32_op)
            out_ref = nfo.output(mw, e - a, c, y, q, rd.scale, rd.route)
            check_output(f.out[a:e].cpu().numpy(), {"out": out_ref, "counts": c}, mw, e - a, W, d,
                         f.pol.decode_mode, tag)
            return e - a

        with ThreadPoolExecutor(POOL) as ex:
            assert sum(ex.map(check_range, range(0, n, RANGE))) == n
        # every injected non-finite value lies in a checked range; they are where the lay says
        assert np.all(~np.isfinite(gh[f.lay.inject_w, f.lay.inject_i]))
    finally:
        del gh


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
