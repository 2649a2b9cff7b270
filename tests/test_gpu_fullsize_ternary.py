"""G-Ternary parity at full workload sizes, in the launch configuration of
`bench.py --format ternary`: one nf_route_buckets call over the whole
stacked buffer, inputs generated on the device.

Nothing is sampled.  GPT-1.3B scale (and the W = 255 fan-in pair, and ViT
scale cut as DDP cuts it): every
bucket checked in full against the oracle's ternary whole bucket (a pool of
threads, one bucket copied to the host at a time).  Stress (W = 64, one 100M-element bucket, forced
low-bit): statistics per worker row over every element, the thresholds from
them, then the oracle's element-wise steps (planes, c+ and c-, FP32 path,
output) over consecutive ranges covering the bucket, every word and value
compared.  Both sides round each worker's exact |g| sum once, so the sums,
the thresholds, the scale, the planes and every decoded value are compared
bit for bit.  The oracle builds its own mask from the layout's segments.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import POOL, check_decision, check_stats, mask_bool, oracle_masks, same_f32
from tests.test_gpu_ternary import check_ternary_bucket

pytestmark = pytest.mark.gpu

RANGE = 1 << 20  # elements per oracle range of the one-bucket stress workload (a multiple of 64)


class FullTernary:
    def __init__(self, name, pol, ddp=False):
        """ddp: buckets cut at tensor boundaries through the bucket-table
        driver; else equal buckets."""
        self.lay = lay = synth.CONFIGS[name]()
        d = torch.device("cuda:0")
        self.W, self.n = lay.W, lay.n_total
        self.off = synth.ddp_offsets(lay) if ddp else \
            np.array(list(range(0, self.n, lay.bucket_n)) + [self.n], np.int64)
        self.nb = len(self.off) - 1
        nw = (self.n + 63) // 64
        print(f"[fullsize-ternary] {name}: W={self.W} n={self.n:,} buckets={self.nb}", flush=True)
        self.g = torch.empty((self.W, lay.stride), dtype=torch.float32, device=d)
        synth.generate_device(lay, self.g)
        mask_dev, self.mask_o = oracle_masks(lay)
        mask = torch.from_numpy(mask_dev.view(np.int64)).to(d)
        self.bits = torch.full((2 * self.W, nw), -1, dtype=torch.int64, device=d)
        self.counts = torch.full((2 * self.n,), 0xAB, dtype=torch.uint8, device=d)
        self.out = torch.full((self.n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.zeros(self.nb * self.W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        dec = torch.zeros(self.nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        self.pol = pol
        if ddp:
            table = torch.empty(nf.nf_bucket_table_bytes(self.W, self.off), dtype=torch.uint8, device=d)
            nf.nf_bucket_table_init(self.W, self.off, table)
            ws = nf.empty_workspace(nf.nf_workspace_bytes_table(self.W, self.off), d)
            nf.nf_route_bucket_table(self.g, self.off, table, mask, pol, self.bits, self.counts, self.out, stats,
                                     dec, ws)
        else:
            ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(self.W, self.n, lay.bucket_n), d)
            nf.nf_route_buckets(self.g, self.n, lay.bucket_n, mask, pol, self.bits, self.counts, self.out, stats,
                                dec, ws)
        torch.cuda.synchronize()
        self.stats = nf.stats_host(stats, self.W, self.nb)
        self.dec = nf.decisions_host(dec, self.nb)
        del mask, ws

    def release(self):
        del self.g, self.bits, self.counts, self.out
        torch.cuda.empty_cache()

    def check_bucket(self, b):
        a, e = int(self.off[b]), int(self.off[b + 1])
        ka, ke = a // 64, (e + 63) // 64
        res = dict(bits=self.bits[:, ka:ke].cpu().numpy().view(np.uint64),
                   counts=np.concatenate([self.counts[a:e].cpu().numpy(),
                                          self.counts[self.n + a:self.n + e].cpu().numpy()]),
                   out=self.out[a:e].cpu().numpy(), stats=self.stats[b:b + 1], dec=self.dec[b:b + 1])
        gh = self.g[:, a:e].cpu().numpy()
        return check_ternary_bucket(res, gh, np.ascontiguousarray(self.mask_o[ka:ke]), e - a, self.pol, 0, e - a,
                                    f"{self.lay.name} bucket {b}")


def test_fullsize_ternary_gpt1p3b_every_bucket():
    f = FullTernary("gpt1p3b", nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5))
    try:
        with ThreadPoolExecutor(POOL) as ex:
            routes = np.array(list(ex.map(f.check_bucket, range(f.nb))))
        assert (routes[:185] == nfo.ROUTE_L).all() and (routes[185:] == nfo.ROUTE_P).all(), routes
        print(f"[fullsize-ternary] gpt1p3b: {f.nb} buckets checked", flush=True)
    finally:
        f.release()


def test_fullsize_ternary_fanin255_every_bucket():
    """W = 255 (four groups of worker rows in the first pass and the plane
    pack): both buckets in full."""
    f = FullTernary("fanin255", nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5))
    try:
        with ThreadPoolExecutor(POOL) as ex:
            routes = list(ex.map(f.check_bucket, range(f.nb)))
        assert all(r == nfo.ROUTE_L for r in routes), routes
    finally:
        f.release()


@pytest.mark.parametrize("name", ["vitb16"])
def test_fullsize_ternary_ddp_buckets_every_bucket(name):
    """G-Ternary over buckets cut as DDP cuts the model, through the
    bucket-table driver, every bucket in full."""
    f = FullTernary(name, nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5), ddp=True)
    try:
        with ThreadPoolExecutor(POOL) as ex:
            routes = list(ex.map(f.check_bucket, range(f.nb)))
        assert set(routes) <= {nfo.ROUTE_L, nfo.ROUTE_P} and nfo.ROUTE_L in routes, routes
    finally:
        f.release()


def test_fullsize_ternary_stress_forced_lowbit():
    f = FullTernary("stress", nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=1))
    try:
        W, n, mask = f.W, f.n, f.mask_o
        n_e = nfo.count_eligible(mask, n)
        gh = f.g[:, :n].cpu().numpy()  # 25.6 GB of host memory, released at the end
        with ThreadPoolExecutor(POOL) as ex:
            ref_st = np.array(list(ex.map(lambda w: nfo.health(gh[w:w + 1], mask)[0], range(W))),
                              dtype=nfo.STATS_DTYPE)
        check_stats(f.stats[0], ref_st, "stress ternary", exact_abs=True)
        d = f.dec[0]
        assert int(d["route"]) == nfo.ROUTE_L
        rd = nfo.decide(ref_st, n, n_e, nfo.policy(force_lowbit=1, format=nfo.FORMAT_TERNARY, tau=0.5))
        check_decision(d, rd, "stress ternary", exact_scale=True)
        th_gpu = nf.nf_ternary_threshold(f.stats[0], n_e, 0.5)
        th_ref = np.array([nfo.ternary_threshold(ref_st[w], n_e, 0.5) for w in range(W)], np.float32)
        assert np.array_equal(th_gpu.view(np.uint32), th_ref.view(np.uint32)), "thresholds"
        q = nfo.ternary_decode_table(W, f.pol.decode_mode)

        def check_range(a):
            e = min(a + RANGE, n)
            ka, ke = a // 64, (e + 63) // 64
            g = gh[:, a:e]
            mw = np.ascontiguousarray(mask[ka:ke])
            tag = f"stress ternary [{a}, {e})"
            pos, neg = nfo.pack_ternary(g, mw, th_ref)
            b = f.bits[:, ka:ke].cpu().numpy().view(np.uint64)
            assert np.array_equal(b[:W], pos) and np.array_equal(b[W:], neg), f"{tag} planes"
            cp, cn = nfo.counts(pos, e - a), nfo.counts(neg, e - a)
            assert np.array_equal(f.counts[a:e].cpu().numpy(), cp), f"{tag} c+"
            assert np.array_equal(f.counts[n + a:n + e].cpu().numpy(), cn), f"{tag} c-"
            y = nfo.fp32_path(g, f.pol.fp32_op)
            ref = nfo.ternary_output(mw, e - a, cp, cn, y, q, rd.scale, W, rd.route)
            out = f.out[a:e].cpu().numpy()
            m = mask_bool(mw, e - a)
            assert same_f32(out[~m], ref[~m]), f"{tag} routed positions"
            assert same_f32(out[m], ref[m]), f"{tag} decoded values"
            return e - a

        with ThreadPoolExecutor(POOL) as ex:
            assert sum(ex.map(check_range, range(0, n, RANGE))) == n
        del gh
    finally:
        f.release()
