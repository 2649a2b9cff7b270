"""G-Ternary parity at full workload sizes, in the launch configuration of
`bench.py --format ternary`: one nf_route_buckets call over the whole
stacked buffer, inputs generated on the device.

GPT-1.3B scale: sampled buckets (the first, a middle one, the last low-bit
bucket, the mixed bucket 184, the first and the last FP32-only buckets)
checked in full against the oracle's ternary whole bucket.  Stress (W = 64,
one 100M-element bucket, forced low-bit): thresholds from the oracle's
statistics over every element, planes, counts and decoded values on sampled
word blocks (the injected non-finite values included).  Bars as in
test_gpu_ternary.py.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import check_stats, mask_bool, oracle_policy, same_f32
from tests.test_gpu_ternary import check_ternary_bucket, unpack

pytestmark = pytest.mark.gpu


class FullTernary:
    def __init__(self, name, pol):
        self.lay = lay = synth.CONFIGS[name]()
        d = torch.device("cuda:0")
        self.W, self.n, self.bn, self.nb = lay.W, lay.n_total, lay.bucket_n, lay.nb
        nw = (self.n + 63) // 64
        print(f"[fullsize-ternary] {name}: W={self.W} n={self.n:,} buckets={self.nb}", flush=True)
        self.g = torch.empty((self.W, lay.stride), dtype=torch.float32, device=d)
        synth.generate_device(lay, self.g)
        self.mask_h = nf.nf_mask_from_segments(*synth.mask_segments(lay), self.n)
        mask = torch.from_numpy(self.mask_h.view(np.int64)).to(d)
        self.bits = torch.full((2 * self.W, nw), -1, dtype=torch.int64, device=d)
        self.counts = torch.full((2 * self.n,), 0xAB, dtype=torch.uint8, device=d)
        self.out = torch.full((self.n,), float("nan"), dtype=torch.float32, device=d)
        stats = torch.zeros(self.nb * self.W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
        dec = torch.zeros(self.nb * nf.DECISION_BYTES, dtype=torch.uint8, device=d)
        ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(self.W, self.n, self.bn), d)
        self.pol = pol
        nf.nf_route_buckets(self.g, self.n, self.bn, mask, pol, self.bits, self.counts, self.out, stats, dec, ws)
        torch.cuda.synchronize()
        self.stats = nf.stats_host(stats, self.W, self.nb)
        self.dec = nf.decisions_host(dec, self.nb)
        del mask, ws

    def release(self):
        del self.g, self.bits, self.counts, self.out
        torch.cuda.empty_cache()

    def check_bucket(self, b):
        a, e = b * self.bn, min((b + 1) * self.bn, self.n)
        ka, ke = a // 64, (e + 63) // 64
        res = dict(bits=self.bits[:, ka:ke].cpu().numpy().view(np.uint64),
                   counts=np.concatenate([self.counts[a:e].cpu().numpy(),
                                          self.counts[self.n + a:self.n + e].cpu().numpy()]),
                   out=self.out[a:e].cpu().numpy(), stats=self.stats[b:b + 1], dec=self.dec[b:b + 1])
        gh = self.g[:, a:e].contiguous().cpu().numpy()
        return check_ternary_bucket(res, gh, np.ascontiguousarray(self.mask_h[ka:ke]), e - a, self.pol, 0, e - a,
                                    f"{self.lay.name} bucket {b}")


def test_fullsize_ternary_gpt1p3b_sampled_buckets():
    f = FullTernary("gpt1p3b", nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5))
    try:
        routes = f.dec["route"].astype(int)
        assert (routes[:185] == nfo.ROUTE_L).all() and (routes[185:] == nfo.ROUTE_P).all()
        for b in (0, 100, 183, 184, 185, 200):
            f.check_bucket(b)
    finally:
        f.release()


def test_fullsize_ternary_stress_forced_lowbit():
    f = FullTernary("stress", nf.policy(format=nf.NF_FORMAT_TERNARY, tau=0.5, force_lowbit=1))
    try:
        W, n, mask = f.W, f.n, f.mask_h
        n_e = nfo.count_eligible(mask, n)

        def row_stats(w):
            return nfo.health(f.g[w:w + 1, :n].cpu().numpy(), mask)[0]
        with ThreadPoolExecutor(8) as ex:
            ref_st = np.array(list(ex.map(row_stats, range(W))), dtype=nfo.STATS_DTYPE)
        check_stats(f.stats[0], ref_st, "stress ternary")
        d = f.dec[0]
        assert int(d["route"]) == nfo.ROUTE_L
        th_gpu = nf.nf_ternary_threshold(f.stats[0], n_e, 0.5)
        th_ref = np.array([nfo.ternary_threshold(ref_st[w], n_e, 0.5) for w in range(W)], np.float32)
        q = nfo.ternary_decode_table(W, f.pol.decode_mode)
        rng = np.random.default_rng(12)
        nw = (n + 63) // 64
        words = set(rng.integers(0, nw, 48).tolist()) | {0, nw - 1}
        words |= {int(i) // 64 for i in f.lay.inject_i[:24]}
        for k in sorted(words):
            a, e = 64 * k, min(64 * k + 64, n)
            gh = f.g[:, a:e].contiguous().cpu().numpy()
            mw = np.ascontiguousarray(mask[k:k + 1])
            pos, neg = nfo.pack_ternary(gh, mw, th_gpu)  # the planes the GPU's thresholds define
            bp = f.bits[:W, k:k + 1].cpu().numpy().view(np.uint64)
            bn_ = f.bits[W:, k:k + 1].cpu().numpy().view(np.uint64)
            assert np.array_equal(bp, pos) and np.array_equal(bn_, neg), f"planes word {k}"
            rp, rn = nfo.pack_ternary(gh, mw, th_ref)  # the oracle's own thresholds
            lo, hi = np.minimum(th_gpu, th_ref), np.maximum(th_gpu, th_ref)
            between = (np.abs(gh) >= lo[:, None]) & (np.abs(gh) < hi[:, None])
            diff = (unpack(pos, e - a) != unpack(rp, e - a)) | (unpack(neg, e - a) != unpack(rn, e - a))
            assert not np.any(diff & ~between), f"planes away from the thresholds, word {k}"
            cp, cn = nfo.counts(pos, e - a), nfo.counts(neg, e - a)
            assert np.array_equal(f.counts[a:e].cpu().numpy(), cp), f"c+ word {k}"
            assert np.array_equal(f.counts[n + a:n + e].cpu().numpy(), cn), f"c- word {k}"
            m = mask_bool(mw, e - a)
            want = np.where(m, (np.float32(d["scale"]) * q[cp.astype(int) - cn.astype(int) + W]).astype(np.float32),
                            nfo.fp32_path(gh, f.pol.fp32_op))
            assert same_f32(f.out[a:e].cpu().numpy(), want), f"output word {k}"
    finally:
        f.release()
