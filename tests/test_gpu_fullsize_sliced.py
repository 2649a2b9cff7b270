"""Parity of the sliced path at the GPT-1.3B scale, in the configuration that
`bench.py --sliced` times: pass 1 over the whole buffer as one bucket,
compaction, per-slice scales from pass 1's chunk partials, and the count +
decode from the compacted rows (every eligible tensor is one slice).

Nothing is sampled.  Every slice's sums and scale are checked against the
two-pass statistics on the GPU, and their total against pass 1's bucket
sums.  Every slice is then checked against the oracle, in a pool of host
threads (its calls release the interpreter lock): sums and scale, the
compacted words that lie inside it, its compacted-order counts and its
decoded values; every compacted word that straddles two slices is checked
from both slices' signs; and every position outside the slices must be
untouched."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import POOL, same_f32

pytestmark = pytest.mark.gpu


def test_fullsize_sliced_gpt1p3b():
    lay = synth.CONFIGS["gpt1p3b"]()
    d = torch.device("cuda:0")
    W, n = lay.W, lay.n_total
    nw = (n + 63) // 64
    print(f"[fullsize sliced] gpt1p3b: W={W} n={n:,}", flush=True)
    g = torch.empty((W, lay.stride), dtype=torch.float32, device=d)
    synth.generate_device(lay, g)
    off, ln, el = synth.mask_segments(lay)
    e = np.asarray(el, bool)
    soff, sln = np.asarray(off, np.int64)[e], np.asarray(ln, np.int64)[e]
    sl = nf.SlicedLayout(soff, sln, n, device=d)
    bits = torch.empty((W, nw), dtype=torch.int64, device=d)
    stats = torch.zeros(W * nf.STATS_BYTES, dtype=torch.uint8, device=d)
    ws = nf.empty_workspace(nf.nf_workspace_bytes(W, n), d)
    nf.nf_pack_signs(g, n, sl.d_mask, bits, stats, ws)
    nwc = (sl.n_eligible + 63) // 64
    cbits = torch.empty((W, nwc), dtype=torch.int64, device=d)
    nf.nf_compact_signs(bits, W, n, sl, cbits)
    del bits
    sums = torch.empty((sl.S, W), dtype=torch.float64, device=d)
    scales = torch.empty(sl.S, dtype=torch.float32, device=d)
    nf.nf_slice_scales_from_pass1(g, n, sl, sums, scales, ws)
    sums2 = torch.empty((sl.S, W), dtype=torch.float64, device=d)
    scales2 = torch.empty(sl.S, dtype=torch.float32, device=d)
    ws2 = nf.empty_workspace(nf.nf_slice_workspace_bytes(W, sl.segments), d)
    nf.nf_slice_scales(g, sl, sums2, scales2, ws2)
    counts_c = torch.empty(sl.n_eligible, dtype=torch.uint8, device=d)
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=d)
    nf.nf_compact_signcount_reduce(cbits, W, sl, scales, nfo.DECODE_SOFT, counts_c, out)
    torch.cuda.synchronize()

    s1, sc = sums.cpu().numpy(), scales.cpu().numpy()
    assert np.allclose(s1, sums2.cpu().numpy(), rtol=1e-12, atol=0), "sums: from pass 1 vs second read"
    sc2 = scales2.cpu().numpy()
    assert np.all(np.abs(sc - sc2) <= 1e-6 * np.abs(sc2)), "scales: from pass 1 vs second read"
    st = nf.stats_host(stats, W)[0]
    assert np.allclose(s1.sum(axis=0), st["sum_abs_elig"], rtol=1e-12, atol=0), "slices add up to the bucket"

    q = nfo.decode_table(W)
    ones = lambda k: np.full(k, np.uint64(0xFFFFFFFFFFFFFFFF))

    def check_slice(s):
        o, L, r0 = int(soff[s]), int(sln[s]), int(sl.rstart[s])
        tag = f"slice {s} ({L:,} elements at {o:,})"
        gh = g[:, o:o + L].contiguous().cpu().numpy()
        ref_sums, ref_sc = nfo.slice_scales(gh, np.zeros(1, np.int64), np.array([L], np.int64))
        assert np.allclose(s1[s], ref_sums[0], rtol=1e-12, atol=0), f"{tag} sums"
        assert abs(sc[s] - ref_sc[0]) <= 1e-6 * abs(ref_sc[0]), f"{tag} scale"
        full = ones((L + 63) // 64)
        if L % 64:
            full[-1] = np.uint64((1 << (L % 64)) - 1)
        sbits = nfo.pack(gh, full)  # the slice's signs, in rank order
        want_c = nfo.counts(sbits, L)
        # compacted words wholly inside the slice's ranks [r0, r0 + L)
        oa, ob = -(-r0 // 64), (r0 + L) // 64
        if ob > oa:
            sub = np.ascontiguousarray(gh[:, 64 * oa - r0:64 * ob - r0])
            want_w = nfo.pack(sub, ones(ob - oa))
            assert np.array_equal(cbits[:, oa:ob].cpu().numpy().view(np.uint64), want_w), f"{tag} compacted words"
        assert np.array_equal(counts_c[r0:r0 + L].cpu().numpy(), want_c), f"{tag} compacted-order counts"
        assert same_f32(out[o:o + L].cpu().numpy(), np.float32(sc[s]) * q[want_c]), f"{tag} decoded values"
        return L

    def check_straddle(s):
        """The compacted word holding the last ranks of slice s: shared with the
        first ranks of the next slice, or (after the last slice) the payload's
        last, zero-padded word.  Every slice is far longer than 64 elements."""
        r_end = int(sl.rstart[s]) + int(sln[s])
        if r_end % 64 == 0:
            return 0
        w0 = r_end // 64
        o, L = int(soff[s]), int(sln[s])
        tail = g[:, o + L - (r_end - 64 * w0):o + L]
        k = min(64 * w0 + 64, sl.n_eligible) - r_end
        if k > 0:
            o2 = int(soff[s + 1])
            assert k <= int(sln[s + 1]), "a word spans three slices"
            both = torch.cat([tail, g[:, o2:o2 + k]], dim=1).contiguous().cpu().numpy()
        else:
            both = tail.contiguous().cpu().numpy()
        m = ones(1)
        if both.shape[1] < 64:
            m[0] = np.uint64((1 << both.shape[1]) - 1)
        want = nfo.pack(both, m)
        assert np.array_equal(cbits[:, w0:w0 + 1].cpu().numpy().view(np.uint64), want), f"word {w0} after slice {s}"
        return 1

    with ThreadPoolExecutor(POOL) as ex:
        assert sum(ex.map(check_slice, range(sl.S))) == sl.n_eligible
        straddles = sum(ex.map(check_straddle, range(sl.S)))
    print(f"[fullsize sliced] {sl.S} slices and {straddles} straddling words checked", flush=True)

    # every position outside the slices: untouched
    elig = np.unpackbits(sl.mask.view(np.uint8), bitorder="little")[:n].astype(bool)
    assert int(elig.sum()) == sl.n_eligible
    oh = out.cpu().numpy()
    assert np.isnan(oh[~elig]).all(), "positions outside the slices written"
