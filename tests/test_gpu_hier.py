"""GPU parity of hierarchical and stock sign counting (§6.1 reducer model,
§6.3 contrast with stock packed-sign transport) against the oracle, through
the C ABI.

The W worker rows form G groups of P workers (a group = one node's GPUs).
Node-local partial counts must equal the oracle's counts over each group's
rows; their sum, and every replica of the stock (replicated) count, must
equal the oracle's count over all W rows; all bit-exact.  Decoded values are
exactly fl32(scale * q[c]) with the oracle's decode table.
"""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests.nfgpu import mask_bool, same_f32, to_dev

pytestmark = pytest.mark.gpu


def payload(W, n, seed):
    """Sign bitmaps of seeded gradients through the oracle's pack (a real
    payload: zero padding, routed positions 0) and the mask."""
    lay = synth.small(W, n, seed, elig_frac=0.8, nruns=7)
    g = synth.generate_host(lay)
    mask = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    return nfo.pack(g, mask), mask


GROUPS = [(8, 1), (8, 4), (8, 8), (12, 3), (16, 4), (64, 8), (255, 5), (255, 51)]


@pytest.mark.parametrize("W,P", GROUPS)
@pytest.mark.parametrize("n", [1, 63, 64, 65, 4097, 131_072, 100_003])
def test_partial_counts_match_oracle(W, P, n):
    bits, _ = payload(W, n, 13 * W + n)
    G = W // P
    stride = (n + 15) // 16 * 16 + 16
    partial = torch.full((G, stride), 0xCD, dtype=torch.uint8, device="cuda:0")
    nf.nf_partial_counts(to_dev(bits.view(np.int64)), W, P, n, partial)
    torch.cuda.synchronize()
    got = partial.cpu().numpy()
    for gr in range(G):
        want = nfo.counts(bits[gr * P:(gr + 1) * P], n)
        assert np.array_equal(got[gr, :n], want), f"group {gr}"
        assert np.all(got[gr, n:] == 0xCD), "bytes past n untouched"
    assert np.array_equal(got[:, :n].sum(axis=0), nfo.counts(bits, n)), "partials sum to the count"


@pytest.mark.parametrize("W,P", GROUPS)
@pytest.mark.parametrize("n", [1, 17, 64, 4097, 131_072 + 9])
@pytest.mark.parametrize("mode", [nfo.DECODE_SOFT, nfo.DECODE_MAJORITY])
def test_partial_count_reduce_matches_direct_count(W, P, n, mode):
    check_partial_count_reduce(W, P, n, mode)


@pytest.mark.parametrize("n", [131_072, 524_288])
def test_paper_local_count_shapes(n):
    """The logical-bucket shapes of the paper's local-count check (8 workers x
    131K and x 524K elements, read as 2 nodes x 4 GPUs)."""
    check_partial_count_reduce(8, 4, n, nfo.DECODE_SOFT)


def check_partial_count_reduce(W, P, n, mode):
    bits, mask = payload(W, n, 7 * W + n + mode)
    G = W // P
    stride = (n + 15) // 16 * 16
    partial = torch.zeros((G, stride), dtype=torch.uint8, device="cuda:0")
    nf.nf_partial_counts(to_dev(bits.view(np.int64)), W, P, n, partial)
    scale = np.float32(2.5e-4)
    counts = torch.full((n,), 0xAB, dtype=torch.uint8, device="cuda:0")
    out = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda:0")
    nf.nf_partial_count_reduce(partial, W, n, to_dev(mask.view(np.int64)), to_dev(np.array([scale])), mode,
                               counts, out)
    torch.cuda.synchronize()
    c = nfo.counts(bits, n)
    assert np.array_equal(counts.cpu().numpy(), c), "counts"
    m = mask_bool(mask, n)
    o = out.cpu().numpy()
    q = nfo.decode_table(W, mode)
    want = (scale * q[c]).astype(np.float32)
    assert same_f32(o[m], want[m]), "decoded values"
    assert np.all(np.isnan(o[~m])), "routed positions untouched"


@pytest.mark.parametrize("W,P", [(16, 4), (64, 8)])
def test_contrast_shapes(W, P):
    """The shapes `bench.py --contrast` times at a full bucket: 4 nodes x 4
    GPUs and 8 x 8, 6,553,600 elements."""
    check_partial_count_reduce(W, P, 6_553_600, nfo.DECODE_SOFT)


@pytest.mark.parametrize("W,R", [(1, 1), (8, 8), (16, 3), (64, 2), (255, 2)])
@pytest.mark.parametrize("n", [1, 65, 4097, 100_003])
def test_stock_replicas_equal_direct_count(W, R, n):
    bits, mask = payload(W, n, 3 * W + n)
    scale = np.float32(1.25e-3)
    stride = n + 7
    counts = torch.full((R * stride,), 0xAB, dtype=torch.uint8, device="cuda:0")
    out = torch.full((R * stride,), float("nan"), dtype=torch.float32, device="cuda:0")
    nf.nf_stock_signcount(to_dev(bits.view(np.int64)), W, n, to_dev(mask.view(np.int64)),
                          to_dev(np.array([scale])), nfo.DECODE_SOFT, R, counts, out, stride)
    torch.cuda.synchronize()
    c = nfo.counts(bits, n)
    m = mask_bool(mask, n)
    want = (scale * nfo.decode_table(W)[c]).astype(np.float32)
    cc, oo = counts.cpu().numpy(), out.cpu().numpy()
    for r in range(R):
        assert np.array_equal(cc[r * stride:r * stride + n], c), f"replica {r} counts"
        o = oo[r * stride:r * stride + n]
        assert same_f32(o[m], want[m]), f"replica {r} decode"
        assert np.all(np.isnan(o[~m]))
        assert np.all(cc[r * stride + n:(r + 1) * stride] == 0xAB)


def test_empty_calls_are_no_ops():
    bits = torch.zeros((8, 1), dtype=torch.int64, device="cuda:0")
    partial = torch.zeros((2, 16), dtype=torch.uint8, device="cuda:0")
    nf.nf_partial_counts(bits, 8, 4, 0, partial)
    nf.nf_partial_count_reduce(partial, 8, 0, None, None, 0, None, None)
    torch.cuda.synchronize()
