"""Host layout tables of the compacted payload and per-slice scales (no GPU):
nf_sliced_layout against tables computed directly from the slice list, and
its argument checks."""
import numpy as np
import pytest

import oracle as nfo
import paper_2606_25759_amd as nf


def random_slices(n, rng, count, max_len):
    """Sorted, disjoint, non-empty intervals inside [0, n)."""
    cuts = np.sort(rng.choice(np.arange(1, n), size=min(2 * count, n - 1), replace=False))
    off, ln = [], []
    for a, b in zip(cuts[0::2], cuts[1::2]):
        b = min(b, a + max_len)
        if b > a:
            off.append(int(a))
            ln.append(int(b - a))
    return np.array(off, np.int64), np.array(ln, np.int64)


@pytest.mark.parametrize("n,count,max_len", [(1, 0, 1), (64, 1, 64), (300, 5, 40), (5000, 40, 300),
                                             (70_000, 3, 70_000), (200_003, 17, 150_000)])
def test_layout_tables(n, count, max_len):
    rng = np.random.default_rng(n)
    off, ln = random_slices(n, rng, count, max_len) if n > 1 else (np.zeros(0, np.int64), np.zeros(0, np.int64))
    lay = nf.SlicedLayout(off, ln, n)
    elig = np.zeros(n, bool)
    for o, l in zip(off, ln):
        elig[o:o + l] = True
    nE = int(elig.sum())
    assert lay.n_eligible == nE and lay.segments == int(sum(-(-l // 65536) for l in ln))
    words = np.packbits(np.concatenate([elig, np.zeros((-n) % 64, bool)]).astype(np.uint8),
                        bitorder="little").view(np.uint64)
    assert np.array_equal(lay.mask, words)
    assert nfo.count_eligible(words, n) == nE
    nw = (n + 63) // 64
    pre = np.concatenate([[0], np.cumsum([int(elig[64 * k:64 * k + 64].sum()) for k in range(nw)])])
    assert np.array_equal(lay.prefix.astype(np.int64), pre)
    ranks = np.flatnonzero(elig)                      # element of each compacted rank
    for o in range((nE + 63) // 64):
        assert lay.start[o] == ranks[64 * o] // 64
    slice_of = np.full(n, len(off))
    for s, (o, l) in enumerate(zip(off, ln)):
        slice_of[o:o + l] = s
    for k in range(nw):
        e = np.flatnonzero(elig[64 * k:64 * k + 64])
        assert lay.wslice[k] == (slice_of[64 * k + e[0]] if len(e) else len(off))
    assert np.array_equal(lay.rstart, np.concatenate([[0], np.cumsum(ln)]).astype(np.int64))


def test_layout_rejects_bad_slices():
    for off, ln, n in [([5, 3], [2, 2], 10), ([0, 2], [3, 3], 10), ([0], [0], 10), ([8], [3], 10), ([-1], [2], 10)]:
        with pytest.raises(nf.NFError):
            nf.SlicedLayout(off, ln, n)
