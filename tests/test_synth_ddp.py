"""The DDP-style bucket cut of the synthetic layouts (CPU): the offsets the
bucket-table tests and `bench.py --ddp-buckets` use.

DDP fills buckets with whole tensors in reverse registration order and
closes a bucket once it holds its capacity (the first bucket a smaller
one); a tensor above the capacity closes the bucket it joins.  The cut then moves each
bucket start down to a multiple of 64 elements."""
import numpy as np
import pytest

import synth

CAP, FIRST = (25 << 20) // 4, (1 << 20) // 4  # elements


@pytest.mark.parametrize("name", ["resnet50", "vitb16", "gpt1p3b", "fanin255", "stress"])
def test_ddp_offsets_invariants(name):
    lay = synth.CONFIGS[name]()
    off = synth.ddp_offsets(lay)
    assert off[0] == 0 and off[-1] == lay.n_total
    assert np.all(np.diff(off) > 0)
    assert np.all(off[:-1] % 64 == 0)
    ends = set(int(e) for e in np.cumsum(lay.lengths))
    for b in range(1, len(off) - 1):
        # each interior start lies at most 63 elements below a tensor boundary
        assert any(int(off[b]) + d in ends for d in range(64)), (name, b, int(off[b]))
    sizes = np.diff(off)
    # every bucket but the last holds at least its capacity (up to the 64-element moves)
    assert sizes[0] >= FIRST - 63
    assert np.all(sizes[1:-1] >= CAP - 126), sizes[1:-1].min()


def test_ddp_offsets_gpt_scale():
    """GPT scale: each layer gives three buckets, each closed by one of its
    large matrices (16.8M elements with the small tensors before it), and the
    last bucket holds the position table and the 102,926,336-element
    embedding."""
    lay = synth.gpt1p3b()
    sizes = np.diff(synth.ddp_offsets(lay))
    assert len(sizes) == 3 * 24 + 1
    assert np.all(np.abs(sizes[:-1] - 2048 * 8192) < 16_384), sizes[:-1]
    assert 102_926_336 + 4_194_304 <= sizes[-1] < 102_926_336 + 4_194_304 + 16_384


def test_ddp_offsets_small_layout():
    """A hand-made layout: tensors of 100k, 2M, 5M, 7M and 10 elements with a
    capacity of 25 MiB (6,553,600 elements) and a first bucket of 1 MiB."""
    t = [(100_000, 1), (2_000_000, 1), (5_000_000, 1), (7_000_000, 1), (10, 0)]
    lay = synth._from_tensors("hand", 2, 1, list(reversed(t)), (1e-3, 1e-3), synth.DIST_NORMAL)
    off = synth.ddp_offsets(lay)
    # first bucket: 100k + 2M >= 262,144 -> closes at 2,100,000 (moved down to a multiple of 64);
    # second: 5M + 7M >= 6,553,600 -> closes at 14,100,000; the last holds the 10-element tensor
    assert off.tolist() == [0, 2_100_000 // 64 * 64, 14_100_000 // 64 * 64, 14_100_010]
