"""The largest bucket count one call takes, 65,535, through the C ABI: the
decision runs one block per bucket and pass 2 a row of blocks per bucket,
so this is the launch grid's limit.

Checked: 65,535 buckets of 64 elements (the last one of 17) give the same
bits, counts, outputs, statistics and decisions through the flat and the
bucket-table drivers, byte for byte, and every bucket equals the oracle on
that bucket, in both formats; 65,535 buckets of ragged sizes (64 to 1,024
elements) through the table driver equal the oracle bucket by bucket.
"""
import numpy as np
import pytest

import paper_2606_25759_amd as nf
from tests import nfgpu as H
from tests.test_gpu_bucket_table import check_table_bucket, flat_route, layout_for, table_route

pytestmark = pytest.mark.gpu

NB = 65_535
W = 3


@pytest.mark.parametrize("fmt", [nf.NF_FORMAT_BINARY, nf.NF_FORMAT_TERNARY])
def test_max_buckets_of_64(fmt):
    assert nf.NF_MAX_BUCKETS == NB
    n = (NB - 1) * 64 + 17
    off = np.append(np.arange(0, NB * 64, 64, dtype=np.int64)[:NB], n)
    g, m = layout_for(W, n, 6000 + fmt, elig_frac=0.8)
    pol = nf.policy(format=fmt, tau=0.5)
    t = table_route(g, m, off, pol)
    f = flat_route(g, m, n, 64, pol)
    for k in ("bits", "counts", "raw_stats", "raw_dec"):
        assert np.array_equal(t[k], f[k]), f"fmt={fmt}: {k} differ between the drivers"
    assert H.same_f32(t["out"], f["out"]), f"fmt={fmt}: out differs between the drivers"
    for b in range(NB):
        check_table_bucket(t, g, m, off, b, pol, f"fmt={fmt} bucket {b} of {NB}")


def test_max_buckets_ragged():
    rng = np.random.default_rng(65535)
    sizes = rng.integers(1, 17, size=NB) * 64
    sizes[-1] -= 23
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    n = int(off[-1])
    g, m = layout_for(W, n, 6100, elig_frac=0.8)
    pol = nf.policy()
    t = table_route(g, m, off, pol)
    for b in range(NB):
        check_table_bucket(t, g, m, off, b, pol, f"ragged bucket {b} of {NB}")
