"""Pass-1 chunks whose elements are all routed to FP32, with more than 16
workers (several workers per wavefront).  Such a chunk is read element-major
in groups of workers, each lane keeping its running FP32 sums from one group
to the next.  The sizes give more than 1,024 chunks, so every chunk has its
full number of tiles (up to 16 steps of 64 elements per wavefront).  Long
FP32 runs hold whole routed chunks; non-finite values sit inside them, in
workers of the first, a middle and the last group.  Every output is checked
against the oracle: statistics, decision, sign words, counts and values."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from tests import nfgpu as H

pytestmark = pytest.mark.gpu


def routed_chunks(m, n, chunk):
    """Full chunks of `chunk` elements with no eligible element (one bucket)."""
    elig = H.mask_bool(m, n)
    full = n // chunk
    return int((~elig[: full * chunk].reshape(full, chunk).any(axis=1)).sum())


@pytest.mark.parametrize("W", [17, 32, 33, 64, 100, 129, 255])
def test_routed_chunks_wide(W):
    # the library's own chunk size for a problem this large (its geometry query)
    chunk, _ = nf.nf_pass1_chunk_elems(W, 1 << 30, 1 << 30)
    n = 1040 * chunk + 777
    got, per_bucket = nf.nf_pass1_chunk_elems(W, n, n)
    assert got == chunk and per_bucket == -(-n // chunk) > 1024, (got, per_bucket)
    lay = synth.small(W, n, 4000 + W, elig_frac=0.5, nruns=40)
    g = synth.generate_host(lay)
    m = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    routed = np.flatnonzero(~H.mask_bool(m, n))
    # the element-major path runs: several whole chunks hold no eligible element
    assert routed_chunks(m, n, chunk) >= 4, routed_chunks(m, n, chunk)
    rng = np.random.default_rng(W)
    bad = [0, W // 2, W - 1]
    vals = np.array([np.nan, np.inf, -np.inf], np.float32)
    g_bad = g.copy()
    for k, w in enumerate(bad):
        pos = rng.choice(routed, 5, replace=False)
        g_bad[w, pos] = vals[(np.arange(5) + k) % 3]
    cases = ((g, nf.policy(), "clean"),
             (g, nf.policy(fp32_op=nf.NF_FP32_MEAN), "mean"),
             (g_bad, nf.policy(), "non-finite"),
             (g_bad, nf.policy(force_lowbit=1), "non-finite forced"))
    # every route on the GPU first, then the oracle checks in a pool of host
    # threads (its calls release the interpreter lock)
    results = []
    for gg, pol, what in cases:
        run = H.Bucket(gg, m, n)
        results.append(run.route(pol))
        del run
        torch.cuda.empty_cache()
    with ThreadPoolExecutor(len(cases)) as ex:
        list(ex.map(lambda k: H.check_route(results[k], cases[k][0], m, n, cases[k][1], what=f"W={W} {cases[k][2]}"),
                    range(len(cases))))
