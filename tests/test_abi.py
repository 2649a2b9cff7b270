"""The C-ABI library on the host (no GPU): it loads, exports every function
include/nf.h declares, its host functions agree with the oracle, and invalid
arguments return error codes before anything is launched."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as nfo
import paper_2606_25759_amd as nf
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "nf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nf_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_function():
    lib = nf.load()
    decl = declared_functions()
    assert len(decl) >= 12
    for name in decl:
        assert hasattr(lib, name), f"{name} not exported"
    assert sorted(nf.EXPORTS) == decl


def test_abi_version_and_struct_sizes():
    assert nf.nf_abi_version() == 2
    assert ctypes.sizeof(nf.nf_worker_stats) == 24 == nf.STATS_DTYPE.itemsize
    assert ctypes.sizeof(nf.nf_route_decision) == 40 == nf.DECISION_DTYPE.itemsize
    assert ctypes.sizeof(nf.nf_route_policy) == 40


@pytest.mark.parametrize("n", [0, 1, 63, 64, 65, 1000, 100_003])
def test_mask_from_segments_matches_oracle(n):
    lay = synth.small(1, n, 31 + n, elig_frac=0.6, nruns=17)
    off, ln, el = synth.mask_segments(lay)
    a = nf.nf_mask_from_segments(off, ln, el, n)
    b = nfo.mask_from_segments(off, ln, el, n)
    assert np.array_equal(a, b)


def test_mask_from_segments_rejects_out_of_range():
    with pytest.raises(nf.NFError) as e:
        nf.nf_mask_from_segments([5], [10], [1], 12)
    assert e.value.status == nf.NF_ERR_INVALID_ARG
    with pytest.raises(nf.NFError):
        nf.nf_mask_from_segments([-1], [1], [1], 12)


def test_route_decide_host_matches_oracle():
    rng = np.random.default_rng(5)
    for trial in range(3000):
        W = int(rng.integers(1, 20))
        st = np.zeros(W, dtype=nf.STATS_DTYPE)
        st["sum_abs_elig"] = rng.choice([0.0, 1.0, 2.5, 1e-7], size=W)
        st["sum_sq"] = rng.choice([0.0, 1.0, 2.0, 16.0, 17.0, 40.0, np.inf, np.nan], size=W)
        st["nonfinite"] = rng.choice([0, 0, 0, 3], size=W)
        n = int(rng.integers(0, 1000))
        ne = int(rng.integers(0, n + 1))
        kw = dict(admitted=int(rng.integers(0, 2)), veto=int(rng.integers(0, 2)),
                  guard_ok=int(rng.integers(0, 2)), force_lowbit=int(rng.integers(0, 2)),
                  kappa=float(rng.choice([1.0, 2.0, 4.0, 3.5])), format=int(rng.integers(0, 2)))
        d = nf.nf_route_decide(st, n, ne, nf.policy(**kw))
        rd = nfo.decide(st, n, ne, nfo.policy(**kw))
        assert (d.route, d.reasons, d.n_eligible) == (rd.route, rd.reasons, rd.n_eligible), trial
        assert d.bytes_route == rd.bytes_route and d.bytes_fp32 == rd.bytes_fp32
        assert np.float32(d.scale) == np.float32(rd.scale)


def test_ternary_threshold_host_matches_oracle():
    rng = np.random.default_rng(6)
    for trial in range(500):
        W = int(rng.integers(1, 40))
        st = np.zeros(W, dtype=nf.STATS_DTYPE)
        st["sum_abs_elig"] = rng.random(W) * 10.0 ** float(rng.integers(-9, 3))
        st["sum_abs_elig"][rng.random(W) < 0.1] = np.nan
        ne = int(rng.integers(0, 10 ** 7))
        tau = float(np.float32(rng.choice([0.0, 0.25, 0.5, 1.0, 3.0, rng.random() * 4])))
        th = nf.nf_ternary_threshold(st, ne, tau)
        want = np.array([nfo.ternary_threshold(st[w], ne, tau) for w in range(W)], dtype=np.float32)
        na, nb = np.isnan(th), np.isnan(want)
        assert np.array_equal(na, nb) and np.array_equal(th[~na].view(np.uint32), want[~nb].view(np.uint32)), trial


def test_route_decide_worked_example():
    """The W=3 worked bucket's statistics give route L, reasons 0."""
    st = np.zeros(3, dtype=nf.STATS_DTYPE)
    st["sum_abs_elig"] = [1.5, 4.0, 4.25]
    st["sum_sq"] = [5.25, 22.5, 74.0625]
    d = nf.nf_route_decide(st, 4, 3)
    assert (d.route, d.reasons) == (nf.NF_ROUTE_LOWBIT, 0)
    assert np.float32(d.scale).view(np.uint32) == 0x3F8AAAAB
    assert d.bytes_route == 8.375 and d.bytes_fp32 == 16.0


def _lib():
    return nf.load()


def test_invalid_arguments_return_codes_without_launch():
    lib = _lib()
    P = ctypes.c_void_p
    fake = P(0x1000)          # never dereferenced: validation fails first
    ws = P(0x100000)
    # W out of range
    assert lib.nf_bucket_health(fake, 64, 0, 64, fake, fake, ws, 1 << 20, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_bucket_health(fake, 64, 256, 64, fake, fake, ws, 1 << 20, None) == nf.NF_ERR_INVALID_ARG
    assert "W=256" in nf.nf_last_error()
    # stride < n
    assert lib.nf_fp32_reduce(fake, 10, 2, 64, fake, 0, 0, fake, None) == nf.NF_ERR_INVALID_ARG
    # misaligned gradients / stride
    assert lib.nf_fp32_reduce(P(0x1004), 64, 2, 64, fake, 0, 0, fake, None) == nf.NF_ERR_ALIGNMENT
    assert lib.nf_fp32_reduce(fake, 66, 2, 64, fake, 0, 0, fake, None) == nf.NF_ERR_ALIGNMENT
    # bad select / op
    assert lib.nf_fp32_reduce(fake, 64, 2, 64, fake, 9, 0, fake, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_fp32_reduce(fake, 64, 2, 64, fake, 0, 9, fake, None) == nf.NF_ERR_INVALID_ARG
    # bits stride too small
    assert lib.nf_pack_signs(fake, 640, 2, 640, fake, fake, 9, None, ws, 1 << 20, None) == nf.NF_ERR_INVALID_ARG
    # the allocation-free driver: sizes beyond its static scratch, bad sizes, before any launch
    big = 100_000_000
    assert nf.nf_workspace_bytes(255, big) > nf.NF_STATIC_SCRATCH_BYTES
    assert lib.nf_route_buckets_noalloc(fake, big, 255, big, big, fake, None, fake, big, None, fake, fake, fake,
                                        None) == nf.NF_ERR_WORKSPACE
    assert "static" in nf.nf_last_error()
    assert lib.nf_route_buckets_noalloc(fake, 640, 0, 640, 640, fake, None, fake, 10, None, fake, fake, fake,
                                        None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_route_buckets_noalloc(fake, 640, 2, 640, 100, fake, None, fake, 10, None, fake, fake, fake,
                                        None) == nf.NF_ERR_INVALID_ARG
    # workspace too small
    need = nf.nf_workspace_bytes(2, 640)
    assert need > 0
    assert lib.nf_pack_signs(fake, 640, 2, 640, fake, fake, 10, None, ws, need - 1, None) == nf.NF_ERR_WORKSPACE
    # policy checks
    pol = nf.policy(kappa=0.0)
    assert lib.nf_route_bucket(fake, 640, 2, 640, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                               ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    pol = nf.policy(decode_mode=5)
    assert lib.nf_route_bucket(fake, 640, 2, 640, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                               ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    pol = nf.policy(format=7)
    assert lib.nf_route_bucket(fake, 640, 2, 640, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                               ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=-1.0)
    assert lib.nf_route_bucket(fake, 640, 2, 640, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                               ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    # flat buffers: bucket_n > 0 and, when there are several buckets, a multiple of 64
    pol = nf.policy()
    assert lib.nf_route_buckets(fake, 640, 2, 640, 0, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                                ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_route_buckets(fake, 640, 2, 640, 100, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                                ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    pol = nf.policy(format=nf.NF_FORMAT_TERNARY, tau=float("nan"))
    assert lib.nf_route_bucket(fake, 640, 2, 640, fake, ctypes.byref(pol), fake, 10, None, fake, fake, fake,
                               ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    # ternary components
    assert lib.nf_pack_ternary(fake, 640, 2, 640, fake, None, fake, 10, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_pack_ternary(fake, 640, 2, 640, fake, P(0x1002), fake, 10, None) == nf.NF_ERR_ALIGNMENT
    assert lib.nf_ternary_reduce(fake, 10, 2, 640, fake, None, 0, None, fake, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_ternary_reduce(fake, 10, 2, 640, fake, fake, 4, None, fake, None) == nf.NF_ERR_INVALID_ARG
    th = (ctypes.c_float * 2)()
    assert lib.nf_ternary_threshold(st_fake := (nf.nf_worker_stats * 2)(), 2, 10, ctypes.c_float(-0.5), th) == \
        nf.NF_ERR_INVALID_ARG
    # bucket size not a multiple of 64
    pol = nf.policy()
    assert lib.nf_route_buckets(fake, 6400, 2, 6400, 100, fake, ctypes.byref(pol), fake, 100, None, fake,
                                fake, fake, ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    # decode counts: W out of range
    assert lib.nf_signcount_reduce(fake, 10, 0, 640, fake, fake, 0, fake, fake, None) == nf.NF_ERR_INVALID_ARG
    # hierarchical counting: group size must divide W; partial stride; alignment of partial rows
    assert lib.nf_partial_counts(fake, 10, 8, 3, 640, fake, 640, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_partial_counts(fake, 10, 8, 0, 640, fake, 640, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_partial_counts(fake, 10, 8, 4, 640, fake, 639, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_partial_counts(fake, 9, 8, 4, 640, fake, 640, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_partial_count_reduce(fake, 640, 3, 8, 640, fake, fake, 0, fake, fake, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_partial_count_reduce(P(0x1008), 640, 2, 8, 640, fake, fake, 0, fake, fake, None) == \
        nf.NF_ERR_ALIGNMENT
    assert lib.nf_partial_count_reduce(fake, 648, 2, 8, 640, fake, fake, 0, fake, fake, None) == \
        nf.NF_ERR_ALIGNMENT
    assert lib.nf_partial_count_reduce(fake, 640, 2, 8, 640, fake, None, 0, fake, fake, None) == \
        nf.NF_ERR_INVALID_ARG
    # compacted payload and per-slice scales
    assert lib.nf_compact_signs(fake, 10, 2, 640, fake, fake, fake, 641, fake, 11, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_compact_signs(fake, 10, 2, 640, fake, fake, fake, 600, fake, 9, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_compact_signs(fake, 10, 2, 640, fake, P(0x1004), fake, 600, fake, 10, None) == nf.NF_ERR_ALIGNMENT
    assert lib.nf_slice_scales(fake, 640, 0, fake, fake, fake, 3, 3, fake, fake, ws, 1 << 20, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_slice_scales(fake, 640, 2, fake, fake, fake, 3, 2, fake, fake, ws, 1 << 20, None) == \
        nf.NF_ERR_INVALID_ARG
    need = nf.nf_slice_workspace_bytes(2, 3)
    assert lib.nf_slice_scales(fake, 640, 2, fake, fake, fake, 3, 3, fake, fake, ws, need - 1, None) == \
        nf.NF_ERR_WORKSPACE
    # slice statistics from pass 1's partials: W, S <= n, stride, NULLs, alignment, workspace; S = 0 is a no-op
    wneed = nf.nf_workspace_bytes(2, 640)
    assert lib.nf_slice_scales_from_pass1(fake, 640, 0, 640, fake, fake, 3, fake, fake, ws, wneed, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_slice_scales_from_pass1(fake, 640, 2, 2, fake, fake, 3, fake, fake, ws, wneed, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_slice_scales_from_pass1(fake, 639, 2, 640, fake, fake, 3, fake, fake, ws, wneed, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_slice_scales_from_pass1(fake, 640, 2, 640, None, fake, 3, fake, fake, ws, wneed, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_slice_scales_from_pass1(fake, 640, 2, 640, P(0x1004), fake, 3, fake, fake, ws, wneed, None) == \
        nf.NF_ERR_ALIGNMENT
    assert lib.nf_slice_scales_from_pass1(fake, 640, 2, 640, fake, fake, 3, fake, fake, ws, wneed - 1, None) == \
        nf.NF_ERR_WORKSPACE
    assert lib.nf_slice_scales_from_pass1(None, 640, 2, 640, None, None, 0, None, None, None, 0, None) == nf.NF_OK
    assert lib.nf_compact_signcount_reduce(fake, 10, 2, 640, fake, fake, fake, fake, 2, 600, fake, 0, None, fake,
                                           None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_compact_signcount_reduce(fake, 10, 2, 640, fake, fake, fake, fake, 0, 600, fake, 0, fake, fake,
                                           None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_compact_signcount_reduce(fake, 10, 2, 640, fake, fake, fake, fake, 2, 600, fake, 7, fake, fake,
                                           None) == nf.NF_ERR_INVALID_ARG
    # stock replicas: count and stride
    assert lib.nf_stock_signcount(fake, 10, 8, 640, fake, fake, 0, 0, fake, fake, 640, None) == \
        nf.NF_ERR_INVALID_ARG
    assert lib.nf_stock_signcount(fake, 10, 8, 640, fake, fake, 0, 2, fake, fake, 639, None) == \
        nf.NF_ERR_INVALID_ARG
    # decision: n_eligible > n
    st = (nf.nf_worker_stats * 2)()
    d = nf.nf_route_decision()
    assert lib.nf_route_decide(st, 2, 10, 11, ctypes.byref(pol), ctypes.byref(d)) == nf.NF_ERR_INVALID_ARG


def test_bucket_table_sizes_and_argument_errors():
    lib = _lib()
    P = ctypes.c_void_p
    fake = P(0x1000)          # never dereferenced: validation fails first
    ws = P(0x100000)
    b = 6_553_600
    # equal buckets through a table: the workspace of the equal-bucket driver
    for W in (4, 16, 64, 255):
        assert nf.nf_workspace_bytes_table(W, [0, b, 2 * b, 3 * b]) == nf.nf_workspace_bytes_buckets(W, 3 * b, b)
    # a short last bucket holds fewer slots than a full one
    assert 0 < nf.nf_workspace_bytes_table(16, [0, b, b + 64]) <= nf.nf_workspace_bytes_buckets(16, b + 64, b)
    # the table: 32-byte rows, then an int32 per pass-1 chunk, each part 256-byte aligned
    _, chunks = nf.nf_pass1_chunk_elems(16, 3 * b, b)
    assert nf.nf_bucket_table_bytes(16, [0, b, 2 * b, 3 * b]) == 256 + -(-3 * chunks * 4 // 256) * 256
    pol = nf.policy()
    for bad in ([0], [1, 64], [0, 64, 64], [0, 100, 200], [0, 128, 64]):
        assert nf.nf_bucket_table_bytes(16, bad) == 0 and nf.nf_workspace_bytes_table(16, bad) == 0, bad
        o = np.array(bad, np.int64)
        op = o.ctypes.data_as(P)
        assert lib.nf_bucket_table_init(16, op, len(bad) - 1, fake, 1 << 20, None) == nf.NF_ERR_INVALID_ARG
        assert lib.nf_route_bucket_table(fake, 1 << 10, 16, op, len(bad) - 1, fake, fake, ctypes.byref(pol),
                                         fake, 16, None, fake, fake, fake, ws, 1 << 24, None) == \
            nf.NF_ERR_INVALID_ARG, bad
    assert "multiple of 64" in (lib.nf_bucket_table_init(16, np.array([0, 100, 200], np.int64).ctypes.data_as(P), 2,
                                                         fake, 1 << 20, None) and nf.nf_last_error())
    o = np.array([0, 640, 1000], np.int64)
    op = o.ctypes.data_as(P)
    need = nf.nf_bucket_table_bytes(16, o)
    assert lib.nf_bucket_table_init(0, op, 2, fake, need, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_bucket_table_init(16, op, 2, fake, need - 1, None) == nf.NF_ERR_WORKSPACE
    assert lib.nf_bucket_table_init(16, op, 2, None, need, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_bucket_table_init(16, op, 2, P(0x1008), need, None) == nf.NF_ERR_ALIGNMENT
    assert lib.nf_route_bucket_table(fake, 1 << 10, 16, op, 2, None, fake, ctypes.byref(pol), fake, 16, None,
                                     fake, fake, fake, ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_route_bucket_table(fake, 1 << 10, 16, op, 2, P(0x1008), fake, ctypes.byref(pol), fake, 16, None,
                                     fake, fake, fake, ws, 1 << 24, None) == nf.NF_ERR_ALIGNMENT
    # more buckets than a launch-grid row holds, in both drivers, before any launch
    many = np.arange(0, 64 * 65_537, 64, dtype=np.int64)  # 65,536 buckets of 64
    assert nf.nf_bucket_table_bytes(16, many) == 0
    assert lib.nf_route_bucket_table(fake, 1 << 23, 16, many.ctypes.data_as(P), len(many) - 1, fake, fake,
                                     ctypes.byref(pol), fake, 1 << 17, None, fake, fake, fake, ws, 1 << 30,
                                     None) == nf.NF_ERR_INVALID_ARG
    assert lib.nf_route_buckets(fake, 1 << 23, 16, 64 * 65_536, 64, fake, ctypes.byref(pol), fake, 1 << 17, None,
                                fake, fake, fake, ws, 1 << 30, None) == nf.NF_ERR_INVALID_ARG
    assert "at most 65535" in nf.nf_last_error()
    # a row stride shorter than n_total = offsets[nb]
    assert lib.nf_route_bucket_table(fake, 996, 16, op, 2, fake, fake, ctypes.byref(pol), fake, 16, None,
                                     fake, fake, fake, ws, 1 << 24, None) == nf.NF_ERR_INVALID_ARG


def test_sliced_sizes():
    ne, seg = ctypes.c_int64(), ctypes.c_int64()
    ln = np.array([1, 65536, 65537, 200_000], dtype=np.int64)
    assert nf.load().nf_sliced_layout_sizes(ln.ctypes.data, 4, ctypes.byref(ne), ctypes.byref(seg)) == nf.NF_OK
    assert ne.value == int(ln.sum()) and seg.value == 1 + 1 + 2 + 4
    assert nf.nf_slice_workspace_bytes(16, 8) == 1024 and nf.nf_slice_workspace_bytes(0, 8) == 0


def test_pass1_launch_counts():
    # GPT-1.3B scale: 201 buckets of 400 chunks (the last 306), 80,306 chunks
    assert nf.nf_pass1_launches(16, 1_315_723_264, 6_553_600) == 314
    assert nf.nf_pass1_launches(16, 1_315_723_264, 6_553_600, sign_words=False) == 79
    # small problems: one launch either way; empty and invalid sizes: none
    assert nf.nf_pass1_launches(4, 1 << 20, 1 << 20) == 1
    assert nf.nf_pass1_launches(4, 1 << 20, 1 << 20, sign_words=False) == 1
    assert nf.nf_pass1_launches(16, 0, 100) == 0
    assert nf.nf_pass1_launches(0, 100, 100) == 0
    assert nf.nf_pass1_launches(256, 100, 100) == 0


def test_pass1_chunk_geometry():
    # W = 16: tiles of 512 elements, 32 per chunk; a 25 MiB bucket has 400 chunks
    assert nf.nf_pass1_chunk_elems(16, 6_553_600 * 201, 6_553_600) == (16_384, 400)
    # W = 64: two row groups of 32, two workers per wavefront, tiles of 256 elements, 32 per chunk
    assert nf.nf_pass1_chunk_elems(64, 100_000_000, 100_000_000) == (8_192, 12_208)
    assert nf.nf_pass1_launches(64, 100_000_000, 100_000_000) == 2 * 48
    # W > 64: rows in ceil(W / 64) near-equal groups, with the geometry of the
    # largest (255: four of 64 or 63 rows; 65: 33 and 32 rows, tiles of 256
    # elements, 31 per chunk)
    assert nf.nf_pass1_chunk_elems(255, 6_553_600 * 2, 6_553_600) == (4_096, 1_600)
    assert nf.nf_pass1_chunk_elems(65, 6_553_600 * 2, 6_553_600) == (7_936, 826)
    assert nf.nf_pass1_launches(255, 6_553_600 * 2, 6_553_600) == 4  # 3,200 chunks: one launch per group
    assert nf.nf_pass1_launches(65, 6_553_600 * 2, 6_553_600) == 2
    # above 4,096 chunks, launches of 256 (1,024 without sign words)
    assert nf.nf_pass1_launches(16, 70_000_000, 30_000_000) == 17  # 4,275 chunks
    assert nf.nf_pass1_launches(16, 70_000_000, 30_000_000, sign_words=False) == 5
    assert nf.nf_pass1_launches(16, 60_000_000, 30_000_000) == 1  # 3,664 chunks
    # a problem of fewer than 1,024 chunks takes shorter ones to fill the chip
    # (at most 1,024 chunks); one of at most 1,024 tiles takes one chunk per
    # compute unit (at most 256, whole tiles)
    for W, n, most in ((4, 1 << 20, 256), (16, 500_000, 256), (64, 200_000, 256), (255, 250_000, 256),
                       (4, 4_000_000, 1024), (16, 8_000_000, 1024), (64, 1_000_000, 1024)):
        e, c = nf.nf_pass1_chunk_elems(W, n, n)
        assert most // 2 < c <= most and e * c >= n and e % 64 == 0, (W, n, e, c)
    assert nf.nf_pass1_chunk_elems(0, 100, 100) == (0, 0)
    assert nf.nf_pass1_chunk_elems(16, 0, 100) == (0, 0)


def test_workspace_sizes():
    assert nf.nf_workspace_bytes(0, 10) == 0
    # One bucket of 6,553,600 elements at W=16 is a small problem: 12,800 tiles
    # in 985 chunks of 13, so 985 partial slots and 493 groups of two;
    # 40-byte partials and 8-byte counts, each array 256-byte aligned.
    a = nf.nf_workspace_bytes(16, 6_553_600)
    assert a == 630_528 + 7_936 + 315_648 + 4_096
    # 201 such buckets: 400 chunks of 32 tiles each, no second level.
    b = nf.nf_workspace_bytes_buckets(16, 6_553_600 * 201, 6_553_600)
    assert b == 51_456_000 + 643_328
    assert nf.nf_workspace_bytes_buckets(16, 100, 0) == 0
    # W = 255, two 25 MiB buckets: 1,600 chunk slots each, summed first in
    # 64 groups of 25 (the decision reads at most 64 partials per worker above
    # 32 workers).
    c = nf.nf_workspace_bytes_buckets(255, 6_553_600 * 2, 6_553_600)
    assert c == 2 * 1_600 * 255 * 40 + 25_600 + 2 * 64 * 255 * 40 + 1_024


def declared_prototypes():
    """name -> list of parameter declarations, from include/nf.h."""
    src = open(os.path.join(ROOT, "include", "nf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    out = {}
    for m in re.finditer(r"\b(nf_[a-z0-9_]+)\s*\(([^;{]*?)\)\s*;", src, flags=re.S):
        params = [p.strip() for p in m.group(2).split(",")]
        out[m.group(1)] = [] if params == ["void"] or params == [""] else params
    return out


def _ctype_class(param):
    if "*" in param:
        return "pointer"
    for c, k in (("int64_t", "i64"), ("int32_t", "i32"), ("size_t", "size"), ("double", "f64"), ("float", "f32"),
                 ("int", "i32")):
        if re.search(rf"\b{c}\b", param):
            return k
    return "other"


def test_binding_signatures_match_the_header():
    lib = nf.load()
    kinds = {ctypes.c_void_p: "pointer", ctypes.c_char_p: "pointer", ctypes.c_int64: "i64", ctypes.c_int32: "i32",
             ctypes.c_size_t: "size", ctypes.c_double: "f64", ctypes.c_float: "f32"}
    protos = declared_prototypes()
    assert sorted(protos) == declared_functions()
    for name, params in protos.items():
        args = getattr(lib, name).argtypes or []
        assert len(args) == len(params), f"{name}: {len(args)} ctypes arguments, {len(params)} declared"
        for a, p in zip(args, params):
            k = kinds.get(a, "pointer" if issubclass(a, (ctypes._Pointer, ctypes.Structure)) else "other")
            assert k == _ctype_class(p), f"{name}: {p!r} bound as {a}"
