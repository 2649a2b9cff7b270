"""Pins of the reference oracle against facts that do not come from the oracle.

Each pin takes a loaded oracle library (a ctypes CDLL) and raises
AssertionError on a mismatch, so the same pins run against the real oracle
(test_oracle_pins.py) and against deliberately broken copies of it
(test_oracle_mutants.py, which requires every planted mistake to be caught).

What pins what:
  * exact rational arithmetic (fractions.Fraction) with a hand-written
    round-to-nearest-even conversion to FP32: scale, decode table, decoded
    values, FP32 sums of two terms, and whole tiny buckets;
  * library routines: numpy float32 elementwise adds in worker order for the
    FP32 path, numpy float64 means and math.fsum for the health sums,
    numpy isfinite for the non-finite counts;
  * closed forms and invariants: counts in [0, W] and zero off the mask,
    sum of counts = total popcount, W = 1 gives sign(g) * scale, negation
    symmetry, exact power-of-two scaling, an all-FP32 mask gives plain FP32,
    MEAN = fl32(SUM / W), the route truth table, route correctness, and the
    modeled-bytes equation of §3.2 on hand-counted buckets;
  * brute force: every W-bit sign pattern for W <= 6 with signed zeros,
    subnormals, infinities and NaN.
"""
import itertools
import math
from fractions import Fraction

import numpy as np

import oracle as nfo

# ---------------------------------------------------------------- exact FP32


def f32_round(x):
    """Round a Fraction to the nearest FP32 value, ties to even (IEEE 754).

    Written from the definition: find the binade, scale to a 24-bit integer
    significand (or the fixed subnormal quantum), round half to even, and
    return +-inf past the largest finite value.
    """
    x = Fraction(x)
    if x == 0:
        return np.float32(0.0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                    # subnormals share the quantum 2^-149
    quantum = Fraction(2) ** (e - 23)
    q, r = divmod(a, quantum)
    q = int(q)
    if r > quantum / 2 or (r == quantum / 2 and q % 2 == 1):
        q += 1
    val = q * quantum
    if val >= Fraction(2) ** 128:
        return np.float32(sign * np.inf)
    return np.float32(sign * float(val))  # exact: val has <= 24 significant bits


def frac(x):
    return Fraction(float(x))


def same_f32(a, b):
    """Bitwise equality of FP32 arrays, any NaN equal to any NaN."""
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    if a.shape != b.shape:
        return False
    na, nb = np.isnan(a), np.isnan(b)
    if not np.array_equal(na, nb):
        return False
    return np.array_equal(a[~na].view(np.uint32), b[~nb].view(np.uint32))


# ------------------------------------------------------------ input helpers


def mask_of(m):
    """Python list/array of 0/1 per element -> LSB-first uint64 words."""
    m = np.asarray(m, dtype=np.uint8)
    n = len(m)
    words = np.zeros(max((n + 63) // 64, 1), dtype=np.uint64)
    for i in range(n):
        if m[i]:
            words[i // 64] |= np.uint64(1) << np.uint64(i % 64)
    return words[: (n + 63) // 64]


def mask_elems(words, n):
    return [int((int(words[i // 64]) >> (i % 64)) & 1) for i in range(n)]


def gauss(rng, W, n, sigma=1e-3):
    return (rng.standard_normal((W, n)) * sigma).astype(np.float32)


SPECIALS = np.array([0.0, -0.0, 1e-45, -1e-45, 1e-40, -1e-40, np.inf, -np.inf, np.nan,
                     3.4028235e38, -3.4028235e38, 1.0, -1.0], dtype=np.float32)


# --------------------------------------------------------- reference models


def model_fp32_sum(g):
    """numpy float32 elementwise adds in worker order (a library routine)."""
    s = g[0].copy()
    with np.errstate(over="ignore", invalid="ignore"):
        for w in range(1, g.shape[0]):
            s = s + g[w]
    return s


def model_bits(g, m):
    W, n = g.shape
    out = []
    for w in range(W):
        bits = [1 if (m[i] and g[w, i] > 0) else 0 for i in range(n)]
        out.append(bits)
    return out


def model_scale_exact(g, m):
    """Exact rational (sum_w (sum_E |g_w| / n_E)) / W rounded once to FP32.

    Matches the oracle bit for bit whenever every FP64 operation of the
    oracle is exact (dyadic inputs with few significant bits)."""
    W, n = g.shape
    nE = sum(m)
    if nE == 0:
        return np.float32(0.0)
    acc = Fraction(0)
    for w in range(W):
        acc += sum((abs(frac(g[w, i])) for i in range(n) if m[i]), Fraction(0)) / nE
    return f32_round(acc / W)


def model_q(W, mode):
    q = []
    for c in range(W + 1):
        margin = 2 * c - W
        if mode == nfo.DECODE_MAJORITY:
            q.append(np.float32(1.0 if margin > 0 else (-1.0 if margin < 0 else 0.0)))
        else:
            q.append(f32_round(Fraction(margin, W)))
    return np.array(q, dtype=np.float32)


# ===================================================================== pins


def pin_mask_from_segments(lib):
    rng = np.random.default_rng(11)
    for n in [1, 63, 64, 65, 200, 1000]:
        cuts = np.sort(rng.choice(np.arange(1, n), size=min(7, n - 1), replace=False)) \
            if n > 1 else np.array([], dtype=np.int64)
        bounds = np.concatenate([[0], cuts, [n]]).astype(np.int64)
        off = bounds[:-1]
        ln = np.diff(bounds)
        el = (np.arange(len(off)) % 2 == 0).astype(np.uint8)
        words = nfo.mask_from_segments(off, ln, el, n, lib=lib)
        want = np.zeros(n, np.uint8)
        for o, l_, e in zip(off, ln, el):
            want[o:o + l_] = e
        assert mask_elems(words, n) == want.tolist(), f"mask layout n={n}"
        # padding bits past n are zero
        if n % 64:
            assert int(words[-1]) >> (n % 64) == 0, "mask padding"
        assert nfo.count_eligible(words, n, lib=lib) == int(want.sum()), "n_E"
    # a segment past the end is an error
    try:
        nfo.mask_from_segments([5], [10], [1], 12, lib=lib)
    except ValueError:
        pass
    else:
        raise AssertionError("segment beyond n accepted")


def pin_pack_bruteforce(lib):
    """Every W-bit sign pattern at some position, plus special values."""
    rng = np.random.default_rng(12)
    for W in range(1, 7):
        pats = np.array(list(itertools.product([0, 1], repeat=W)), dtype=np.uint8).T  # W x 2^W
        npat = pats.shape[1]
        mag = np.abs(rng.standard_normal((W, npat))).astype(np.float32) + np.float32(1e-3)
        g = np.where(pats == 1, mag, -mag).astype(np.float32)
        extra = rng.choice(SPECIALS, size=(W, 90)).astype(np.float32)
        g = np.concatenate([g, extra, gauss(rng, W, 77)], axis=1)
        n = g.shape[1]
        m = (rng.random(n) < 0.8).astype(np.uint8)
        m[:npat] = 1
        words = mask_of(m)
        bits = nfo.pack(g, words, lib=lib)
        want = model_bits(g, m)
        for w in range(W):
            got = mask_elems(bits[w], n)
            assert got == want[w], f"pack W={W} w={w}"
            if n % 64:
                assert int(bits[w, -1]) >> (n % 64) == 0, "pack padding"
        c = nfo.counts(bits, n, lib=lib)
        # every pattern's count is its popcount
        assert c[:npat].tolist() == pats.sum(axis=0).tolist(), f"counts of patterns W={W}"


def pin_counts_invariants(lib):
    rng = np.random.default_rng(13)
    for W in [1, 2, 3, 7, 16, 64, 255]:
        n = 257
        g = gauss(rng, W, n)
        m = (rng.random(n) < 0.7).astype(np.uint8)
        words = mask_of(m)
        bits = nfo.pack(g, words, lib=lib)
        c = nfo.counts(bits, n, lib=lib)
        assert c.max() <= W, "I1 upper bound"
        assert np.all(c[m == 0] == 0), "I1 zero off the mask"
        total = sum(bin(int(x)).count("1") for x in bits.ravel())
        assert int(c.astype(np.int64).sum()) == total, "I2 sum of counts = popcount"
        want = np.array(model_bits(g, m), dtype=np.int64).sum(axis=0)
        assert np.array_equal(c.astype(np.int64), want), f"counts W={W}"
    # a bitmap row stride larger than the row: the counts read the right words
    g = gauss(rng, 3, 130)
    words = mask_of(np.ones(130, np.uint8))
    bits = nfo.pack(g, words, lib=lib)
    wide = np.zeros((3, 9), np.uint64)
    wide[:, :3] = bits
    c1 = nfo.counts(bits, 130, lib=lib)
    c2 = nfo.counts(wide, 130, lib=lib)
    assert np.array_equal(c1, c2), "bits stride"


def pin_fp32_path(lib):
    rng = np.random.default_rng(14)
    for W in [1, 2, 3, 5, 16, 64]:
        g = (rng.standard_normal((W, 301)) * np.logspace(-6, 2, 301)).astype(np.float32)
        g[:, :13] = SPECIALS[:13]
        y = nfo.fp32_path(g, nfo.OP_SUM, lib=lib)
        assert same_f32(y, model_fp32_sum(g)), f"FP32 SUM W={W}"
        ym = nfo.fp32_path(g, nfo.OP_MEAN, lib=lib)
        assert same_f32(ym, model_fp32_sum(g) / np.float32(W)), f"FP32 MEAN W={W} (I9)"
    # W = 2 is one correctly rounded IEEE addition: check against exact arithmetic
    g = (rng.standard_normal((2, 200)) * np.logspace(-30, 30, 200)).astype(np.float32)
    y = nfo.fp32_path(g, nfo.OP_SUM, lib=lib)
    want = np.array([f32_round(frac(g[0, i]) + frac(g[1, i])) for i in range(200)], np.float32)
    assert same_f32(y, want), "W=2 exact sum"
    # the sum is taken in worker order, not another order: (a + b) + c with
    # a = 1, b = 2^-24, c = 2^-24 keeps 1; reassociating gives 1 + 2^-23
    g = np.array([[1.0], [2.0 ** -24], [2.0 ** -24]], dtype=np.float32)
    assert nfo.fp32_path(g, nfo.OP_SUM, lib=lib)[0] == np.float32(1.0), "worker order"
    g = np.array([[2.0 ** -24], [2.0 ** -24], [1.0]], dtype=np.float32)
    assert nfo.fp32_path(g, nfo.OP_SUM, lib=lib)[0] == np.float32(1.0 + 2.0 ** -23), "order 2"
    # MEAN uses a division: fl(7/3) differs from fl(7 * fl(1/3))
    g = np.array([[7.0], [0.0], [0.0]], dtype=np.float32)
    want = f32_round(Fraction(7, 3))
    assert nfo.fp32_path(g, nfo.OP_MEAN, lib=lib)[0] == want, "MEAN by division"


def f64_round(x):
    """Round a positive Fraction to the nearest FP64 value, ties to even.

    Written from the definition, for values inside FP64's normal range: find
    the binade, scale to a 53-bit integer significand, round half to even.
    """
    x = Fraction(x)
    assert x > 0
    e = x.numerator.bit_length() - x.denominator.bit_length()
    if Fraction(2) ** e > x:
        e -= 1
    while Fraction(2) ** (e + 1) <= x:
        e += 1
    quantum = Fraction(2) ** (e - 52)
    q, r = divmod(x, quantum)
    q = int(q)
    if r > quantum / 2 or (r == quantum / 2 and q % 2 == 1):
        q += 1
    return float(q * quantum)  # exact: q * quantum has at most 53 significant bits


def exact_sum64(vals):
    """The exact sum of FP32 values (as Fractions), rounded once to FP64."""
    t = sum((Fraction(float(v)) for v in vals), Fraction(0))
    return 0.0 if t == 0 else f64_round(t)


def pin_health(lib):
    """R8: non-finite counts, and both sums exact and rounded once to FP64."""
    rng = np.random.default_rng(15)
    W, n = 5, 1000
    g = (rng.standard_normal((W, n)) * 1e-3).astype(np.float32)
    g[1, 10] = np.nan
    g[1, 20] = np.inf
    g[3, 999] = -np.inf
    m = (rng.random(n) < 0.6).astype(np.uint8)
    m[10] = m[20] = 1  # a NaN and an infinity, both eligible
    m[999] = 0
    words = mask_of(m)
    st = nfo.health(g, words, lib=lib)
    assert st["nonfinite"].tolist() == (~np.isfinite(g)).sum(axis=1).tolist(), "nonfinite"
    for w in range(W):
        x = g[w].astype(np.float64)
        if np.all(np.isfinite(x)):
            # math.fsum returns the correctly rounded sum of its terms, and
            # each term (|g|, or g*g: 48 significant bits) is exact in FP64
            assert st["sum_sq"][w] == math.fsum((x * x).tolist()), f"ssq w={w}"
            assert st["sum_abs_elig"][w] == math.fsum(np.abs(x[m == 1]).tolist()), f"sabs w={w}"
    # IEEE semantics of non-finite terms: NaN wins, else +Inf; |g| only where eligible
    assert np.isnan(st["sum_sq"][1]) and np.isnan(st["sum_abs_elig"][1]), "NaN in worker 1"
    assert st["sum_sq"][3] == np.inf, "-Inf squared"
    assert st["sum_abs_elig"][3] == math.fsum(np.abs(g[3, m == 1].astype(np.float64)).tolist()), \
        "an infinity off the mask leaves |g| finite"
    # exact rationals on the full FP32 range: the largest finite value,
    # subnormals, and sums that land on or next to a rounding midpoint
    cases = [
        [1.0, 2.0 ** -53],                          # midpoint, even below: 1
        [1.0, 2.0 ** -52, 2.0 ** -53],              # midpoint, even above: 1 + 2^-51
        [1.0, 2.0 ** -53, 2.0 ** -149],             # just past the midpoint: up
        [2.0 ** -53, 1.0, 2.0 ** -149],
        [3.4028234663852886e38] * 7 + [2.0 ** -149] * 3,
        [2.0 ** -149, 2.0 ** -140, 2.0 ** -126, 1.5e-45],
        [1.0, 2.0 ** -27, 2.0 ** -27],              # g*g: 1 + 2 * 2^-54, a midpoint
        [1.0, 2.0 ** -27, 2.0 ** -27, 2.0 ** -27],  # g*g: 1 + 3 * 2^-54, up
        [7.0, -2.0 ** -60, 2.0 ** -49, -3.0e-39, 1e30, -1e-30],
    ]
    for k, vals in enumerate(cases):
        g = np.array([vals], dtype=np.float32)
        m = np.ones(len(vals), np.uint8)
        m[-1] = 0 if len(vals) > 3 else 1
        st = nfo.health(g, mask_of(m), lib=lib)
        want_abs = exact_sum64([abs(float(v)) for v, e in zip(g[0], m) if e])
        want_sq = exact_sum64([float(v) * float(v) for v in g[0]])
        assert st["sum_abs_elig"][0] == want_abs, f"sabs exact case {k}"
        assert st["sum_sq"][0] == want_sq, f"ssq exact case {k}"
    # the exact sum depends on no order: a permutation gives the same bits
    g = (rng.standard_normal((3, 777)) * np.exp(rng.uniform(-40, 40, (3, 777)))).astype(np.float32)
    m = (rng.random(777) < 0.8).astype(np.uint8)
    st = nfo.health(g, mask_of(m), lib=lib)
    perm = rng.permutation(777)
    st2 = nfo.health(np.ascontiguousarray(g[:, perm]), mask_of(m[perm]), lib=lib)
    assert st.tobytes() == st2.tobytes(), "order"
    for w in range(3):
        x = g[w].astype(np.float64)
        assert st["sum_sq"][w] == math.fsum((x * x).tolist()), "ssq wide range"
        assert st["sum_abs_elig"][w] == math.fsum(np.abs(x[m == 1]).tolist()), "sabs wide range"


def pin_scale(lib):
    rng = np.random.default_rng(16)
    # dyadic inputs: the oracle's FP64 steps are exact up to the divisions by
    # n_E and W, so compare with the exact rational rounded once; choose n_E
    # and W as powers of two so every division is exact as well
    for W, n in [(1, 64), (2, 128), (4, 256), (8, 64)]:
        g = rng.integers(-1024, 1025, size=(W, n)).astype(np.float32) / np.float32(4096)
        m = np.zeros(n, np.uint8)
        m[rng.choice(n, size=n // 2, replace=False)] = 1
        st = nfo.health(g, mask_of(m), lib=lib)
        s = nfo.scale(st, int(m.sum()), lib=lib)
        assert s == model_scale_exact(g, m), f"scale exact W={W}"
    # the combination is carried in FP64 and rounded once: worker means
    # 0.5 + 2^-25 and 2^-25 give exactly 0.25 + 2^-25, while rounding each
    # partial to FP32 (ties to even) would give 0.25
    g = np.array([[1.0, 2.0 ** -24], [2.0 ** -24, 0.0]], dtype=np.float32)
    m = np.array([1, 1], np.uint8)
    st = nfo.health(g, mask_of(m), lib=lib)
    s = nfo.scale(st, 2, lib=lib)
    assert s == model_scale_exact(g, m) == np.float32(0.25 + 2.0 ** -25), "scale rounded once"
    # I7: constant |g| = a on E gives scale = a
    for a in [np.float32(0.75), np.float32(1e-3), np.float32(3.0e-7)]:
        W, n = 6, 300
        g = np.where(rng.random((W, n)) < 0.5, a, -a).astype(np.float32)
        m = (rng.random(n) < 0.5).astype(np.uint8)
        nE = int(m.sum())
        st = nfo.health(g, mask_of(m), lib=lib)
        assert nfo.scale(st, nE, lib=lib) == a, f"I7 a={a}"
    # general data: numpy float64 mean over eligible, mean over workers
    W, n = 7, 999
    g = gauss(rng, W, n) * np.linspace(0.5, 2.0, W, dtype=np.float32)[:, None]
    m = (rng.random(n) < 0.9).astype(np.uint8)
    st = nfo.health(g, mask_of(m), lib=lib)
    s = nfo.scale(st, int(m.sum()), lib=lib)
    ref = np.abs(g[:, m == 1].astype(np.float64)).mean(axis=1).mean()
    assert abs(float(s) - ref) <= 1e-7 * ref, "scale vs numpy mean"
    assert nfo.scale(st, 0, lib=lib) == 0.0, "scale with no eligible element"


def pin_decode_table(lib):
    for W in list(range(1, 40)) + [63, 64, 100, 127, 128, 200, 254, 255]:
        q = nfo.decode_table(W, nfo.DECODE_SOFT, lib=lib)
        assert same_f32(q, model_q(W, nfo.DECODE_SOFT)), f"SOFT table W={W}"
        qm = nfo.decode_table(W, nfo.DECODE_MAJORITY, lib=lib)
        assert same_f32(qm, model_q(W, nfo.DECODE_MAJORITY)), f"MAJORITY table W={W}"


def _exact_bucket(g, m, pol):
    """Whole tiny bucket with exact rationals where the oracle rounds once."""
    W, n = g.shape
    bits = np.array(model_bits(g, m), dtype=np.int64)
    c = bits.sum(axis=0)
    y = model_fp32_sum(g)
    if pol.fp32_op == nfo.OP_MEAN:
        y = y / np.float32(W)
    return bits, c, y


def pin_whole_bucket_bruteforce(lib):
    """Tiny buckets: every output of nfo_reduce_bucket against the models."""
    rng = np.random.default_rng(17)
    for trial in range(40):
        W = int(rng.integers(1, 7))
        n = int(rng.integers(1, 300))
        g = rng.integers(-512, 513, size=(W, n)).astype(np.float32) / np.float32(256)
        m = (rng.random(n) < rng.random()).astype(np.uint8)
        mode = nfo.DECODE_MAJORITY if trial % 3 == 0 else nfo.DECODE_SOFT
        op = nfo.OP_MEAN if trial % 4 == 1 else nfo.OP_SUM
        pol = nfo.policy(decode_mode=mode, fp32_op=op, force_lowbit=1)
        r = nfo.reduce_bucket(g, mask_of(m), pol, lib=lib)
        bits, c, y = _exact_bucket(g, m, pol)
        for w in range(W):
            assert mask_elems(r["bits"][w], n) == bits[w].tolist(), "bucket bits"
        assert r["counts"].astype(np.int64).tolist() == c.tolist(), "bucket counts"
        d = r["decision"]
        nE = int(m.sum())
        assert d.n_eligible == nE, "n_E"
        # scale: integers / 256 make every per-worker FP64 sum exact; the
        # division by n_E and the worker sum may round in FP64, so compare the
        # exact value within one FP32 ulp and require equality when n_E and W
        # are powers of two
        exact_scale = model_scale_exact(g, m)
        if nE and (nE & (nE - 1)) == 0 and (W & (W - 1)) == 0:
            assert d.scale == exact_scale, "bucket scale exact"
        else:
            assert abs(float(d.scale) - float(exact_scale)) <= abs(float(exact_scale)) * 2 ** -23, \
                "bucket scale"
        q = model_q(W, mode)
        if nE == 0:
            assert d.route == nfo.ROUTE_P, "no eligible -> P"
        for i in range(n):
            if d.route == nfo.ROUTE_L and m[i]:
                want = f32_round(frac(d.scale) * frac(q[c[i]]))
            else:
                want = y[i]
            assert same_f32([r["out"][i]], [want]), f"bucket out[{i}] trial {trial}"


def pin_appendix_example(lib):
    """The hand-worked W=3, n=4 bucket (tests/golden/worked_example_w3.json)."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "worked_example_w3.json")
    ex = json.load(open(path))
    g = np.array(ex["grads"], dtype=np.float32)
    m = np.array(ex["mask"], dtype=np.uint8)
    r = nfo.reduce_bucket(g, mask_of(m), nfo.policy(), lib=lib)
    W, n = g.shape
    bits, c, y = _exact_bucket(g, m, nfo.policy())
    # exact rational re-derivation of every stored value
    s = model_scale_exact(g, m)
    q = model_q(W, nfo.DECODE_SOFT)
    out = [f32_round(frac(s) * frac(q[c[i]])) if m[i] else y[i] for i in range(n)]
    exp = ex["expected"]
    assert [int(v, 16) for v in exp["bits_word0"]] == \
        [int(sum(int(b) << i for i, b in enumerate(bits[w]))) for w in range(W)], "example bits model"
    assert exp["counts"] == c.tolist(), "example counts model"
    assert int(exp["scale_hex"], 16) == int(np.float32(s).view(np.uint32)), "example scale model"
    assert [int(v, 16) for v in exp["out_hex"]] == \
        [int(np.float32(v).view(np.uint32)) for v in out], "example out model"
    # the oracle reproduces the stored values
    assert [int(v, 16) for v in exp["bits_word0"]] == [int(r["bits"][w, 0]) for w in range(W)], \
        "example bits"
    assert r["counts"].tolist() == exp["counts"], "example counts"
    assert int(np.float32(r["decision"].scale).view(np.uint32)) == int(exp["scale_hex"], 16), \
        "example scale"
    assert r["out"].view(np.uint32).tolist() == [int(v, 16) for v in exp["out_hex"]], "example out"
    assert r["decision"].route == nfo.ROUTE_L and r["decision"].reasons == 0, "example route"
    assert r["decision"].bytes_route == exp["bytes_route"], "example route bytes"
    assert r["decision"].bytes_fp32 == exp["bytes_fp32"], "example fp32 bytes"
    assert r["stats"]["sum_sq"].tolist() == exp["sum_sq"], "example ssq"
    assert r["stats"]["sum_abs_elig"].tolist() == exp["sum_abs"], "example sabs"
    pm = nfo.reduce_bucket(g, mask_of(m), nfo.policy(fp32_op=nfo.OP_MEAN), lib=lib)
    assert int(pm["out"].view(np.uint32)[3]) == int(exp["mean_out3_hex"], 16), "example MEAN"


def pin_w1(lib):
    """I4: W = 1 decodes to sign(g) * scale (+0, -0 and NaN vote negative)."""
    rng = np.random.default_rng(18)
    g = gauss(rng, 1, 500)
    g[0, :4] = [0.0, -0.0, 1e-45, -1e-45]
    m = np.ones(500, np.uint8)
    r = nfo.reduce_bucket(g, mask_of(m), nfo.policy(), lib=lib)
    s = r["decision"].scale
    want = np.where(g[0] > 0, s, -s).astype(np.float32)
    assert same_f32(r["out"], want), "I4 W=1"
    assert np.array_equal(r["counts"], (g[0] > 0).astype(np.uint8)), "I4 counts"


def pin_negation(lib):
    """I5: negating every gradient (no zeros or NaN) mirrors the bucket."""
    rng = np.random.default_rng(19)
    for W in [2, 3, 8, 17]:
        n = 333
        g = gauss(rng, W, n)
        g[g == 0] = np.float32(1e-6)
        m = (rng.random(n) < 0.8).astype(np.uint8)
        words = mask_of(m)
        a = nfo.reduce_bucket(g, words, nfo.policy(), lib=lib)
        b = nfo.reduce_bucket(-g, words, nfo.policy(), lib=lib)
        assert a["decision"].route == nfo.ROUTE_L == b["decision"].route, "I5 route"
        assert np.array_equal(b["counts"][m == 1].astype(int), W - a["counts"][m == 1].astype(int)), \
            "I5 counts"
        # a tie (2c = W) decodes to +0 both ways; every other value flips sign
        tie = (m == 1) & (2 * a["counts"].astype(int) == W)
        assert same_f32(b["out"][~tie], -a["out"][~tie]), f"I5 out W={W}"
        assert same_f32(b["out"][tie], a["out"][tie]) and not a["out"][tie].any(), "I5 ties"
        assert a["stats"].tobytes() == b["stats"].tobytes(), "I5 stats"


def pin_scaling(lib):
    """I6: g * 2^k leaves bits and counts and multiplies every float by 2^k."""
    rng = np.random.default_rng(20)
    W, n = 5, 400
    g = gauss(rng, W, n)
    m = (rng.random(n) < 0.85).astype(np.uint8)
    words = mask_of(m)
    a = nfo.reduce_bucket(g, words, nfo.policy(), lib=lib)
    for k in [-3, 5]:
        f = np.float32(2.0 ** k)
        b = nfo.reduce_bucket(g * f, words, nfo.policy(), lib=lib)
        assert np.array_equal(a["bits"], b["bits"]) and np.array_equal(a["counts"], b["counts"]), \
            "I6 bits"
        assert b["decision"].scale == a["decision"].scale * f, "I6 scale"
        assert same_f32(b["out"], a["out"] * f), "I6 out"
        assert np.array_equal(b["stats"]["sum_abs_elig"], a["stats"]["sum_abs_elig"] * float(f)), \
            "I6 sabs"
        assert np.array_equal(b["stats"]["sum_sq"], a["stats"]["sum_sq"] * float(f) ** 2), "I6 ssq"


def pin_all_fp32_mask(lib):
    """I8: M = 0 everywhere gives route P and the plain sequential sum."""
    rng = np.random.default_rng(21)
    for W in [1, 2, 9]:
        g = gauss(rng, W, 200)
        r = nfo.reduce_bucket(g, mask_of(np.zeros(200, np.uint8)), nfo.policy(), lib=lib)
        assert r["decision"].route == nfo.ROUTE_P, "I8 route"
        assert r["decision"].reasons & nfo.R_NO_ELIGIBLE, "I8 reason"
        assert r["decision"].scale == 0.0, "I8 scale"
        assert same_f32(r["out"], model_fp32_sum(g)), "I8 plain sum"
        assert not r["counts"].any() and not r["bits"].any(), "I8 no payload"


def _stats(W, sabs=1.0, ssq=1.0):
    st = np.zeros(W, dtype=nfo.STATS_DTYPE)
    st["sum_abs_elig"] = sabs
    st["sum_sq"] = ssq
    return st


def pin_route_truth_table(lib):
    """I10: every combination of controller inputs and health conditions."""
    W, n = 5, 1000
    for adm, veto, gok, force, has_e, nonf, zero, spike in itertools.product([0, 1], repeat=8):
        st = _stats(W)
        if nonf:
            st["nonfinite"][2] = 3
            st["sum_sq"][2] = np.inf
        if zero:
            st["sum_abs_elig"][1] = 0.0
        if spike:
            st["sum_sq"][4] = 17.0
        nE = 500 if has_e else 0
        pol = nfo.policy(admitted=adm, veto=veto, guard_ok=gok, force_lowbit=force)
        d = nfo.decide(st, n, nE, pol, lib=lib)
        want = 0
        want |= 0 if adm else nfo.R_NOT_ADMITTED
        want |= 0 if has_e else nfo.R_NO_ELIGIBLE
        want |= nfo.R_VETO if veto else 0
        want |= 0 if gok else nfo.R_GUARD
        want |= nfo.R_NONFINITE if nonf else 0
        want |= nfo.R_ZERO_WORKER if (zero and has_e) else 0
        want |= nfo.R_NORM_SPIKE if spike else 0
        if not adm or not has_e:
            route = nfo.ROUTE_P
        elif force:
            route = nfo.ROUTE_L
            want |= nfo.R_FORCED
        elif veto or not gok or nonf or (zero and has_e) or spike:
            route = nfo.ROUTE_F
        else:
            route = nfo.ROUTE_L
        key = (adm, veto, gok, force, has_e, nonf, zero, spike)
        assert d.route == route, f"I10 route {key}"
        assert d.reasons == want, f"I10 reasons {key}: {d.reasons} != {want}"
        assert d.bytes_fp32 == 4.0 * n, "I12 fp32 bytes"
        if route == nfo.ROUTE_L:
            assert d.bytes_route == nE / 8 + 4 + 4 * (n - nE), "I12 route bytes"
        else:
            assert d.bytes_route == 4.0 * n, "I12 fallback bytes"


def pin_norm_spike_median(lib):
    """R12 on explicit statistics: lower median, finite values only, at least two."""
    def spikes(ssq, kappa=4.0):
        st = _stats(len(ssq))
        st["sum_sq"] = ssq
        d = nfo.decide(st, 100, 50, nfo.policy(kappa=kappa), lib=lib)
        return bool(d.reasons & nfo.R_NORM_SPIKE)
    assert not spikes([1.0, 16.0]), "two workers, ratio exactly 16"
    assert spikes([1.0, 16.5]), "two workers, lower median 1"
    assert not spikes([16.5, 1.0, 2.0, 30.0]), "lower median of 4 is 2 (16*2=32)"
    assert spikes([16.5, 1.0, 2.0, 33.0]), "33 > 32"
    assert not spikes([5.0, 9.0, 3.0]), "median 5"
    assert spikes([5.0, 81.0, 3.0]), "81 > 80"
    assert not spikes([np.inf, 1.0, np.nan, 16.0]), "non-finite ignored"
    assert spikes([1.0, np.inf, 1e9]), "two finite values"
    assert not spikes([1e9]), "one worker never spikes"
    assert not spikes([np.inf, 1e9]), "one finite value never spikes"
    assert spikes([0.0, 0.0, 1e-300]), "zero median"
    assert not spikes([1.0, 9.0], kappa=3.0), "kappa 3: 9 is not > 9"
    assert spikes([1.0, 9.5], kappa=3.0), "kappa 3"


def pin_spike_construction(lib):
    """Worker 2 = c * worker 0 elementwise: L2 ratio c, ssq ratio c^2 (kappa = 4)."""
    rng = np.random.default_rng(22)
    base = gauss(rng, 1, 256)[0]
    m = mask_of(np.ones(256, np.uint8))
    for c, expect in [(3.9, False), (4.1, True), (4.0, False)]:
        g = np.stack([base, base, base * np.float32(c), base]).astype(np.float32)
        r = nfo.reduce_bucket(g, m, nfo.policy(), lib=lib)
        got = bool(r["decision"].reasons & nfo.R_NORM_SPIKE)
        assert got == expect, f"spike x{c}"
        assert r["decision"].route == (nfo.ROUTE_F if expect else nfo.ROUTE_L), f"route x{c}"


def pin_route_correctness(lib):
    """I11: routed positions always carry the FP32 path; F and P carry it everywhere."""
    rng = np.random.default_rng(23)
    W, n = 6, 500
    g = gauss(rng, W, n)
    m = (rng.random(n) < 0.7).astype(np.uint8)
    words = mask_of(m)
    y = model_fp32_sum(g)
    for pol, route in [(nfo.policy(), nfo.ROUTE_L), (nfo.policy(veto=1), nfo.ROUTE_F),
                       (nfo.policy(guard_ok=0), nfo.ROUTE_F), (nfo.policy(admitted=0), nfo.ROUTE_P)]:
        r = nfo.reduce_bucket(g, words, pol, lib=lib)
        assert r["decision"].route == route, "I11 route"
        assert same_f32(r["out"][m == 0], y[m == 0]), "I11 routed positions"
        if route != nfo.ROUTE_L:
            assert same_f32(r["out"], y), "I11 fallback everywhere"
        else:
            s = r["decision"].scale
            assert np.all(np.abs(r["out"][m == 1]) <= s), "I11 decoded magnitude"


def pin_health_routes(lib):
    """Non-finite values, a zero worker and a x10 worker each force F (R10-R12)."""
    rng = np.random.default_rng(24)
    W, n = 8, 640
    m = (rng.random(n) < 0.9).astype(np.uint8)
    words = mask_of(m)
    cases = []
    g = gauss(rng, W, n); g[3, 7] = np.nan; cases.append((g, nfo.R_NONFINITE))
    g = gauss(rng, W, n); g[5, 100] = -np.inf; cases.append((g, nfo.R_NONFINITE))
    g = gauss(rng, W, n); g[6, :] = 0.0; cases.append((g, nfo.R_ZERO_WORKER))
    g = gauss(rng, W, n); g[6, m == 1] = -0.0; cases.append((g, nfo.R_ZERO_WORKER))
    g = gauss(rng, W, n); g[1] *= 10; cases.append((g, nfo.R_NORM_SPIKE))
    for g, bit in cases:
        r = nfo.reduce_bucket(g, words, nfo.policy(), lib=lib)
        assert r["decision"].route == nfo.ROUTE_F, f"health route {bit}"
        assert r["decision"].reasons == bit, f"health reasons {r['decision'].reasons} != {bit}"
        assert same_f32(r["out"], model_fp32_sum(g)), "health fallback output"
        r = nfo.reduce_bucket(g, words, nfo.policy(force_lowbit=1), lib=lib)
        assert r["decision"].route == nfo.ROUTE_L, "forced L"
        assert r["decision"].reasons == bit | nfo.R_FORCED, "forced reasons"


# ------------------------------------------------------------- G-Ternary


def model_theta(S, nE, tau):
    """R18 from IEEE arithmetic: double division, then FP32 rounding, then an
    FP32 product (numpy float32 scalars)."""
    if nE <= 0:
        return np.float32(0.0)
    return np.float32(np.float32(tau) * np.float32(float(S) / nE))


def model_planes(g, m, theta):
    """R19 written from its definition, element by element."""
    W, n = g.shape
    pos = np.zeros((W, n), dtype=np.uint8)
    neg = np.zeros((W, n), dtype=np.uint8)
    with np.errstate(invalid="ignore"):
        for w in range(W):
            for i in range(n):
                x = np.float32(g[w, i])
                if not m[i] or np.abs(x) < theta[w]:
                    continue
                pos[w, i] = 1 if x > 0 else 0
                neg[w, i] = 1 if x < 0 else 0
    return pos, neg


def unpack_rows(words, n):
    words = np.atleast_2d(np.asarray(words, dtype=np.uint64))
    return np.array([[int((int(r[i // 64]) >> (i % 64)) & 1) for i in range(n)] for r in words], dtype=np.uint8)


def stats_rec(S):
    st = np.zeros(1, dtype=nfo.STATS_DTYPE)
    st["sum_abs_elig"] = S
    return st


def pin_ternary_threshold(lib):
    """R18 against IEEE arithmetic and exact rationals, including a case where
    rounding once (instead of twice) gives a different threshold."""
    rng = np.random.default_rng(31)
    for _ in range(200):
        S = float(rng.random() * 10.0 ** int(rng.integers(-8, 4)))
        nE = int(rng.integers(1, 10 ** 6))
        tau = float(np.float32(rng.random() * 3))
        got = nfo.ternary_threshold(stats_rec(S), nE, tau, lib=lib)
        assert same_f32(got, model_theta(S, nE, tau)), f"theta S={S} nE={nE} tau={tau}"
    assert nfo.ternary_threshold(stats_rec(5.0), 0, 0.5, lib=lib) == 0.0, "theta without eligible elements"
    # dyadic: (3/4) * 0.5 exactly
    assert nfo.ternary_threshold(stats_rec(3.0), 4, 0.5, lib=lib) == np.float32(0.375), "theta dyadic"
    # S / n_E = 1 + 2^-24 + 2^-30: fl32 rounds it up to 1 + 2^-23; times 3 is
    # 3 + 1.5 ulp, a tie that goes to 3 + 2^-21.  Rounding the exact product
    # once would give 3 + 2^-22.
    S = 1.0 + 2.0 ** -24 + 2.0 ** -30
    want = f32_round(Fraction(3) * Fraction(float(np.float32(S))))
    assert want == np.float32(3 + 2.0 ** -21)
    got = nfo.ternary_threshold(stats_rec(S), 1, 3.0, lib=lib)
    assert same_f32(got, want), f"theta double rounding: {got!r} != {want!r}"


def pin_pack_ternary_bruteforce(lib):
    """Every value class around the threshold, with signed zeros, NaN and
    infinities, masks with holes, a different threshold per worker."""
    for W in (1, 2, 3):
        theta = np.array([0.25, 1.0, 2.5][:W], dtype=np.float32)
        vals = []
        for t in theta:
            for v in (t, np.nextafter(t, np.float32(0)), np.nextafter(t, np.float32(np.inf)), 2 * t, t / 2):
                vals += [v, -v]
        vals += [0.0, -0.0, np.nan, np.inf, -np.inf, 1e-45, -1e-45, 3.4e38, -3.4e38]
        vals = np.array(vals, dtype=np.float32)
        n = 3 * len(vals)
        rng = np.random.default_rng(W)
        g = np.stack([np.concatenate([np.roll(vals, w + k) for k in range(3)]) for w in range(W)]).astype(np.float32)
        m = (rng.random(n) < 0.8).astype(np.uint8)
        pos, neg = nfo.pack_ternary(g, mask_of(m), theta, lib=lib)
        mp, mn = model_planes(g, m, theta)
        assert np.array_equal(unpack_rows(pos, n), mp), f"pos plane W={W}"
        assert np.array_equal(unpack_rows(neg, n), mn), f"neg plane W={W}"
        assert not np.any(unpack_rows(pos, n) & unpack_rows(neg, n)), "an element in both planes"


def pin_ternary_decode_table(lib):
    for W in (1, 2, 3, 5, 16, 64, 127, 255):
        q = nfo.ternary_decode_table(W, nfo.DECODE_SOFT, lib=lib)
        want = np.array([f32_round(Fraction(d, W)) for d in range(-W, W + 1)], dtype=np.float32)
        assert same_f32(q, want), f"ternary SOFT table W={W}"
        q = nfo.ternary_decode_table(W, nfo.DECODE_MAJORITY, lib=lib)
        want = np.array([np.sign(d) for d in range(-W, W + 1)], dtype=np.float32)
        assert same_f32(q, want), f"ternary MAJORITY table W={W}"


def pin_ternary_tau0_is_binary(lib):
    """tau = 0 and no zero or NaN: the vote difference is 2c - W, so every
    output equals the binary route's bit for bit."""
    rng = np.random.default_rng(33)
    for W in (1, 2, 5, 16):
        for mode in (nfo.DECODE_SOFT, nfo.DECODE_MAJORITY):
            n = 333
            g = gauss(rng, W, n)
            g[g == 0] = 1e-3
            m = (rng.random(n) < 0.85).astype(np.uint8)
            words = mask_of(m)
            rb = nfo.reduce_bucket(g, words, nfo.policy(decode_mode=mode), lib=lib)
            rt = nfo.reduce_bucket_ternary(g, words, nfo.policy(decode_mode=mode, format=1, tau=0.0), lib=lib)
            assert same_f32(rt["out"], rb["out"]), f"tau=0 output W={W} mode={mode}"
            assert np.array_equal(rt["pos"], rb["bits"]), "tau=0 pos plane = sign bits"
            assert np.array_equal(rt["cpos"], rb["counts"]), "tau=0 c+"
            assert np.array_equal(rt["cneg"], np.where(m == 1, W - rb["counts"].astype(int), 0)), "tau=0 c-"


def pin_ternary_gate_all(lib):
    """A threshold above every value gates everything: no votes, output 0 at
    eligible positions, FP32 at routed ones."""
    rng = np.random.default_rng(34)
    W, n = 6, 200
    g = gauss(rng, W, n)
    m = (rng.random(n) < 0.7).astype(np.uint8)
    r = nfo.reduce_bucket_ternary(g, mask_of(m), nfo.policy(format=1, tau=1e30), lib=lib)
    assert not r["pos"].any() and not r["neg"].any(), "gate all: planes"
    assert not r["cpos"].any() and not r["cneg"].any(), "gate all: counts"
    e = m == 1
    assert np.all(r["out"][e] == 0.0), "gate all: decoded 0"
    assert same_f32(r["out"][~e], model_fp32_sum(g)[~e]), "gate all: routed positions"


def pin_ternary_whole_bucket(lib):
    """Dyadic tiny buckets (every FP64 step of the oracle exact): all outputs
    against the models, plus the two-plane MGTR bytes of R21."""
    rng = np.random.default_rng(35)
    for trial in range(24):
        W = int(rng.integers(1, 6))
        n = int(rng.integers(1, 140))
        g = (rng.integers(-40, 41, (W, n)) / 64.0).astype(np.float32)
        m = (rng.random(n) < 0.75).astype(np.uint8)
        tau = float([0.0, 0.5, 1.0, 1.5][trial % 4])
        mode = nfo.DECODE_SOFT if trial % 3 else nfo.DECODE_MAJORITY
        r = nfo.reduce_bucket_ternary(g, mask_of(m), nfo.policy(format=1, tau=tau, decode_mode=mode,
                                                                  force_lowbit=1), lib=lib)
        nE = int(m.sum())
        theta = np.array([model_theta(sum(abs(frac(g[w, i])) for i in range(n) if m[i]), nE, tau)
                          for w in range(W)], dtype=np.float32)
        mp, mn = model_planes(g, m, theta)
        assert np.array_equal(unpack_rows(r["pos"], n), mp) and np.array_equal(unpack_rows(r["neg"], n), mn), \
            f"planes trial {trial}"
        cp, cn = mp.sum(axis=0), mn.sum(axis=0)
        assert np.array_equal(r["cpos"], cp) and np.array_equal(r["cneg"], cn), f"counts trial {trial}"
        scale = model_scale_exact(g, m)
        assert same_f32(r["decision"].scale, scale), f"scale trial {trial}"
        y = model_fp32_sum(g)
        for i in range(n):
            if m[i]:
                d = int(cp[i]) - int(cn[i])
                q = np.float32(np.sign(d)) if mode == nfo.DECODE_MAJORITY else f32_round(Fraction(d, W))
                want = f32_round(frac(scale) * frac(q))
            else:
                want = y[i]
            assert same_f32(r["out"][i], want), f"output trial {trial} i={i}"
        assert r["decision"].bytes_route == 2 * nE / 8 + 4 + 4 * (n - nE), f"MGTR bytes trial {trial}"


def pin_ternary_negation(lib):
    """Negating every gradient swaps the planes and negates the decoded values."""
    rng = np.random.default_rng(36)
    W, n = 7, 257
    g = gauss(rng, W, n)
    m = (rng.random(n) < 0.8).astype(np.uint8)
    words = mask_of(m)
    pol = nfo.policy(format=1, tau=0.5)
    a = nfo.reduce_bucket_ternary(g, words, pol, lib=lib)
    b = nfo.reduce_bucket_ternary(-g, words, pol, lib=lib)
    assert np.array_equal(a["pos"], b["neg"]) and np.array_equal(a["neg"], b["pos"]), "negation planes"
    e = m == 1
    assert np.array_equal(a["out"][e], -b["out"][e]), "negation decoded values"


# ------------------------------------- compacted payload, per-slice scales

def np_compact(g, mask_bool_row):
    """Reference compacted rows from numpy: the (g > 0) bits at eligible positions, repacked LSB-first."""
    W = g.shape[0]
    rows = []
    for w in range(W):
        b = (g[w] > 0) & mask_bool_row
        sel = b[mask_bool_row].astype(np.uint8)
        nE = len(sel)
        padded = np.zeros(((nE + 63) // 64) * 64, dtype=np.uint8)
        padded[:nE] = sel
        rows.append(np.packbits(padded, bitorder="little").view(np.uint64))
    return np.array(rows).reshape(W, -1)


def pin_pack_compact(lib):
    # hand example: mask bits 1, 2, 4, 5, 7; signs there - + - + -  -> ranks 1 and 3 set
    g = np.array([[1.0, -1.0, 2.0, 3.0, -4.0, 5.0, 6.0, -7.0]], dtype=np.float32)
    m = np.array([0b10110110], dtype=np.uint64)
    assert nfo.pack_compact(g, m, lib=lib)[0, 0] == 0b01010, "hand example"
    rng = np.random.default_rng(21)
    for W, n, dens in [(1, 1, 1.0), (3, 63, 0.5), (5, 64, 0.9), (2, 65, 0.3), (7, 1000, 0.7), (4, 4097, 0.95),
                       (3, 3000, 0.02)]:
        g = rng.normal(size=(W, n)).astype(np.float32)
        g[rng.random((W, n)) < 0.05] = 0.0
        mb = rng.random(n) < dens
        words = np.packbits(np.concatenate([mb, np.zeros((-n) % 64, bool)]).astype(np.uint8),
                            bitorder="little").view(np.uint64)
        got = nfo.pack_compact(g, words, lib=lib)
        assert np.array_equal(got, np_compact(g, mb)), f"compact W={W} n={n}"
        if dens == 1.0 or mb.all():
            assert np.array_equal(got, nfo.pack(g, words, lib=lib)), "all eligible: compact = positional"
    assert nfo.pack_compact(np.ones((2, 10), np.float32), np.zeros(1, np.uint64), lib=lib).shape == (2, 0)


def pin_slice_scales(lib):
    rng = np.random.default_rng(22)
    # one slice over the whole eligible region: the bucket scale of R5
    W, n = 5, 3000
    g = rng.normal(0, 1e-3, (W, n)).astype(np.float32)
    off, ln = np.array([700]), np.array([1800])
    mb = np.zeros(n, bool)
    mb[700:2500] = True
    words = np.packbits(np.concatenate([mb, np.zeros((-n) % 64, bool)]).astype(np.uint8),
                        bitorder="little").view(np.uint64)
    st = nfo.health(g, words, lib=lib)
    _, sc = nfo.slice_scales(g, off, ln, lib=lib)
    assert sc[0] == nfo.scale(st, 1800, lib=lib), "one slice = bucket scale"
    # constant |g| = a on a slice: scale a exactly
    g2 = np.where(rng.random((W, n)) < 0.5, 0.375, -0.375).astype(np.float32)
    _, sc = nfo.slice_scales(g2, [0, 100, 2999], [50, 900, 1], lib=lib)
    assert np.all(sc == np.float32(0.375)), "constant magnitude"
    # dyadic values: FP64 sums exact; the scale is the exact rational rounded once
    g3 = (rng.integers(-64, 65, (3, 200)) / 64.0).astype(np.float32)
    offs, lens = np.array([0, 10, 150]), np.array([7, 120, 50])
    sums, sc = nfo.slice_scales(g3, offs, lens, lib=lib)
    for s_ in range(3):
        exact = [sum(Fraction(abs(float(x))) for x in g3[w, offs[s_]:offs[s_] + lens[s_]]) for w in range(3)]
        assert all(sums[s_, w] == float(exact[w]) for w in range(3)), "exact slice sums"
        want = f32_round(sum(e / lens[s_] for e in exact) / 3)
        got = sc[s_]
        # the oracle divides and adds in FP64 (R31): within one FP32 rounding of the exact value
        assert got == want or abs(float(got) - float(want)) <= np.spacing(np.float32(want)), "slice scale"


def pin_sliced_output(lib):
    rng = np.random.default_rng(23)
    W, n = 6, 5000
    g = rng.normal(0, 1e-3, (W, n)).astype(np.float32)
    offs, lens = np.array([100, 900, 4000]), np.array([800, 2500, 999])  # slices 0 and 1 adjacent
    mb = np.zeros(n, bool)
    for o, l in zip(offs, lens):
        mb[o:o + l] = True
    words = np.packbits(np.concatenate([mb, np.zeros((-n) % 64, bool)]).astype(np.uint8),
                        bitorder="little").view(np.uint64)
    bits = nfo.pack(g, words, lib=lib)
    c = nfo.counts(bits, n, lib=lib)
    y = nfo.fp32_path(g, lib=lib)
    q = nfo.decode_table(W, lib=lib)
    scales = np.array([1.5e-4, 2.5e-3, 7.0e-1], dtype=np.float32)
    out = nfo.sliced_output(words, c, y, q, offs, lens, scales, lib=lib)
    for o, l, sc in zip(offs, lens, scales):
        assert np.array_equal(out[o:o + l], (sc * q[c[o:o + l]]).astype(np.float32)), "slice decode"
    assert np.array_equal(out[~mb], y[~mb]), "routed positions carry the FP32 path"
    # one slice with the bucket scale reproduces the G-Binary bucket output
    r = nfo.reduce_bucket(g[:, 1000:3500], np.packbits(np.ones(2500 + (-2500) % 64, np.uint8)[:2560],
                                                      bitorder="little").view(np.uint64), lib=lib)
    gs = g[:, 1000:3500]
    m1 = np.packbits(np.concatenate([np.ones(2500, bool), np.zeros(60, bool)]).astype(np.uint8),
                     bitorder="little").view(np.uint64)
    _, sc1 = nfo.slice_scales(gs, [0], [2500], lib=lib)
    o1 = nfo.sliced_output(m1, r["counts"], nfo.fp32_path(gs, lib=lib), q, [0], [2500], sc1, lib=lib)
    assert sc1[0] == np.float32(r["decision"].scale) and np.array_equal(o1, r["out"]), "one slice = G-Binary"
    # a route other than L gives the FP32 path everywhere
    assert np.array_equal(nfo.sliced_output(words, c, y, q, offs, lens, scales, route=nfo.ROUTE_F, lib=lib), y)


ALL_PINS = [pin_mask_from_segments, pin_pack_bruteforce, pin_counts_invariants, pin_fp32_path,
            pin_health, pin_scale, pin_decode_table, pin_whole_bucket_bruteforce,
            pin_appendix_example, pin_w1, pin_negation, pin_scaling, pin_all_fp32_mask,
            pin_route_truth_table, pin_norm_spike_median, pin_spike_construction,
            pin_route_correctness, pin_health_routes,
            pin_ternary_threshold, pin_pack_ternary_bruteforce, pin_ternary_decode_table,
            pin_ternary_tau0_is_binary, pin_ternary_gate_all, pin_ternary_whole_bucket,
            pin_ternary_negation, pin_pack_compact, pin_slice_scales, pin_sliced_output]


def run_all(lib):
    """Run every pin; returns the list of (pin name, message) that failed."""
    failures = []
    for pin in ALL_PINS:
        try:
            pin(lib)
        except AssertionError as e:
            failures.append((pin.__name__, str(e)))
        except Exception as e:  # a broken variant may also crash a model
            failures.append((pin.__name__, f"{type(e).__name__}: {e}"))
    return failures
