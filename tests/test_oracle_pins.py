"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Every check compares the oracle with something other than itself: a printed
worked example, a closed form, a textbook routine (numpy / scipy / Python
fractions), a hand-derived fixture, or exhaustive brute force.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def h(v):
    """fp16 bit pattern of an exactly representable value (numpy's cast)."""
    return int(np.array(v, dtype=np.float16).view(np.uint16))


# --------------------------------------------------------------------------
# binary16 conversions (the coefficient precision of the format)
# --------------------------------------------------------------------------

def test_fp16_to_double_matches_numpy_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.fp16_to_double(int(b)) for b in bits])
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite], ref[finite])
    assert np.array_equal(np.isinf(got), np.isinf(ref))
    assert np.array_equal(np.isnan(got), np.isnan(ref))


def test_fp16_rne_matches_numpy():
    rng = np.random.default_rng(7)
    vals = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.uniform(-9, 5, 20000),
        rng.uniform(-1e-7, 1e-7, 2000),           # subnormal range
        rng.uniform(65000, 66000, 2000),          # overflow boundary
        [0.0, -0.0, 65504.0, 65519.99, 65520.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26],
    ])
    # exact ties between consecutive halves must round to even
    halves = np.arange(0x0001, 0x7BFF, 97, dtype=np.uint16).view(np.float16).astype(np.float64)
    nxt = (np.arange(0x0001, 0x7BFF, 97, dtype=np.uint16) + 1).view(np.float16).astype(np.float64)
    vals = np.concatenate([vals, (halves + nxt) / 2, -(halves + nxt) / 2])
    with np.errstate(over="ignore"):
        ref = vals.astype(np.float16).view(np.uint16)
    got = np.array([oracle.fp16_from_double(v) for v in vals], dtype=np.uint16)
    assert np.array_equal(got, ref)


# --------------------------------------------------------------------------
# Search space, Eqs. 5-11
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n", [8, 128, 37])
def test_q95_matches_numpy_linear_quantile(n):
    rng = np.random.default_rng(n)
    for _ in range(50):
        D = rng.standard_normal(n)
        assert oracle.quantile_linear(D, 0.95) == pytest.approx(
            np.quantile(D, 0.95, method="linear"), rel=1e-14, abs=1e-15)


def test_candidate_sets_match_hand_fixture():
    fx = json.load(open(os.path.join(GOLDEN, "search_grid_fixture.json")))
    D = np.array(fx["D"])
    assert oracle.quantile_linear(D, 0.95) == pytest.approx(fx["q95"], abs=1e-15)
    for K in (2, 4):
        R, S, B = oracle.candidate_sets(D, K)
        np.testing.assert_allclose(S, fx["S"], rtol=0, atol=1e-15)
        np.testing.assert_allclose(B, fx["B"][str(K)], rtol=0, atol=1e-15)
        np.testing.assert_allclose(R, fx["R"], rtol=0, atol=1e-15)
    assert oracle.DEFAULT.size == 1024


# --------------------------------------------------------------------------
# AllSubsetSums: the Sec. 4.1 worked example, Fig. 4 caption, Eq. 12
# --------------------------------------------------------------------------

def test_subset_sums_worked_example():
    # [a, b, c] -> [0, a, b, c, a+b, a+c, b+c, a+b+c]
    a, b, c = 0.5, 0.25, -3.0
    sums = oracle.subset_sums([h(a), h(b), h(c)])
    expect = [0, a, b, c, a + b, a + c, b + c, a + b + c]
    assert sorted(sums) == sorted(expect)
    # index p = sum_i bit_i 2^i: bit 0 <-> a, bit 1 <-> b, bit 2 <-> c
    assert list(sums) == [0, a, b, a + b, c, a + c, b + c, a + b + c]


def _fig4_points(r):
    coeffs, ok = oracle.entry_coeffs(r, 1.0, 0.0, 4, normalise=False)
    assert ok
    return oracle.subset_sums(coeffs)


def test_fig4_kurtosis_binomial_at_r_minus_one():
    pts = _fig4_points(-1.0)
    # coefficients 1, -1, 1, -1: binomial multiset {-2, -1 x4, 0 x6, 1 x4, 2}
    vals, counts = np.unique(pts, return_counts=True)
    assert list(vals) == [-2, -1, 0, 1, 2] and list(counts) == [1, 4, 6, 4, 1]
    assert stats.kurtosis(pts, fisher=True, bias=True) == pytest.approx(-0.5, abs=1e-12)


def test_fig4_kurtosis_uniform_at_r_minus_half():
    pts = np.sort(_fig4_points(-0.5))
    np.testing.assert_array_equal(pts, -0.625 + 0.125 * np.arange(16))
    n = 16
    expect = -6 * (n * n + 1) / (5 * (n * n - 1))  # discrete uniform, -> -1.2
    assert stats.kurtosis(pts, fisher=True, bias=True) == pytest.approx(expect, abs=1e-12)
    assert expect == pytest.approx(-1.2094, abs=1e-4)


def test_fig4_kurtosis_tunable_between():
    k_mid = stats.kurtosis(_fig4_points(-0.75), fisher=True, bias=True)
    assert -1.2094 < k_mid < -0.5


def test_eq12_coefficients_give_twos_complement():
    s = 2.0 ** -5
    coeffs = [h(-8 * s), h(s), h(2 * s), h(4 * s)]
    sums = np.sort(oracle.subset_sums(coeffs))
    np.testing.assert_array_equal(sums, s * np.arange(-8, 8))


def test_span_normalised_coefficients_span_s():
    for r in (-0.9375, -0.75, -0.5, -2.0, -1.5, -1.125):
        for s in (0.1, 3.3, 17.0):
            c, ok = oracle.entry_coeffs(r, s, 0.0, 4, normalise=True)
            assert ok
            sums = oracle.subset_sums(c)
            assert sums.max() - sums.min() == pytest.approx(s, rel=2e-3)
            # the geometric ratio survives fp16 rounding
            cf = c.view(np.float16).astype(np.float64)
            assert cf[1] / cf[0] == pytest.approx(r, rel=2e-3)


def test_literal_coefficients_are_geometric_plus_bias():
    c, ok = oracle.entry_coeffs(-0.5, 2.0, 0.25, 4, normalise=False)
    assert ok
    np.testing.assert_array_equal(c.view(np.float16).astype(np.float64),
                                  [2.25, -0.75, 0.75, 0.0])


# --------------------------------------------------------------------------
# Nearest and Algorithm 1 by brute force
# --------------------------------------------------------------------------

def test_nearest_matches_argmin_first_minimum():
    rng = np.random.default_rng(3)
    for _ in range(300):
        K = rng.integers(1, 5)
        coeffs = rng.standard_normal(K).astype(np.float16).view(np.uint16)
        sums = oracle.subset_sums(coeffs)
        for x in rng.standard_normal(10) * 2:
            d = np.abs(x - sums)
            assert oracle.nearest(sums, x) == int(np.argmin(d))  # argmin: first minimum
    # duplicate sums (r = -1): ties go to the lowest pattern index
    sums = oracle.subset_sums([h(1.0), h(-1.0), h(1.0), h(-1.0)])
    assert oracle.nearest(sums, 0.0) == 0
    assert oracle.nearest(sums, 1.0) == 1
    assert oracle.nearest(sums, 0.5) == 0  # |0.5-0| == |0.5-1|: first (p=0) wins


def _entries(D, K, params):
    R, S, B = oracle.candidate_sets(D, K, params)
    out = []
    for r in R:
        for s in S:
            for b in B:
                if not s > 0:
                    continue
                c, ok = oracle.entry_coeffs(r, s, b, K, params.normalise)
                if ok:
                    out.append(c)
    return out


@pytest.mark.parametrize("K", [1, 2, 3])
def test_encoder_mse_equals_exhaustive_minimum_group8(K):
    rng = np.random.default_rng(100 + K)
    for trial in range(6):
        D = rng.standard_normal(8) * 0.02 + (0.01 if trial % 2 else 0.0)
        coeffs, codes, mse, entry = oracle.encode_group(D, K)
        best = np.inf
        for c in _entries(D, K, oracle.DEFAULT):
            sums = oracle.subset_sums(c)
            # every element independently tries all 2^K patterns
            err = (D[:, None] - sums[None, :]) ** 2
            best = min(best, err.min(axis=1).sum() / D.size)
        assert mse == pytest.approx(best, rel=1e-12, abs=0)
        # reported MSE is the MSE of the emitted coefficients and codes
        sums = oracle.subset_sums(coeffs)
        assert mse == pytest.approx(np.mean((D - sums[codes]) ** 2), rel=1e-12)


@pytest.mark.parametrize("K", [1, 2])
def test_encoder_joint_assignment_brute_force_group8(K):
    """Enumerate all (2^K)^8 joint bit assignments per entry: the separable
    per-element choice of Algorithm 1 must reach the same minimum."""
    small = oracle.SearchParams(n_ratio1=2, n_ratio2=2, n_scale=4, n_bias=2)
    rng = np.random.default_rng(200 + K)
    n = 8
    joint = np.array(list(itertools.product(range(1 << K), repeat=n)), dtype=np.int64)
    for _ in range(3):
        D = rng.standard_normal(n)
        _, _, mse, _ = oracle.encode_group(D, K, small)
        best = np.inf
        for c in _entries(D, K, small):
            sums = oracle.subset_sums(c)
            e = ((D[None, :] - sums[joint]) ** 2).sum(axis=1) / n
            best = min(best, e.min())
        assert mse == pytest.approx(best, rel=1e-12)


def test_encoder_k4_group128_per_element_brute_force():
    W = synth.weights(2, 256, 0.02, seed=55)
    for D in W.reshape(-1, 128).astype(np.float64):
        _, _, mse, _ = oracle.encode_group(D, 4)
        best = np.inf
        for c in _entries(D, 4, oracle.DEFAULT):
            sums = oracle.subset_sums(c)
            best = min(best, ((D[:, None] - sums[None, :]) ** 2).min(axis=1).mean())
        assert mse == pytest.approx(best, rel=1e-12)


def test_encoder_first_strict_minimum_wins():
    # constant-span data where several entries tie exactly: the first is kept
    D = np.zeros(8)
    D[::2] = 1.0
    _, _, mse0, e0 = oracle.encode_group(D, 1)
    # entries visited before e0 must all be strictly worse or inadmissible
    ents = []
    R, S, B = oracle.candidate_sets(D, 1)
    idx = 0
    for r in R:
        for s in S:
            for b in B:
                c, ok = oracle.entry_coeffs(r, s, b, 1, True)
                if s > 0 and ok:
                    ents.append((idx, oracle.entry_mse(D, c)))
                idx += 1
    best = min(m for _, m in ents)
    first = min(i for i, m in ents if m == best)
    assert e0 == first and mse0 == best


def test_degenerate_groups():
    # all-zero group: every s is 0 -> no admissible entry -> (fp16(mean), 0, ...)
    c, codes, mse, e = oracle.encode_group(np.zeros(128), 4)
    assert e == -1 and list(c) == [0, 0, 0, 0] and mse == 0.0
    # constant negative group: s_max = 0 and s_min = 2 q95 < 0, so every
    # s = s_min + (j+1) s_gran lies in (s_min, 0]: same fallback, every
    # element decodes to fp16(mean)
    c, codes, mse, e = oracle.encode_group(np.full(128, -0.3), 3)
    assert e == -1 and c[0] == h(-0.3) and list(c[1:]) == [0, 0]
    sums = oracle.subset_sums(c)
    assert np.all(sums[codes] == np.float16(-0.3).astype(np.float64))
    # constant positive group: the S grid runs downwards from 2 q95 to 0,
    # so entries remain admissible and the search still runs
    c, codes, mse, e = oracle.encode_group(np.full(128, 0.3), 3)
    assert e >= 0 and mse < 1e-4
    # all-negative group: q95 < 0 -> some s <= 0 are skipped, rest still searched
    D = -np.abs(synth.weights(1, 128, 0.02, seed=9)[0]).astype(np.float64) - 0.05
    c, codes, mse, e = oracle.encode_group(D, 4)
    assert e >= 0 and np.isfinite(mse)


# --------------------------------------------------------------------------
# Whole-matrix invariants, decompression, the fp64 GEMV
# --------------------------------------------------------------------------

@pytest.fixture(scope="module")
def encoded_small():
    W = synth.weights(24, 512, 0.02, seed=11, outlier_frac=0.001)
    planes, coeffs, mse = oracle.encode_matrix(W, 4, want_mse=True)
    return W, planes, coeffs, mse


def test_decoded_weights_are_subset_sums_of_their_group(encoded_small):
    W, planes, coeffs, _ = encoded_small
    What = oracle.decompress(planes, coeffs)
    O, G, K, _ = planes.shape
    for o in range(O):
        for g in range(G):
            sums = oracle.subset_sums(coeffs[o, g])
            w = What[o, g * 128:(g + 1) * 128]
            assert np.all(np.isin(w, sums))
            # and each element took the sum nearest to its original weight
            D = W[o, g * 128:(g + 1) * 128].astype(np.float64)
            nearest = np.array([sums[oracle.nearest(sums, x)] for x in D])
            np.testing.assert_array_equal(w, nearest)


def test_plane_bit_order_and_plane_coefficient_pairing():
    # element j of group g <-> word j // 32, bit j % 32 (LSB first); plane i <-> c_i
    planes = np.zeros((1, 1, 3, 4), dtype=np.uint32)
    planes[0, 0, 0, 0] = 1 << 5          # element 5 in plane 0
    planes[0, 0, 1, 2] = 1 << 31         # element 95 in plane 1
    planes[0, 0, 2, 3] = (1 << 0) | (1 << 31)  # elements 96 and 127 in plane 2
    planes[0, 0, 0, 3] = 1 << 31         # element 127 also in plane 0
    coeffs = np.array([[[h(1.0), h(2.0), h(4.0)]]], dtype=np.uint16)
    w = oracle.decompress(planes, coeffs)[0]
    expect = np.zeros(128)
    expect[5], expect[95], expect[96], expect[127] = 1.0, 2.0, 4.0, 5.0
    np.testing.assert_array_equal(w, expect)


def test_decompress_matches_fractions(encoded_small):
    _, planes, coeffs, _ = encoded_small
    What = oracle.decompress(planes, coeffs)
    rng = np.random.default_rng(1)
    O, G, K, _ = planes.shape
    for _ in range(200):
        o, j = rng.integers(O), rng.integers(G * 128)
        g, jj = divmod(int(j), 128)
        total = Fraction(0)
        for i in range(K):
            if (int(planes[o, g, i, jj // 32]) >> (jj % 32)) & 1:
                hb = int(coeffs[o, g, i])
                sign = -1 if hb >> 15 else 1
                e, m = (hb >> 10) & 31, hb & 1023
                v = Fraction(m, 2 ** 24) if e == 0 else Fraction(1024 + m, 2 ** 10) * Fraction(2) ** (e - 15)
                total += sign * v
        assert Fraction(What[o, j]) == total


def test_gemv_matches_numpy_float64(encoded_small):
    _, planes, coeffs, _ = encoded_small
    What = oracle.decompress(planes, coeffs)
    x = synth.activations(What.shape[1], seed=5)
    ref = What @ x.astype(np.float64)
    y = oracle.sbvr_gemv(planes, coeffs, x)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14 * np.abs(ref).max())
    yd = oracle.gemv_dense(What, x.astype(np.float64))
    np.testing.assert_allclose(yd, ref, rtol=1e-12, atol=1e-14 * np.abs(ref).max())
    # row subsets and batches give the same values
    X = synth.activations(What.shape[1], seed=6, batch=3)
    Y = oracle.sbvr_gemv(planes, coeffs, X)
    rows = [0, 7, 23]
    Ys = oracle.sbvr_gemv(planes, coeffs, X, rows=rows)
    np.testing.assert_array_equal(Ys, Y[:, rows])
    np.testing.assert_allclose(Y, X.astype(np.float64) @ What.T, rtol=1e-12,
                               atol=1e-14 * np.abs(Y).max())


# --------------------------------------------------------------------------
# Quality sanity (Sec. 3.1) and determinism
# --------------------------------------------------------------------------

def test_quality_against_rtn_and_rate_distortion(encoded_small):
    W = synth.weights(32, 1024, 1.0, seed=77)
    groups = W.reshape(-1, 128).astype(np.float64)
    for K, lo, hi in ((2, 0.10, 0.16), (3, 0.045, 0.065), (4, 0.0085, 0.011)):
        _, _, mse = oracle.encode_matrix(W, K, want_mse=True)
        m = mse.mean()
        assert lo < m < hi, (K, m)
        assert m > 2.0 ** (-2 * K)                       # Eq. 1: D >= sigma^2 2^(-2R)
        sym = np.mean([oracle.rtn_sym_mse(d, K) for d in groups])
        assert m < sym                                   # beats symmetric RTN
    # literal reading of Eq. 4 is worse at 4 bits (why span-normalised is the default)
    _, _, lit = oracle.encode_matrix(W[:4], 4, oracle.SearchParams(normalise=False), want_mse=True)
    assert lit.mean() > 0.014


def test_encoding_is_deterministic_across_thread_counts():
    W = synth.weights(8, 384, 0.02, seed=3)
    p1, c1 = oracle.encode_matrix(W, 3, nthreads=1)
    p8, c8 = oracle.encode_matrix(W, 3, nthreads=8)
    assert np.array_equal(p1, p8) and np.array_equal(c1, c8)


def test_synth_is_deterministic_and_sane():
    a = synth.weights(64, 1024, 0.02, seed=1001, outlier_frac=0.001)
    b = synth.weights(64, 1024, 0.02, seed=1001, outlier_frac=0.001)
    assert a.tobytes() == b.tobytes()
    out = np.isclose(np.abs(a), np.float32(8 * 0.02), rtol=0, atol=0)
    assert out.sum() == round(0.001 * a.size)
    g = a[~out].astype(np.float64)
    assert abs(g.mean()) < 5 * 0.02 / np.sqrt(g.size)
    assert abs(g.std() / 0.02 - 1) < 5 / np.sqrt(2 * g.size)
    x = synth.activations(4096, seed=synth.X_SEED_OFFSET)
    assert x.dtype == np.float16 and abs(float(x.astype(np.float64).std()) - 1) < 0.05


# --------------------------------------------------------------------------
# Online activation conversion to SBVR-8 (Sec. 4.3, Eq. 12) and the W4A8
# reference (readings R11-R13 of the oracle)
# --------------------------------------------------------------------------

def test_eq12_eight_bit_coefficients_are_twos_complement():
    """l = 8: {-128, 1, 2, ..., 64} (s = 1) has every integer -128..127 as
    exactly one subset sum -- two's complement."""
    coeffs = np.array([oracle.fp16_from_double(v) for v in (-128, 1, 2, 4, 8, 16, 32, 64)], dtype=np.uint16)
    sums = oracle.subset_sums(coeffs)
    assert sorted(sums.tolist()) == list(range(-128, 128))


def test_act_bitvectors_decode_every_code():
    q = np.arange(-127, 128, dtype=np.int32)
    q = np.concatenate([q, np.zeros(128 * 2 - q.size, dtype=np.int32)])   # two groups
    planes = oracle.act_planes(q)
    assert planes.shape == (256, 8) and set(np.unique(planes)) <= {0, 1}
    s = np.array([1.0, 0.375], dtype=np.float32)
    x_hat = oracle.act_decode(planes, s)
    np.testing.assert_array_equal(x_hat, q.astype(np.float64) * np.repeat(s.astype(np.float64), 128))
    # the bit patterns are the two's-complement bytes of q
    byte = (planes[:, 0].astype(int) << 7) | sum(planes[:, i].astype(int) << (i - 1) for i in range(1, 8))
    np.testing.assert_array_equal(byte.astype(np.uint8), q.astype(np.int8).view(np.uint8))


def test_act_quantize_nearest_grid_point():
    """Each element maps to the nearest point of {k s : |k| <= 127} (fp64
    check; the binary32 decision may differ only within rounding of a tie),
    the error is at most s/2, and the group's absmax element maps to +-127."""
    rng = np.random.default_rng(5)
    for trial in range(20):
        x = (rng.standard_normal(512) * 10 ** rng.uniform(-4, 3)).astype(np.float16)
        if trial == 0:
            x[:128] = 0           # a zero group
        q, s = oracle.act_quantize(x)
        xd = x.astype(np.float64)
        for g in range(4):
            sl = slice(128 * g, 128 * g + 128)
            sg = float(s[g])
            if np.abs(xd[sl]).max() == 0:
                assert sg == 0 and np.all(q[sl] == 0)
                continue
            assert np.abs(q[sl]).max() == 127
            err = np.abs(xd[sl] - q[sl] * sg)
            assert err.max() <= sg / 2 * (1 + 2 ** -20)
            t = xd[sl] / sg
            clear = np.abs(np.abs(t - np.floor(t)) - 0.5) > 1e-4   # not near a tie
            assert np.array_equal(q[sl][clear], np.clip(np.round(t[clear]), -127, 127).astype(np.int32))


def test_act_quantize_power_of_two_scaling():
    x = synth.activations(384, seed=8)
    q1, s1 = oracle.act_quantize(x)
    q2, s2 = oracle.act_quantize((x.astype(np.float32) * 4).astype(np.float16))
    np.testing.assert_array_equal(q1, q2)
    np.testing.assert_array_equal(s2, s1 * 4)


def test_w4a8_reference_equals_fp16_reference_on_grid_activations():
    """Activations that already lie on the grid (integers with absmax 127, so
    s = 1) convert exactly: the W4A8 reference equals the fp16 one."""
    O, I, K = 24, 512, 4
    planes, coeffs = synth.random_sbvr(O, I, K, seed=4)
    rng = np.random.default_rng(2)
    x = rng.integers(-127, 128, size=I).astype(np.float16)
    x[::128] = 127.0
    q, s = oracle.act_quantize(x)
    assert np.all(s == 1.0) and np.array_equal(q, x.astype(np.int32))
    np.testing.assert_array_equal(oracle.sbvr_gemv_w4a8(planes, coeffs, x), oracle.sbvr_gemv(planes, coeffs, x))


def test_w4a8_reference_is_dense_gemv_of_decoded_operands():
    O, I, K = 16, 640, 3
    planes, coeffs = synth.random_sbvr(O, I, K, seed=9)
    x = synth.activations(I, seed=10)
    q, s = oracle.act_quantize(x)
    x_hat = oracle.act_decode(oracle.act_planes(q), s)
    y = oracle.sbvr_gemv_w4a8(planes, coeffs, x)
    np.testing.assert_allclose(y, oracle.decompress(planes, coeffs) @ x_hat, rtol=1e-12, atol=1e-15)
    rows = [3, 0, 15]
    np.testing.assert_array_equal(oracle.sbvr_gemv_w4a8(planes, coeffs, x, rows=rows), y[rows])


# --------------------------------------------------------------------------
# Coefficient cache + per-group index (Sec. 4.4)
# --------------------------------------------------------------------------

def _bit(planes, o, g, i, j):
    return (int(planes[o, g, i, j // 32]) >> (j % 32)) & 1


def test_coefficient_cache_worked_example():
    """Three groups over two rows, two of them with the same set: the cache
    holds the two distinct sets in order of first appearance."""
    h = lambda v: np.float16(v).view(np.uint16)
    a = [h(0.5), h(-0.25)]
    b = [h(1.0), h(2.0)]
    coeffs = np.array([[a, b, a], [b, b, a]], dtype=np.uint16)   # [O=2][G=3][k=2]
    index, table = oracle.coefficient_cache(coeffs)
    assert index.tolist() == [[0, 1, 0], [1, 1, 0]]
    assert table.tolist() == [a, b]
    assert np.array_equal(oracle.gather_coefficients(index, table), coeffs)


def test_gathered_decompression_brute_force():
    """Decoded weights of the cache format from the definition, element by
    element: w[o][128 g + j] = sum_i table[index[o][g]][i] * b[o][g][i][j],
    with exact rational arithmetic (asymmetric O, G, k, N so that a
    transposed index or table fails)."""
    O, G, K, N = 3, 2, 3, 5
    planes, index, table = synth.random_indexed_sbvr(O, G * 128, K, N, seed=12)
    assert index.shape == (O, G) and table.shape == (N, K)
    What = oracle.decompress(planes, oracle.gather_coefficients(index, table))
    tab = [[Fraction(float(np.uint16(v).view(np.float16))) for v in row] for row in table]
    for o in range(O):
        for g in range(G):
            c = tab[int(index[o, g])]
            for j in range(128):
                w = sum((c[i] for i in range(K) if _bit(planes, o, g, i, j)), Fraction(0))
                assert Fraction(What[o, 128 * g + j]) == w


def test_coefficient_cache_round_trip_and_distinct_sets():
    """Per-group coefficients drawn from a small pool of sets: the cache is
    lossless, its sets are distinct and equal numpy's unique rows, and every
    index is in range."""
    rng = np.random.default_rng(3)
    pool = (rng.standard_normal((37, 4)) * 0.01).astype(np.float16).view(np.uint16)
    pick = rng.integers(0, 37, size=(64, 9))
    coeffs = pool[pick]                                  # [64][9][4]
    index, table = oracle.coefficient_cache(coeffs)
    assert np.array_equal(oracle.gather_coefficients(index, table), coeffs)
    assert table.shape[0] == len(np.unique(coeffs.reshape(-1, 4), axis=0))
    assert len({r.tobytes() for r in table}) == table.shape[0]
    assert index.dtype == np.uint16 and int(index.max()) < table.shape[0]
    # first appearance order
    first = [coeffs.reshape(-1, 4)[int(np.flatnonzero(index.reshape(-1) == n)[0])] for n in range(table.shape[0])]
    assert np.array_equal(np.array(first), table)
    with pytest.raises(ValueError):
        oracle.gather_coefficients(np.array([[table.shape[0]]]), table)


def test_indexed_generator_shapes_and_range():
    planes, index, table = synth.random_indexed_sbvr(7, 384, 2, 65536, seed=1)
    assert planes.shape == (7, 3, 2, 4) and index.shape == (7, 3) and table.shape == (65536, 2)
    _, index1, _ = synth.random_indexed_sbvr(7, 384, 2, 1, seed=1)
    assert np.all(index1 == 0)


def test_rtn_comparators_hand_values():
    """The RTN comparators (Sec. 3.1, Eq. 2 with the step read as
    max|w| / (2^(b-1) - 1), reading R7; asymmetric min-max RTN with 2^b
    levels) on D = {-3, ..., 4} * 2^-6, every quotient exact in binary64:
      symmetric 2 bits: delta = 2^-4, q = (-1, 0, 0, 0, 0, 0, 1, 1) (the
        ties -0.5 and 0.5 go to even), errors (1, -2, -1, 0, 1, 2, -1, 0) *
        2^-6, MSE = 12 / 8 * 2^-12;
      asymmetric 2 bits: delta = 7/3 * 2^-6, q = (0, 0, 1, 1, 2, 2, 3, 3),
        errors (0, 1, -1/3, 2/3, -2/3, 1/3, -1, 0) * 2^-6, MSE = 7/18 * 2^-12;
      asymmetric 3 bits: delta = 2^-6, every point on the grid, MSE = 0."""
    D = np.arange(-3, 5, dtype=np.float64) * 2.0 ** -6
    assert oracle.rtn_sym_mse(D, 2) == 1.5 * 2.0 ** -12
    np.testing.assert_allclose(oracle.rtn_asym_mse(D, 2), 7.0 / 18.0 * 2.0 ** -12, rtol=1e-12)
    assert oracle.rtn_asym_mse(D, 3) == 0.0
    # a constant group and an all-zero group have nothing to round away
    assert oracle.rtn_asym_mse(np.full(8, 0.3), 2) == 0.0
    assert oracle.rtn_sym_mse(np.zeros(8), 3) == 0.0
