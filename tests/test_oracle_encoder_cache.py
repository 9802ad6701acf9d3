"""Pins of the oracle's encoder with the cache of Sec. 4.2 (last paragraph and
its footnote; reading R14), on the CPU.

The cached encoder is checked against what the paper and the reading fix,
group by group, using only functions pinned elsewhere (Algorithm 1 per group
and its MSE, `test_oracle_pins.py`):

  * a group either ran Algorithm 1 (its coefficients, patterns and MSE are
    the exhaustive search's) or took a set that the search chose for one of
    the row's last `slots` searched groups -- the best of them on this group,
    with an MSE strictly below the mean MSE of the row's earlier groups;
  * a searched group had no such cached set (the cache could not serve it);
  * the first group of a row always searches; slots = 0 is the plain encoder;
  * the paper's two effects: a large share of hits on Gaussian weights, and
    fewer distinct coefficient sets (at most one per searched group).
A mistake in the ring order, the threshold, its strictness, what enters the
average or what enters the cache changes some group's decision and fails
the walk below.
"""
import numpy as np
import pytest

import oracle
import synth

GROUP = 128


def planes_of(codes, K):
    """Canonical planes [K][4] of one group from its 128 pattern codes."""
    pl = np.zeros((K, 4), dtype=np.uint32)
    for j, p in enumerate(codes):
        for i in range(K):
            if (int(p) >> i) & 1:
                pl[i, j // 32] |= np.uint32(1 << (j % 32))
    return pl


def nearest_codes(D, coeffs):
    sums = oracle.subset_sums(coeffs)
    return [oracle.nearest(sums, float(x)) for x in D]


def walk_row(W_row, K, slots, planes, coeffs, mse, hits, params=oracle.DEFAULT):
    """Check one row's decisions group by group; returns the hit count."""
    G = W_row.size // GROUP
    searched = []   # coefficient sets chosen by the search, in order (fallbacks excluded)
    total = 0.0     # binary64 sum of the earlier groups' MSEs, in group order
    n_hits = 0
    for g in range(G):
        D = W_row[g * GROUP:(g + 1) * GROUP].astype(np.float64)
        window = searched[-slots:] if slots > 0 else []
        scores = [oracle.entry_mse(D, c) for c in window]        # oldest first
        best = min(scores) if scores else np.inf
        avg = total / g if g > 0 else np.inf
        if hits[g]:
            assert g > 0 and window, ("hit without a cache", g)
            j = scores.index(best)                                 # oldest among equal ones
            assert np.array_equal(coeffs[g], window[j]), ("hit took another set", g)
            assert best < avg, ("hit at or above the moving average", g, best, avg)
            assert mse[g] == best, g
            assert np.array_equal(planes[g], planes_of(nearest_codes(D, coeffs[g]), K)), g
            n_hits += 1
        else:
            assert not (window and best < avg), ("a cached set was good enough", g, best, avg)
            c_ref, codes_ref, m_ref, entry = oracle.encode_group(D, K, params)
            assert np.array_equal(coeffs[g], c_ref) and mse[g] == m_ref, ("search result differs", g)
            assert np.array_equal(planes[g], planes_of(codes_ref, K)), g
            if entry >= 0:
                searched.append(c_ref.copy())
        total += float(mse[g])
    return n_hits


@pytest.mark.parametrize("K,slots,O,I", [(4, 64, 6, 2048), (4, 3, 6, 2048), (3, 1, 5, 1536),
                                         (2, 8, 4, 2048), (1, 64, 4, 1024), (4, 2, 3, 4096)])
def test_cached_encoder_decisions(K, slots, O, I):
    W = synth.weights(O, I, 0.02, seed=synth.seed_for(2, K, slots), outlier_frac=0.001)
    planes, coeffs, mse, hits = oracle.encode_matrix_cached(W, K, slots)
    n = 0
    for o in range(O):
        n += walk_row(W[o], K, slots, planes[o], coeffs[o], mse[o], hits[o])
    assert n == int(hits.sum())
    assert n > 0, "no hit at all: the cache never served"


def test_cached_encoder_degenerate_rows():
    """Constant, zero and extreme groups inside rows: R6 fallbacks are not
    cached, and decisions still follow the rule."""
    rng = np.random.default_rng(3)
    groups = [np.zeros(128), np.full(128, 0.0125), rng.standard_normal(128) * 0.02,
              rng.standard_normal(128) * 1e30, rng.standard_normal(128) * 0.02, np.zeros(128),
              rng.standard_normal(128) * 0.02, np.full(128, -3.5)]
    W = np.concatenate(groups).astype(np.float32)[None, :]
    for K in (1, 2, 4):
        for slots in (1, 4):
            planes, coeffs, mse, hits = oracle.encode_matrix_cached(W, K, slots)
            walk_row(W[0], K, slots, planes[0], coeffs[0], mse[0], hits[0])


@pytest.mark.parametrize("K", [1, 2, 3, 4])
def test_zero_slots_is_the_plain_encoder(K):
    W = synth.weights(7, 1024, 0.02, seed=11 + K, outlier_frac=0.001)
    p, c, m = oracle.encode_matrix(W, K, want_mse=True)
    pc, cc, mc, hc = oracle.encode_matrix_cached(W, K, 0)
    assert np.array_equal(p, pc) and np.array_equal(c, cc)
    assert np.array_equal(m.view(np.uint64), mc.view(np.uint64))
    assert not hc.any()


def test_threshold_is_strict():
    """Three identical groups: the first searches; the cached set then scores
    exactly the running mean (m, then (m + m) / 2 = m), which is not strictly
    below it, so the next two search as well."""
    D = synth.weights(1, 128, 0.02, seed=5)[0]
    W = np.tile(D, 3)[None, :].astype(np.float32)
    planes, coeffs, mse, hits = oracle.encode_matrix_cached(W, 4, 8)
    assert hits.tolist() == [[0, 0, 0]]
    assert mse[0, 0] == mse[0, 1] == mse[0, 2]
    assert (coeffs[0] == coeffs[0, 0]).all()


def test_rows_are_independent_and_first_group_searches():
    W = synth.weights(6, 1024, 0.02, seed=21)
    full = oracle.encode_matrix_cached(W, 4, 16)
    assert not full[3][:, 0].any()
    for o in (0, 3, 5):
        one = oracle.encode_matrix_cached(W[o:o + 1], 4, 16)
        for a, b in zip(full, one):
            assert np.array_equal(a[o:o + 1], b)


def test_paper_effects_hit_share_and_fewer_sets():
    """Gaussian weights (N(0, 0.02^2), 0.1 % outliers at +-8 sigma) at the
    Llama-3-8B inner dimension: a large share of groups reuse a cached set
    (the paper reports up to 90 %), every hit shares an earlier group's set,
    so the distinct sets number at most the searched groups, and the error
    grows by a bounded factor."""
    W = synth.weights(16, 4096, 0.02, seed=synth.seed_for(1, 0, 0), outlier_frac=0.001)
    _, c0, m0 = oracle.encode_matrix(W, 4, want_mse=True)
    _, c, m, h = oracle.encode_matrix_cached(W, 4, 64)
    rate = float(h.mean())
    distinct = len({x.tobytes() for x in c.reshape(-1, 4)})
    assert rate >= 0.4, rate
    assert distinct <= int((h == 0).sum()), (distinct, int((h == 0).sum()))
    assert distinct < len({x.tobytes() for x in c0.reshape(-1, 4)})
    assert m.mean() >= m0.mean()          # the exhaustive search is the minimum per group
    assert m.mean() <= 1.5 * m0.mean(), m.mean() / m0.mean()


def test_bad_arguments():
    W = np.zeros((2, 256), dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.encode_matrix_cached(W, 4, 65)
    with pytest.raises(ValueError):
        oracle.encode_matrix_cached(W, 4, -1)
    with pytest.raises(ValueError):
        oracle.encode_matrix_cached(W[:, :200], 4, 4)
