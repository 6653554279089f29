"""Pins of the token-exact pattern sets (Sec. 2.1, Sec. 3.1)."""
import json
import os

import numpy as np

from oracle import patterns as P

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _loop_ashape(n, s, w):
    m = np.zeros((n, n), bool)
    for i in range(n):
        for j in range(i + 1):
            m[i, j] = j < s or i - j < w
    return m


def _loop_vs(n, V, D):
    m = np.zeros((n, n), bool)
    for i in range(n):
        for j in range(i + 1):
            m[i, j] = (j in V) or ((i - j) in D)
    return m


def test_ashape_matches_loops_and_closed_form():
    for n, s, w in [(50, 3, 7), (64, 0, 1), (70, 10, 100), (33, 40, 5)]:
        m = P.ashape_mask(np.arange(n), n, s, w)
        np.testing.assert_array_equal(m, _loop_ashape(n, s, w))
        assert m.sum() == P.ashape_pairs(n, s, w)


def test_ashape_wide_window_is_dense():
    n = 77
    np.testing.assert_array_equal(P.ashape_mask(np.arange(n), n, 0, n), P.dense_mask(np.arange(n), n))


def test_vs_matches_loops_and_degenerates_to_dense():
    n = 60
    r = np.random.default_rng(1)
    V = set(r.choice(n, 7, replace=False).tolist())
    D = set(r.choice(n, 9, replace=False).tolist()) | {0}
    np.testing.assert_array_equal(P.vs_mask(np.arange(n), n, sorted(V), sorted(D)), _loop_vs(n, V, D))
    dense = P.dense_mask(np.arange(n), n)
    np.testing.assert_array_equal(P.vs_mask(np.arange(n), n, np.arange(n), []), dense)
    np.testing.assert_array_equal(P.vs_mask(np.arange(n), n, [], np.arange(n)), dense)


def test_bs_matches_loops_and_degenerates_to_dense():
    n, B = 200, 16
    nb = (n + B - 1) // B
    r = np.random.default_rng(2)
    sel = {bq: sorted(set(r.choice(bq + 1, min(bq + 1, 3), replace=False).tolist()) | {bq})
           for bq in range(nb)}
    m = P.bs_mask(np.arange(n), n, B, lambda bq: sel[bq])
    for i in range(n):
        for j in range(n):
            assert m[i, j] == (j <= i and (j // B) in sel[i // B])
    np.testing.assert_array_equal(P.bs_mask(np.arange(n), n, B, lambda bq: range(bq + 1)),
                                  P.dense_mask(np.arange(n), n))


def test_workload_pair_counts():
    """Per-head kept pairs of the A-shape (128, 1024) layer at n = 8192 and of the
    block-sparse top-100 layer at n = 131072 (64-token blocks), from their closed forms."""
    with open(os.path.join(GOLD, "pair_counts.json")) as f:
        gold = json.load(f)
    assert P.ashape_pairs(8192, 128, 1024) == gold["ashape_n8192_s128_w1024"]
    B, k, n = 64, 100, 131072
    nb = n // B
    tot = 0
    for bq in range(nb):
        ns = min(bq + 1, k)
        tot += (ns - 1) * B * B + B * (B + 1) // 2
    assert tot == gold["bs_n131072_b64_k100"]
    # enumeration on a scaled-down block-sparse case with the same rule
    n2, B2, k2 = 640, 8, 5
    m = P.bs_mask(np.arange(n2), n2, B2, lambda bq: range(max(0, bq - k2 + 1), bq + 1))
    tot2 = sum((min(bq + 1, k2) - 1) * B2 * B2 + B2 * (B2 + 1) // 2 for bq in range(n2 // B2))
    assert m.sum() == tot2


def test_masks_on_column_subsets_equal_full_mask_columns():
    """Evaluating a pattern on a subset of key positions gives exactly those columns of the
    full mask, for every family (used to check long prefixes on the kept keys only)."""
    r = np.random.default_rng(9)
    s1 = 700
    rows = np.sort(r.choice(s1, 60, replace=False))
    cols = np.sort(r.choice(s1, 250, replace=False))
    V = r.choice(s1, 40, replace=False)
    D = np.concatenate([[0], r.choice(s1, 30, replace=False)])
    sel = {b: sorted(set(r.choice(b + 1, min(b + 1, 4), replace=False).tolist()) | {b}) for b in range(11)}
    cases = [(P.dense_mask, ()), (P.ashape_mask, (64, 100)), (P.vs_mask, (V, D)),
             (P.bs_mask, (64, lambda b: sel[b]))]
    for fn, args in cases:
        full = fn(rows, s1, *args)
        sub = fn(rows, s1, *args, cols=cols)
        assert sub.shape == (rows.size, cols.size)
        assert np.array_equal(sub, full[:, cols]), fn.__name__
