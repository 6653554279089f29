"""Pins of the index rules (Sec. 3.1): total order, forced sets, nesting."""
import numpy as np

from oracle import indices as IX


def _brute_rank(scores, cand):
    return [c for _, _, c in sorted((-scores[c], bool(np.signbit(scores[c])), c) for c in cand)]


def test_rank_order_matches_full_sort_with_ties():
    r = np.random.default_rng(1)
    s = np.round(r.random(500) * 20) / 20          # many exact ties
    s[[3, 10, 40]] = 0.0
    s[[5, 11]] = -0.0
    cand = np.arange(500)
    assert IX.rank_order(s, cand).tolist() == _brute_rank(s, cand)
    t = np.array([1.0, 2.0, 2.0, 0.5, 2.0])
    assert IX.rank_order(t, np.arange(5)).tolist() == [1, 2, 4, 0, 3]
    z = np.array([0.0, -0.0, 0.0, -0.0])
    assert IX.rank_order(z, np.arange(4)).tolist() == [0, 2, 1, 3]


def test_vs_indices_forced_nested_sorted():
    r = np.random.default_rng(2)
    s1 = 300
    col, diag = r.random(s1), r.random(s1)
    diag[0] = -1.0                                   # forced despite the lowest score
    V1, D1, vr, dr = IX.vs_indices(col, diag, s1, 10, 20)
    V2, D2, _, _ = IX.vs_indices(col, diag, s1, 40, 60)
    assert 0 in D1 and dr[0] == 0
    assert set(V1) <= set(V2) and set(D1) <= set(D2)
    assert np.all(np.diff(V1) > 0) and np.all(np.diff(D2) > 0)
    assert V1.tolist() == sorted(_brute_rank(col, range(s1))[:10])
    assert D1.tolist() == sorted([0] + [c for c in _brute_rank(diag, range(s1)) if c != 0][:19])
    V3, D3, _, _ = IX.vs_indices(col, diag, 30, 1000, 1000)
    assert V3.tolist() == list(range(30)) and D3.tolist() == list(range(30))


def test_bs_indices_diagonal_first_and_budget():
    r = np.random.default_rng(3)
    nb = 40
    L = r.standard_normal((nb, nb))
    L[np.triu_indices(nb, 1)] = np.nan
    sel, ranks = IX.bs_indices(L, 5)
    for bq in range(nb):
        assert ranks[bq][0] == bq
        assert len(sel[bq]) == min(bq + 1, 5)
        exp = sorted([bq] + _brute_rank(L[bq], range(bq))[:4])
        assert sel[bq].tolist() == exp
