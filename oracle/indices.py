"""Candidate index rules (oracle; test infrastructure only).

Sec. 3.1: recent queries score global columns and diagonals (vertical-slash), pooled
queries and keys score coarse blocks (block-sparse), A-shape needs no content-dependent
indices.  Reading of the open choices:

* one total order for every selection: score descending, then -0.0 after +0.0, then
  position ascending;
* vertical-slash: V = F_v + top (n_v - |F_v|) columns of the rest, D = F_s + top
  (n_s - |F_s|) diagonals of the rest, with forced sets F_v = {} and F_s = {0} (the
  main diagonal keeps every row non-empty); forced items count toward the budget;
* block-sparse: Sel(bq) = {bq} + top (k - 1) of the blocks bk < bq by pooled score;
* when fewer candidates exist than the budget, all are taken;
* budgets of one family are prefixes of one ranking (nested); outputs are also given in
  ascending order.
"""
from __future__ import annotations

import numpy as np


def rank_order(scores, cand):
    """``cand`` ordered by (score desc, +0.0 before -0.0, index asc)."""
    cand = np.asarray(cand, dtype=np.int64)
    if cand.size == 0:
        return cand
    s = np.asarray(scores, dtype=np.float64)[cand]
    order = np.lexsort((cand, np.signbit(s), -s))
    return cand[order]


def _forced_then_ranked(scores, s1, forced):
    forced = np.array(sorted({int(f) for f in forced if 0 <= int(f) < s1}), dtype=np.int64)
    rest = np.setdiff1d(np.arange(s1, dtype=np.int64), forced, assume_unique=True)
    return np.concatenate([forced, rank_order(scores, rest)])


def vs_ranking(col, diag, s1, F_v=(), F_s=(0,)):
    """Full rankings (forced first) of columns and diagonals over [0, s1)."""
    return _forced_then_ranked(col, s1, F_v), _forced_then_ranked(diag, s1, F_s)


def vs_indices(col, diag, s1, n_v, n_s, F_v=(), F_s=(0,)):
    """Vertical-slash index sets for budget (n_v, n_s): (V, D) ascending, plus rankings."""
    vr, dr = vs_ranking(col, diag, s1, F_v, F_s)
    return np.sort(vr[:n_v]), np.sort(dr[:n_s]), vr, dr


def bs_ranking_row(lrow, bq):
    """Ranking of key blocks for query block bq: bq first, then blocks < bq by score."""
    return np.concatenate([[bq], rank_order(lrow, np.arange(bq, dtype=np.int64))]).astype(np.int64)


def bs_indices(L, k):
    """Block-sparse selection for every query block of a pooled-score matrix ``L``
    (lower triangle valid): list of ascending arrays and list of rankings."""
    nb = L.shape[0]
    sel, ranks = [], []
    for bq in range(nb):
        r = bs_ranking_row(L[bq], bq)
        ranks.append(r)
        sel.append(np.sort(r[:k]))
    return sel, ranks
