"""Token-exact key sets of the pattern library (oracle; test infrastructure only).

Each function returns a boolean [len(rows), s1] mask whose row r is the kept set S_i of
query position i = rows[r] over keys [0, s1).  Every set is intersected with the causal
set {j <= i} (Sec. 2.1).  Block granularity in a kernel is an implementation detail: the
semantics are token-exact.
"""
from __future__ import annotations

import numpy as np


def _grid(rows, s1, cols=None):
    rows = np.asarray(rows, dtype=np.int64)
    i = rows[:, None]
    j = (np.arange(s1, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64))[None, :]
    return i, j


# Every mask function takes an optional ``cols`` (key positions in [0, s1)): the mask is then
# evaluated on those columns only, i.e. equals the full mask's columns ``cols``.


def dense_mask(rows, s1, cols=None):
    """Dense candidate / fallback: the full causal set C_i (Sec. 3.1)."""
    i, j = _grid(rows, s1, cols)
    return j <= i


def ashape_mask(rows, s1, sink, window, cols=None):
    """A-shape (Sec. 2.1, Sec. 3.1): initial tokens [0, sink) together with a local window.

    Reading: the window holds ``window`` keys including the diagonal, (i - window, i].
    """
    i, j = _grid(rows, s1, cols)
    return (j <= i) & ((j < sink) | (j > i - window))


def vs_mask(rows, s1, V, D, cols=None):
    """Vertical-slash (Sec. 2.1): S_i = {j in V : j <= i} U {i - delta : delta in D, delta <= i}."""
    i, j = _grid(rows, s1, cols)
    vb = np.zeros(s1, dtype=bool)
    V = np.asarray(V, dtype=np.int64)
    vb[V[(V >= 0) & (V < s1)]] = True
    db = np.zeros(s1, dtype=bool)
    D = np.asarray(D, dtype=np.int64)
    db[D[(D >= 0) & (D < s1)]] = True
    delta = i - j
    in_d = np.zeros(delta.shape, dtype=bool)
    ok = (delta >= 0) & (delta < s1)
    in_d[ok] = db[delta[ok]]
    return (j <= i) & (vb[j] | in_d)


def bs_mask(rows, s1, block, sel, cols=None):
    """Block-sparse (Sec. 2.1): S_i = {j <= i : floor(j/B) in Sel(floor(i/B))}.

    ``sel`` maps a query block index to an iterable of selected key block indices.
    """
    rows = np.asarray(rows, dtype=np.int64)
    j = np.arange(s1, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    out = np.zeros((rows.size, j.size), dtype=bool)
    jb = j // block
    # rows of one query block share its selection
    for b in np.unique(rows // block):
        r = np.nonzero(rows // block == b)[0]
        chosen = np.zeros((s1 + block - 1) // block, dtype=bool)
        s = np.asarray(list(sel(int(b))), dtype=np.int64)
        s = s[(s >= 0) & (s < chosen.size)]
        chosen[s] = True
        out[r] = chosen[jb][None, :] & (j[None, :] <= rows[r][:, None])
    return out


def ashape_pairs(n, sink, window):
    """Closed form for sum_i |S_i| of A-shape over rows [0, n) with keys [0, n)."""
    total = 0
    # row i keeps min(i+1, window) window keys, plus sinks j < sink that lie outside the window
    for i in range(n):
        w = min(i + 1, window)
        lo = i - w + 1                     # first window key
        total += w + max(0, min(sink, lo))
    return total
