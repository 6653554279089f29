"""Shared attention probe and block-mean estimator (oracle; test infrastructure only).

Follows Sec. 3.2 (Eq. 3) and the index builders of Sec. 3.1.  Reading of the open
choices (the paper gives no proportions, pooling width or descriptor formulas):

* sampled rows of a unit (rows [s0, s1), keys [0, s1)) are the union of
  R = the last r_rec rows of the segment, U = r_uni uniformly spaced rows and
  Bd = r_bnd rows just after the segment start (never below row 64);
* sampled rows are scored at token resolution (pooling width g = 1): the vertical-slash
  builder needs single columns and diagonals;
* the block-sparse builder scores coarse blocks with mean-pooled queries and keys
  (block width B, last partial block averaged over its actual tokens);
* descriptors per sampled row: entropy of the 64-key block masses divided by the log of
  the number of visible blocks (0 when only one block is visible), and the local mass
  within the last ``local_w`` keys (i - local_w, i].
"""
from __future__ import annotations

import numpy as np

from .attention import dense_probs, default_scale

SUB_R, SUB_U, SUB_B = 0, 1, 2


def sample_rows(s0, s1, r_rec, r_uni, r_bnd):
    """Probe rows (R, U, Bd) of segment [s0, s1), each ascending and pairwise disjoint."""
    R = np.arange(max(s0, s1 - r_rec), s1, dtype=np.int64)
    L = s1 - s0
    if r_uni > 0 and L > 0:
        U = s0 + ((2 * np.arange(r_uni, dtype=np.int64) + 1) * L) // (2 * r_uni)
        U = np.unique(U)
        U = U[~np.isin(U, R)]
    else:
        U = np.zeros(0, dtype=np.int64)
    if r_bnd > 0:
        B = max(s0, 64) + np.arange(r_bnd, dtype=np.int64)
        B = B[(B >= s0) & (B < s1)]
        B = B[~np.isin(B, R) & ~np.isin(B, U)]
    else:
        B = np.zeros(0, dtype=np.int64)
    return R, U, B


def probe_rows(s0, s1, r_rec, r_uni, r_bnd):
    """All sampled rows ascending, with their subset label (0 = R, 1 = U, 2 = Bd)."""
    R, U, B = sample_rows(s0, s1, r_rec, r_uni, r_bnd)
    rows = np.concatenate([R, U, B])
    lab = np.concatenate([np.full(R.size, SUB_R), np.full(U.size, SUB_U), np.full(B.size, SUB_B)])
    order = np.argsort(rows, kind="stable")
    return rows[order], lab[order].astype(np.int64)


def col_diag_scores(a, rows, is_recent, s1):
    """Column and diagonal scores of the vertical-slash builder (Sec. 3.1): with
    R the recent rows, col[j] = sum_{i in R} a_ij and diag[delta] = sum_{i in R} a_{i,i-delta}
    for j, delta in [0, s1)."""
    col = np.zeros(s1, dtype=np.float64)
    diag = np.zeros(s1, dtype=np.float64)
    for r in np.nonzero(is_recent)[0]:
        i = int(rows[r])
        col += a[r, :s1]
        # a_{i, i - delta} for delta = 0..i
        diag[:i + 1] += a[r, i::-1]
    return col, diag


def row_descriptors(a, rows, local_w=1024, block=64):
    """Per sampled row: normalised 64-block entropy and local-band mass (Sec. 3.2)."""
    ent = np.zeros(len(rows))
    loc = np.zeros(len(rows))
    for r, i in enumerate(rows):
        i = int(i)
        nvis = i // block + 1
        bm = np.zeros(nvis)
        np.add.at(bm, np.arange(i + 1) // block, a[r, :i + 1])
        nz = bm[bm > 0]
        h = -(nz * np.log(nz)).sum()
        ent[r] = h / np.log(nvis) if nvis > 1 else 0.0
        loc[r] = a[r, max(0, i - local_w + 1):i + 1].sum()
    return ent, loc


def probe_unit(q, k, s0, s1, r_rec, r_uni, r_bnd, scale=None, local_w=1024):
    """The probe of one unit (query head, segment): exact fp64 rows for the sampled set,
    the recent-row column/diagonal scores and the descriptors (Sec. 3.2, Eq. 3 with g = 1)."""
    rows, lab = probe_rows(s0, s1, r_rec, r_uni, r_bnd)
    a = dense_probs(q, k, rows, s1, scale)
    col, diag = col_diag_scores(a, rows, lab == SUB_R, s1)
    ent, loc = row_descriptors(a, rows, local_w)
    return dict(rows=rows, subset=lab, a=a, col=col, diag=diag, entropy=ent, local=loc,
                entropy_mean=float(ent.mean()) if ent.size else 0.0,
                local_mean=float(loc.mean()) if loc.size else 0.0)


def block_means(x, block=64):
    """Mean of each block of ``block`` consecutive rows; the last block uses its actual count."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    nb = (n + block - 1) // block
    out = np.zeros((nb, x.shape[1]))
    for b in range(nb):
        out[b] = x[b * block:min(n, (b + 1) * block)].mean(axis=0)
    return out


def block_mean_logits(q, k, block=64, scale=None):
    """Pooled-query x pooled-key scores of the block-sparse builder (Sec. 3.1):
    L[bq, bk] = (mean q over block bq) . (mean k over block bk) * scale for bk <= bq,
    NaN above the diagonal."""
    scale = default_scale(q.shape[1]) if scale is None else scale
    qb = block_means(q, block)
    kb = block_means(k, block)
    lg = (qb @ kb.T) * scale
    nb = lg.shape[0]
    lg[np.triu_indices(nb, 1)] = np.nan
    return lg
