"""Dense and masked causal attention in fp64 (oracle; test infrastructure only).

One head at a time: ``q`` is [n, d] (rows of one query head), ``k``/``v`` are [n, d]
(the key/value head that query head reads), ``rows`` are absolute query positions and
``s1`` bounds the keys considered, [0, s1).  The causal visible set of row i is
{0, ..., i}.
"""
from __future__ import annotations

import numpy as np


def default_scale(d: int) -> float:
    return 1.0 / np.sqrt(float(d))


def logits(q, k, rows, s1, scale=None):
    """l_ij = (q_i . k_j) * scale for i in rows, j in [0, s1)  (Sec. 2.1, Eq. 1)."""
    rows = np.asarray(rows, dtype=np.int64)
    scale = default_scale(q.shape[1]) if scale is None else scale
    qr = np.asarray(q)[rows].astype(np.float64)
    kk = np.asarray(k)[:s1].astype(np.float64)
    return (qr @ kk.T) * scale


def causal_visible(rows, s1):
    rows = np.asarray(rows, dtype=np.int64)
    return np.arange(s1)[None, :] <= rows[:, None]


def dense_probs(q, k, rows, s1=None, scale=None):
    """Exact causal attention rows a_ij (Sec. 2.1, Eq. 1); a_ij = 0 for j > i."""
    rows = np.asarray(rows, dtype=np.int64)
    s1 = int(rows.max()) + 1 if s1 is None else s1
    lg = logits(q, k, rows, s1, scale)
    vis = causal_visible(rows, s1)
    lg = np.where(vis, lg, -np.inf)
    mx = lg.max(axis=1, keepdims=True)
    e = np.where(vis, np.exp(lg - mx), 0.0)
    return e / e.sum(axis=1, keepdims=True)


def masked_softmax(q, k, rows, mask, scale=None):
    """Masked attention probabilities: logits outside ``mask`` become minus infinity
    and each row is a softmax over its kept set S_i (Sec. 2.1).  ``mask`` is a boolean
    [len(rows), s1] array; it is intersected with the causal set.  Rows with an empty
    kept set get all-zero probabilities and log-sum-exp minus infinity.

    Returns (probabilities, lse) with lse_i = log sum_{j in S_i} exp(l_ij).
    """
    rows = np.asarray(rows, dtype=np.int64)
    mask = np.asarray(mask, dtype=bool)
    s1 = mask.shape[1]
    keep = mask & causal_visible(rows, s1)
    lg = np.where(keep, logits(q, k, rows, s1, scale), -np.inf)
    mx = lg.max(axis=1, keepdims=True)
    empty = ~keep.any(axis=1)
    mx = np.where(empty[:, None], 0.0, mx)
    e = np.where(keep, np.exp(lg - mx), 0.0)
    den = e.sum(axis=1, keepdims=True)
    p = np.where(empty[:, None], 0.0, e / np.where(den > 0, den, 1.0))
    lse = np.where(empty, -np.inf, mx[:, 0] + np.log(np.where(den[:, 0] > 0, den[:, 0], 1.0)))
    return p, lse


def dense_attention(q, k, v, rows=None, scale=None, block=512):
    """O_i = sum_{j<=i} a_ij v_j (Sec. 2.1, Eq. 1), computed in row blocks."""
    n = q.shape[0]
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, v.shape[1]), dtype=np.float64)
    vv = np.asarray(v, dtype=np.float64)
    for b in range(0, rows.size, block):
        rb = rows[b:b + block]
        s1 = int(rb.max()) + 1
        out[b:b + block] = dense_probs(q, k, rb, s1, scale) @ vv[:s1]
    return out


def masked_attention(q, k, v, rows, mask, scale=None):
    """O~_i = softmax over S_i of l_i. times V (Sec. 2.1): the sparse-mask output."""
    p, lse = masked_softmax(q, k, rows, mask, scale)
    return p @ np.asarray(v)[:p.shape[1]].astype(np.float64), lse


def masked_attention_cols(q, k, v, rows, cols, keep, scale=None):
    """Masked attention (Sec. 2.1) whose kept sets lie among the key positions ``cols``
    (ascending): S_i = {cols[c] : keep[r, c] and cols[c] <= i}.  The result equals
    masked_attention with the mask that is ``keep`` on ``cols`` and False elsewhere; only the
    logits of the listed keys are formed, so sparse sets over long prefixes stay cheap.  The
    same fp64 steps as masked_softmax, taken with torch CPU operations (multi-threaded).

    Returns (output, lse) as masked_attention does (empty rows: 0 and minus infinity)."""
    import torch
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    scale = default_scale(q.shape[1]) if scale is None else scale
    keep = torch.from_numpy(np.asarray(keep, dtype=bool) & (cols[None, :] <= rows[:, None]))
    qr = torch.from_numpy(np.asarray(q)[rows]).to(torch.float64)
    kc = torch.from_numpy(np.asarray(k)[cols]).to(torch.float64)
    vc = torch.from_numpy(np.asarray(v)[cols]).to(torch.float64)
    lg = (qr @ kc.T) * scale
    lg = lg.masked_fill(~keep, float("-inf"))
    empty = ~keep.any(dim=1)
    zero = torch.zeros((), dtype=torch.float64)
    mx = torch.where(empty, zero, lg.amax(dim=1) if cols.size else zero)[:, None]
    e = torch.exp(lg - mx).masked_fill(~keep, 0.0)
    den = e.sum(dim=1, keepdim=True)
    p = e / torch.where(den > 0, den, torch.ones_like(den))  # empty rows: e = 0, so p = 0
    lse = torch.where(empty, float("-inf"), mx[:, 0] + torch.log(torch.where(den[:, 0] > 0, den[:, 0],
                                                                           torch.ones_like(den[:, 0]))))
    return (p @ vc).numpy(), lse.numpy()


def retained_mass(a, mask):
    """m_i = sum_{j in S_i} a_ij: exact attention mass kept by the mask (Sec. 3.3)."""
    return np.where(mask, a, 0.0).sum(axis=1)


def renormalized_attention(a, mask, v):
    """Second form of the masked output: a~_ij = a_ij / m_i on S_i (Sec. 3.3)."""
    m = retained_mass(a, mask)
    at = np.where(mask, a, 0.0) / np.where(m > 0, m, 1.0)[:, None]
    return at @ np.asarray(v, dtype=np.float64)[:a.shape[1]], at, m


def certificate(a, mask, v, rows):
    """Omitted-mass certificate (Sec. 3.3, Eq. 5), per row.

    Returns (err, bound, l1) with err = ||a_i V - a~_i V||_2,
    bound = 2 (1 - m_i) max_{j<=i} ||v_j||_2 and l1 = ||a_i - a~_i||_1, which equals
    2 (1 - m_i) exactly.
    """
    rows = np.asarray(rows, dtype=np.int64)
    vv = np.asarray(v, dtype=np.float64)[:a.shape[1]]
    ot, at, m = renormalized_attention(a, mask, vv)
    o = a @ vv
    err = np.linalg.norm(o - ot, axis=1)
    norms = np.linalg.norm(vv, axis=1)
    vmax = np.maximum.accumulate(norms)[rows]
    bound = 2.0 * (1.0 - m) * vmax
    l1 = np.abs(a - at).sum(axis=1)
    return err, bound, l1


def e_rel(o, o_tilde, eps=1e-12):
    """E_rel = ||O - O~||_F / (||O||_F + eps) (Sec. 4.2, Eq. 9); eps is not given in the
    paper, 1e-12 is used."""
    o = np.asarray(o, dtype=np.float64)
    o_tilde = np.asarray(o_tilde, dtype=np.float64)
    return float(np.linalg.norm(o - o_tilde) / (np.linalg.norm(o) + eps))
