"""Candidate coverage, uncertainty, lower mass and risk (oracle; test infrastructure only).

Sec. 3.2 defines the covered probe mass of a candidate and the agreement between probe
subsets; Sec. 3.3 defines the risk (Eq. 4) and the lower confidence mass.  Reading:

* m_i(c) = sum_{j in S_i(c)} a_ij for every sampled row i, with S_i(c) the token-exact
  key set of candidate c (for the vertical-slash family the sets built from the recent
  rows are applied to every sampled row);
* m_hat(c) is the mean over all sampled rows, m_R, m_U, m_B the means over each probe
  subset;
* u(c) = max - min of the subset means over the non-empty subsets (0 with one subset);
* m_lower = max(0, m_hat - delta_q);
* risk R(c) = (1 - m_hat) + alpha * u + beta * e (Eq. 4), e the optional calibrated
  error predictor; the dense candidate has m_hat = 1, u = 0 and risk 0 by definition.

Reading of e (Sec. 3.3 asks only for a small monotone regressor fitted offline on dense
calibration runs, fed with probe descriptors and candidate metadata): with omega = 1 - m_hat,
H and L the means over the unit's sampled rows of the normalised block entropy and of the
local-band mass, the features are (omega, u, omega * H, omega * (1 - L)) and
e = sum_k w[family][k] x_k with non-negative weights, hence monotone non-decreasing in every
feature; dense candidates get 0.  Sums in fp64, e rounded to fp32.  The features and the model
form are this reading, not the paper's: parity unpinned beyond the invariants its tests check.
"""
from __future__ import annotations

import numpy as np

from .attention import retained_mass
from .probe import SUB_R, SUB_U, SUB_B


def row_coverage(a, mask):
    """m_i for each sampled row (Sec. 3.3)."""
    return retained_mass(a, mask)


def subset_means(m_rows, subset):
    """(m_hat, [m_R, m_U, m_B], [n_R, n_U, n_B]); a mean over an empty subset is 0."""
    m_rows = np.asarray(m_rows, dtype=np.float64)
    subset = np.asarray(subset)
    means, counts = [], []
    for s in (SUB_R, SUB_U, SUB_B):
        sel = subset == s
        counts.append(int(sel.sum()))
        means.append(float(m_rows[sel].mean()) if sel.any() else 0.0)
    return float(m_rows.mean()), means, counts


def disagreement(sub_means, sub_counts):
    """u = max - min over the non-empty probe subsets (Sec. 3.2)."""
    vals = [m for m, c in zip(sub_means, sub_counts) if c > 0]
    if len(vals) <= 1:
        return 0.0
    return max(vals) - min(vals)


def lower_mass(m_hat, delta_q):
    """m_lower = max(0, m_hat - delta_q) (Sec. 3.3)."""
    return max(0.0, m_hat - delta_q)


def risk(m_hat, u, e, alpha, beta):
    """Risk score of Eq. (4): (1 - m_hat) + alpha * u + beta * e."""
    return (1.0 - m_hat) + alpha * u + beta * e


def error_features(m_hat, sub_means, sub_counts, entropy_rows, local_rows):
    """(omega, u, omega * H, omega * (1 - L)) of one (unit, candidate)."""
    om = 1.0 - float(m_hat)
    uu = disagreement(sub_means, sub_counts)
    ent = [float(x) for x in entropy_rows]
    loc = [float(x) for x in local_rows]
    H = sum(ent) / len(ent) if ent else 0.0
    L = sum(loc) / len(loc) if loc else 0.0
    return [om, uu, om * H, om * (1.0 - L)]


def predict_error(features, weights):
    """e = sum_k w_k x_k (fp64, in feature order), rounded to fp32."""
    acc = 0.0
    for w, x in zip(weights, features):
        acc = acc + float(np.float32(w)) * float(x)
    return float(np.float32(acc))
