"""Pins of coverage, risk and the router (Sec. 3.2-3.4, Eqs. 4, 6-8)."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import attention as A
from oracle import coverage as CV
from oracle import patterns as P
from oracle import probe as PR
from oracle import router as RT

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_coverage_all_rows_equals_exact_mean_retained_mass():
    r = np.random.default_rng(1)
    n, d = 128, 16
    q, k = r.standard_normal((n, d)), r.standard_normal((n, d))
    res = PR.probe_unit(q, k, 0, n, r_rec=n, r_uni=0, r_bnd=0)
    mask = P.ashape_mask(res["rows"], n, 4, 16)
    m = CV.row_coverage(res["a"], mask)
    # retained mass from logsumexp of masked vs causal logits, independent of the probabilities
    from scipy.special import logsumexp
    lg = A.logits(q, k, np.arange(n), n)
    ref = np.exp(logsumexp(np.where(mask, lg, -np.inf), 1) - logsumexp(np.where(P.dense_mask(np.arange(n), n), lg, -np.inf), 1))
    mh, means, counts = CV.subset_means(m, res["subset"])
    assert abs(mh - ref.mean()) < 1e-12 and counts == [n, 0, 0]
    assert CV.disagreement(means, counts) == 0.0


def test_disagreement_and_risk_by_hand():
    assert CV.disagreement([0.9, 0.7, 0.8], [4, 2, 1]) == pytest.approx(0.2)
    assert CV.disagreement([0.9, 0.1, 0.8], [4, 0, 1]) == pytest.approx(0.1)
    assert CV.risk(0.9, 0.1, 0.0, 1.0, 0.0) == pytest.approx(0.2)
    assert CV.risk(0.9, 0.1, 0.5, 1.0, 0.2) == pytest.approx(0.3)
    assert CV.lower_mass(0.03, 0.05) == 0.0


def _exact_mckp(R, t, t_probe, T):
    U, C = R.shape
    best = None
    for ch in itertools.product(range(C), repeat=U):
        tot = t_probe + sum(t[u, c] for u, c in enumerate(ch))
        if tot <= T:
            rk = sum(R[u, c] for u, c in enumerate(ch))
            if best is None or rk < best:
                best = rk
    return best


@pytest.mark.parametrize("seed", range(40))
def test_greedy_vs_exhaustive_mckp(seed):
    r = np.random.default_rng(seed)
    U, C = int(r.integers(1, 6)), int(r.integers(2, 5))
    fam = [RT.DENSE] + [int(x) for x in r.integers(1, 4, C - 1)]
    R = r.random((U, C)) * 0.5
    R[:, 0] = 0.0
    t = r.uniform(1, 10, (U, C))
    t[:, 0] = r.uniform(10, 20, U)
    tp = 1.0
    T = tp + t.min(1).sum() + r.uniform(-3, 0.6) * U * 5
    choice, over = RT.greedy(R, t, [0] * U, tp, T)
    exact = _exact_mckp(R, t, tp, T)
    assert over == (exact is None)
    if exact is not None:
        assert RT.total_time(t, choice, tp) <= T
        assert sum(R[u, c] for u, c in enumerate(choice)) >= exact - 1e-12


def test_router_hand_worked_example():
    with open(os.path.join(GOLD, "router_two_units.json")) as f:
        g = json.load(f)
    out = RT.route_layer(np.array(g["mhat"]), np.array(g["msub"]), np.array(g["nsub"]),
                         np.zeros((2, 3)), np.array(g["t"]), g["fam"], g["brank"], g["t_probe"],
                         g["T_layer"], g["tau"], g["alpha"], 0.0, g["delta_q"])
    assert out["choice"] == g["expect_choice"]
    assert out["total"] == pytest.approx(g["expect_total"])
    assert out["over_budget"] == g["expect_over_budget"]
    assert out["n_fallback"] == g["expect_n_fallback"]


def test_tau_expands_then_falls_back():
    fam = [RT.DENSE, RT.VSLASH, RT.VSLASH, RT.VSLASH]
    brank = [0, 0, 1, 2]
    ML = np.array([[1, 0.5, 0.96, 0.99], [1, 0.5, 0.6, 0.7], [1, 0.97, 0.98, 0.99]])
    t = np.ones((3, 4))
    out, nfb = RT.expand_or_fallback([1, 1, 1], fam, brank, ML, 0.95, 0, t)
    assert out == [2, 0, 1] and nfb == 1


def test_tau_switches_to_cheapest_passing_sparse_candidate():
    # A-shape fails tau at both budgets; vertical-slash (two budgets) and block-sparse pass:
    # the cheaper passing candidate is taken, dense only when no sparse candidate passes
    fam = [RT.DENSE, RT.ASHAPE, RT.ASHAPE, RT.VSLASH, RT.VSLASH, RT.BSPARSE]
    brank = [0, 0, 1, 0, 1, 0]
    ML = np.array([[1, 0.5, 0.6, 0.96, 0.99, 0.97],
                   [1, 0.5, 0.6, 0.90, 0.99, 0.97],
                   [1, 0.5, 0.6, 0.90, 0.91, 0.92]])
    t = np.array([[100, 2, 5, 30, 40, 20],
                  [100, 2, 5, 30, 40, 50],
                  [100, 2, 5, 30, 40, 50]], dtype=float)
    out, nfb = RT.expand_or_fallback([1, 1, 1], fam, brank, ML, 0.95, 0, t)
    assert out == [5, 4, 0] and nfb == 1


def test_grouping():
    assert RT.group([2, 0, 2, 1, 0], 4) == [(0, [1, 4]), (1, [3]), (2, [0, 2])]


def test_error_predictor_by_hand_and_invariants():
    """The calibrated error predictor e of Eq. 4 (features and model are a reading; see the
    module docstring): a hand-worked case, and the invariants that pin the reading: zero
    omitted mass and no disagreement give 0, and e never decreases when the omitted mass,
    the disagreement, the entropy grow or the local mass shrinks."""
    # m_hat 0.9, subset means (0.95, 0.85, 0.9) -> u = 0.1; mean entropy 0.5, mean local 0.8
    x = CV.error_features(0.9, [0.95, 0.85, 0.9], [64, 64, 32], [0.25, 0.75], [0.7, 0.9])
    assert np.allclose(x, [0.1, 0.1, 0.05, 0.02], atol=1e-15)
    assert abs(CV.predict_error(x, [1.0, 2.0, 4.0, 8.0]) - 0.66) < 1e-7
    # an empty subset does not enter u; no sampled rows give H = L = 0
    x = CV.error_features(0.8, [0.7, 0.0, 0.9], [10, 0, 5], [], [])
    assert np.allclose(x, [0.2, 0.2, 0.0, 0.2], atol=1e-15)
    assert CV.predict_error(CV.error_features(1.0, [1.0, 1.0, 1.0], [1, 1, 1], [0.9], [0.1]), [3, 3, 3, 3]) == 0.0
    r = np.random.default_rng(7)
    for _ in range(200):
        w = r.random(4)
        mh, mh2 = sorted(r.random(2))[::-1]  # mh >= mh2: more omitted mass in the second
        subs = list(r.random(3))
        ent, loc = list(r.random(5)), list(r.random(5))
        e1 = CV.predict_error(CV.error_features(mh, subs, [3, 3, 3], ent, loc), w)
        e2 = CV.predict_error(CV.error_features(mh2, subs, [3, 3, 3], ent, loc), w)
        assert e2 >= e1
        e3 = CV.predict_error(CV.error_features(mh, subs, [3, 3, 3], [x + 0.1 for x in ent],
                                                [x - 0.1 for x in loc]), w)
        assert e3 >= e1
        assert CV.predict_error(CV.error_features(mh, subs, [3, 3, 3], ent, loc), [0, 0, 0, 0]) == 0.0
