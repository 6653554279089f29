"""Pins of the dense / masked attention oracle (Sec. 2.1 Eq. 1, Sec. 3.3 Eq. 5, Sec. 4.2 Eq. 9)."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import patterns as P


def _rand(n, d, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((n, d)), r.standard_normal((n, d)), r.standard_normal((n, d))


def _brute_dense(q, k, v):
    n, d = q.shape
    out = np.zeros((n, d))
    for i in range(n):
        lg = [sum(q[i, t] * k[j, t] for t in range(d)) / math.sqrt(d) for j in range(i + 1)]
        mx = max(lg)
        w = [math.exp(x - mx) for x in lg]
        s = sum(w)
        for j in range(i + 1):
            for t in range(d):
                out[i, t] += w[j] / s * v[j, t]
    return out


def test_dense_matches_brute_force_loops():
    q, k, v = _rand(40, 8, 1)
    np.testing.assert_allclose(A.dense_attention(q, k, v), _brute_dense(q, k, v), atol=1e-12, rtol=0)


def test_dense_matches_torch_sdpa_fp64():
    q, k, v = _rand(300, 64, 2)
    t = lambda x: torch.from_numpy(x)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True)[0, 0].numpy()
    np.testing.assert_allclose(A.dense_attention(q, k, v, block=64), ref, atol=1e-12, rtol=0)


def test_dense_rows_sum_to_one_and_row0_is_v0():
    q, k, v = _rand(100, 16, 3)
    a = A.dense_probs(q, k, np.arange(100), 100)
    np.testing.assert_allclose(a.sum(1), 1.0, atol=1e-13)
    assert np.all(a[np.triu_indices(100, 1)] == 0)
    np.testing.assert_allclose(A.dense_attention(q, k, v)[0], v[0], atol=1e-14)


def test_dense_value_affine_invariance():
    q, k, v = _rand(80, 16, 4)
    o = A.dense_attention(q, k, v)
    np.testing.assert_allclose(A.dense_attention(q, k, 2.5 * v - 0.75), 2.5 * o - 0.75, atol=1e-12)


def test_masked_two_forms_agree_and_causal_mask_is_dense():
    q, k, v = _rand(120, 16, 5)
    rows = np.arange(120)
    mask = np.random.default_rng(6).random((120, 120)) < 0.3
    mask[rows, rows] = True
    o1, _ = A.masked_attention(q, k, v, rows, mask)
    a = A.dense_probs(q, k, rows, 120)
    o2, _, _ = A.renormalized_attention(a, mask & P.dense_mask(rows, 120), v)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    od, _ = A.masked_attention(q, k, v, rows, np.ones((120, 120), bool))
    np.testing.assert_allclose(od, A.dense_attention(q, k, v), atol=1e-12)


def test_masked_single_key_and_constant_values():
    q, k, v = _rand(50, 8, 7)
    rows = np.arange(50)
    mask = np.zeros((50, 50), bool)
    pick = np.random.default_rng(8).integers(0, rows + 1)
    mask[rows, pick] = True
    o, lse = A.masked_attention(q, k, v, rows, mask)
    np.testing.assert_allclose(o, v[pick], atol=1e-14)
    lg = A.logits(q, k, rows, 50)
    np.testing.assert_allclose(lse, lg[rows, pick], atol=1e-12)
    vc = np.tile(np.arange(8.0), (50, 1))
    m2 = np.random.default_rng(9).random((50, 50)) < 0.5
    m2[rows, rows] = True
    o2, _ = A.masked_attention(q, k, vc, rows, m2)
    np.testing.assert_allclose(o2, vc, atol=1e-13)


def test_masked_empty_row_is_zero_with_minus_inf_lse():
    q, k, v = _rand(10, 4, 10)
    mask = np.ones((10, 10), bool)
    mask[3] = False
    o, lse = A.masked_attention(q, k, v, np.arange(10), mask)
    assert np.all(o[3] == 0) and lse[3] == -np.inf and np.isfinite(lse[[0, 1, 2, 4]]).all()


def test_retained_mass_is_lse_difference():
    # m_i = exp(LSE over S_i - LSE over C_i): an identity independent of the probability path
    from scipy.special import logsumexp
    q, k, v = _rand(90, 16, 11)
    rows = np.arange(90)
    mask = np.random.default_rng(12).random((90, 90)) < 0.4
    mask[rows, rows] = True
    mask &= P.dense_mask(rows, 90)
    lg = A.logits(q, k, rows, 90)
    ref = np.exp(logsumexp(np.where(mask, lg, -np.inf), axis=1)
                 - logsumexp(np.where(P.dense_mask(rows, 90), lg, -np.inf), axis=1))
    m = A.retained_mass(A.dense_probs(q, k, rows, 90), mask)
    np.testing.assert_allclose(m, ref, atol=1e-12)


@pytest.mark.parametrize("seed", [13, 14, 15])
def test_certificate_identity_and_bound(seed):
    r = np.random.default_rng(seed)
    n = 128
    q, k, v = r.standard_normal((n, 32)) * 2, r.standard_normal((n, 32)), r.standard_normal((n, 32))
    rows = np.arange(n)
    mask = (r.random((n, n)) < r.uniform(0.05, 0.9)) & P.dense_mask(rows, n)
    mask[rows, rows] = True
    a = A.dense_probs(q, k, rows, n)
    err, bound, l1 = A.certificate(a, mask, v, rows)
    m = A.retained_mass(a, mask)
    np.testing.assert_allclose(l1, 2 * (1 - m), atol=1e-12)
    assert np.all(err <= bound + 1e-12)


def test_e_rel_values():
    o = np.random.default_rng(16).standard_normal((20, 8))
    assert A.e_rel(o, o) == 0.0
    assert abs(A.e_rel(o, np.zeros_like(o)) - 1.0) < 1e-12
    assert abs(A.e_rel(o, 3 * o) - 2.0) < 1e-12


def _brute_masked(q, k, v, rows, keep_fn):
    """Per-element loops: softmax over the kept keys of each row, times V."""
    n, d = q.shape
    out = np.zeros((len(rows), v.shape[1]))
    for r, i in enumerate(rows):
        S = [j for j in range(i + 1) if keep_fn(r, j)]
        if not S:
            continue
        lg = [sum(q[i, t] * k[j, t] for t in range(d)) / math.sqrt(d) for j in S]
        mx = max(lg)
        w = [math.exp(x - mx) for x in lg]
        s = sum(w)
        for jj, j in enumerate(S):
            out[r] += w[jj] / s * v[j]
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_masked_cols_matches_brute_force_and_full_mask(seed):
    """masked_attention_cols over a column subset equals per-element loops and the full-width
    masked_attention with the mask embedded (columns outside ``cols`` dropped); rows left with
    no kept key give 0 and minus infinity."""
    n, d = 50, 8
    q, k, v = _rand(n, d, 40 + seed)
    r = np.random.default_rng(seed)
    rows = np.sort(r.choice(n, 20, replace=False))
    cols = np.sort(r.choice(n, 23, replace=False))
    keep = r.random((rows.size, cols.size)) < 0.6
    keep[0] = False                                   # an empty row
    got, lse = A.masked_attention_cols(q, k, v, rows, cols, keep)
    full = np.zeros((rows.size, n), bool)
    full[:, cols] = keep
    ref, rl = A.masked_attention(q, k, v, rows, full)
    colpos = {int(c): x for x, c in enumerate(cols)}
    brute = _brute_masked(q, k, v, rows, lambda rr, j: j in colpos and keep[rr, colpos[j]])
    np.testing.assert_allclose(got, brute, atol=1e-12, rtol=0)
    np.testing.assert_allclose(got, ref, atol=1e-13, rtol=0)
    assert np.isneginf(lse[0]) and np.all(got[0] == 0)
    np.testing.assert_allclose(lse[1:], rl[1:], atol=1e-12)
