"""Pins of the probe oracle (Sec. 3.1, Sec. 3.2 Eq. 3)."""
import math

import numpy as np
import torch

from oracle import probe as PR


def _rand(n, d, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((n, d)), r.standard_normal((n, d))


def test_sample_rows_disjoint_sorted_in_segment():
    for s0, s1, rr, ru, rb in [(0, 2048, 64, 0, 0), (16384, 32768, 64, 64, 32), (0, 100, 64, 64, 32),
                               (0, 50, 64, 8, 8), (100, 300, 16, 300, 4)]:
        R, U, B = PR.sample_rows(s0, s1, rr, ru, rb)
        allr = np.concatenate([R, U, B])
        assert np.unique(allr).size == allr.size
        assert allr.size == 0 or (allr.min() >= s0 and allr.max() < s1)
        assert np.array_equal(R, np.arange(max(s0, s1 - rr), s1))
        assert np.all(np.diff(U) > 0) and np.all(np.diff(B) > 0)
    R, U, B = PR.sample_rows(0, 2048, 64, 0, 0)
    assert R.size == 64 and U.size == 0 and B.size == 0
    R, U, B = PR.sample_rows(16384, 32768, 64, 64, 32)
    assert U.size == 64 and B.size == 32 and B[0] == 16384
    assert U[0] == 16384 + 16384 // 128


def test_col_diag_against_torch_attention_matrix():
    n, d = 150, 16
    q, k = _rand(n, d, 1)
    res = PR.probe_unit(q, k, 0, n, r_rec=n, r_uni=0, r_bnd=0)
    lg = torch.from_numpy(q) @ torch.from_numpy(k).T / math.sqrt(d)
    lg = lg.masked_fill(torch.triu(torch.ones(n, n, dtype=torch.bool), 1), float("-inf"))
    a = torch.softmax(lg, dim=1).numpy()
    np.testing.assert_allclose(res["col"], a.sum(0), atol=1e-12)
    diag = np.array([np.trace(a, offset=-dl) for dl in range(n)])
    np.testing.assert_allclose(res["diag"], diag, atol=1e-12)


def test_col_diag_invariants_and_loops():
    n, d = 300, 8
    q, k = _rand(n, d, 2)
    res = PR.probe_unit(q, k, 100, 260, r_rec=40, r_uni=10, r_bnd=5)
    nR = int((res["subset"] == PR.SUB_R).sum())
    assert nR == 40
    assert abs(res["col"].sum() - nR) < 1e-10 and abs(res["diag"].sum() - nR) < 1e-10
    assert res["col"].shape == (260,)
    # loop definition of diag on the recent rows
    diag = np.zeros(260)
    for r, i in enumerate(res["rows"]):
        if res["subset"][r] != PR.SUB_R:
            continue
        for dl in range(i + 1):
            diag[dl] += res["a"][r, i - dl]
    np.testing.assert_allclose(res["diag"], diag, atol=1e-13)


def test_block_mean_logits_against_loops():
    n, d, B = 200, 8, 64
    q, k = _rand(n, d, 3)
    L = PR.block_mean_logits(q, k, B)
    nb = 4
    for bq in range(nb):
        for bk in range(nb):
            if bk > bq:
                assert np.isnan(L[bq, bk])
                continue
            qm = [sum(q[t, c] for t in range(bq * B, min(n, bq * B + B))) / len(range(bq * B, min(n, bq * B + B)))
                  for c in range(d)]
            km = [sum(k[t, c] for t in range(bk * B, min(n, bk * B + B))) / len(range(bk * B, min(n, bk * B + B)))
                  for c in range(d)]
            assert abs(L[bq, bk] - sum(a * b for a, b in zip(qm, km)) / math.sqrt(d)) < 1e-12


def test_descriptors_on_uniform_attention():
    # q = 0 makes every visible key equally likely: entropy of full blocks normalises to 1
    n, d = 640, 4
    q = np.zeros((n, d))
    k = np.random.default_rng(4).standard_normal((n, d))
    rows = np.array([63, 127, 255, 639, 600])
    from oracle.attention import dense_probs
    a = dense_probs(q, k, rows, n)
    ent, loc = PR.row_descriptors(a, rows, local_w=100)
    np.testing.assert_allclose(ent[:4], [0.0, 1.0, 1.0, 1.0], atol=1e-12)
    np.testing.assert_allclose(loc, np.minimum(rows + 1, 100) / (rows + 1), atol=1e-12)
