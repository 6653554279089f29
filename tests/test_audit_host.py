"""Host checks of the dense-audit helpers (Sec. 3.3 certificate, Sec. 4.2 E_rel) against the
fp64 oracle: the helpers take the kernels' LSE and outputs, so here they are fed the
oracle's exact masked attention and must reproduce the oracle's retained mass, E_rel and
certificate."""
from types import SimpleNamespace

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import patterns as P
from paper_2608_29058_amd import audit as AU


def _layer(seed=0, n=256, hq=2, d=16, seg=64):
    r = np.random.default_rng(seed)
    q = r.standard_normal((hq, n, d)) * 1.5
    k = r.standard_normal((1, n, d))
    v = r.standard_normal((1, n, d)) * (1.0 + r.random((1, n, 1)))
    RL = SimpleNamespace(n=n, hq=hq, hkv=1, d=d, nunits=hq * (n // seg),
                         unit_list=[(h, s * seg, (s + 1) * seg) for s in range(n // seg) for h in range(hq)])
    rows = np.arange(n)
    out = dict(q=q, k=k, v=v, RL=RL, rows=rows, o=[], lse=[], ot=[], lse_s=[], a=[], mask=[])
    for h in range(hq):
        a = A.dense_probs(q[h], k[0], rows, n)
        od, lse_d = A.masked_attention(q[h], k[0], v[0], rows, P.dense_mask(rows, n))
        mask = P.ashape_mask(rows, n, 4, 16)
        ot, lse_s = A.masked_attention(q[h], k[0], v[0], rows, mask)
        for key, val in (("o", od), ("lse", lse_d), ("ot", ot), ("lse_s", lse_s), ("a", a), ("mask", mask)):
            out[key].append(val)
    return out


def _t(x):
    return torch.tensor(np.asarray(x), dtype=torch.float64)


def test_mass_from_lse_difference_is_retained_mass():
    L = _layer(1)
    m_row, m_unit = AU.true_mass(L["RL"], _t(L["lse_s"]), _t(L["lse"]))
    for h in range(2):
        ref = A.retained_mass(L["a"][h], L["mask"][h])
        assert np.abs(m_row[h].numpy() - ref).max() <= 1e-12
    # unit order: segment-major, head-minor; unit mass is the mean over its rows
    for u, (h, s0, s1) in enumerate(L["RL"].unit_list):
        ref = A.retained_mass(L["a"][h], L["mask"][h])[s0:s1].mean()
        assert abs(float(m_unit[u]) - ref) <= 1e-12


def test_vmax_is_prefix_max_of_value_norms():
    L = _layer(2)
    vm = AU.vmax_units(L["RL"], _t(L["v"]))
    norms = np.linalg.norm(L["v"][0], axis=1)
    for s in range(4):
        assert abs(float(vm[0, s]) - norms[:64 * (s + 1)].max()) <= 1e-5
        assert float(vm[1, s]) == float(vm[0, s])   # both query heads share the one K/V head


def test_unit_metrics_match_oracle_certificate_and_e_rel():
    L = _layer(3)
    met = AU.unit_metrics(L["RL"], _t(L["ot"]), _t(L["lse_s"]), _t(L["o"]), _t(L["lse"]), _t(L["v"]))
    for u, (h, s0, s1) in enumerate(L["RL"].unit_list):
        ref = A.e_rel(L["o"][h][s0:s1], L["ot"][h][s0:s1])
        assert abs(met["e_rel"][u] - ref) <= 1e-5 * max(ref, 1e-3)
        err, bound, l1 = A.certificate(L["a"][h][s0:s1], L["mask"][h][s0:s1], L["v"][0], np.arange(s0, s1))
        assert abs(met["mean_err"][u] - err.mean()) <= 1e-5
        assert met["row_bound_ok"][u] == 1.0
        # the unit-level form: mean error under 2 (1 - mean m) V_max(s1)
        assert met["mean_err"][u] <= 2.0 * (1.0 - met["m_true"][u]) * met["vmax"][u] + 1e-9
    assert met["e_rel"].max() > 0.0


def test_identical_outputs_give_zero_error():
    L = _layer(4)
    o = _t(L["o"])
    met = AU.unit_metrics(L["RL"], o, _t(L["lse"]), o, _t(L["lse"]), _t(L["v"]))
    assert np.all(met["e_rel"] == 0.0) and np.all(met["mean_err"] == 0.0)
    assert np.allclose(met["m_true"], 1.0) and np.all(met["row_bound_ok"] == 1.0)


def test_row_bound_check_rejects_a_planted_error():
    L = _layer(5)
    ot = np.array(L["ot"])
    ot[1, 200] += 10.0 * np.linalg.norm(L["v"][0], axis=1).max()
    met = AU.unit_metrics(L["RL"], _t(ot), _t(L["lse_s"]), _t(L["o"]), _t(L["lse"]), _t(L["v"]))
    u = [i for i, (h, s0, s1) in enumerate(L["RL"].unit_list) if h == 1 and s0 <= 200 < s1][0]
    assert met["row_bound_ok"][u] == pytest.approx(63 / 64)
    assert all(met["row_bound_ok"][i] == 1.0 for i in range(len(L["RL"].unit_list)) if i != u)


def test_predicted_flops_table_prices_nominal_pairs():
    RL = SimpleNamespace(d=128, ncand=4, unit_list=[(0, 0, 16384)],
                         grid=[(0, 0, 0), (1, 128, 1024), (2, 500, 256), (3, 50, 64)])
    edges = np.array([16384, 32768], np.int32)
    t = AU.flops_table(RL, edges, 1.0)
    dense = lambda s0, s1: (s1 * (s1 + 1) - s0 * (s0 + 1)) // 2
    assert t[0, 0] == 4 * 128 * dense(0, 16384) and t[0, 1] == 4 * 128 * dense(16384, 32768)
    # past the cap every row keeps exactly sink + window (A-shape) or k blocks (block-sparse)
    assert t[1, 1] == 4 * 128 * 16384 * (128 + 1024)
    assert t[2, 1] == 4 * 128 * 16384 * 756
    assert t[3, 1] == 4 * 128 * 16384 * 3200
    rows1 = np.arange(1, 16385, dtype=np.float64)
    assert t[1, 0] == 4 * 128 * np.minimum(rows1, 1152).sum()


def test_bf16_allowance_formula():
    assert AU.bf16_allowance(64.0, 1.0, 3.0) == pytest.approx(1.0 + 4.0 / 512)
