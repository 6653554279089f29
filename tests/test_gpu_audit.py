"""The dense-audited quality measurements (Sec. 3.3 certificate, Eq. 5; Sec. 3.5 calibration of
delta_q; Sec. 4.2 E_rel, Eq. 9) computed from kernel outputs, against the fp64 oracle on the
same index sets: a small routed layer (n = 4096, 4 segments, GQA 4/1) with every sparse
candidate launched over every unit.

* m_true (from the LSE of the sparse and the dense kernel) vs the oracle's retained mass;
* E_rel per unit vs the oracle's masked-vs-dense E_rel;
* the row bound ||O_i - O~_i|| <= 2 (1 - m_i) V_max holds on every row (oracle) and the
  kernel-side check agrees;
* delta_q from calibrate() vs the quantile of the oracle's residuals m_hat - m_true."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import patterns as P
from paper_2608_29058_amd import _rs
from paper_2608_29058_amd import audit as AU
from paper_2608_29058_amd.pipeline import RoutedLayer
from synth import gen as G

pytestmark = pytest.mark.gpu

GRID = [(0, 0, 0), (1, 16, 256), (2, 64, 128), (3, 4, 64), (3, 8, 64)]


def _oracle_mask(RL, c, u, rows, s1):
    fam, a_, b_ = GRID[c]
    h = RL.unit_list[u][0]
    cl = sum(1 for g in GRID[:c] if g[0] == fam)
    if fam == 1:
        return P.ashape_mask(rows, s1, a_, b_)
    if fam == 2:
        cnt = RL.ib.vs_count[u, cl].cpu().numpy()
        V = RL.ib.vs_vsorted[u, cl].cpu().numpy()[:cnt[0]]
        D = RL.ib.vs_dsorted[u, cl].cpu().numpy()[:cnt[1]]
        return P.vs_mask(rows, s1, V, D)
    srt = RL.ib.bs_sorted[h, cl].cpu().numpy()
    cnt = RL.ib.bs_count[h, cl].cpu().numpy()
    return P.bs_mask(rows, s1, 64, lambda bq: srt[bq, :cnt[bq]])


def test_audit_metrics_and_delta_q_match_oracle():
    import torch
    n, hq, hkv, d, seg = 4096, 4, 1, 128, 1024
    r = np.random.default_rng(12)
    q = G.bf16_round((r.standard_normal((hq, n, d)) * 1.2).astype(np.float32))
    k = r.standard_normal((hkv, n, d)).astype(np.float32)
    k[:, :4] += 2.0 * q.mean(axis=(0, 1))
    k = G.bf16_round(k)
    v = G.bf16_round((r.standard_normal((hkv, n, d)) * (1.0 + r.random((hkv, n, 1)))).astype(np.float32))
    qd, kd, vd = (torch.from_numpy(x).to(torch.bfloat16).cuda() for x in (q, k, v))
    RL = RoutedLayer(n, hq, hkv, d, seg, GRID, r_rec=64, r_uni=32, r_bnd=16)
    ref = AU.DenseRef(RL)
    qkv = RL.qkv(qd, kd, vd)
    o_d, lse_d = ref(qkv)
    o_d = o_d.clone()
    lse_d = lse_d.clone()
    RL.probe_and_index(qkv)
    torch.cuda.synchronize()
    m_hat = RL.pb.cov[:, :, 0].double().cpu().numpy()
    lse_c = torch.empty((hq, n), dtype=torch.float32, device="cuda")
    all_u = list(range(RL.nunits))
    resid = []
    dense_rows = {}
    for u, (h, s0, s1) in enumerate(RL.unit_list):
        rows = np.arange(s0, s1)
        a = A.dense_probs(q[h], k[0], rows, s1)
        o_ref = a @ v[0][:s1].astype(np.float64)
        dense_rows[u] = (rows, a, o_ref)
    for c, g in enumerate(GRID):
        if g[0] == _rs.RS_DENSE:
            continue
        RL.run_group(qkv, c, all_u, lse_c)
        torch.cuda.synchronize()
        met = AU.unit_metrics(RL, RL.o, lse_c, o_d, lse_d, vd)
        for u, (h, s0, s1) in enumerate(RL.unit_list):
            rows, a, o_ref = dense_rows[u]
            mask = _oracle_mask(RL, c, u, rows, s1)
            m_rows = A.retained_mass(a, mask)
            ot, _ = A.masked_attention(q[h], k[0], v[0], rows, mask)
            # true kept mass from the two kernels' LSE: fp32 logits of bf16 products, |dm| <= 2e-3
            assert abs(met["m_true"][u] - m_rows.mean()) <= 2e-3, (c, u, met["m_true"][u], m_rows.mean())
            # E_rel of the unit against the oracle's (bf16 outputs on both kernels)
            e_ref = A.e_rel(o_ref, ot)
            assert abs(met["e_rel"][u] - e_ref) <= 5e-3 + 0.05 * e_ref, (c, u, met["e_rel"][u], e_ref)
            # the certificate holds on every row in the oracle, and the kernel-side check agrees
            err, bound, l1 = A.certificate(a, mask, v[0][:s1], rows)
            assert np.all(err <= bound + 1e-12)
            np.testing.assert_allclose(l1, 2.0 * (1.0 - m_rows), atol=1e-12)
            assert met["row_bound_ok"][u] == 1.0, (c, u)
            resid.append(m_hat[u, c] - m_rows.mean())
    # calibrate() on the same layer: the one-sided quantile of m_hat - m_true
    dq, r_gpu, _ = AU.calibrate(RL, ref, [(qd, kd, vd)], 0.95, lambda *a: None)
    dq_ref = max(0.0, float(np.quantile(np.array(resid), 0.95)))
    assert r_gpu.size == len(resid)
    assert abs(dq - dq_ref) <= 3e-3, (dq, dq_ref)
