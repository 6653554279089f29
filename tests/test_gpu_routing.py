"""GPU parity of the device side of routing: the calibrated error predictor e (Sec. 3.3,
Eq. 4), the device router (Sec. 3.4, Eqs. 6-8; bit for bit against the fp64 oracle router
and the host router) and the routed attention launch from a device route (equal to one launch
per (pattern, budget) group, which the attention tests check against the oracle)."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import coverage as CV
from oracle import patterns as P
from oracle import router as RT
from paper_2608_29058_amd import _rs
from synth import gen as G

from gpu_helpers import check_close, dev, with_vt
from test_abi_host import GRID, _brank, _random_instance, _t_of

pytestmark = pytest.mark.gpu


def _dev_arrays(cov, nsub, e=None):
    import torch
    out = [torch.from_numpy(np.ascontiguousarray(cov, np.float32)).cuda(),
           torch.from_numpy(np.ascontiguousarray(nsub, np.int32)).cuda()]
    out.append(torch.from_numpy(np.ascontiguousarray(e, np.float32)).cuda() if e is not None else None)
    return out


def test_error_predict_matches_oracle():
    import torch
    r = np.random.default_rng(11)
    U, Cn, rmax = 37, len(GRID), 20
    pb = _rs.ProbeBuffers(U, rmax, 256, 1, Cn)
    cov = r.uniform(0.5, 1.0, (U, Cn, 4)).astype(np.float32)
    nsub = r.integers(0, 7, (U, 3)).astype(np.int32)   # at most 18 <= rmax sampled rows
    nsub[0] = 0                      # a unit without sampled rows
    nsub[1] = [7, 0, 0]              # one non-empty subset: u = 0
    ent = r.random((U, rmax)).astype(np.float32)
    loc = r.random((U, rmax)).astype(np.float32)
    pb.cov.copy_(torch.from_numpy(cov))
    pb.nsub.copy_(torch.from_numpy(nsub))
    pb.entropy.copy_(torch.from_numpy(ent))
    pb.local.copy_(torch.from_numpy(loc))
    w = r.random((4, 4)).astype(np.float32)
    e = torch.full((U, Cn), float("nan"), dtype=torch.float32, device="cuda")
    _rs.rs_error_predict(pb, _rs.make_grid(GRID), Cn, _rs.make_error_model(w), e)
    got = e.cpu().numpy()
    for u in range(U):
        nr = int(nsub[u].sum())
        for c, g in enumerate(GRID):
            if g[0] == RT.DENSE:
                assert got[u, c] == 0.0
                continue
            x = CV.error_features(cov[u, c, 0], [float(v) for v in cov[u, c, 1:]], [int(v) for v in nsub[u]],
                                  ent[u, :nr], loc[u, :nr])
            ref = CV.predict_error(x, w[g[0]])
            assert abs(got[u, c] - ref) <= 1e-6 * max(1.0, abs(ref)), (u, c, got[u, c], ref)


def _check_device_route(cov, nsub, s1, edges, tt, t_probe, T, tau, alpha, beta, dq, e=None):
    import torch
    U = cov.shape[0]
    rb = _rs.RouteDevBuffers(GRID, s1, tt, edges)
    cd, nd, ed = _dev_arrays(cov, nsub, e)
    _rs.rs_route_layer_device(rb, cd, nd, t_probe, T, tau, alpha, beta, dq, e=ed)
    torch.cuda.synchronize()
    got = rb.result()
    t = _t_of(s1, edges, tt)
    e0 = e if e is not None else np.zeros(cov.shape[:2], np.float32)
    ref = RT.route_layer(cov[:, :, 0], cov[:, :, 1:], nsub, e0, t, [g[0] for g in GRID], _brank(GRID), t_probe, T,
                         tau, alpha, beta, dq)
    assert got["choice"] == ref["choice"]
    assert got["groups"] == [(c, us) for c, us in ref["groups"]]
    assert got["total"] == ref["total"] and got["risk"] == ref["risk"]
    assert got["n_fallback"] == ref["n_fallback"] and got["over_budget"] == ref["over_budget"]
    assert np.array_equal(got["R"], ref["R"]) and np.array_equal(got["ML"], ref["ML"])
    st, host = _rs.rs_route_layer(GRID, cov, nsub, s1, tt, edges, t_probe, T, tau, alpha, beta, dq, e=e)
    assert host["choice"] == got["choice"] and host["total"] == got["total"]
    assert host["infeasible"] == got["infeasible"]
    return got


@pytest.mark.parametrize("seed", range(8))
def test_device_router_matches_oracle_bit_for_bit(seed):
    U = [64, 256, 455, 1][seed % 4]
    cov, nsub, s1, edges, tt = _random_instance(seed, U=U)
    t = _t_of(s1, edges, tt)
    dense_total = 30.0 + t[:, 0].sum()
    frac = [1.2, 0.5, 1 / 6.5, 0.05][seed % 4]
    tau = [0.95, 0.9, 0.0, 0.99][seed % 3]
    beta, dq = 0.3 * (seed % 2), 0.01 * (seed % 3)
    e = np.random.default_rng(seed + 100).random(cov.shape[:2]).astype(np.float32)
    _check_device_route(cov, nsub, s1, edges, tt, 30.0, dense_total * frac, tau, 1.0, beta, dq, e=e)


@pytest.mark.parametrize("seed", range(4))
def test_device_router_ties_and_exact_budgets(seed):
    """Equal ratios everywhere (ties to the lowest unit, then candidate) and budgets equal to
    totals at which the solve stops, and their floating-point neighbours."""
    r = np.random.default_rng(2000 + seed)
    U, Cn = 96, len(GRID)
    cov = np.zeros((U, Cn, 4), np.float32)
    base = r.choice([0.875, 0.9375, 0.96875, 1.0], (U, Cn)).astype(np.float32)
    for s in range(4):
        cov[:, :, s] = base
    cov[:, 0, :] = 1.0
    nsub = np.tile(np.array([64, 64, 32], np.int32), (U, 1))
    s1 = r.choice([16384, 32768], U).astype(np.int32)
    edges = np.array([16384, 32768], np.int32)
    tt = np.array([[64.0, 128.0]] + [[float(r.choice([4, 8, 16])), float(r.choice([8, 16, 32]))]
                                     for _ in range(Cn - 1)])
    t = _t_of(s1, edges, tt)
    e0 = np.zeros((U, Cn), np.float32)
    for frac in (0.2, 0.5):
        r0 = RT.route_layer(cov[:, :, 0], cov[:, :, 1:], nsub, e0, t, [g[0] for g in GRID], _brank(GRID), 2.0,
                            2.0 + t[:, 0].sum() * frac, 0.0, 1.0, 0.0, 0.0)
        for T in (r0["total"], np.nextafter(r0["total"], 0.0), np.nextafter(r0["total"], np.inf)):
            for tau in (0.0, 0.95):
                _check_device_route(cov, nsub, s1, edges, tt, 2.0, float(T), tau, 1.0, 0.0, 0.0)


def test_device_router_limits():
    """The largest instances the device router takes: 2048 units x 3 candidates and
    512 units x 9 candidates (4096 moves each), and an infeasible budget."""
    import torch
    grid3 = [GRID[0], GRID[1], GRID[6]]
    for U, grid in ((2048, grid3), (512, GRID)):
        r = np.random.default_rng(U)
        Cn = len(grid)
        cov = np.zeros((U, Cn, 4), np.float32)
        base = r.uniform(0.85, 1.0, (U, Cn)).astype(np.float32)
        for s in range(4):
            cov[:, :, s] = np.clip(base + r.normal(0, 0.01, (U, Cn)), 0, 1) if s else base
        cov[:, 0, :] = 1.0
        nsub = np.tile(np.array([64, 64, 32], np.int32), (U, 1))
        s1 = r.choice([16384 * k for k in range(1, 9)], U).astype(np.int32)
        edges = np.array([16384 * k for k in range(1, 9)], np.int32)
        tt = np.array([[100.0 * (k + 1) for k in range(8)]] +
                      [[float(r.integers(5, 60)) + k for k in range(8)] for _ in range(Cn - 1)])
        t = _t_of(s1, edges, tt)
        for T in (t[:, 0].sum() / 5.0, 1.0):
            rb = _rs.RouteDevBuffers(grid, s1, tt, edges)
            cd, nd, _ = _dev_arrays(cov, nsub)
            _rs.rs_route_layer_device(rb, cd, nd, 10.0, float(T), 0.95, 1.0, 0.0, 0.01)
            torch.cuda.synchronize()
            got = rb.result()
            ref = RT.route_layer(cov[:, :, 0], cov[:, :, 1:], nsub, np.zeros((U, Cn), np.float32), t,
                                 [g[0] for g in grid], _brank(grid), 10.0, float(T), 0.95, 1.0, 0.0, 0.01)
            assert got["choice"] == ref["choice"] and got["total"] == ref["total"]
            assert got["over_budget"] == ref["over_budget"]
            if T == 1.0:
                assert got["infeasible"]


def _layer(n, hq, hkv, d, seed):
    r = np.random.default_rng(seed)
    q = G.bf16_round(r.standard_normal((hq, n, d)).astype(np.float32))
    k = G.bf16_round(r.standard_normal((hkv, n, d)).astype(np.float32) * 1.5)
    v = G.bf16_round(r.standard_normal((hkv, n, d)).astype(np.float32))
    return q, k, v


@pytest.mark.parametrize("vt", [False, True])
def test_routed_attention_equals_group_launches(vt):
    """Every family and budget in one routed call, against one call per group on the same
    probe-built index sets: O and LSE bitwise equal; a unit with an invalid choice is left
    untouched; a few rows checked against the oracle's masked attention (with and without the
    transposed V operand)."""
    import torch
    n, hq, hkv, d, seg = 4096, 4, 2, 128, 1024
    q, k, v = _layer(n, hq, hkv, d, 5)
    qd, kd, vd = dev(q), dev(k), dev(v)
    qkv = _rs.make_qkv(qd, kd, vd)
    if vt:
        qkv, _vt = with_vt(qkv)
    grid = [(0, 0, 0), (1, 64, 256), (1, 64, 1024), (2, 64, 128), (2, 128, 512), (3, 4, 64), (3, 8, 64)]
    g = _rs.make_grid(grid)
    unit_list = [(h, s, s + seg) for s in range(0, n, seg) for h in range(hq)]
    U = len(unit_list)
    units = _rs.make_units([(h, s0, s1, 0, i) for i, (h, s0, s1) in enumerate(unit_list)])
    cfg = _rs.RsProbeCfg(r_rec=64, r_uni=16, r_bnd=8, bs_block=64, local_w=1024,
                         flags=_rs.RS_PROBE_ROWS | _rs.RS_PROBE_BLOCKMEAN)
    pb = _rs.ProbeBuffers(U, 88, n, hq, len(grid), blockmean=True)
    ib = _rs.IndexBuffers(U, n, hq, grid)
    ws = _rs.workspace(max(_rs.rs_probe_workspace_size(qkv, units, U, cfg),
                           _rs.rs_build_indices_workspace_size(pb, g, len(grid))))
    _rs.rs_probe(qkv, units, U, cfg, None, 0, None, ws, pb)
    _rs.rs_build_indices(pb, units, U, g, len(grid), ws, ib)
    choice = [i % len(grid) for i in range(U)]
    choice[5] = -1
    # reference: one call per group
    o1 = torch.full((hq, n, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    l1 = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda")
    for c in range(len(grid)):
        us = [i for i in range(U) if choice[i] == c]
        if not us:
            continue
        gu = _rs.make_units([(unit_list[i][0], unit_list[i][1], unit_list[i][2], c, i) for i in us])
        wsa = _rs.workspace(_rs.rs_attn_workspace_size(qkv, gu, len(us)))
        if grid[c][0] == 0:
            _rs.rs_dense_attn_prefill(qkv, gu, len(us), o1, l1, wsa)
        else:
            _rs.rs_sparse_attn_prefill(qkv, gu, len(us), g, len(grid), ib, o1, l1, wsa)
        torch.cuda.synchronize()
    o2 = torch.full((hq, n, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    l2 = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda")
    ch = torch.tensor(choice, dtype=torch.int32, device="cuda")
    wsr = _rs.workspace(_rs.rs_routed_attn_workspace_size(qkv, units, U))
    _rs.rs_routed_attn_prefill(qkv, units, U, g, len(grid), ib, ch, o2, l2, wsr)
    torch.cuda.synchronize()
    a1, a2 = o1.float().cpu().numpy(), o2.float().cpu().numpy()
    b1, b2 = l1.cpu().numpy(), l2.cpu().numpy()
    assert np.array_equal(a1, a2, equal_nan=True)
    assert np.array_equal(b1, b2, equal_nan=True)
    h5, s05, s15 = unit_list[5]
    assert np.isnan(a2[h5, s05:s15]).all() and np.isnan(b2[h5, s05:s15]).all()
    # oracle on a few rows of an A-shape, a vertical-slash and a block-sparse unit
    grp = hq // hkv
    for i in (1, 3, 6):
        h, s0, s1 = unit_list[i]
        c = choice[i]
        fam, a_, b_ = grid[c]
        rows = np.array([s0, s0 + 1, (s0 + s1) // 2, s1 - 1])
        if fam == 1:
            mask = P.ashape_mask(rows, s1, a_, b_)
        elif fam == 2:
            cl = sum(1 for x in grid[:c] if x[0] == 2)
            cnt = ib.vs_count[i, cl].cpu().numpy()
            V = ib.vs_vsorted[i, cl].cpu().numpy()[:cnt[0]]
            D = ib.vs_dsorted[i, cl].cpu().numpy()[:cnt[1]]
            mask = P.vs_mask(rows, s1, V, D)
        else:
            cl = sum(1 for x in grid[:c] if x[0] == 3)
            srt = ib.bs_sorted[h, cl].cpu().numpy()
            cnt = ib.bs_count[h, cl].cpu().numpy()
            mask = P.bs_mask(rows, s1, 64, lambda bq: srt[bq, :cnt[bq]])
        ref, _ = A.masked_attention(q[h], k[h // grp], v[h // grp], rows, mask)
        check_close(a2[h, rows], ref, f"routed unit {i}")


def test_unit_tables_give_the_same_layer_bit_for_bit():
    """A routed layer whose calls read the unit tables (no per-call uploads) gives bitwise the
    same probe scores, indices, coverage, device route and attention output as the same layer
    with the tables built and uploaded per call."""
    import torch
    from paper_2608_29058_amd.pipeline import RoutedLayer, RouteKnobs
    n, hq, hkv, d, seg = 4096, 4, 2, 128, 1024
    q, k, v = _layer(n, hq, hkv, d, 9)
    qd, kd, vd = dev(q), dev(k), dev(v)
    grid = [(0, 0, 0), (1, 64, 256), (2, 64, 128), (2, 128, 512), (3, 4, 64), (3, 8, 64)]
    edges = np.array([seg * (b + 1) for b in range(n // seg)], np.int32)
    tt = np.array([[e / 1000.0 * (1.0 if g[0] == 0 else 0.2 + 0.03 * c) for e in edges] for c, g in enumerate(grid)])
    snaps = []
    for use_tables in (True, False):
        RL = RoutedLayer(n, hq, hkv, d, seg, grid, r_rec=64, r_uni=16, r_bnd=8, use_tables=use_tables)
        RL.t_table, RL.edges, RL.t_probe_us = tt, edges, 3.0
        RL.knobs = RouteKnobs(T_layer_us=float(tt[0].sum()) * hq / 5, tau=0.9)
        RL.o.fill_(float("nan"))
        assert RL.run(qd, kd, vd, device_route=True) is None
        torch.cuda.synchronize()
        assert (RL.tables is not None) == use_tables
        snap = {"o": RL.o.view(torch.int16).clone(), "choice": RL.rb.choice.clone()}
        for name in ("rows", "subset", "nsub", "row_max", "row_sum", "col", "diag", "lbs", "cov_rows", "cov", "entropy",
                     "local"):
            snap["pb_" + name] = getattr(RL.pb, name).clone()
        for name in ("vs_vsorted", "vs_dsorted", "vs_count", "vs_vbits", "vs_dbits", "bs_rank", "bs_sorted",
                     "bs_count", "bs_bits"):
            snap["ib_" + name] = getattr(RL.ib, name).clone()
        snaps.append(snap)
    for name, a in snaps[0].items():
        b = snaps[1][name]
        if a.is_floating_point():
            a, b = a.view(torch.int32), b.view(torch.int32)
        assert torch.equal(a, b), name
