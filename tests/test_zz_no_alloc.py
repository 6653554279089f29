"""rs_route_layer_device_noalloc (the router's scratch in a fixed library-owned device array)
against rs_route_layer_device (caller workspace) on the same inputs: identical routes, risks,
lower masses, groups, status and totals, bit for bit, on two calls in a row, the second with
fewer units and candidates than the first (the scratch keeps the first call's contents).
Sizes beyond the fixed array are rejected on the host, before any launch."""
import ctypes as C

import numpy as np
import pytest

from paper_2608_29058_amd import _rs

pytestmark = pytest.mark.gpu

GRID = [(0, 0, 0), (1, 128, 1024), (1, 128, 4096), (2, 500, 256), (2, 1000, 512), (2, 2000, 2048),
        (3, 50, 64), (3, 100, 64), (3, 200, 64)]


def _instance(seed, U, grid):
    import torch
    r = np.random.default_rng(seed)
    Cn = len(grid)
    cov = np.zeros((U, Cn, 4), np.float32)
    base = r.choice([0.8, 0.9, 0.95, 0.97, 0.99, 1.0], (U, Cn)).astype(np.float32)
    cov[:, :, 0] = base
    for s in range(3):
        cov[:, :, 1 + s] = np.clip(base + r.normal(0, 0.02, (U, Cn)), 0, 1).astype(np.float32)
    cov[:, 0, :] = 1.0
    nsub = np.tile(np.array([64, 64, 32], np.int32), (U, 1))
    s1 = r.choice([16384 * k for k in range(1, 9)], U).astype(np.int32)
    edges = np.array([16384 * k for k in range(1, 9)], np.int32)
    tt = np.array([[(e / 131072) * (1000.0 if g[0] == 0 else 40.0 + 25.0 * c + 10 * r.random())
                    for e in edges] for c, g in enumerate(grid)])
    T = float(sum(tt[0, int(np.searchsorted(edges, x))] for x in s1)) / 6.5
    return (torch.from_numpy(cov).cuda(), torch.from_numpy(nsub).cuda(), s1, edges, tt, T)


def _route(noalloc, grid, cov, nsub, s1, edges, tt, T):
    import torch
    rb = _rs.RouteDevBuffers(grid, s1, tt, edges)
    for t in (rb.choice, rb.group_cand, rb.group_start, rb.group_units, rb.status):
        t.fill_(-7)
    for t in (rb.risk, rb.m_lower, rb.totals):
        t.fill_(float("nan"))
    fn = _rs.rs_route_layer_device_noalloc if noalloc else _rs.rs_route_layer_device
    fn(rb, cov, nsub, 250.0, T, 0.95, 1.0, 0.0, 0.02)
    torch.cuda.synchronize()
    return {name: getattr(rb, name).clone() for name in ("choice", "group_cand", "group_start", "group_units",
                                                         "risk", "m_lower", "status", "totals")}


def test_noalloc_route_equals_workspace_route_twice():
    import torch
    calls = [(256, GRID, 1), (40, GRID[:1] + GRID[3:6] + GRID[7:], 2)]   # the second call smaller
    for U, grid, seed in calls:
        args = _instance(seed, U, grid)
        want = _route(False, grid, *args)
        got = _route(True, grid, *args)
        for name in want:
            a, b = want[name], got[name]
            if a.is_floating_point():
                a, b = a.view(torch.uint8), b.view(torch.uint8)
            assert torch.equal(a, b), (U, name)
        assert int(got["status"][0]) >= 1


def test_noalloc_route_rejects_sizes_beyond_its_scratch():
    L = _rs.lib()
    grid = _rs.make_grid(GRID)
    out = _rs.RsRouteDevOut(choice=16, group_cand=16, group_start=16, group_units=16, risk=16, m_lower=16,
                            status=16, totals=16)
    cfg = _rs.RsRouteCfg(T_layer_us=1.0, tau=0.9, alpha=1.0, beta=0.0, delta_q=0.0)
    for U in (2049, 1024):     # too many units; too many moves (1024 x 8 > 4096)
        rin = _rs.RsRouteIn(nunits=U, ncand=len(GRID), grid=C.cast(grid, C.c_void_p), cov=16, nsub=16, s1=16,
                            t_table=16, bucket_edge=16, nbucket=1)
        st = L.rs_route_layer_device_noalloc(C.byref(rin), C.byref(cfg), C.byref(out), None)
        assert st == _rs.RS_ERR_UNSUPPORTED, U
