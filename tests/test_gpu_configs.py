"""GPU parity at the full workload sizes (configs 2-5), in the launch configuration the
benchmark times, on sampled outputs the fp64 oracle computes row by row: four whole
128-row query tiles plus random rows per checked head (rows are independent, so these are
exact checks of those rows), bit-exact index sets when the oracle's rule runs on the GPU's
fp32 scores, and exact routing when the oracle's router runs on the GPU's coverage."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import indices as IX
from oracle import patterns as P
from oracle import probe as PR
from oracle import router as RT
from paper_2608_29058_amd import _rs
from synth import gen as G

from gpu_helpers import check_close

pytestmark = pytest.mark.gpu


def _layer(cfg, layer=0):
    import torch
    t = G.make_layer_torch(cfg, layer, device="cuda")
    torch.cuda.synchronize()
    return t


def _host(t, h):
    return t[h].float().cpu().numpy()


def _sample_rows(s0, s1, seed, n_rand=512, n_tiles=4):
    """``n_tiles`` whole 128-row query tiles of [s0, s1) (first, middle, last and random ones)
    plus ``n_rand`` random rows."""
    r = np.random.default_rng(seed)
    t_lo, t_hi = s0 // 128, (s1 - 1) // 128
    tiles = {t_lo, (s0 + s1) // 256, t_hi}
    while len(tiles) < min(n_tiles, t_hi - t_lo + 1):
        tiles.add(int(r.integers(t_lo, t_hi + 1)))
    rows = set()
    for t in tiles:
        rows.update(range(max(s0, 128 * t), min(s1, 128 * t + 128)))
    rows.update(r.integers(s0, s1, n_rand).tolist())
    return np.array(sorted(rows), dtype=np.int64)


# Key positions that contain every kept key of the given rows (the oracle evaluates the
# pattern's own mask on them: a missing kept key would change the oracle's output, never
# hide a kernel error).
def _cols_dense(rb):
    return np.arange(int(rb.max()) + 1)


def _cols_ashape(sink, w):
    return lambda rb: np.unique(np.concatenate([np.arange(min(sink, int(rb.max()) + 1)),
                                                np.arange(max(0, int(rb.min()) - w + 1), int(rb.max()) + 1)]))


def _cols_vs(V, D):
    V, D = np.asarray(V, np.int64), np.asarray(D, np.int64)

    def f(rb):
        c = np.concatenate([V[V <= rb.max()], (rb[:, None] - D[None, :]).ravel()])
        return np.unique(c[c >= 0])
    return f


def _cols_bs(sel):
    def f(rb):
        blocks = np.unique(np.concatenate([np.asarray(sel(int(b)), np.int64) for b in np.unique(rb // 64)]))
        return (blocks[:, None] * 64 + np.arange(64)[None, :]).ravel()
    return f


def _masked_rows(qh, kh, vh, rows, s1, mask_fn, cols_fn, block=128):
    """fp64 masked attention of ``rows`` (row blocks of 128), with the kept set of each row
    given by ``mask_fn(rows, s1, cols=...)`` on the key positions ``cols_fn(rows)``."""
    out = np.zeros((rows.size, qh.shape[1]))
    for b in range(0, rows.size, block):
        rb = rows[b:b + block]
        cols = cols_fn(rb)
        cols = cols[cols < s1]
        out[b:b + block], _ = A.masked_attention_cols(qh, kh, vh, rb, cols, mask_fn(rb, s1, cols=cols))
    return out


def test_config2_ashape_all_heads():
    """n = 8192, GQA 32/8, every head A-shape (128 sink + 1024 window); every head checked on
    four whole query tiles and 512 random rows."""
    import torch
    t = _layer(2)
    q, k, v = t["q"], t["k"], t["v"]
    n = q.shape[1]
    qkv = _rs.make_qkv(q, k, v)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_ASHAPE, 128, 1024)]
    units = _rs.make_units([(h, 0, n, 1, h) for h in range(32)])
    ws = _rs.workspace(_rs.rs_attn_workspace_size(qkv, units, 32))
    o = torch.full_like(q, float("nan"))
    _rs.rs_sparse_attn_prefill(qkv, units, 32, _rs.make_grid(grid), 2, None, o, None, ws)
    torch.cuda.synchronize()
    assert torch.isfinite(o.float()).all()
    for h in range(32):
        rows = _sample_rows(0, n, h)
        ref = _masked_rows(_host(q, h), _host(k, h // 4), _host(v, h // 4), rows, n,
                           lambda rb, s1, cols: P.ashape_mask(rb, s1, 128, 1024, cols=cols), _cols_ashape(128, 1024))
        check_close(_host(o, h)[rows], ref, f"A-shape 8K h={h}")


@pytest.mark.timeout(900)
def test_config3_probe_vs_and_forced_dense():
    """n = 32768: probe on the last 64 queries, vertical-slash (1000, 6096) on 28 heads,
    heads 0, 5, 10, 15 forced dense.  Every head: scores, bit-exact sets, four whole query
    tiles and 512 random rows."""
    import torch
    t = _layer(3)
    q, k, v = t["q"], t["k"], t["v"]
    n = q.shape[1]
    qkv = _rs.make_qkv(q, k, v)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_VSLASH, 1000, 6096)]
    g = _rs.make_grid(grid)
    dense_heads = [0, 5, 10, 15]
    vs_heads = [h for h in range(32) if h not in dense_heads]
    units = _rs.make_units([(h, 0, n, 1, i) for i, h in enumerate(vs_heads)])
    cfg = _rs.RsProbeCfg(r_rec=64, r_uni=0, r_bnd=0, bs_block=64, local_w=1024, flags=_rs.RS_PROBE_ROWS)
    pb = _rs.ProbeBuffers(len(vs_heads), 64, n, 32)
    ib = _rs.IndexBuffers(len(vs_heads), n, 32, grid)
    ws = _rs.workspace(max(_rs.rs_probe_workspace_size(qkv, units, len(vs_heads), cfg),
                           _rs.rs_attn_workspace_size(qkv, units, len(vs_heads))))
    _rs.rs_probe(qkv, units, len(vs_heads), cfg, None, 0, None, ws, pb)
    _rs.rs_build_indices(pb, units, len(vs_heads), g, 2, ws, ib)
    o = torch.full_like(q, float("nan"))
    _rs.rs_sparse_attn_prefill(qkv, units, len(vs_heads), g, 2, ib, o, None, ws)
    du = _rs.make_units([(h, 0, n) for h in dense_heads])
    _rs.rs_dense_attn_prefill(qkv, du, 4, o, None, ws)
    torch.cuda.synchronize()
    assert torch.isfinite(o.float()).all()
    col = pb.col.cpu().numpy().astype(np.float64)
    diag = pb.diag.cpu().numpy().astype(np.float64)
    for slot, h in enumerate(vs_heads):
        qh, kh, vh = _host(q, h), _host(k, h // 4), _host(v, h // 4)
        ref = PR.probe_unit(qh, kh, 0, n, 64, 0, 0)
        assert np.abs(col[slot] - ref["col"]).max() <= 1e-4 and np.abs(diag[slot] - ref["diag"]).max() <= 1e-4
        V, D, _, _ = IX.vs_indices(col[slot], diag[slot], n, 1000, 6096)
        cnt = ib.vs_count[slot, 0].cpu().numpy()
        assert np.array_equal(ib.vs_vsorted[slot, 0].cpu().numpy()[:cnt[0]], V), h
        assert np.array_equal(ib.vs_dsorted[slot, 0].cpu().numpy()[:cnt[1]], D), h
        rows = _sample_rows(0, n, h)
        out = _masked_rows(qh, kh, vh, rows, n, lambda rb, s1, cols: P.vs_mask(rb, s1, V, D, cols=cols),
                           _cols_vs(V, D))
        check_close(_host(o, h)[rows], out, f"vertical-slash 32K h={h}")
    for h in dense_heads:
        rows = _sample_rows(0, n, h)
        ref = _masked_rows(_host(q, h), _host(k, h // 4), _host(v, h // 4), rows, n,
                           lambda rb, s1, cols: P.dense_mask(rb, s1, cols=cols), _cols_dense)
        check_close(_host(o, h)[rows], ref, f"dense 32K h={h}")


def _config4_layer():
    import torch
    t = _layer(4)
    q, k, v = t["q"], t["k"], t["v"]
    n = q.shape[1]
    qkv = _rs.make_qkv(q, k, v)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, 100, 64)]
    g = _rs.make_grid(grid)
    units = _rs.make_units([(h, 0, n, 1, h) for h in range(32)])
    cfg = _rs.RsProbeCfg(r_rec=0, r_uni=0, r_bnd=0, bs_block=64, local_w=1024, flags=_rs.RS_PROBE_BLOCKMEAN)
    pb = _rs.ProbeBuffers(32, 0, n, 32, blockmean=True)
    ib = _rs.IndexBuffers(32, n, 32, grid)
    ws = _rs.workspace(max(_rs.rs_probe_workspace_size(qkv, units, 32, cfg),
                           _rs.rs_attn_workspace_size(qkv, units, 32)))
    _rs.rs_probe(qkv, units, 32, cfg, None, 0, None, ws, pb)
    _rs.rs_build_indices(pb, units, 32, g, 2, ws, ib)
    o = torch.full_like(q, float("nan"))
    _rs.rs_sparse_attn_prefill(qkv, units, 32, g, 2, ib, o, None, ws)
    torch.cuda.synchronize()
    return q, k, v, pb, ib, o


def _lbs_matrix(lbs_h, nb):
    L = np.full((nb, nb), np.nan)
    off = 0
    for bq in range(nb):
        L[bq, :bq + 1] = lbs_h[off:off + bq + 1]
        off += bq + 1
    return L


@pytest.mark.timeout(900)
def test_config4_block_sparse_128k():
    """n = 131072: block-mean estimator (64-token blocks), top-100 key blocks per query
    block, block-sparse attention on all 32 heads.  Every head: block logits, bit-exact
    selections, four whole query tiles and 512 random rows."""
    import torch
    q, k, v, pb, ib, o = _config4_layer()
    n = q.shape[1]
    nb = n // 64
    assert torch.isfinite(o.float()).all()
    lbs = pb.lbs.cpu().numpy().astype(np.float64)
    for h in range(32):
        qh, kh, vh = _host(q, h), _host(k, h // 4), _host(v, h // 4)
        Lref = PR.block_mean_logits(qh, kh, 64)
        L = _lbs_matrix(lbs[h], nb)
        tri = np.tril_indices(nb)
        np.testing.assert_allclose(L[tri], Lref[tri], atol=2e-4, rtol=1e-4)
        sel, _ = IX.bs_indices(L, 100)
        srt = ib.bs_sorted[h, 0].cpu().numpy()
        cnt = ib.bs_count[h, 0].cpu().numpy()
        for bq in range(nb):
            assert cnt[bq] == sel[bq].size and np.array_equal(srt[bq, :cnt[bq]], sel[bq]), (h, bq)
        rows = _sample_rows(0, n, h)
        out = _masked_rows(qh, kh, vh, rows, n,
                           lambda rb, s1, cols: P.bs_mask(rb, s1, 64, lambda b: sel[b], cols=cols),
                           _cols_bs(lambda b: sel[b]))
        check_close(_host(o, h)[rows], out, f"block-sparse 128K h={h}")


@pytest.mark.timeout(900)
def test_config4_whole_head_every_row():
    """Every one of the 131072 rows of one head of the 128K block-sparse layer against the
    oracle (one query block of 64 rows at a time, over the keys of its selected blocks)."""
    q, k, v, pb, ib, o = _config4_layer()
    n = q.shape[1]
    nb = n // 64
    h = 21
    qh, kh, vh = _host(q, h), _host(k, h // 4), _host(v, h // 4)
    L = _lbs_matrix(pb.lbs[h].cpu().numpy().astype(np.float64), nb)
    sel, _ = IX.bs_indices(L, 100)
    got = _host(o, h)
    out = _masked_rows(qh, kh, vh, np.arange(n), n,
                       lambda rb, s1, cols: P.bs_mask(rb, s1, 64, lambda b: sel[b], cols=cols),
                       _cols_bs(lambda b: sel[b]), block=64)
    check_close(got, out, f"block-sparse 128K head {h}, all rows")


@pytest.mark.timeout(900)
def test_config5_routed_layer_decisions_and_outputs():
    """One 128K layer of the 32-layer workload through the whole pipeline (probe, indices,
    coverage, route with the bench's grid, grouped launches): the route equals the oracle
    router on the GPU's coverage arrays, and every unit matches the masked oracle with the
    GPU's sets on two whole query tiles and 64 random rows."""
    import torch
    from paper_2608_29058_amd.pipeline import RoutedLayer, RouteKnobs
    import bench as B
    t = _layer(5, 3)
    q, k, v = t["q"], t["k"], t["v"]
    RL = RoutedLayer(B.N, B.HQ, B.HKV, B.D, B.SEG, B.GRID)
    edges = np.array([B.SEG * (b + 1) for b in range(B.N // B.SEG)], np.int32)
    # a fixed synthetic latency table (us per unit) shaped like the profiled one
    frac = {0: 1.0, 1: 0.02, 2: 0.25, 3: 0.1}
    tt = np.array([[edges[b] / 131072 * 1200 * (frac[gc[0]] + 0.01 * ci) for b in range(len(edges))]
                   for ci, gc in enumerate(B.GRID)])
    RL.t_table, RL.edges, RL.t_probe_us = tt, edges, 5000.0
    dense_us = sum(tt[0, int(np.searchsorted(edges, u[2]))] for u in RL.unit_list)
    RL.knobs = RouteKnobs(T_layer_us=dense_us / 6.5, tau=0.95)
    RL.o.fill_(float("nan"))
    route = RL.run(q, k, v)
    torch.cuda.synchronize()
    cov = RL.cov_host.numpy().astype(np.float64)
    nsub = RL.nsub_host.numpy()
    tu = np.array([tt[:, int(np.searchsorted(edges, u[2]))] for u in RL.unit_list])
    ref = RT.route_layer(cov[:, :, 0], cov[:, :, 1:], nsub, np.zeros(cov.shape[:2]), tu, [gg[0] for gg in B.GRID],
                         [sum(1 for g2 in B.GRID[:c] if g2[0] == B.GRID[c][0]) for c in range(len(B.GRID))],
                         5000.0, dense_us / 6.5, 0.95, 1.0, 0.0, 0.0)
    assert route["choice"] == ref["choice"] and route["total"] == ref["total"]
    assert torch.isfinite(RL.o.float()).all()
    by_head = {}
    for u, (h, s0, s1) in enumerate(RL.unit_list):
        by_head.setdefault(h, []).append(u)
    for h, us in sorted(by_head.items()):
        qh, kh, vh, oh = _host(q, h), _host(k, h // 4), _host(v, h // 4), _host(RL.o, h)
        for u in us:
            _, s0, s1 = RL.unit_list[u]
            cand = route["choice"][u]
            fam, a_, b_ = B.GRID[cand]
            cl = sum(1 for gg in B.GRID[:cand] if gg[0] == fam)
            if fam == 0:
                mf, cf = (lambda rb, e1, cols: P.dense_mask(rb, e1, cols=cols)), _cols_dense
            elif fam == 1:
                mf = lambda rb, e1, cols: P.ashape_mask(rb, e1, a_, b_, cols=cols)
                cf = _cols_ashape(a_, b_)
            elif fam == 2:
                cnt = RL.ib.vs_count[u, cl].cpu().numpy()
                V = RL.ib.vs_vsorted[u, cl].cpu().numpy()[:cnt[0]]
                Dd = RL.ib.vs_dsorted[u, cl].cpu().numpy()[:cnt[1]]
                mf, cf = (lambda rb, e1, cols: P.vs_mask(rb, e1, V, Dd, cols=cols)), _cols_vs(V, Dd)
            else:
                srt = RL.ib.bs_sorted[h, cl].cpu().numpy()
                cnt = RL.ib.bs_count[h, cl].cpu().numpy()
                sf = lambda bq: srt[bq, :cnt[bq]]
                mf, cf = (lambda rb, e1, cols: P.bs_mask(rb, e1, 64, sf, cols=cols)), _cols_bs(sf)
            rows = _sample_rows(s0, s1, u, 64, 2)
            out = _masked_rows(qh, kh, vh, rows, s1, mf, cf)
            check_close(oh[rows], out, f"routed 128K unit {u} cand {cand}")
    # the launch configuration the benchmark times: device route, one persistent launch per
    # family; the same route and bitwise the same output as the grouped launches above
    o_groups = RL.o.clone()
    RL.o.fill_(float("nan"))
    assert RL.run(q, k, v, device_route=True) is None
    torch.cuda.synchronize()
    assert RL.rb.choice[:RL.nunits].cpu().tolist() == route["choice"]
    assert torch.equal(RL.o.view(torch.int16), o_groups.view(torch.int16))
