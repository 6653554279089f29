"""GPU parity of the kernel instantiations the C ABI can reach beyond the benchmark's path,
against the fp64 oracle:

* sparse attention (A-shape, block-sparse, vertical-slash; Sec. 2.1 mask semantics) at head
  dim 64 and with fp32 inputs (rounded to bf16 on load), with and without the transposed V;
* probe scores, block-mean logits and coverage (Sec. 3.1-3.3) at head dim 64 / fp32;
* the coverage pass on grids with more than two A-shape or three vertical-slash /
  block-sparse candidates (the variants that read the index bitmaps inside the key loop),
  up to the 16-candidate limit, including a 16K-row segment at the end of a 128K prefix;
* vertical-slash selection when the largest slash budget exceeds what the selection keeps
  in LDS (every budget then selected from the whole array);
* bitwise repeatability of rs_probe (scores and coverage), rs_build_indices and
  rs_route_layer_device.

Tolerances as everywhere: probe values |delta| <= 1e-4, index sets bit-exact on the GPU's
fp32 scores, attention max-abs 2e-2 / rel-F 1e-2."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import coverage as CV
from oracle import indices as IX
from oracle import patterns as P
from oracle import probe as PR
from oracle import router as RT
from paper_2608_29058_amd import _rs
from synth import gen as G

from gpu_helpers import check_close, dev, fill_bs, fill_vs, out_tensor, with_vt, words_of

pytestmark = pytest.mark.gpu

DENSE, ASHAPE, VSLASH, BSPARSE = _rs.RS_DENSE, _rs.RS_ASHAPE, _rs.RS_VSLASH, _rs.RS_BSPARSE


def _inputs(n, hq, hkv, d, seed, dtype="bf16", kscale=1.0):
    r = np.random.default_rng(seed)
    q = r.standard_normal((hq, n, d)).astype(np.float32)
    k = (r.standard_normal((hkv, n, d)) * kscale).astype(np.float32)
    v = r.standard_normal((hkv, n, d)).astype(np.float32)
    k[:, :4] += 2.5 * q.mean(axis=(0, 1))          # a mild sink the probe can find
    if dtype == "bf16":
        q, k, v = G.bf16_round(q), G.bf16_round(k), G.bf16_round(v)
    return q, k, v


# ---- sparse attention at head dim 64 and with fp32 inputs ---------------------------------

def _run_sparse(q, k, v, units, grid, ib, dtype, vt):
    import torch
    hq, n, d = q.shape
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    qkv = _rs.make_qkv(qd, kd, vd)
    keep = None
    if vt:
        qkv, keep = with_vt(qkv)
    u = _rs.make_units(units)
    ws = _rs.workspace(_rs.rs_attn_workspace_size(qkv, u, len(units)))
    o = out_tensor(hq, n, d)
    lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda")
    _rs.rs_sparse_attn_prefill(qkv, u, len(units), _rs.make_grid(grid), len(grid), ib, o, lse, ws)
    torch.cuda.synchronize()
    del keep
    return o.float().cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("fam", ["ashape", "bs", "vs"])
@pytest.mark.parametrize("d,dtype", [(64, "bf16"), (128, "f32"), (64, "f32")])
@pytest.mark.parametrize("vt", [False, True])
def test_sparse_families_at_head_dim_64_and_fp32(fam, d, dtype, vt):
    n, hq, hkv = 1900, 4, 2           # ragged last tile, GQA group of 2
    q, k, v = _inputs(n, hq, hkv, d, seed=d + (7 if dtype == "f32" else 0) + len(fam), dtype=dtype)
    g = hq // hkv
    r = np.random.default_rng(d)
    units = [(0, 0, n, 1, 0), (1, 300, 1500, 1, 1), (2, 640, n, 1, 2), (3, 0, 777, 1, 3)]
    if fam == "ashape":
        grid, ib = [(DENSE, 0, 0), (ASHAPE, 100, 300)], None
        masks = {u[0]: (lambda rb, s1: P.ashape_mask(rb, s1, 100, 300)) for u in units}
    elif fam == "bs":
        grid = [(DENSE, 0, 0), (BSPARSE, 7, 64)]
        ib = _rs.IndexBuffers(len(units), n, hq, grid)
        nb = (n + 63) // 64
        masks = {}
        for h in range(hq):
            sel = [sorted(set(r.permutation(bq)[:6].tolist()) | {bq}) for bq in range(nb)]
            fill_bs(ib, h, 0, sel)
            masks[h] = (lambda rb, s1, sel=sel: P.bs_mask(rb, s1, 64, lambda b: sel[b]))
    else:
        grid = [(DENSE, 0, 0), (VSLASH, 90, 160)]
        ib = _rs.IndexBuffers(len(units), n, hq, grid)
        masks = {}
        for slot, (h, s0, s1, _, _) in enumerate(units):
            V = np.sort(r.choice(s1, 90, replace=False))
            D = np.unique(np.concatenate([np.arange(64), r.choice(s1, 96, replace=False)]))[:160]
            fill_vs(ib, slot, 0, V, D)
            masks[h] = (lambda rb, s1, V=V, D=D: P.vs_mask(rb, s1, V, D))
    o, lse = _run_sparse(q, k, v, units, grid, ib, dtype, vt)
    # fp32 inputs are rounded to bf16 on load: outputs are checked against the oracle on the
    # fp32 values, the log-sum-exp (which a few-key row carries the logit rounding of in
    # full) against the oracle on the rounded values the kernel computes with
    qr, kr = (G.bf16_round(q), G.bf16_round(k)) if dtype == "f32" else (q, k)
    for h, s0, s1, _, _ in units:
        rows = np.arange(s0, s1)
        ref, _ = A.masked_attention(q[h], k[h // g], v[h // g], rows, masks[h](rows, s1))
        check_close(o[h, s0:s1], ref, f"{fam} d={d} {dtype} h={h}")
        _, rl = A.masked_softmax(qr[h], kr[h // g], rows, masks[h](rows, s1))
        np.testing.assert_allclose(lse[h, s0:s1], rl, atol=4e-3, rtol=1e-4)


# ---- probe, block-mean and coverage: head dim 64, fp32, and the general coverage grids -------

def _probe_scores(q, k, v, units, rcfg, dtype):
    import torch
    hq, n, d = q.shape
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    qkv = _rs.make_qkv(qd, kd, vd)
    u = _rs.make_units(units)
    cfg = _rs.RsProbeCfg(r_rec=rcfg[0], r_uni=rcfg[1], r_bnd=rcfg[2], bs_block=64, local_w=1024,
                         flags=_rs.RS_PROBE_ROWS | _rs.RS_PROBE_BLOCKMEAN)
    pb = _rs.ProbeBuffers(len(units), sum(rcfg), n, hq, 0, blockmean=True)
    ws = _rs.workspace(_rs.rs_probe_workspace_size(qkv, u, len(units), cfg))
    _rs.rs_probe(qkv, u, len(units), cfg, None, 0, None, ws, pb)
    torch.cuda.synchronize()
    return dict(keep=(qd, kd, vd), qkv=qkv, u=u, cfg=cfg, pb=pb, ws=ws)


def _coverage(res, units, grid, rcfg):
    """Index sets for ``grid`` from the scores call, then the coverage call."""
    import torch
    pb = res["pb"]
    n, hq = pb.c.n, pb.c.hq
    g = _rs.make_grid(grid)
    ib = _rs.IndexBuffers(len(units), n, hq, grid)
    ws = _rs.workspace(_rs.rs_build_indices_workspace_size(pb, g, len(grid)))
    _rs.rs_build_indices(pb, res["u"], len(units), g, len(grid), ws, ib)
    pc = _rs.ProbeBuffers(len(units), sum(rcfg), n, hq, len(grid), blockmean=False)
    for name in ("rows", "subset", "nsub"):
        getattr(pc, name).copy_(getattr(pb, name))
    _rs.rs_probe(res["qkv"], res["u"], len(units), res["cfg"], g, len(grid), ib, res["ws"], pc)
    torch.cuda.synchronize()
    return ib, pc


def _lbs_matrix(lbs_h, nb):
    L = np.full((nb, nb), np.nan)
    off = 0
    for bq in range(nb):
        L[bq, :bq + 1] = lbs_h[off:off + bq + 1]
        off += bq + 1
    return L


def _check_coverage(q, k, units, grid, rcfg, ib, pc, group):
    """m_i(c) of every sampled row and candidate, subset means and descriptors vs the oracle,
    with the GPU's index sets (which are checked bit-exact elsewhere)."""
    cov_rows, cov = pc.cov_rows.cpu().numpy(), pc.cov.cpu().numpy()
    fam = [gg[0] for gg in grid]
    cl = [sum(1 for g2 in grid[:c] if g2[0] == grid[c][0]) for c in range(len(grid))]
    for ui, (h, s0, s1) in enumerate(units):
        ref = PR.probe_unit(q[h], k[h // group], s0, s1, *rcfg)
        rows, a = ref["rows"], ref["a"]
        nr = rows.size
        np.testing.assert_allclose(pc.entropy[ui, :nr].cpu().numpy(), ref["entropy"], atol=1e-3)
        np.testing.assert_allclose(pc.local[ui, :nr].cpu().numpy(), ref["local"], atol=1e-4)
        for c, gg in enumerate(grid):
            if fam[c] == DENSE:
                assert np.all(cov_rows[ui, c, :nr] == 1.0)
                continue
            if fam[c] == ASHAPE:
                m = P.ashape_mask(rows, s1, gg[1], gg[2])
            elif fam[c] == VSLASH:
                cnt = ib.vs_count[ui, cl[c]].cpu().numpy()
                V = ib.vs_vsorted[ui, cl[c]].cpu().numpy()[:cnt[0]]
                D = ib.vs_dsorted[ui, cl[c]].cpu().numpy()[:cnt[1]]
                m = P.vs_mask(rows, s1, V, D)
            else:
                srt = ib.bs_sorted[h, cl[c]].cpu().numpy()
                cnt = ib.bs_count[h, cl[c]].cpu().numpy()
                m = P.bs_mask(rows, s1, 64, lambda bq: srt[bq, :cnt[bq]])
            mi = A.retained_mass(a, m)
            err = np.abs(cov_rows[ui, c, :nr] - mi).max()
            assert err <= 1e-4, (ui, c, gg, err)
            mh, means, _ = CV.subset_means(mi, ref["subset"])
            assert abs(cov[ui, c, 0] - mh) <= 1e-4, (ui, c)
            assert np.abs(cov[ui, c, 1:] - np.array(means)).max() <= 1e-4, (ui, c)


@pytest.mark.parametrize("d,dtype", [(64, "bf16"), (128, "f32"), (64, "f32")])
def test_probe_blockmean_and_coverage_at_head_dim_64_and_fp32(d, dtype):
    n, hq, hkv = 2300, 4, 2
    rcfg = (64, 16, 8)
    q, k, v = _inputs(n, hq, hkv, d, seed=31 + d, dtype=dtype, kscale=1.5)
    units = [(0, 0, n), (1, 0, n), (3, 700, 2100)]
    res = _probe_scores(q, k, v, units, rcfg, dtype)
    # fp32 inputs are rounded to bf16 on load: the probe computes the scores of the rounded
    # values, which the oracle is given (the fp32-vs-bf16 difference is the input rounding,
    # not the probe's arithmetic)
    if dtype == "f32":
        q, k = G.bf16_round(q), G.bf16_round(k)
    pb = res["pb"]
    g = hq // hkv
    col, diag = pb.col.cpu().numpy(), pb.diag.cpu().numpy()
    for ui, (h, s0, s1) in enumerate(units):
        ref = PR.probe_unit(q[h], k[h // g], s0, s1, *rcfg)
        assert np.abs(col[ui, :s1] - ref["col"]).max() <= 1e-4
        assert np.abs(diag[ui, :s1] - ref["diag"]).max() <= 1e-4
    nb = (n + 63) // 64
    lbs = pb.lbs.cpu().numpy().astype(np.float64)
    for h in range(hq):
        L = PR.block_mean_logits(q[h], k[h // g], 64)
        tri = np.concatenate([L[bq, :bq + 1] for bq in range(nb)])
        np.testing.assert_allclose(lbs[h], tri, atol=1e-4, rtol=1e-5)
    grid = [(DENSE, 0, 0), (ASHAPE, 64, 256), (VSLASH, 40, 120), (BSPARSE, 5, 64)]
    ib, pc = _coverage(res, units, grid, rcfg)
    _check_coverage(q, k, units, grid, rcfg, ib, pc, g)


# grids that select each coverage instantiation: <2, A-shape only>, <4> (three candidates
# without prefetched bitmap words: a vertical-slash and a block-sparse one among them), <16>
# (five), and the 16-candidate limit (nine)
GRID_C4 = [(DENSE, 0, 0), (ASHAPE, 64, 256), (VSLASH, 20, 40), (VSLASH, 30, 80), (VSLASH, 40, 120),
           (VSLASH, 60, 300), (BSPARSE, 2, 64), (BSPARSE, 3, 64), (BSPARSE, 5, 64), (BSPARSE, 8, 64)]
GRID_C16 = [(DENSE, 0, 0), (ASHAPE, 16, 64), (ASHAPE, 64, 256), (ASHAPE, 128, 1024), (VSLASH, 20, 40),
            (VSLASH, 30, 80), (VSLASH, 40, 120), (VSLASH, 60, 300), (BSPARSE, 2, 64), (BSPARSE, 3, 64),
            (BSPARSE, 5, 64), (BSPARSE, 8, 64)]
GRID_MAX = [(DENSE, 0, 0), (ASHAPE, 16, 64), (ASHAPE, 64, 256), (ASHAPE, 128, 1024), (VSLASH, 10, 20),
            (VSLASH, 20, 40), (VSLASH, 30, 80), (VSLASH, 40, 120), (VSLASH, 60, 300), (VSLASH, 90, 500),
            (BSPARSE, 2, 64), (BSPARSE, 3, 64), (BSPARSE, 5, 64), (BSPARSE, 8, 64), (BSPARSE, 12, 64),
            (BSPARSE, 20, 64)]


@pytest.mark.parametrize("grid", [GRID_C4, GRID_C16, GRID_MAX], ids=["cover4", "cover16", "cover16_full"])
@pytest.mark.parametrize("rcfg", [(64, 16, 8), (100, 0, 0)])
def test_coverage_general_grids_match_oracle(grid, rcfg):
    n, hq, hkv, d = 2600, 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=5, kscale=1.5)
    units = [(0, 0, n), (1, 512, 2400), (0, 1000, 1100)]
    res = _probe_scores(q, k, v, units, rcfg, "bf16")
    ib, pc = _coverage(res, units, grid, rcfg)
    _check_coverage(q, k, units, grid, rcfg, ib, pc, hq // hkv)


def test_coverage_staged_and_fetched_bitmap_words():
    """The coverage pass stages a pair's diagonal-bitmap words in LDS when they fit (rows spread
    over at most ~17K positions) and fetches them with each tile otherwise: a 24K-row unit
    (fetched) and a 16K-row unit (staged) in one call, three prefetched vertical-slash
    candidates, against the oracle."""
    n, hq, hkv, d = 24576, 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=11, kscale=1.5)
    rcfg = (64, 64, 32)
    units = [(0, 0, n), (1, 8192, n)]
    res = _probe_scores(q, k, v, units, rcfg, "bf16")
    grid = [(DENSE, 0, 0), (ASHAPE, 64, 256), (VSLASH, 40, 120), (VSLASH, 80, 300), (VSLASH, 200, 900),
            (BSPARSE, 5, 64)]
    ib, pc = _coverage(res, units, grid, rcfg)
    _check_coverage(q, k, units, grid, rcfg, ib, pc, hq // hkv)


def test_coverage_general_grid_on_128k_segments():
    """The 16-candidate coverage variant over 16K-row segments of a 128K prefix (the last
    segment sees every key) on the 32-layer workload's synthetic layer."""
    import torch
    t = G.make_layer_torch(5, 9, device="cuda")
    q, k, v = t["q"], t["k"], t["v"]
    n = q.shape[1]
    rcfg = (64, 64, 32)
    units = [(0, n - 16384, n), (1, 0, 16384), (6, 49152, 65536)]
    qkv = _rs.make_qkv(q, k, v)
    u = _rs.make_units(units)
    cfg = _rs.RsProbeCfg(r_rec=64, r_uni=64, r_bnd=32, bs_block=64, local_w=1024,
                         flags=_rs.RS_PROBE_ROWS | _rs.RS_PROBE_BLOCKMEAN)
    pb = _rs.ProbeBuffers(len(units), 160, n, 32, 0, blockmean=True)
    ws = _rs.workspace(_rs.rs_probe_workspace_size(qkv, u, len(units), cfg))
    _rs.rs_probe(qkv, u, len(units), cfg, None, 0, None, ws, pb)
    res = dict(qkv=qkv, u=u, cfg=cfg, pb=pb, ws=ws)
    grid = [(DENSE, 0, 0), (ASHAPE, 128, 1024), (ASHAPE, 128, 4096), (ASHAPE, 256, 8192), (VSLASH, 500, 256),
            (VSLASH, 1000, 512), (VSLASH, 2000, 2048), (VSLASH, 2000, 6096), (BSPARSE, 50, 64),
            (BSPARSE, 100, 64), (BSPARSE, 200, 64), (BSPARSE, 256, 64)]
    ib, pc = _coverage(res, units, grid, rcfg)
    # the oracle reads only the heads of the units
    qh = {h: q[h].float().cpu().numpy() for h in {x[0] for x in units}}
    kh = {h // 4: k[h // 4].float().cpu().numpy() for h in qh}
    _check_coverage(qh, kh, units, grid, rcfg, ib, pc, 4)


def test_vs_selection_beyond_the_lds_gather_limit():
    """A slash budget above the selection's LDS capacity (8192): every vertical-slash budget
    is then selected from the whole score array; sets stay bit-exact against the oracle's
    rule on the GPU's scores, and nested."""
    import torch
    n, hq, hkv, d = 20000, 1, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=8)
    q[0, -64:] *= 0.05          # nearly uniform recent rows: many close scores
    units = [(0, 0, n), (0, 2000, 15000)]
    res = _probe_scores(q, k, v, units, (64, 0, 0), "bf16")
    pb = res["pb"]
    grid = [(DENSE, 0, 0), (VSLASH, 300, 2000), (VSLASH, 1000, 9000), (VSLASH, 2048, 12288)]
    g = _rs.make_grid(grid)
    ib = _rs.IndexBuffers(len(units), n, hq, grid)
    ws = _rs.workspace(_rs.rs_build_indices_workspace_size(pb, g, len(grid)))
    _rs.rs_build_indices(pb, res["u"], len(units), g, len(grid), ws, ib)
    torch.cuda.synchronize()
    col, diag = pb.col.cpu().numpy().astype(np.float64), pb.diag.cpu().numpy().astype(np.float64)
    nw = (n + 31) // 32
    for ui, (h, s0, s1) in enumerate(units):
        prev = None
        for cl, (_, nv, ns) in enumerate(grid[1:]):
            Vr, Dr, _, _ = IX.vs_indices(col[ui], diag[ui], s1, nv, ns)
            cnt = ib.vs_count[ui, cl].cpu().numpy()
            V = ib.vs_vsorted[ui, cl].cpu().numpy()
            D = ib.vs_dsorted[ui, cl].cpu().numpy()
            assert np.array_equal(V[:cnt[0]], Vr) and np.array_equal(D[:cnt[1]], Dr), (ui, cl)
            assert np.all(V[cnt[0]:] == -1) and np.all(D[cnt[1]:] == -1)
            assert np.array_equal(ib.vs_vbits[ui, cl].cpu().numpy(), words_of(Vr, nw))
            assert np.array_equal(ib.vs_dbits[ui, cl].cpu().numpy(), words_of(Dr, nw))
            if prev is not None:
                assert set(prev[0]) <= set(Vr.tolist()) and set(prev[1]) <= set(Dr.tolist())
            prev = (Vr.tolist(), Dr.tolist())


# ---- bitwise repeatability -----------------------------------------------------------------

def test_probe_indices_and_device_route_repeat_bitwise():
    """Identical inputs give bitwise-identical probe scores, block-mean logits, index sets,
    coverage, descriptors and device routes, call after call (every cross-workgroup reduction
    sums fixed partials in a fixed order)."""
    import torch
    n, hq, hkv, d = 12000, 4, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=17, kscale=1.5)
    seg = 4000
    units = [(h, s, s + seg) for s in range(0, n, seg) for h in range(hq)]
    rcfg = (64, 32, 16)
    grid = [(DENSE, 0, 0), (ASHAPE, 64, 512), (ASHAPE, 64, 2048), (VSLASH, 50, 100), (VSLASH, 100, 400),
            (BSPARSE, 8, 64), (BSPARSE, 16, 64)]
    outs = []
    for rep in range(3):
        res = _probe_scores(q, k, v, units, rcfg, "bf16")
        ib, pc = _coverage(res, units, grid, rcfg)
        s1 = np.array([u[2] for u in units], np.int32)
        edges = np.array([seg, 2 * seg, 3 * seg], np.int32)
        tt = np.array([[e / 1000.0 * (1.0 if gg[0] == DENSE else 0.1 + 0.05 * c) for e in edges]
                       for c, gg in enumerate(grid)])
        rb = _rs.RouteDevBuffers(grid, s1, tt, edges)
        T = float(sum(tt[0, int(np.searchsorted(edges, x))] for x in s1)) / 4
        _rs.rs_route_layer_device(rb, pc.cov, pc.nsub, 5.0, T, 0.95, 1.0, 0.0, 0.01)
        torch.cuda.synchronize()
        pb = res["pb"]
        snap = {name: getattr(pb, name).clone() for name in ("rows", "subset", "nsub", "row_max", "row_sum", "col",
                                                             "diag", "lbs")}
        snap.update({"cov_" + name: getattr(pc, name).clone() for name in ("cov_rows", "cov", "entropy", "local",
                                                                           "row_max", "row_sum")})
        snap.update({"ib_" + name: getattr(ib, name).clone() for name in ("vs_vsorted", "vs_dsorted", "vs_count",
                                                                          "vs_vbits", "vs_dbits", "bs_rank",
                                                                          "bs_sorted", "bs_count", "bs_bits")})
        snap.update({"rt_" + name: getattr(rb, name).clone() for name in ("choice", "group_cand", "group_start",
                                                                          "group_units", "risk", "m_lower", "status",
                                                                          "totals")})
        outs.append(snap)
    for rep in (1, 2):
        for name, t0 in outs[0].items():
            t1 = outs[rep][name]
            assert torch.equal(t0.view(torch.uint8) if t0.is_floating_point() else t0,
                               t1.view(torch.uint8) if t1.is_floating_point() else t1), (rep, name)
    # and the route is the oracle's on those coverage arrays
    cov = outs[0]["cov_cov"].cpu().numpy().astype(np.float64)
    nsub = outs[0]["nsub"].cpu().numpy()
    s1 = np.array([u[2] for u in units])
    edges = np.array([seg, 2 * seg, 3 * seg])
    tt = np.array([[e / 1000.0 * (1.0 if gg[0] == DENSE else 0.1 + 0.05 * c) for e in edges]
                   for c, gg in enumerate(grid)])
    tu = np.array([tt[:, int(np.searchsorted(edges, x))] for x in s1])
    ref = RT.route_layer(cov[:, :, 0], cov[:, :, 1:], nsub, np.zeros(cov.shape[:2]), tu, [gg[0] for gg in grid],
                         [sum(1 for g2 in grid[:c] if g2[0] == grid[c][0]) for c in range(len(grid))], 5.0,
                         T, 0.95, 1.0, 0.0, 0.01)
    assert outs[0]["rt_choice"][:len(units)].cpu().tolist() == ref["choice"]
