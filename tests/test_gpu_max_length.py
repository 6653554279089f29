"""The whole path at the maximum supported length (262144 tokens, 4096 key blocks), against
the oracle with the bars of the small-size tests: the probe's column and diagonal scores
(Sec. 3.2, Eq. 3) and block-mean logits, the index rules run on the GPU's scores (Sec. 3.1),
coverage of every family's sets (Sec. 3.2-3.3), and the attention of every family on the
sets the GPU built (Sec. 2.1)."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import coverage as CV
from oracle import indices as IX
from oracle import patterns as P
from oracle import probe as PR
from paper_2608_29058_amd import _rs

from gpu_helpers import check_close, out_tensor, with_vt, words_of
from test_gpu_probe import _gpu_vs_sets, _inputs, _probe

pytestmark = pytest.mark.gpu


def test_path_at_the_maximum_length():
    import torch
    n, hq, hkv, d = 262144, 2, 1, 128
    nb, nw = n // 64, n // 32
    q, k, v = _inputs(n, hq, hkv, d, 9)
    # the last 16K segment of head 0 and a short last unit of head 1 (whose 128-row items
    # include the sequence's last rows and key blocks)
    units = [(0, n - 16384, n), (1, n - 700, n)]
    rc = (64, 16, 8)
    res = _probe(q, k, v, units, rc, _rs.RS_PROBE_ROWS | _rs.RS_PROBE_BLOCKMEAN)
    pb = res["pb"]
    col, diag = pb.col.cpu().numpy().astype(np.float64), pb.diag.cpu().numpy().astype(np.float64)
    refs = []
    for ui, (h, s0, s1) in enumerate(units):
        ref = PR.probe_unit(q[h], k[0], s0, s1, *rc)
        refs.append(ref)
        assert np.abs(col[ui, :s1] - ref["col"]).max() <= 1e-4, ui
        assert np.abs(diag[ui, :s1] - ref["diag"]).max() <= 1e-4, ui

    # block-mean logits (lower triangle, row-major): the last 64 query blocks of each head
    lbs = pb.lbs.cpu().numpy().astype(np.float64)
    Lg = {}
    for h in range(hq):
        L = PR.block_mean_logits(q[h], k[0], 64)
        for bq in range(nb - 64, nb):
            off = bq * (bq + 1) // 2
            np.testing.assert_allclose(lbs[h, off:off + bq + 1], L[bq, :bq + 1], atol=1e-4, rtol=1e-5)
        G = np.full((nb, nb), np.nan)
        for bq in range(nb):
            off = bq * (bq + 1) // 2
            G[bq, :bq + 1] = lbs[h, off:off + bq + 1]
        Lg[h] = G

    # index sets from the GPU's scores: bit-exact against the oracle's rules on the same scores
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_ASHAPE, 128, 1024), (_rs.RS_VSLASH, 500, 256), (_rs.RS_BSPARSE, 100, 64)]
    g = _rs.make_grid(grid)
    ib = _rs.IndexBuffers(len(units), n, hq, grid)
    ws = _rs.workspace(_rs.rs_build_indices_workspace_size(pb, g, len(grid)))
    _rs.rs_build_indices(pb, res["u"], len(units), g, len(grid), ws, ib)
    torch.cuda.synchronize()
    sets = []
    for ui, (h, s0, s1) in enumerate(units):
        Vr, Dr, _, _ = IX.vs_indices(col[ui], diag[ui], s1, 500, 256)
        V, D, Vpad, Dpad = _gpu_vs_sets(ib, ui, 0)
        assert np.array_equal(V, Vr) and np.array_equal(D, Dr), ui
        assert np.all(Vpad == -1) and np.all(Dpad == -1)
        assert np.array_equal(ib.vs_vbits[ui, 0].cpu().numpy(), words_of(Vr, nw))
        assert np.array_equal(ib.vs_dbits[ui, 0].cpu().numpy(), words_of(Dr, nw))
        sel, _ = IX.bs_indices(Lg[h], 100)
        srt, cnt = ib.bs_sorted[h, 0].cpu().numpy(), ib.bs_count[h, 0].cpu().numpy()
        for bq in range(s0 // 64, nb):
            assert cnt[bq] == sel[bq].size and np.array_equal(srt[bq, :cnt[bq]], sel[bq]), (h, bq)
        sets.append((V, D, srt, cnt))

    # coverage of every candidate on the sampled rows
    pc = _rs.ProbeBuffers(len(units), sum(rc), n, hq, len(grid), blockmean=False)
    for name in ("rows", "subset", "nsub"):
        getattr(pc, name).copy_(getattr(pb, name))
    _rs.rs_probe(res["qkv"], res["u"], len(units), res["cfg"], g, len(grid), ib, res["ws"], pc)
    torch.cuda.synchronize()
    cov_rows, cov = pc.cov_rows.cpu().numpy(), pc.cov.cpu().numpy()
    for ui, (h, s0, s1) in enumerate(units):
        rows, a = refs[ui]["rows"], refs[ui]["a"]
        nr = rows.size
        V, D, srt, cnt = sets[ui]
        masks = [None, P.ashape_mask(rows, s1, 128, 1024), P.vs_mask(rows, s1, V, D),
                 P.bs_mask(rows, s1, 64, lambda bq: srt[bq, :cnt[bq]])]
        assert np.all(cov_rows[ui, 0, :nr] == 1.0)
        for c in range(1, len(grid)):
            mi = A.retained_mass(a, masks[c])
            assert np.abs(cov_rows[ui, c, :nr] - mi).max() <= 1e-4, (ui, c)
            mh, means, _ = CV.subset_means(mi, refs[ui]["subset"])
            assert abs(cov[ui, c, 0] - mh) <= 1e-4 and np.abs(cov[ui, c, 1:] - np.array(means)).max() <= 1e-4

    # attention of every family on head 1's unit, with the sets above, on sampled rows
    h, s0, s1 = units[1]
    qkv, _vt = with_vt(res["qkv"])
    rows = np.unique(np.concatenate([np.arange(s0, s0 + 16), np.arange(s1 - 48, s1),
                                     np.random.default_rng(1).choice(np.arange(s0, s1), 64, replace=False)]))
    V, D, srt, cnt = sets[1]
    fam_masks = {1: P.ashape_mask(rows, s1, 128, 1024), 2: P.vs_mask(rows, s1, V, D),
                 3: P.bs_mask(rows, s1, 64, lambda bq: srt[bq, :cnt[bq]])}
    for c, m in fam_masks.items():
        u = _rs.make_units([(h, s0, s1, c, 1)])
        ws_a = _rs.workspace(_rs.rs_attn_workspace_size(qkv, u, 1))
        o = out_tensor(hq, n, d)
        _rs.rs_sparse_attn_prefill(qkv, u, 1, g, len(grid), ib, o, None, ws_a)
        torch.cuda.synchronize()
        ref, _ = A.masked_attention(q[h], k[0], v[0], rows, m)
        check_close(o[h].float().cpu().numpy()[rows], ref, f"family {c} at n={n}")
    u = _rs.make_units([(h, s0, s1)])
    ws_a = _rs.workspace(_rs.rs_attn_workspace_size(qkv, u, 1))
    o = out_tensor(hq, n, d)
    _rs.rs_dense_attn_prefill(qkv, u, 1, o, None, ws_a)
    torch.cuda.synchronize()
    check_close(o[h].float().cpu().numpy()[rows], A.dense_attention(q[h], k[0], v[0], rows=rows), f"dense at n={n}")
