"""GPU parity of the dense and sparse attention kernels against the fp64 oracle
(Sec. 2.1 Eq. 1 and the masked-softmax semantics; pattern sets of Sec. 3.1).

Index sets are written host-side here so each kernel is checked on its own; the
probe-built sets are covered by the probe tests.  Tolerance: max-abs 2e-2 and
relative Frobenius 1e-2 (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import patterns as P
from paper_2608_29058_amd import _rs
from synth import gen as G

from gpu_helpers import check_close, dev, fill_bs, fill_vs, out_tensor, with_vt

pytestmark = pytest.mark.gpu


def _inputs(n, hq, hkv, d, seed, dtype="bf16"):
    r = np.random.default_rng(seed)
    q = r.standard_normal((hq, n, d)).astype(np.float32)
    k = r.standard_normal((hkv, n, d)).astype(np.float32)
    v = r.standard_normal((hkv, n, d)).astype(np.float32)
    k[:, :3] += 3.0 * q[:, -1:].mean(0)[:1] if hq else 0       # a mild sink
    if dtype == "bf16":
        q, k, v = G.bf16_round(q), G.bf16_round(k), G.bf16_round(v)
    return q, k, v


def _run_dense(q, k, v, units, dtype="bf16", lse=False, vt=False):
    import torch
    hq, n, d = q.shape
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    qkv = _rs.make_qkv(qd, kd, vd)
    if vt:
        qkv, _vt = with_vt(qkv)
    u = _rs.make_units(units)
    ws = _rs.workspace(_rs.rs_attn_workspace_size(qkv, u, len(units)))
    o = out_tensor(hq, n, d)
    ls = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda") if lse else None
    _rs.rs_dense_attn_prefill(qkv, u, len(units), o, ls, ws)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), (ls.cpu().numpy() if lse else None)


@pytest.mark.parametrize("n,hq,hkv,d,dtype", [(1000, 4, 2, 128, "bf16"), (4097, 2, 1, 128, "bf16"),
                                              (700, 2, 2, 64, "bf16"), (2048, 1, 1, 64, "f32"),
                                              (64, 1, 1, 128, "bf16"), (1, 1, 1, 128, "bf16")])
@pytest.mark.parametrize("vt", [False, True])
def test_dense_matches_oracle(n, hq, hkv, d, dtype, vt):
    q, k, v = _inputs(n, hq, hkv, d, seed=n + d)
    units = [(h, 0, n) for h in range(hq)]
    o, lse = _run_dense(q, k, v, units, dtype, lse=True, vt=vt)
    g = hq // hkv
    for h in range(hq):
        ref = A.dense_attention(q[h], k[h // g], v[h // g])
        check_close(o[h], ref, f"dense h={h}")
        lg = A.logits(q[h], k[h // g], np.arange(n), n)
        lg = np.where(P.dense_mask(np.arange(n), n), lg, -np.inf)
        from scipy.special import logsumexp
        np.testing.assert_allclose(lse[h], logsumexp(lg, axis=1), atol=2e-3, rtol=1e-4)


@pytest.mark.parametrize("vt", [False, True])
def test_dense_segments_write_only_their_rows(vt):
    n, hq, hkv, d = 1500, 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=7)
    units = [(0, 100, 700), (1, 640, 1500), (0, 1200, 1201)]
    o, _ = _run_dense(q, k, v, units, vt=vt)
    written = np.zeros((hq, n), bool)
    for h, s0, s1 in units:
        written[h, s0:s1] = True
        rows = np.arange(s0, s1)
        check_close(o[h, s0:s1], A.dense_attention(q[h], k[0], v[0], rows=rows), f"seg {h},{s0},{s1}")
    assert np.isnan(o[~written]).all()


def _run_sparse(q, k, v, units, grid, ib, dtype="bf16", vt=False):
    import torch
    hq, n, d = q.shape
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    qkv = _rs.make_qkv(qd, kd, vd)
    if vt:
        qkv, _vt = with_vt(qkv)
    u = _rs.make_units(units)
    g = _rs.make_grid(grid)
    ws = _rs.workspace(_rs.rs_attn_workspace_size(qkv, u, len(units)))
    o = out_tensor(hq, n, d)
    lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda")
    _rs.rs_sparse_attn_prefill(qkv, u, len(units), g, len(grid), ib, o, lse, ws)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("n,sink,window", [(3000, 128, 1024), (2500, 0, 1), (1800, 100, 300),
                                           (700, 4, 64), (5000, 130, 1000)])
@pytest.mark.parametrize("vt", [False, True])
def test_ashape_matches_oracle(n, sink, window, vt):
    hq, hkv, d = 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=sink + window)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_ASHAPE, sink, window)]
    units = [(0, 0, n, 1), (1, 640, n, 1)]
    o, lse = _run_sparse(q, k, v, units, grid, None, vt=vt)
    for h, s0, s1, _ in units:
        rows = np.arange(s0, s1)
        ref, rl = A.masked_attention(q[h], k[0], v[0], rows, P.ashape_mask(rows, s1, sink, window))
        check_close(o[h, s0:s1], ref, f"ashape h={h}")
        np.testing.assert_allclose(lse[h, s0:s1], rl, atol=2e-3, rtol=1e-4)


@pytest.mark.parametrize("n,k_blocks", [(2000, 5), (4096, 12), (1100, 40)])
@pytest.mark.parametrize("vt", [False, True])
def test_block_sparse_matches_oracle(n, k_blocks, vt):
    hq, hkv, d = 4, 2, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=n)
    nb = (n + 63) // 64
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, k_blocks, 64)]
    ib = _rs.IndexBuffers(hq, n, hq, grid)
    r = np.random.default_rng(3)
    sels = {}
    for h in range(hq):
        sel = []
        for bq in range(nb):
            others = r.permutation(bq)[:k_blocks - 1]
            sel.append(sorted(set(others.tolist()) | {bq}))
        sels[h] = sel
        fill_bs(ib, h, 0, sel)
    units = [(h, 0 if h % 2 == 0 else 320, n, 1) for h in range(hq)]
    o, _ = _run_sparse(q, k, v, units, grid, ib, vt=vt)
    g = hq // hkv
    for h, s0, s1, _ in units:
        rows = np.arange(s0, s1)
        mask = P.bs_mask(rows, s1, 64, lambda bq, h=h: sels[h][bq])
        ref, _ = A.masked_attention(q[h], k[h // g], v[h // g], rows, mask)
        check_close(o[h, s0:s1], ref, f"bs h={h}")


@pytest.mark.parametrize("n,s0,k_blocks,hq,hkv", [(2000, 0, 7, 4, 2), (2600, 96, 30, 4, 2), (4160, 640, 64, 4, 2),
                                                  (2600, 96, 30, 6, 2)])
@pytest.mark.parametrize("vt", [False, True])
def test_block_sparse_mates_match_single_units(n, s0, k_blocks, hq, hkv, vt):
    """Block-sparse units of heads 2m and 2m + 1 with the same rows and key/value head run as
    mates (64-row items, one selection per wave pair): every row's output and LSE equal, bit
    for bit, those of the same units launched one by one (128-row items), and the oracle's
    masked attention (Sec. 3.1 block-sparse mask).  With three heads per key/value head,
    heads 2 and 3 read different key/value heads and stay unpaired."""
    d = 128
    q, k, v = _inputs(n, hq, hkv, d, seed=n + s0)
    nb = (n + 63) // 64
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, k_blocks, 64)]
    ib = _rs.IndexBuffers(hq, n, hq, grid)
    r = np.random.default_rng(n)
    sels = {}
    for h in range(hq):
        # head 1 shares part of head 0's selections, heads 2 and 3 are independent
        sel = []
        for bq in range(nb):
            others = r.permutation(bq)[:k_blocks - 1]
            if h == 1 and bq < len(sels[0]):
                keep = [b for b in sels[0][bq] if b != bq][: (k_blocks - 1) // 2]
                others = np.array(sorted(set(keep) | set(others.tolist()[: k_blocks - 1 - len(keep)])), dtype=np.int64)
            sel.append(sorted(set(others.tolist()) | {bq}))
        sels[h] = sel
        fill_bs(ib, h, 0, sel)
    units = [(h, s0, n, 1) for h in range(hq)]
    o, lse = _run_sparse(q, k, v, units, grid, ib, vt=vt)
    g = hq // hkv
    for h in range(hq):
        o1, lse1 = _run_sparse(q, k, v, [units[h]], grid, ib, vt=vt)
        assert np.array_equal(o[h, s0:n], o1[h, s0:n]) and np.array_equal(lse[h, s0:n], lse1[h, s0:n]), h
        rows = np.arange(s0, n)
        mask = P.bs_mask(rows, n, 64, lambda bq, h=h: sels[h][bq])
        ref, rl = A.masked_attention(q[h], k[h // g], v[h // g], rows, mask)
        check_close(o[h, s0:n], ref, f"bs mates h={h}")
        np.testing.assert_allclose(lse[h, s0:n], rl, atol=2e-3, rtol=1e-4)


def test_block_sparse_mates_at_the_maximum_length():
    """The last 64-row query blocks of a sequence of the maximum length (262144 tokens, 4096
    key blocks) run as mates: their key-block bitmaps reach block 4096 (one past the last),
    and the rows match the same units launched one by one and the oracle."""
    n, hq, hkv, d, kb = 262144, 2, 1, 128, 5
    q, k, v = _inputs(n, hq, hkv, d, seed=11)
    nb = n // 64
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, kb, 64)]
    ib = _rs.IndexBuffers(hq, n, hq, grid)
    r = np.random.default_rng(3)
    sels = {}
    for h in range(hq):
        sel = [[bq] for bq in range(nb)]
        for bq in (nb - 2, nb - 1):
            sel[bq] = sorted({bq, 0, *r.choice(bq, kb - 2, replace=False).tolist()})
        sels[h] = sel
        fill_bs(ib, h, 0, sel)
    s0 = n - 128
    units = [(h, s0, n, 1) for h in range(hq)]
    o, lse = _run_sparse(q, k, v, units, grid, ib, vt=True)
    for h in range(hq):
        o1, lse1 = _run_sparse(q, k, v, [units[h]], grid, ib, vt=True)
        assert np.array_equal(o[h, s0:n], o1[h, s0:n]) and np.array_equal(lse[h, s0:n], lse1[h, s0:n]), h
        rows = np.arange(s0, n)
        mask = P.bs_mask(rows, n, 64, lambda bq, h=h: sels[h][bq])
        ref, rl = A.masked_attention(q[h], k[0], v[0], rows, mask)
        check_close(o[h, s0:n], ref, f"bs mates max length h={h}")
        np.testing.assert_allclose(lse[h, s0:n], rl, atol=2e-3, rtol=1e-4)


@pytest.mark.parametrize("n,nv,ns,spread", [(3000, 40, 300, "local"), (2048, 64, 256, "scatter"),
                                            (4100, 200, 1500, "mixed"), (900, 0, 1, "diag_only"),
                                            # the most vertical columns a set may hold (2048), nearly all
                                            # gathered (only the local diagonals give contiguous tiles)
                                            (6000, 2048, 4, "local")])
@pytest.mark.parametrize("vt", [False, True])   # the vertical-slash kernel ignores vt
def test_vertical_slash_matches_oracle(n, nv, ns, spread, vt):
    hq, hkv, d = 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=nv + ns)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_VSLASH, nv, ns)]
    units = [(0, 0, n, 1, 0), (1, 500, n, 1, 1)]
    ib = _rs.IndexBuffers(2, n, hq, grid)
    r = np.random.default_rng(5)
    sets = []
    for slot, (h, s0, s1, _, _) in enumerate(units):
        V = np.sort(r.choice(s1, min(nv, s1), replace=False))
        if spread == "local":
            D = np.arange(min(ns, s1))
        elif spread == "scatter":
            D = np.sort(np.unique(np.concatenate([[0], r.choice(s1, ns - 1, replace=False)])))[:ns]
        elif spread == "mixed":
            D = np.unique(np.concatenate([np.arange(ns // 2), r.choice(s1, ns - ns // 2, replace=False)]))[:ns]
        else:
            D = np.array([0])
        fill_vs(ib, slot, 0, V, D)
        sets.append((V, D))
    o, _ = _run_sparse(q, k, v, units, grid, ib, vt=vt)
    for slot, (h, s0, s1, _, _) in enumerate(units):
        rows = np.arange(s0, s1)
        V, D = sets[slot]
        ref, _ = A.masked_attention(q[h], k[0], v[0], rows, P.vs_mask(rows, s1, V, D))
        check_close(o[h, s0:s1], ref, f"vs slot={slot}")


def test_index_counts_beyond_their_arrays_are_clamped():
    """A set whose count runs past its array (vertical-slash: |V|, |D| above nv_max, ns_max;
    block-sparse: the -1 pads counted, and a count above k_max) gives exactly the output of
    the well-formed set: counts are read clamped to the arrays and entries outside the causal
    key blocks are skipped.  Only unit 0 / head 0 is altered, which is not the last row of
    its buffer, so every read stays inside the allocation either way."""
    import torch
    n, hq, hkv, d = 1500, 2, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=77)
    r = np.random.default_rng(11)

    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_VSLASH, 40, 64)]
    units = [(0, 0, n, 1, 0), (1, 200, n, 1, 1)]
    ib = _rs.IndexBuffers(2, n, hq, grid)
    for slot in range(2):
        fill_vs(ib, slot, 0, np.sort(r.choice(n, 40, replace=False)), np.arange(64))
    ref, _ = _run_sparse(q, k, v, units, grid, ib)
    nvm, nsm = ib.vs_vsorted.shape[2], ib.vs_dsorted.shape[2]
    ib.vs_count[0, 0] = torch.tensor([nvm + 100, nsm + 100], dtype=torch.int32).cuda()
    got, _ = _run_sparse(q, k, v, units, grid, ib)
    assert np.array_equal(got, ref, equal_nan=True), "vertical-slash counts above the arrays"

    nb = (n + 63) // 64
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, 6, 64)]
    ib = _rs.IndexBuffers(hq, n, hq, grid)
    for h in range(hq):
        fill_bs(ib, h, 0, [sorted(set(r.permutation(bq)[:3].tolist()) | {bq}) for bq in range(nb)])
    units = [(h, 0, n, 1) for h in range(hq)]
    ref, _ = _run_sparse(q, k, v, units, grid, ib)
    kmax = ib.bs_sorted.shape[3]
    ib.bs_count[0, 0] = kmax             # the -1 pads after each set counted
    got, _ = _run_sparse(q, k, v, units, grid, ib)
    assert np.array_equal(got, ref, equal_nan=True), "block-sparse counts over the pads"
    ib.bs_count[0, 0] = kmax + 5         # and beyond the array
    got, _ = _run_sparse(q, k, v, units, grid, ib)
    assert np.array_equal(got, ref, equal_nan=True), "block-sparse counts above k_max"


def test_empty_rows_give_zero_and_minus_inf_lse():
    # vertical-slash with no diagonals and columns only late: early rows keep nothing
    n, d = 300, 128
    q, k, v = _inputs(n, 1, 1, d, seed=11)
    grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_VSLASH, 2, 0)]
    ib = _rs.IndexBuffers(1, n, 1, grid)
    fill_vs(ib, 0, 0, [200, 250], [])
    o, lse = _run_sparse(q, k, v, [(0, 0, n, 1, 0)], grid, ib)
    assert np.all(o[0, :200] == 0) and np.all(np.isneginf(lse[0, :200]))
    rows = np.arange(200, n)
    ref, _ = A.masked_attention(q[0], k[0], v[0], rows, P.vs_mask(rows, n, [200, 250], []))
    check_close(o[0, 200:], ref, "late rows")


def test_deterministic_bitwise():
    n, hq, hkv, d = 2000, 4, 1, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=19)
    units = [(h, 0, n) for h in range(hq)]
    a, _ = _run_dense(q, k, v, units)
    b, _ = _run_dense(q, k, v, units)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("fam", ["dense", "ashape", "bs"])
def test_repeated_runs_bitwise_identical(fam):
    """Many key tiles per workgroup and several repetitions: every LDS tile must be fully
    resident before it is read, so repeated runs agree bit for bit."""
    import torch
    n, hq, hkv, d = 6000, 8, 2, 128
    q, k, v = _inputs(n, hq, hkv, d, seed=23)
    units = [(h, 0, n, 1, h) for h in range(hq)]
    if fam == "dense":
        grid, ib = [(_rs.RS_DENSE, 0, 0)], None
        runs = [_run_dense(q, k, v, [u[:3] for u in units])[0] for _ in range(4)]
    else:
        if fam == "ashape":
            grid, ib = [(_rs.RS_DENSE, 0, 0), (_rs.RS_ASHAPE, 64, 2048)], None
        else:
            grid = [(_rs.RS_DENSE, 0, 0), (_rs.RS_BSPARSE, 30, 64)]
            ib = _rs.IndexBuffers(hq, n, hq, grid)
            nb = (n + 63) // 64
            r = np.random.default_rng(1)
            for h in range(hq):
                fill_bs(ib, h, 0, [sorted(set(r.permutation(bq)[:29].tolist()) | {bq}) for bq in range(nb)])
        runs = [_run_sparse(q, k, v, units, grid, ib)[0] for _ in range(4)]
    for o in runs[1:]:
        assert np.array_equal(o, runs[0])


@pytest.mark.parametrize("n,hkv,d,dtype", [(1000, 2, 128, "bf16"), (64, 1, 64, "bf16"), (130, 3, 128, "f32"),
                                           (1, 1, 64, "bf16")])
def test_transpose_v_layout(n, hkv, d, dtype):
    """rs_transpose_v: [hkv][d][npad] bf16, keys permuted within groups of 16, zero past n."""
    import torch
    r = np.random.default_rng(n + d)
    v = r.standard_normal((hkv, n, d)).astype(np.float32)
    vd = dev(v, dtype)
    qkv = _rs.make_qkv(vd, vd, vd)
    npad = (n + 63) // 64 * 64
    assert _rs.rs_vt_bytes(qkv) == hkv * d * npad * 2
    buf = torch.full((hkv * d * npad * 2,), 0xAB, dtype=torch.uint8, device="cuda")
    _rs.rs_transpose_v(qkv, buf)
    torch.cuda.synchronize()
    got = buf.cpu().numpy().view(np.uint16).reshape(hkv, d, npad)
    perm = np.array([0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15])
    keys = (np.arange(npad) // 16) * 16 + perm[np.arange(npad) % 16]
    want = np.zeros((hkv, d, npad), np.uint16)
    vb = G.bf16_bits(v)                                 # round to nearest even, as on load
    ok = keys < n
    want[:, :, ok] = np.transpose(vb[:, keys[ok], :], (0, 2, 1))
    np.testing.assert_array_equal(got, want)
