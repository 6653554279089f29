"""Helpers shared by the GPU tests: device copies of seeded inputs and host-built index
sets (so the attention kernels can be checked independently of the probe)."""
import numpy as np

from paper_2608_29058_amd import _rs


def dev(x, dtype="bf16"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.cuda()


def words_of(idx, nwords):
    w = np.zeros(nwords, np.uint32)
    idx = np.asarray(idx, dtype=np.int64)
    if idx.size:
        np.bitwise_or.at(w, idx >> 5, (np.uint32(1) << (idx & 31).astype(np.uint32)))
    return w.view(np.int32)


def fill_vs(ib, slot, cl, V, D):
    """Write one unit's vertical-slash sets into IndexBuffers ``ib``."""
    import torch
    V = np.sort(np.asarray(V, np.int64))
    D = np.sort(np.asarray(D, np.int64))
    nv, ns = ib.vs_vsorted.shape[2], ib.vs_dsorted.shape[2]
    a = np.full(nv, -1, np.int32); a[:V.size] = V
    b = np.full(ns, -1, np.int32); b[:D.size] = D
    ib.vs_vsorted[slot, cl] = torch.from_numpy(a).cuda()
    ib.vs_dsorted[slot, cl] = torch.from_numpy(b).cuda()
    ib.vs_count[slot, cl] = torch.tensor([V.size, D.size], dtype=torch.int32).cuda()
    nw = ib.vs_vbits.shape[2]
    ib.vs_vbits[slot, cl] = torch.from_numpy(words_of(V, nw)).cuda()
    ib.vs_dbits[slot, cl] = torch.from_numpy(words_of(D, nw)).cuda()


def fill_bs(ib, head, cl, sel):
    """sel: list over query blocks of selected key blocks."""
    import torch
    nb, kmax, nbw = ib.bs_sorted.shape[2], ib.bs_sorted.shape[3], ib.bs_bits.shape[3]
    srt = np.full((nb, kmax), -1, np.int32)
    cnt = np.zeros(nb, np.int32)
    bits = np.zeros((nb, nbw), np.int32)
    for bq in range(nb):
        s = np.sort(np.asarray(list(sel[bq]), np.int64))
        srt[bq, :s.size] = s
        cnt[bq] = s.size
        bits[bq] = words_of(s, nbw)
    ib.bs_sorted[head, cl] = torch.from_numpy(srt).cuda()
    ib.bs_count[head, cl] = torch.from_numpy(cnt).cuda()
    ib.bs_bits[head, cl] = torch.from_numpy(bits).cuda()


def out_tensor(hq, n, d):
    import torch
    return torch.full((hq, n, d), float("nan"), dtype=torch.bfloat16, device="cuda")


def check_close(got, ref, tag, max_abs=2e-2, rel_f=1e-2):
    """Tolerance of the routed-prefill outputs: bf16 in, fp32 accumulate."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.isfinite(got).all(), f"{tag}: non-finite output"
    err = np.abs(got - ref).max() if got.size else 0.0
    rf = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert err <= max_abs and rf <= rel_f, f"{tag}: max-abs {err:.3e} rel-F {rf:.3e}"
    return err, rf


def with_vt(qkv):
    """Return ``(qkv, buffer)`` with V also written in the transposed operand layout
    (rs_transpose_v) and qkv.vt pointing at it; keep the buffer alive while qkv is used."""
    import torch
    buf = torch.empty(_rs.rs_vt_bytes(qkv), dtype=torch.uint8, device="cuda")
    _rs.rs_transpose_v(qkv, buf)
    qkv.vt = buf.data_ptr()
    return qkv, buf
