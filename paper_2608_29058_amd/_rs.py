"""ctypes binding of librs.so (include/rs.h): argument marshalling only.

Every computation runs in the library.  torch supplies device memory and the stream;
the helpers here only allocate caller-owned buffers with the dimensions the header
documents and fill the C structs.  The library must have been built in-tree
(``python -m paper_2608_29058_amd.build``); there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librs.so")

RS_OK, RS_ERR_INVALID_ARG, RS_ERR_UNSUPPORTED, RS_ERR_HIP, RS_ERR_WORKSPACE, RS_ERR_BUDGET_INFEASIBLE = range(6)
RS_BF16, RS_F32 = 0, 1
RS_DENSE, RS_ASHAPE, RS_VSLASH, RS_BSPARSE = 0, 1, 2, 3
RS_PROBE_ROWS, RS_PROBE_BLOCKMEAN = 1, 2

EXPORTS = ["rs_unit_table_size", "rs_unit_table_init",
           "rs_probe_workspace_size", "rs_probe", "rs_build_indices_workspace_size",
           "rs_build_indices", "rs_route_layer", "rs_attn_workspace_size",
           "rs_sparse_attn_prefill", "rs_dense_attn_prefill", "rs_error_predict",
           "rs_route_layer_device_workspace_size", "rs_route_layer_device", "rs_route_layer_device_noalloc",
           "rs_routed_attn_workspace_size", "rs_routed_attn_prefill", "rs_vt_bytes", "rs_transpose_v",
           "rs_last_error", "rs_version"]

P = C.c_void_p
I32 = C.c_int32
I64 = C.c_int64


class RsQkv(C.Structure):
    _fields_ = [("q", P), ("k", P), ("v", P), ("dtype", I32), ("n", I32), ("hq", I32),
                ("hkv", I32), ("d", I32), ("_pad0", I32), ("sq_h", I64), ("sq_t", I64),
                ("sk_h", I64), ("sk_t", I64), ("sv_h", I64), ("sv_t", I64),
                ("scale", C.c_float), ("_pad1", I32), ("vt", P), ("tables", P)]


class RsUnit(C.Structure):
    _fields_ = [("head", I32), ("s0", I32), ("s1", I32), ("cand", I32), ("slot", I32),
                ("_pad", I32 * 3)]


class RsCandidate(C.Structure):
    _fields_ = [("fam", I32), ("a", I32), ("b", I32), ("_pad", I32)]


class RsProbeCfg(C.Structure):
    _fields_ = [("r_rec", I32), ("r_uni", I32), ("r_bnd", I32), ("bs_block", I32),
                ("local_w", I32), ("flags", C.c_uint32)]


class RsProbeOut(C.Structure):
    _fields_ = [("nunits", I32), ("rmax", I32), ("n", I32), ("nb", I32), ("ncand", I32),
                ("hq", I32), ("rows", P), ("subset", P), ("nsub", P), ("row_max", P),
                ("row_sum", P), ("col", P), ("diag", P), ("entropy", P), ("local", P),
                ("lbs", P), ("cov_rows", P), ("cov", P), ("tables", P)]


class RsUnitTable(C.Structure):
    _fields_ = [("dev", P), ("key_units", C.c_uint64), ("key_cfg", C.c_uint64), ("nunits", I32), ("rmax", I32),
                ("ngroups", I32), ("n", I32), ("hq", I32), ("hkv", I32)]


class RsIndexSet(C.Structure):
    _fields_ = [("nunits", I32), ("n", I32), ("nb", I32), ("hq", I32), ("nv_max", I32),
                ("ns_max", I32), ("k_max", I32), ("nwords", I32), ("ncand_vs", I32),
                ("ncand_bs", I32), ("nbw", I32), ("_pad", I32),
                ("vs_vsorted", P), ("vs_dsorted", P), ("vs_count", P), ("vs_vbits", P),
                ("vs_dbits", P), ("bs_rank", P), ("bs_sorted", P), ("bs_count", P),
                ("bs_bits", P)]


class RsRouteIn(C.Structure):
    _fields_ = [("nunits", I32), ("ncand", I32), ("grid", P), ("cov", P), ("nsub", P), ("e", P),
                ("s1", P), ("t_table", P), ("bucket_edge", P), ("nbucket", I32), ("_pad", I32),
                ("t_probe_us", C.c_double)]


class RsRouteCfg(C.Structure):
    _fields_ = [("T_layer_us", C.c_double), ("tau", C.c_double), ("alpha", C.c_double),
                ("beta", C.c_double), ("delta_q", C.c_double)]


class RsRouteOut(C.Structure):
    _fields_ = [("choice", P), ("group_cand", P), ("group_start", P), ("group_units", P),
                ("risk", P), ("m_lower", P), ("ngroups", I32), ("n_fallback", I32),
                ("over_budget", I32), ("infeasible", I32), ("total_us", C.c_double),
                ("total_risk", C.c_double)]


class RsErrorModel(C.Structure):
    _fields_ = [("w", (C.c_float * 4) * 4)]


class RsRouteDevOut(C.Structure):
    _fields_ = [("choice", P), ("group_cand", P), ("group_start", P), ("group_units", P),
                ("risk", P), ("m_lower", P), ("status", P), ("totals", P)]


_lib = None


def lib():
    """The loaded librs.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2608_29058_amd.build`")
        L = C.CDLL(LIB_PATH)
        L.rs_last_error.restype = C.c_char_p
        L.rs_version.restype = C.c_char_p
        for name in ("rs_unit_table_size", "rs_probe_workspace_size", "rs_build_indices_workspace_size",
                     "rs_attn_workspace_size", "rs_route_layer_device_workspace_size",
                     "rs_routed_attn_workspace_size", "rs_vt_bytes"):
            getattr(L, name).restype = C.c_size_t
        L.rs_unit_table_size.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsProbeCfg)]
        L.rs_unit_table_init.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsProbeCfg), P,
                                         C.c_size_t, C.POINTER(RsUnitTable), P]
        L.rs_vt_bytes.argtypes = [C.POINTER(RsQkv)]
        L.rs_transpose_v.argtypes = [C.POINTER(RsQkv), P, P]
        L.rs_probe_workspace_size.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsProbeCfg)]
        L.rs_probe.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsProbeCfg),
                               C.POINTER(RsCandidate), I32, C.POINTER(RsIndexSet), P, C.c_size_t,
                               C.POINTER(RsProbeOut), P]
        L.rs_build_indices_workspace_size.argtypes = [C.POINTER(RsProbeOut), C.POINTER(RsCandidate), I32]
        L.rs_build_indices.argtypes = [C.POINTER(RsProbeOut), C.POINTER(RsUnit), I32, C.POINTER(RsCandidate),
                                       I32, P, C.c_size_t, C.POINTER(RsIndexSet), P]
        L.rs_route_layer.argtypes = [C.POINTER(RsRouteIn), C.POINTER(RsRouteCfg), C.POINTER(RsRouteOut)]
        L.rs_attn_workspace_size.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32]
        L.rs_sparse_attn_prefill.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsCandidate),
                                             I32, C.POINTER(RsIndexSet), P, I64, I64, P, P, C.c_size_t, P]
        L.rs_dense_attn_prefill.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, P, I64, I64, P, P,
                                            C.c_size_t, P]
        L.rs_error_predict.argtypes = [C.POINTER(RsProbeOut), C.POINTER(RsCandidate), I32,
                                       C.POINTER(RsErrorModel), P, P]
        L.rs_route_layer_device_workspace_size.argtypes = [I32, I32]
        L.rs_route_layer_device.argtypes = [C.POINTER(RsRouteIn), C.POINTER(RsRouteCfg), C.POINTER(RsRouteDevOut),
                                            P, C.c_size_t, P]
        L.rs_route_layer_device_noalloc.argtypes = [C.POINTER(RsRouteIn), C.POINTER(RsRouteCfg),
                                                    C.POINTER(RsRouteDevOut), P]
        L.rs_routed_attn_workspace_size.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32]
        L.rs_routed_attn_prefill.argtypes = [C.POINTER(RsQkv), C.POINTER(RsUnit), I32, C.POINTER(RsCandidate),
                                             I32, C.POINTER(RsIndexSet), P, P, I64, I64, P, P, C.c_size_t,
                                             C.POINTER(P), P]
        for name in ("rs_unit_table_init", "rs_probe", "rs_build_indices", "rs_route_layer", "rs_sparse_attn_prefill",
                     "rs_dense_attn_prefill", "rs_error_predict", "rs_route_layer_device",
                     "rs_route_layer_device_noalloc",
                     "rs_routed_attn_prefill", "rs_transpose_v"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


class RsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"librs status {status}: {msg}")
        self.status = status


def _check(st, allow=()):
    if st != RS_OK and st not in allow:
        raise RsError(st, lib().rs_last_error().decode())
    return st


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


# ---- argument builders ------------------------------------------------------------------

def make_qkv(q, k, v, scale: float = 0.0, vt=None) -> RsQkv:
    """q: [hq, n, d], k/v: [hkv, n, d] device tensors (bf16 or float32, last dim contiguous);
    vt: optional uint8 device tensor holding V in the rs_transpose_v layout."""
    import torch
    dt = {torch.bfloat16: RS_BF16, torch.float32: RS_F32}[q.dtype]
    assert k.dtype == q.dtype and v.dtype == q.dtype
    return RsQkv(q=q.data_ptr(), k=k.data_ptr(), v=v.data_ptr(), dtype=dt, n=q.shape[1], hq=q.shape[0],
                 hkv=k.shape[0], d=q.shape[2], sq_h=q.stride(0), sq_t=q.stride(1), sk_h=k.stride(0),
                 sk_t=k.stride(1), sv_h=v.stride(0), sv_t=v.stride(1), scale=scale,
                 vt=vt.data_ptr() if vt is not None else None)


def rs_vt_bytes(qkv) -> int:
    return lib().rs_vt_bytes(C.byref(qkv))


def rs_transpose_v(qkv, vt, stream=None):
    """vt: uint8 device tensor of rs_vt_bytes(qkv) bytes (or more)."""
    return _check(lib().rs_transpose_v(C.byref(qkv), _ptr(vt), _stream(stream)))


class UnitTable:
    """Device unit tables of one unit list (rs_unit_table_init): set ``qkv.tables`` and the
    probe output's ``tables`` to ``ptr`` so the layer's calls read them instead of uploading."""

    def __init__(self, qkv, units, nunits, cfg=None, device="cuda", stream=None):
        import torch
        cp = C.byref(cfg) if cfg is not None else None
        nbytes = lib().rs_unit_table_size(C.byref(qkv), units, nunits, cp)
        self.dev = torch.empty(max(256, int(nbytes)), dtype=torch.uint8, device=device)
        self.c = RsUnitTable()
        _check(lib().rs_unit_table_init(C.byref(qkv), units, nunits, cp, _ptr(self.dev), self.dev.numel(),
                                        C.byref(self.c), _stream(stream)))

    @property
    def ptr(self):
        return C.cast(C.pointer(self.c), P).value


def make_units(units) -> C.Array:
    """units: iterable of (head, s0, s1[, cand[, slot]])."""
    units = list(units)
    arr = (RsUnit * max(1, len(units)))()
    for i, u in enumerate(units):
        u = tuple(u) + (0,) * (5 - len(u))
        arr[i].head, arr[i].s0, arr[i].s1, arr[i].cand, arr[i].slot = [int(x) for x in u[:5]]
    return arr


def make_grid(grid) -> C.Array:
    """grid: iterable of (family, a, b)."""
    grid = list(grid)
    arr = (RsCandidate * len(grid))()
    for i, g in enumerate(grid):
        arr[i].fam, arr[i].a, arr[i].b = int(g[0]), int(g[1]), int(g[2])
    return arr


def workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(256, int(nbytes)), dtype=torch.uint8, device=device)


class ProbeBuffers:
    """Caller-owned probe output arrays (rs_probe_out)."""

    def __init__(self, nunits, rmax, n, hq, ncand=0, blockmean=False, device="cuda"):
        import torch
        f, i = torch.float32, torch.int32
        nb = (n + 63) // 64
        self.rows = torch.full((nunits, rmax), -1, dtype=i, device=device)
        self.subset = torch.full((nunits, rmax), -1, dtype=i, device=device)
        self.nsub = torch.zeros((nunits, 3), dtype=i, device=device)
        self.row_max = torch.zeros((nunits, rmax), dtype=f, device=device)
        self.row_sum = torch.zeros((nunits, rmax), dtype=f, device=device)
        self.col = torch.zeros((nunits, n), dtype=f, device=device)
        self.diag = torch.zeros((nunits, n), dtype=f, device=device)
        self.entropy = torch.zeros((nunits, rmax), dtype=f, device=device)
        self.local = torch.zeros((nunits, rmax), dtype=f, device=device)
        self.lbs = torch.zeros((hq, nb * (nb + 1) // 2), dtype=f, device=device) if blockmean else None
        self.cov_rows = torch.zeros((nunits, max(ncand, 1), rmax), dtype=f, device=device)
        self.cov = torch.zeros((nunits, max(ncand, 1), 4), dtype=f, device=device)
        self.c = RsProbeOut(nunits=nunits, rmax=rmax, n=n, nb=nb, ncand=ncand, hq=hq,
                            rows=self.rows.data_ptr(), subset=self.subset.data_ptr(),
                            nsub=self.nsub.data_ptr(), row_max=self.row_max.data_ptr(),
                            row_sum=self.row_sum.data_ptr(), col=self.col.data_ptr(),
                            diag=self.diag.data_ptr(), entropy=self.entropy.data_ptr(),
                            local=self.local.data_ptr(),
                            lbs=self.lbs.data_ptr() if self.lbs is not None else None,
                            cov_rows=self.cov_rows.data_ptr(), cov=self.cov.data_ptr())


class IndexBuffers:
    """Caller-owned index-set arrays (rs_index_set) sized for a candidate grid."""

    def __init__(self, nunits, n, hq, grid, device="cuda"):
        import torch
        i = torch.int32
        grid = list(grid)
        vs = [g for g in grid if g[0] == RS_VSLASH]
        bs = [g for g in grid if g[0] == RS_BSPARSE]
        nb = (n + 63) // 64
        nwords, nbw = (n + 31) // 32, (nb + 31) // 32
        nv_max = max([g[1] for g in vs], default=0)
        ns_max = max([g[2] for g in vs], default=0)
        k_max = max([g[1] for g in bs], default=0)
        z = lambda *s: torch.zeros(s, dtype=i, device=device)
        self.vs_vsorted = z(nunits, len(vs), max(nv_max, 1)) if vs else None
        self.vs_dsorted = z(nunits, len(vs), max(ns_max, 1)) if vs else None
        self.vs_count = z(nunits, len(vs), 2) if vs else None
        self.vs_vbits = z(nunits, len(vs), nwords) if vs else None
        self.vs_dbits = z(nunits, len(vs), nwords) if vs else None
        self.bs_rank = z(hq, nb, k_max) if bs else None
        self.bs_sorted = z(hq, len(bs), nb, k_max) if bs else None
        self.bs_count = z(hq, len(bs), nb) if bs else None
        self.bs_bits = z(hq, len(bs), nb, nbw) if bs else None
        self.c = RsIndexSet(nunits=nunits, n=n, nb=nb, hq=hq, nv_max=nv_max, ns_max=ns_max,
                            k_max=k_max, nwords=nwords, ncand_vs=len(vs), ncand_bs=len(bs), nbw=nbw)
        for name in ("vs_vsorted", "vs_dsorted", "vs_count", "vs_vbits", "vs_dbits", "bs_rank",
                     "bs_sorted", "bs_count", "bs_bits"):
            t = getattr(self, name)
            setattr(self.c, name, t.data_ptr() if t is not None else None)


# ---- the C ABI, same names --------------------------------------------------------------

def rs_probe_workspace_size(qkv, units, nunits, cfg):
    return lib().rs_probe_workspace_size(C.byref(qkv), units, nunits, C.byref(cfg))


def rs_probe(qkv, units, nunits, cfg, grid, ncand, idx, ws, out, stream=None):
    return _check(lib().rs_probe(C.byref(qkv), units, nunits, C.byref(cfg), grid, ncand,
                                 C.byref(idx.c) if idx is not None else None, _ptr(ws),
                                 ws.numel() if ws is not None else 0, C.byref(out.c), _stream(stream)))


def rs_build_indices_workspace_size(scores, grid, ncand):
    return lib().rs_build_indices_workspace_size(C.byref(scores.c), grid, ncand)


def rs_build_indices(scores, units, nunits, grid, ncand, ws, out, stream=None):
    return _check(lib().rs_build_indices(C.byref(scores.c), units, nunits, grid, ncand, _ptr(ws),
                                         ws.numel() if ws is not None else 0, C.byref(out.c),
                                         _stream(stream)))


def rs_attn_workspace_size(qkv, units, nunits):
    return lib().rs_attn_workspace_size(C.byref(qkv), units, nunits)


def rs_sparse_attn_prefill(qkv, units, nunits, grid, ncand, idx, o, lse, ws, stream=None):
    return _check(lib().rs_sparse_attn_prefill(
        C.byref(qkv), units, nunits, grid, ncand, C.byref(idx.c) if idx is not None else None,
        _ptr(o), o.stride(0), o.stride(1), _ptr(lse), _ptr(ws), ws.numel() if ws is not None else 0,
        _stream(stream)))


def rs_dense_attn_prefill(qkv, units, nunits, o, lse, ws, stream=None):
    return _check(lib().rs_dense_attn_prefill(
        C.byref(qkv), units, nunits, _ptr(o), o.stride(0), o.stride(1), _ptr(lse), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def rs_route_layer(grid, cov, nsub, s1, t_table, bucket_edge, t_probe_us, T_layer_us, tau, alpha,
                   beta, delta_q, e=None):
    """Host-only router.  cov: float32 [U, C, 4], nsub: int32 [U, 3], s1: int32 [U],
    t_table: float64 [C, nbucket], bucket_edge: int32 [nbucket], e: float32 [U, C] or None.
    Returns (status, dict of outputs)."""
    import numpy as np
    cov = np.ascontiguousarray(cov, dtype=np.float32)
    U, Cn = cov.shape[0], cov.shape[1]
    nsub = np.ascontiguousarray(nsub, dtype=np.int32)
    s1 = np.ascontiguousarray(s1, dtype=np.int32)
    t_table = np.ascontiguousarray(t_table, dtype=np.float64)
    bucket_edge = np.ascontiguousarray(bucket_edge, dtype=np.int32)
    e_arr = None if e is None else np.ascontiguousarray(e, dtype=np.float32)
    g = make_grid(grid)
    rin = RsRouteIn(nunits=U, ncand=Cn, grid=C.cast(g, P), cov=cov.ctypes.data, nsub=nsub.ctypes.data,
                    e=e_arr.ctypes.data if e_arr is not None else None, s1=s1.ctypes.data,
                    t_table=t_table.ctypes.data, bucket_edge=bucket_edge.ctypes.data,
                    nbucket=len(bucket_edge), t_probe_us=t_probe_us)
    cfg = RsRouteCfg(T_layer_us=T_layer_us, tau=tau, alpha=alpha, beta=beta, delta_q=delta_q)
    choice = np.zeros(max(U, 1), np.int32)
    gc = np.zeros(Cn, np.int32)
    gs = np.zeros(Cn + 1, np.int32)
    gu = np.zeros(max(U, 1), np.int32)
    risk = np.zeros((max(U, 1), Cn), np.float64)
    ml = np.zeros((max(U, 1), Cn), np.float64)
    out = RsRouteOut(choice=choice.ctypes.data, group_cand=gc.ctypes.data, group_start=gs.ctypes.data,
                     group_units=gu.ctypes.data, risk=risk.ctypes.data, m_lower=ml.ctypes.data)
    st = _check(lib().rs_route_layer(C.byref(rin), C.byref(cfg), C.byref(out)),
                allow=(RS_ERR_BUDGET_INFEASIBLE,))
    ng = out.ngroups
    groups = [(int(gc[k]), [int(x) for x in gu[gs[k]:gs[k + 1]]]) for k in range(ng)]
    return st, dict(choice=[int(x) for x in choice[:U]], groups=groups, total=out.total_us,
                    risk=out.total_risk, n_fallback=out.n_fallback, over_budget=bool(out.over_budget),
                    infeasible=bool(out.infeasible), R=risk[:U], ML=ml[:U])


def make_error_model(w) -> RsErrorModel:
    """w: [4][4] non-negative weights, [family][feature]."""
    m = RsErrorModel()
    for f in range(4):
        for k in range(4):
            m.w[f][k] = float(w[f][k])
    return m


def rs_error_predict(probe, grid, ncand, model, e, stream=None):
    """e: float32 device tensor [nunits, ncand]."""
    return _check(lib().rs_error_predict(C.byref(probe.c), grid, ncand, C.byref(model), _ptr(e),
                                         _stream(stream)))


class RouteDevBuffers:
    """Device inputs and outputs of rs_route_layer_device for a fixed layer shape: the unit key
    lengths, the latency table and its bucket edges (uploaded once), the route outputs and the
    workspace."""

    def __init__(self, grid, s1, t_table, bucket_edge, device="cuda"):
        import numpy as np
        import torch
        grid = list(grid)
        U, Cn = len(s1), len(grid)
        self.U, self.C = U, Cn
        self.grid = make_grid(grid)
        i, d = torch.int32, torch.float64
        self.s1 = torch.as_tensor(np.asarray(s1, np.int32), device=device)
        self.t_table = torch.as_tensor(np.ascontiguousarray(t_table, np.float64), device=device)
        self.bucket_edge = torch.as_tensor(np.asarray(bucket_edge, np.int32), device=device)
        self.nbucket = len(bucket_edge)
        self.choice = torch.zeros(max(U, 1), dtype=i, device=device)
        self.group_cand = torch.zeros(Cn, dtype=i, device=device)
        self.group_start = torch.zeros(Cn + 1, dtype=i, device=device)
        self.group_units = torch.zeros(max(U, 1), dtype=i, device=device)
        self.risk = torch.zeros((max(U, 1), Cn), dtype=d, device=device)
        self.m_lower = torch.zeros((max(U, 1), Cn), dtype=d, device=device)
        self.status = torch.zeros(4, dtype=i, device=device)
        self.totals = torch.zeros(2, dtype=d, device=device)
        self.ws = workspace(lib().rs_route_layer_device_workspace_size(U, Cn), device=device)
        self.out = RsRouteDevOut(choice=self.choice.data_ptr(), group_cand=self.group_cand.data_ptr(),
                                 group_start=self.group_start.data_ptr(), group_units=self.group_units.data_ptr(),
                                 risk=self.risk.data_ptr(), m_lower=self.m_lower.data_ptr(),
                                 status=self.status.data_ptr(), totals=self.totals.data_ptr())

    def result(self):
        """The route as rs_route_layer returns it (copies to the host; synchronises)."""
        st = self.status.cpu().tolist()
        tot = self.totals.cpu().tolist()
        gc = self.group_cand.cpu().tolist()
        gs = self.group_start.cpu().tolist()
        gu = self.group_units.cpu().tolist()
        ng = st[0]
        return dict(choice=self.choice[:self.U].cpu().tolist(),
                    groups=[(gc[k], gu[gs[k]:gs[k + 1]]) for k in range(ng)],
                    total=tot[0], risk=tot[1], n_fallback=st[1], over_budget=bool(st[2]),
                    infeasible=bool(st[3]), R=self.risk[:self.U].cpu().numpy(),
                    ML=self.m_lower[:self.U].cpu().numpy())


def rs_route_layer_device(rb, cov, nsub, t_probe_us, T_layer_us, tau, alpha, beta, delta_q, e=None,
                          stream=None):
    """cov: float32 device [U, C, 4], nsub: int32 device [U, 3], e: float32 device [U, C] or None."""
    rin = RsRouteIn(nunits=rb.U, ncand=rb.C, grid=C.cast(rb.grid, P), cov=cov.data_ptr(), nsub=nsub.data_ptr(),
                    e=e.data_ptr() if e is not None else None, s1=rb.s1.data_ptr(),
                    t_table=rb.t_table.data_ptr(), bucket_edge=rb.bucket_edge.data_ptr(), nbucket=rb.nbucket,
                    t_probe_us=t_probe_us)
    cfg = RsRouteCfg(T_layer_us=T_layer_us, tau=tau, alpha=alpha, beta=beta, delta_q=delta_q)
    return _check(lib().rs_route_layer_device(C.byref(rin), C.byref(cfg), C.byref(rb.out), _ptr(rb.ws),
                                              rb.ws.numel(), _stream(stream)))


def rs_route_layer_device_noalloc(rb, cov, nsub, t_probe_us, T_layer_us, tau, alpha, beta, delta_q, e=None,
                                  stream=None):
    """As rs_route_layer_device, with the library's fixed scratch instead of rb.ws."""
    rin = RsRouteIn(nunits=rb.U, ncand=rb.C, grid=C.cast(rb.grid, P), cov=cov.data_ptr(), nsub=nsub.data_ptr(),
                    e=e.data_ptr() if e is not None else None, s1=rb.s1.data_ptr(),
                    t_table=rb.t_table.data_ptr(), bucket_edge=rb.bucket_edge.data_ptr(), nbucket=rb.nbucket,
                    t_probe_us=t_probe_us)
    cfg = RsRouteCfg(T_layer_us=T_layer_us, tau=tau, alpha=alpha, beta=beta, delta_q=delta_q)
    return _check(lib().rs_route_layer_device_noalloc(C.byref(rin), C.byref(cfg), C.byref(rb.out), _stream(stream)))


def rs_routed_attn_workspace_size(qkv, units, nunits):
    return lib().rs_routed_attn_workspace_size(C.byref(qkv), units, nunits)


def rs_routed_attn_prefill(qkv, units, nunits, grid, ncand, idx, choice, o, lse, ws, events=None, stream=None):
    """choice: int32 device tensor [nunits]; events: five torch.cuda.Event (timing enabled) or
    None.  Each event is recorded once here first so that it exists."""
    ev = None
    if events is not None:
        assert len(events) == 5
        for e in events:
            e.record()
        ev = (P * 5)(*[C.c_void_p(e.cuda_event) for e in events])
    return _check(lib().rs_routed_attn_prefill(
        C.byref(qkv), units, nunits, grid, ncand, C.byref(idx.c) if idx is not None else None, _ptr(choice),
        _ptr(o), o.stride(0), o.stride(1), _ptr(lse), _ptr(ws), ws.numel() if ws is not None else 0, ev,
        _stream(stream)))
