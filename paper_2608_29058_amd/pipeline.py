"""Sequencing of one routed layer through the C ABI (inference-procedure steps 1-6).

No arithmetic happens here: this module allocates caller-owned buffers once and calls the
library in the order of the per-layer procedure (Sec. 3.4 and its table):
  0. rs_transpose_v (V in the operand layout of the dense, A-shape and block-sparse kernels)
  1. rs_probe (scores: sampled rows, col/diag, descriptors, block-mean logits)
  2. rs_build_indices, then rs_probe (coverage of every candidate)
  3-5. rs_route_layer on the host after copying the coverage back (latency lookup, greedy
       solve, expand/fallback, grouping), or rs_route_layer_device on the stream
  6. one rs_sparse_attn_prefill / rs_dense_attn_prefill launch per (pattern, budget) group, or
     after device routing one rs_routed_attn_prefill call (one launch per family, work lists
     built on the device: no host synchronisation in the layer).
With beta > 0 the calibrated error predictor (rs_error_predict) runs after the coverage.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import _rs


@dataclass
class RouteKnobs:
    T_layer_us: float = 1e30
    tau: float = 0.95
    alpha: float = 1.0
    beta: float = 0.0
    delta_q: float = 0.0
    error_model: object = None   # [4][4] non-negative weights of the error predictor (beta > 0)


@dataclass
class LayerTimes:
    phases_ms: dict = field(default_factory=dict)
    groups: list = field(default_factory=list)  # (cand, n_units, ms)


class RoutedLayer:
    """Buffers and call order of one routed layer for fixed shapes."""

    def __init__(self, n, hq, hkv, d, seg_len, grid, r_rec=64, r_uni=64, r_bnd=32, local_w=1024,
                 device="cuda", use_vt=True, use_tables=True):
        import torch
        self.n, self.hq, self.hkv, self.d = n, hq, hkv, d
        self.grid = list(grid)
        self.g = _rs.make_grid(self.grid)
        self.ncand = len(self.grid)
        segs = [(s, min(n, s + seg_len)) for s in range(0, n, seg_len)]
        self.unit_list = [(h, s0, s1) for (s0, s1) in segs for h in range(hq)]
        self.nunits = len(self.unit_list)
        self.units = _rs.make_units([(h, s0, s1, 0, i) for i, (h, s0, s1) in enumerate(self.unit_list)])
        self.cfg = _rs.RsProbeCfg(r_rec=r_rec, r_uni=r_uni, r_bnd=r_bnd, bs_block=64, local_w=local_w,
                                  flags=_rs.RS_PROBE_ROWS | _rs.RS_PROBE_BLOCKMEAN)
        self.rmax = r_rec + r_uni + r_bnd
        self.pb = _rs.ProbeBuffers(self.nunits, self.rmax, n, hq, self.ncand, blockmean=True, device=device)
        self.ib = _rs.IndexBuffers(self.nunits, n, hq, self.grid, device=device)
        self.o = torch.empty((hq, n, d), dtype=torch.bfloat16, device=device)
        # V in the transposed operand layout of rs_transpose_v (rewritten by every qkv() call)
        self.vt = (torch.empty(hkv * d * ((n + 63) // 64 * 64) * 2, dtype=torch.uint8, device=device)
                   if use_vt else None)
        self.s1 = np.array([u[2] for u in self.unit_list], np.int32)
        self.cov_host = torch.empty((self.nunits, self.ncand, 4), dtype=torch.float32, pin_memory=True)
        self.nsub_host = torch.empty((self.nunits, 3), dtype=torch.int32, pin_memory=True)
        self.e = torch.zeros((self.nunits, self.ncand), dtype=torch.float32, device=device)
        self.e_host = torch.empty((self.nunits, self.ncand), dtype=torch.float32, pin_memory=True)
        self.rb = None
        self._rb_table = None
        self.tables = None   # device unit tables (rs_unit_table_init), built with the first qkv()
        self.use_tables = use_tables
        self._ws = None
        self._ws_routed = None
        self.t_table = None
        self.edges = None
        self.t_probe_us = 0.0
        self.knobs = RouteKnobs()

    def qkv(self, q, k, v):
        """The layer's rs_qkv.  With the transposed-V layout on, this also (re)writes V^T of this
        layer into self.vt on the stream (rs_transpose_v): the returned descriptor is valid until
        the next qkv() call.  The descriptor carries the unit tables of the layer's unit list
        (built once, on the first call), so the layer's calls upload nothing."""
        qkv = _rs.make_qkv(q, k, v, vt=self.vt)
        if self.use_tables:
            if self.tables is None:
                self.tables = _rs.UnitTable(qkv, self.units, self.nunits, self.cfg)
                self.pb.c.tables = self.tables.ptr
            qkv.tables = self.tables.ptr
        if self.vt is None:
            return qkv
        assert _rs.rs_vt_bytes(qkv) == self.vt.numel()
        _rs.rs_transpose_v(qkv, self.vt)
        return qkv

    def workspace(self, qkv):
        if self._ws is None:
            need = max(_rs.rs_probe_workspace_size(qkv, self.units, self.nunits, self.cfg),
                       _rs.rs_build_indices_workspace_size(self.pb, self.g, self.ncand),
                       _rs.rs_attn_workspace_size(qkv, self.units, self.nunits))
            self._ws = _rs.workspace(need)
        return self._ws

    # -- steps ---------------------------------------------------------------------------
    def probe_and_index(self, qkv, mark=None):
        """Scores probe, index construction, coverage probe (``mark(name)`` after each)."""
        mark = mark or (lambda name: None)
        ws = self.workspace(qkv)
        _rs.rs_probe(qkv, self.units, self.nunits, self.cfg, None, 0, None, ws, self.pb)
        mark("probe_scores")
        _rs.rs_build_indices(self.pb, self.units, self.nunits, self.g, self.ncand, ws, self.ib)
        mark("indices")
        _rs.rs_probe(qkv, self.units, self.nunits, self.cfg, self.g, self.ncand, self.ib, ws, self.pb)

    def _use_e(self):
        return self.knobs.beta > 0 and self.knobs.error_model is not None

    def predict_error(self):
        """e of the risk score from this layer's probe (rs_error_predict), on the stream."""
        _rs.rs_error_predict(self.pb, self.g, self.ncand, _rs.make_error_model(self.knobs.error_model),
                             self.e)

    def route(self):
        import torch
        if self._use_e():
            self.predict_error()
            self.e_host.copy_(self.e, non_blocking=True)
        self.cov_host.copy_(self.pb.cov, non_blocking=True)
        self.nsub_host.copy_(self.pb.nsub, non_blocking=True)
        torch.cuda.current_stream().synchronize()
        k = self.knobs
        st, out = _rs.rs_route_layer(self.grid, self.cov_host.numpy(), self.nsub_host.numpy(), self.s1,
                                     self.t_table, self.edges, self.t_probe_us, k.T_layer_us, k.tau,
                                     k.alpha, k.beta, k.delta_q, e=self.e_host.numpy() if self._use_e() else None)
        return out

    def route_device(self):
        """rs_route_layer_device on the stream; the route stays in self.rb (device)."""
        if self.rb is None or self._rb_table is not self.t_table:   # latency table uploaded once
            self.rb = _rs.RouteDevBuffers(self.grid, self.s1, self.t_table, self.edges)
            self._rb_table = self.t_table
        k = self.knobs
        if self._use_e():
            self.predict_error()
        _rs.rs_route_layer_device(self.rb, self.pb.cov, self.pb.nsub, self.t_probe_us, k.T_layer_us, k.tau, k.alpha,
                                  k.beta, k.delta_q, e=self.e if self._use_e() else None)

    def run_routed(self, qkv, lse=None, family_events=None):
        """All units with the device route's choices: one rs_routed_attn_prefill call
        (``family_events``: five timing events around its per-family launches)."""
        if self._ws_routed is None:
            self._ws_routed = _rs.workspace(_rs.rs_routed_attn_workspace_size(qkv, self.units, self.nunits))
        _rs.rs_routed_attn_prefill(qkv, self.units, self.nunits, self.g, self.ncand, self.ib, self.rb.choice,
                                   self.o, lse, self._ws_routed, events=family_events)

    def group_units(self, cand, unit_idx):
        return _rs.make_units([(self.unit_list[u][0], self.unit_list[u][1], self.unit_list[u][2], cand, u)
                               for u in unit_idx])

    def run_group(self, qkv, cand, unit_idx, lse=None):
        ws = self.workspace(qkv)
        us = self.group_units(cand, unit_idx)
        if self.grid[cand][0] == _rs.RS_DENSE:
            _rs.rs_dense_attn_prefill(qkv, us, len(unit_idx), self.o, lse, ws)
        else:
            _rs.rs_sparse_attn_prefill(qkv, us, len(unit_idx), self.g, self.ncand, self.ib, self.o, lse, ws)

    def run(self, q, k, v, events=None, lse=None, per_unit=False, fixed_route=None, device_route=False,
            family_events=None):
        """One routed layer; returns the route (None with ``device_route``: it stays on the
        device, in self.rb).  ``events`` (optional) is a callable ``mark(name)`` used to record
        stream events between phases; ``lse`` (optional, float32 [hq, n]) receives the
        log-sum-exp of every row; ``per_unit`` launches each unit on its own instead of one
        launch per (pattern, budget) group; ``fixed_route`` (a route returned earlier) replaces
        the input-conditional routing decision while the index sets are still built from this
        input; ``device_route`` routes on the device and launches the attention from that route
        with no host synchronisation (``family_events``: see run_routed)."""
        mark = events or (lambda name: None)
        mark("start")
        qkv = self.qkv(q, k, v)
        if self.vt is not None:
            mark("transpose_v")
        self.probe_and_index(qkv, mark)
        mark("probe")
        if device_route:
            self.route_device()
            mark("route")
            self.run_routed(qkv, lse, family_events)
            mark("attention")
            return None
        route = self.route() if fixed_route is None else fixed_route
        mark("route")
        for ci, (cand, us) in enumerate(route["groups"]):
            if per_unit:
                for u in us:
                    self.run_group(qkv, cand, [u], lse)
            else:
                self.run_group(qkv, cand, us, lse)
            mark(f"group{ci}")
        return route

    # -- offline calibration (untimed) ---------------------------------------------------
    def profile_latency(self, qkv, edges, reps=3, tail=None):
        """Kernel latency table t_ker[candidate][bucket] in us per unit: for every candidate
        and key-length bucket, the time of one launch over every unit of that bucket (all
        query heads, as the routed launches hold many units) divided by their number; the
        median of ``reps`` launches.  Launches over one key/value group's heads alone price
        the families differently from the routed launches (measured: their routes ran ~3%
        slower and varied from run to run).  ``tail`` (optional dict) receives the 0.95
        quantile of the same launches under key "p95"."""
        import torch
        stream = torch.cuda.current_stream()
        t = np.zeros((self.ncand, len(edges)))
        t95 = np.zeros((self.ncand, len(edges)))
        for c in range(self.ncand):
            for b in range(len(edges)):
                us = [i for i, u in enumerate(self.unit_list) if u[2] == edges[b]]
                if not us:
                    continue
                ts = []
                for _ in range(reps):
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    self.run_group(qkv, c, us)
                    e1.record(stream)
                    e1.synchronize()
                    ts.append(e0.elapsed_time(e1))
                t[c, b] = float(np.median(ts)) / len(us) * 1e3
                t95[c, b] = float(np.quantile(ts, 0.95)) / len(us) * 1e3
        if tail is not None:
            tail["p95"] = t95
        return t

    def profile_probe(self, qkv, reps=3):
        """Median time of the V transpose (when on) + probe + indices + coverage, in us."""
        import torch
        stream = torch.cuda.current_stream()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if self.vt is not None:
                _rs.rs_transpose_v(qkv, self.vt)
            self.probe_and_index(qkv)
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts)) * 1e3
