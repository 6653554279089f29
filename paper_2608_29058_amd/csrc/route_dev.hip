// Device side of routing (Sec. 3.3 error predictor; Sec. 3.4 router; inference-procedure
// steps 3-6 without a host round trip), for gfx950.  Compiled with floating-point
// contraction disabled: the router's fp64 operations are those of the host router, in the
// same order, so both give bit-identical routes.
//
//   error_predict_kernel  e(u, c) of the risk score from the probe's coverage and descriptors
//   route_kernel          the greedy latency-constrained solve, the tau step and the grouping,
//                         one workgroup
//   plan_kernel           per family, the work queues of the attention launch (query tiles of
//                         the units routed to the family, one queue per key/value bucket, longest
//                         first; block-sparse units of two heads with the same rows and key/value
//                         head share 64-row items), one workgroup per family
//
// Greedy on the device.  The host solve repeatedly applies the (unit, candidate)
// substitution of minimum ratio rho = (R(c) - R(cur)) / (t(cur) - t(c)) over strictly cheaper
// candidates, ties to the lowest unit and then the lowest candidate, until the unit-order
// total is within the budget.  A unit's next move depends only on its own current choice, so
// every unit's sequence of moves (its path) is fixed in advance; the solve merges the paths,
// always taking the smallest head.  That merge takes the moves in increasing order of
// (K, unit, position), K being the running maximum of rho along the unit's path: a move whose
// rho is below an earlier move of its unit is taken right after that move.  The kernel builds
// the paths (one thread per unit), sorts the moves by that key, and finds by bisection the
// first prefix of the order after which the total (recomputed in unit order, non-increasing
// in the prefix length) is within the budget.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace rs {

constexpr int kRouteMaxUnits = 2048;
constexpr int kRouteMaxMoves = 4096;
constexpr int kMaxCandR = 16;

// ---- error predictor ---------------------------------------------------------------------
struct EpArgs {
  int nunits, rmax, ncand;
  int fam[kMaxCandR];
  float w[4][4];
  const float *cov, *entropy, *local;
  const int *nsub;
  float *e;
};

__global__ void __launch_bounds__(64) error_predict_kernel(const EpArgs a) {
  const int u = blockIdx.x, lane = threadIdx.x;
  __shared__ double sHL[2];
  if (lane == 0) {
    const int nr = min(a.rmax, a.nsub[u * 3 + 0] + a.nsub[u * 3 + 1] + a.nsub[u * 3 + 2]);
    double h = 0.0, l = 0.0;
    for (int r = 0; r < nr; ++r) {
      h = h + (double)a.entropy[(long long)u * a.rmax + r];
      l = l + (double)a.local[(long long)u * a.rmax + r];
    }
    sHL[0] = nr > 0 ? h / (double)nr : 0.0;
    sHL[1] = nr > 0 ? l / (double)nr : 0.0;
  }
  __syncthreads();
  const int c = lane;
  if (c >= a.ncand) return;
  const int f = a.fam[c];
  float out = 0.f;
  if (f != RS_DENSE) {
    const float *cv = a.cov + ((long long)u * a.ncand + c) * 4;
    double vmax = 0.0, vmin = 0.0;
    int nv = 0;
    for (int s = 0; s < 3; ++s) {
      if (a.nsub[u * 3 + s] <= 0) continue;
      const double x = (double)cv[1 + s];
      if (nv == 0) {
        vmax = x;
        vmin = x;
      } else {
        vmax = vmax < x ? x : vmax;
        vmin = x < vmin ? x : vmin;
      }
      ++nv;
    }
    const double om = 1.0 - (double)cv[0];
    const double uu = nv <= 1 ? 0.0 : vmax - vmin;
    const double x[4] = {om, uu, om * sHL[0], om * (1.0 - sHL[1])};
    double acc = 0.0;
    for (int k = 0; k < 4; ++k) acc = acc + (double)a.w[f][k] * x[k];
    out = (float)acc;
  }
  a.e[(long long)u * a.ncand + c] = out;
}

// ---- router ------------------------------------------------------------------------------
struct RouteArgs {
  int U, C, nbucket, dense_c;
  int fam[kMaxCandR], brank[kMaxCandR];
  const float *cov, *e;
  const int *nsub, *s1, *bucket_edge;
  const double *t_table;
  double t_probe, T, tau, alpha, beta, delta_q;
  int *choice, *group_cand, *group_start, *group_units, *status;
  double *risk, *m_lower, *totals;
  double *t;    // [U][C] latency per (unit, candidate)
  int *path;    // [U][C-1] candidates along the unit's path
  int *rank;    // [U][C-1] position of each move in the merged order
  int *plen;    // [U] moves on the unit's path
};

__global__ void __launch_bounds__(1024) route_kernel(const RouteArgs a) {
  const int U = a.U, C = a.C, W = C - 1;
  const int tid = threadIdx.x, NT = blockDim.x;
  __shared__ double sKey[kRouteMaxMoves];  // sort keys; later the per-unit times of a total
  __shared__ int sId[kRouteMaxMoves];
  __shared__ double sTot;
  __shared__ int sPlen[kRouteMaxUnits];
  __shared__ int sFb, sNvalid, sCnt[kMaxCandR], sStart[kMaxCandR + 1];

  // latency, risk and lower mass per (unit, candidate)
  for (int i = tid; i < U * C; i += NT) {
    const int u = i / C, c = i % C;
    int b = a.nbucket - 1;
    for (int k = 0; k < a.nbucket; ++k)
      if (a.bucket_edge[k] >= a.s1[u]) {
        b = k;
        break;
      }
    a.t[i] = a.t_table[(long long)c * a.nbucket + b];
    double R = 0.0, ML = 1.0;
    if (a.fam[c] != RS_DENSE) {
      const float *cv = a.cov + (long long)i * 4;
      const double mh = (double)cv[0];
      double vmax = 0.0, vmin = 0.0;
      int nv = 0;
      for (int s = 0; s < 3; ++s) {
        if (a.nsub[u * 3 + s] <= 0) continue;
        const double x = (double)cv[1 + s];
        if (nv == 0) {
          vmax = x;
          vmin = x;
        } else {
          vmax = vmax < x ? x : vmax;
          vmin = x < vmin ? x : vmin;
        }
        ++nv;
      }
      const double uu = nv <= 1 ? 0.0 : vmax - vmin;
      const double e = a.e ? (double)a.e[i] : 0.0;
      R = (1.0 - mh) + a.alpha * uu + a.beta * e;
      const double lm = mh - a.delta_q;
      ML = 0.0 < lm ? lm : 0.0;
    }
    a.risk[i] = R;
    a.m_lower[i] = ML;
  }
  if (tid == 0) sFb = 0;
  __syncthreads();

  // each unit's path: from dense, repeatedly its best strictly cheaper candidate
  int Mp = 1;
  while (Mp < U * W) Mp <<= 1;
  for (int u = tid; u < U; u += NT) {
    int cur = a.dense_c, len = 0;
    double K = 0.0;
    for (;;) {
      const double tc = a.t[(long long)u * C + cur], rc = a.risk[(long long)u * C + cur];
      int bc = -1;
      double br = 0.0;
      for (int c = 0; c < C; ++c) {
        const double tn = a.t[(long long)u * C + c];
        if (!(tn < tc)) continue;
        const double rho = (a.risk[(long long)u * C + c] - rc) / (tc - tn);
        if (bc < 0 || rho < br) {
          br = rho;
          bc = c;
        }
      }
      if (bc < 0) break;
      K = (len == 0 || br > K) ? br : K;
      a.path[u * W + len] = bc;
      sKey[u * W + len] = K;
      sId[u * W + len] = u * W + len;
      ++len;
      cur = bc;
    }
    a.plen[u] = len;
    sPlen[u] = len;
    for (int j = len; j < W; ++j) {
      sKey[u * W + j] = INFINITY;
      sId[u * W + j] = 0x7fffffff;
    }
  }
  for (int i = U * W + tid; i < Mp; i += NT) {
    sKey[i] = INFINITY;
    sId[i] = 0x7fffffff;
  }
  __syncthreads();

  // bitonic sort of the moves by (K, unit, position); unused slots sort last
  for (int k = 2; k <= Mp; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < Mp; i += NT) {
        const int l = i ^ j;
        if (l <= i) continue;
        const bool up = (i & k) == 0;
        const double ki = sKey[i], kl = sKey[l];
        const int ii = sId[i], il = sId[l];
        const bool gt = ki > kl || (ki == kl && ii > il);
        if (gt == up) {
          sKey[i] = kl;
          sKey[l] = ki;
          sId[i] = il;
          sId[l] = ii;
        }
      }
      __syncthreads();
    }
  for (int i = tid; i < Mp; i += NT) {
    const int id = sId[i];
    if (id != 0x7fffffff) a.rank[id] = i;
  }
  if (tid == 0) {
    int nv = 0;
    for (int u = 0; u < U; ++u) nv += sPlen[u];
    sNvalid = nv;
  }
  __syncthreads();
  const int nvalid = sNvalid;

  // unit-order total after the first k moves of the merged order
  double *sTu = sKey;
  auto total_after = [&](int k) -> double {
    __syncthreads();
    for (int u = tid; u < U; u += NT) {
      int cnt = 0;
      for (int j = 0; j < sPlen[u]; ++j) cnt += a.rank[u * W + j] < k;
      const int ch = cnt == 0 ? a.dense_c : a.path[u * W + cnt - 1];
      sTu[u] = a.t[(long long)u * C + ch];
    }
    __syncthreads();
    if (tid == 0) {
      double tot = a.t_probe;
      for (int u = 0; u < U; ++u) tot = tot + sTu[u];
      sTot = tot;
    }
    __syncthreads();
    return sTot;
  };
  int kstar = 0;
  bool infeasible = false;
  if (total_after(0) > a.T) {
    if (total_after(nvalid) > a.T) {
      kstar = nvalid;
      infeasible = true;
    } else {
      int lo = 0, hi = nvalid;  // total(lo) > T >= total(hi)
      while (hi - lo > 1) {
        const int mid = lo + (hi - lo) / 2;
        if (total_after(mid) > a.T) lo = mid;
        else hi = mid;
      }
      kstar = hi;
    }
  }
  __syncthreads();

  // the solve's choice, then expand or fall back
  for (int u = tid; u < U; u += NT) {
    int cnt = 0;
    for (int j = 0; j < sPlen[u]; ++j) cnt += a.rank[u * W + j] < kstar;
    int ch = cnt == 0 ? a.dense_c : a.path[u * W + cnt - 1];
    const double *ml = a.m_lower + (long long)u * C;
    if (a.fam[ch] != RS_DENSE && !(ml[ch] >= a.tau)) {
      int pick = -1, pick_rank = 1 << 30;
      for (int c2 = 0; c2 < C; ++c2) {
        if (a.fam[c2] != a.fam[ch] || a.brank[c2] <= a.brank[ch]) continue;
        if (ml[c2] >= a.tau && a.brank[c2] < pick_rank) {
          pick = c2;
          pick_rank = a.brank[c2];
        }
      }
      if (pick < 0) {
        double best_t = 0.0;
        for (int c2 = 0; c2 < C; ++c2) {
          if (a.fam[c2] == RS_DENSE || !(ml[c2] >= a.tau)) continue;
          const double tt = a.t[(long long)u * C + c2];
          if (pick < 0 || tt < best_t) {
            best_t = tt;
            pick = c2;
          }
        }
      }
      if (pick < 0) {
        pick = a.dense_c;
        atomicAdd(&sFb, 1);
      }
      ch = pick;
    }
    a.choice[u] = ch;
    sId[u] = ch;                                   // the choice, for the serial loops below
    sKey[u] = a.t[(long long)u * C + ch];          // its time
    sKey[kRouteMaxUnits + u] = a.risk[(long long)u * C + ch];  // its risk
  }
  for (int c = tid; c < C; c += NT) sCnt[c] = 0;
  __syncthreads();
  for (int u = tid; u < U; u += NT) atomicAdd(&sCnt[sId[u]], 1);
  __syncthreads();
  if (tid == 0) {
    double tot = a.t_probe, rsum = 0.0;
    for (int u = 0; u < U; ++u) {
      tot = tot + sKey[u];
      rsum = rsum + sKey[kRouteMaxUnits + u];
    }
    int ng = 0, pos = 0;
    for (int c = 0; c < C; ++c) {
      sStart[c] = pos;
      if (sCnt[c] > 0) {
        a.group_cand[ng] = c;
        a.group_start[ng] = pos;
        ++ng;
      }
      pos += sCnt[c];
    }
    a.group_start[ng] = pos;
    a.status[0] = ng;
    a.status[1] = sFb;
    a.status[3] = infeasible ? 1 : 0;
    a.status[2] = (infeasible || tot > a.T) ? 1 : 0;
    a.totals[0] = tot;
    a.totals[1] = rsum;
  }
  __syncthreads();
  // group members in ascending unit order, one thread per candidate
  for (int c = tid; c < C; c += NT) {
    int pos = sStart[c];
    for (int u = 0; u < U; ++u)
      if (sId[u] == c) a.group_units[pos++] = u;
  }
}

// ---- work lists of the routed attention launches -------------------------------------------
struct PlanArgs {
  int U, C, group, bm;
  int fam[kMaxCandR], cl[kMaxCandR], ca[kMaxCandR], cb[kMaxCandR];
  const rs_unit *units;
  const int *choice;
  DevUnit *dunits;  // [4][U]
  int *order;       // [4][max_items], bucket-major
  int max_items;
  int *qsize, *qoff, *qcount;  // [4][8] each
};

__global__ void __launch_bounds__(1024) plan_kernel(const PlanArgs a) {
  const int f = blockIdx.x, tid = threadIdx.x, NT = blockDim.x;
  __shared__ int sLu2u[kRouteMaxUnits];   // local unit -> unit
  __shared__ int sOff[kRouteMaxUnits + 1];  // local unit -> first flat item
  __shared__ int sBl[kRouteMaxUnits];     // units of each bucket, ascending
  // items of a unit: n of them, the j-th starting at row 64 (k0 + g j); g = 2 for 128-row
  // query tiles, 1 for the 64-row query blocks of a block-sparse unit with a mate
  __shared__ int sK0[kRouteMaxUnits], sN[kRouteMaxUnits], sG[kRouteMaxUnits];
  __shared__ int sBk[kRouteMaxUnits];     // bucket of a unit, -1 when routed to another family
  __shared__ int sMate[kRouteMaxUnits];   // unit taken along (block-sparse), -2 taken along, -1
  __shared__ int sBs[9], sSize[8], sNl;
  const int U = a.U, bm = a.bm;
  // per unit, in parallel: bucket and whether the unit is routed to this family
  for (int u = tid; u < U; u += NT) {
    const rs_unit un = a.units[u];
    const int c = a.choice[u];
    sBk[u] = (c >= 0 && c < a.C && a.fam[c] == f) ? (un.head / a.group) & 7 : -1;
    sMate[u] = -1;
  }
  __syncthreads();
  // block-sparse mates: the first unit of an even head h takes along the first unit of head
  // h + 1 with the same rows when both are routed here and read the same key/value head
  if (f == RS_BSPARSE) {
    for (int u = tid; u < U; u += NT) {
      const rs_unit un = a.units[u];
      const int h = un.head;
      if (sBk[u] < 0 || (h & 1) || (h + 1) / a.group != h / a.group) continue;
      int v = -1;
      bool first = true;
      for (int w = 0; w < U && first; ++w) {
        if (sBk[w] != sBk[u]) continue;  // a mate reads the same key/value head: same bucket
        const rs_unit x = a.units[w];
        if (x.s0 != un.s0 || x.s1 != un.s1) continue;
        if (x.head == h && w < u) first = false;
        if (x.head == h + 1 && v < 0) v = w;
      }
      if (first && v >= 0) {
        sMate[u] = v;
        sMate[v] = -2;
      }
    }
    __syncthreads();
  }
  for (int u = tid; u < U; u += NT) {
    const rs_unit un = a.units[u];
    if (sMate[u] >= 0) {
      sK0[u] = un.s0 / 64;
      sN[u] = (un.s1 - 1) / 64 - un.s0 / 64 + 1;
      sG[u] = 1;
    } else {
      sK0[u] = 2 * (un.s0 / bm);
      sN[u] = sMate[u] == -2 ? 0 : (un.s1 - 1) / bm - un.s0 / bm + 1;
      sG[u] = 2;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int nl = 0, cntb[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int b = 0; b < 8; ++b) sSize[b] = 0;
    sOff[0] = 0;
    for (int u = 0; u < U; ++u) {
      const int b = sBk[u];
      if (b < 0 || sMate[u] == -2) continue;
      const int nt = sN[u];
      sLu2u[nl] = u;
      sOff[nl + 1] = sOff[nl] + nt;
      sSize[b] += nt;
      ++cntb[b];
      ++nl;
    }
    sBs[0] = 0;
    for (int b = 0; b < 8; ++b) sBs[b + 1] = sBs[b] + cntb[b];
    int fill[8];
    for (int b = 0; b < 8; ++b) fill[b] = sBs[b];
    for (int l = 0; l < nl; ++l) {
      const int u = sLu2u[l];
      sBl[fill[sBk[u]]++] = u;
    }
    sNl = nl;
    int off = 0;
    for (int b = 0; b < 8; ++b) {
      a.qsize[f * 8 + b] = sSize[b];
      a.qoff[f * 8 + b] = off;
      a.qcount[f * 8 + b] = 0;
      off += sSize[b];
    }
  }
  __syncthreads();
  const int nl = sNl, total = sOff[nl];
  DevUnit *dunits = a.dunits + (long long)f * U;
  int *order = a.order + (long long)f * a.max_items;
  for (int l = tid; l < nl; l += NT) {
    const int u = sLu2u[l];
    const rs_unit &un = a.units[u];
    const int c = a.choice[u];
    const int m = sMate[u];
    dunits[l] = DevUnit{un.head, un.s0, un.s1, a.cl[c], un.slot, f == RS_ASHAPE ? a.ca[c] : 0,
                        f == RS_ASHAPE ? a.cb[c] : 0, m >= 0 ? a.units[m].head + 1 : 0,
                        m >= 0 ? a.cl[a.choice[m]] : 0};
  }
  for (int i = tid; i < total; i += NT) {
    int lo = 0, hi = nl - 1;  // local unit holding flat item i
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sOff[mid] <= i) lo = mid;
      else hi = mid - 1;
    }
    const int u = sLu2u[lo], t = i - sOff[lo];
    const int key = sK0[u] + sG[u] * t;  // first row / 64
    const int b = sBk[u];
    // rank in the bucket: later query rows first, then units ascending
    int r = 0;
    for (int x = sBs[b]; x < sBs[b + 1]; ++x) {
      const int v = sBl[x];
      const int k0 = sK0[v], g = sG[v], n = sN[v];
      const int below = key < k0 ? 0 : min(n, (key - k0) / g + 1);  // items of v starting at or before key
      r += n - below;
      r += (v < u && key >= k0 && (key - k0) % g == 0 && (key - k0) / g < n) ? 1 : 0;
    }
    int off = 0;
    for (int bb = 0; bb < b; ++bb) off += sSize[bb];
    order[off + r] = (lo << 16) | t;
  }
}

// ---- host launchers ----------------------------------------------------------------------
static int tiles128(const rs_unit &u) { return (u.s1 - 1) / 128 - u.s0 / 128 + 1; }

rs_status error_predict_launch(const rs_probe_out *p, const rs_candidate *grid, int32_t ncand,
                               const rs_error_model *m, float *e, hipStream_t st) {
  EpArgs a{};
  a.nunits = p->nunits;
  a.rmax = p->rmax;
  a.ncand = ncand;
  for (int c = 0; c < ncand; ++c) a.fam[c] = grid[c].fam;
  for (int f = 0; f < 4; ++f)
    for (int k = 0; k < 4; ++k) a.w[f][k] = m->w[f][k];
  a.cov = p->cov;
  a.entropy = p->entropy;
  a.local = p->local;
  a.nsub = p->nsub;
  a.e = e;
  if (p->nunits == 0) return RS_OK;
  hipLaunchKernelGGL(error_predict_kernel, dim3(p->nunits), dim3(64), 0, st, a);
  RS_HIP(hipGetLastError());
  return RS_OK;
}

size_t route_dev_ws_bytes(int32_t nunits, int32_t ncand) {
  Arena ar(nullptr, 0);
  ar.take<double>((size_t)nunits * ncand);
  ar.take<int>((size_t)nunits * (ncand > 1 ? ncand - 1 : 1));
  ar.take<int>((size_t)nunits * (ncand > 1 ? ncand - 1 : 1));
  ar.take<int>((size_t)nunits);
  return ar.off + 256;
}

// ---- allocation-free device routing ------------------------------------------------------
// The router's scratch (per-(unit, candidate) latency, the units' greedy paths and the merged
// order's ranks) in a fixed device array instead of a caller workspace.  Every element the
// kernel reads it has written earlier in the same launch, so nothing needs clearing between
// calls.  The largest workspace the limits allow (nunits <= 2048, nunits * (ncand - 1) <=
// 4096, ncand <= 16) is 16 U (C - 1) + 12 U <= 90112 bytes plus alignment: 96 KiB holds it.
constexpr size_t kRouteScratchBytes = 96 * 1024;
static __device__ __align__(256) char scratch[kRouteScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each GPU, once known

// Device address of this GPU's copy of the scratch array (the host symbol is only a
// stand-in): looked up once per device, with that device current.
static rs_status route_scratch(void **ptr) {
  int dev = 0;
  RS_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(RS_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    RS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(RS_ERR_HIP, "hipGetSymbolAddress returned no address for the routing scratch");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return RS_OK;
}

rs_status route_dev_launch(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                           const int *fam, const int *brank, int dense_c, void *ws, size_t ws_bytes,
                           hipStream_t st);

rs_status route_dev_launch_noalloc(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                                   const int *fam, const int *brank, int dense_c, hipStream_t st) {
  const int U = in->nunits, C = in->ncand;
  if (U > kRouteMaxUnits || U * (C - 1) > kRouteMaxMoves)
    return fail(RS_ERR_UNSUPPORTED, "device routing supports nunits <= 2048 and nunits * (ncand - 1) <= 4096");
  if (route_dev_ws_bytes(U, C) > kRouteScratchBytes)
    return fail(RS_ERR_UNSUPPORTED, "routing scratch needs " + std::to_string(route_dev_ws_bytes(U, C)) +
                                        " bytes, more than the fixed " + std::to_string(kRouteScratchBytes));
  void *ptr = nullptr;
  rs_status s = route_scratch(&ptr);
  if (s != RS_OK) return s;
  return route_dev_launch(in, cfg, out, fam, brank, dense_c, ptr, kRouteScratchBytes, st);
}

rs_status route_dev_launch(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                           const int *fam, const int *brank, int dense_c, void *ws, size_t ws_bytes,
                           hipStream_t st) {
  const int U = in->nunits, C = in->ncand;
  if (U > kRouteMaxUnits || U * (C - 1) > kRouteMaxMoves)
    return fail(RS_ERR_UNSUPPORTED, "device routing supports nunits <= 2048 and nunits * (ncand - 1) <= 4096");
  const size_t need = route_dev_ws_bytes(U, C);
  if (!ws || ws_bytes < need)
    return fail(RS_ERR_WORKSPACE, "device routing workspace too small: need " + std::to_string(need) + " bytes");
  RouteArgs a{};
  a.U = U;
  a.C = C;
  a.nbucket = in->nbucket;
  a.dense_c = dense_c;
  for (int c = 0; c < C; ++c) {
    a.fam[c] = fam[c];
    a.brank[c] = brank[c];
  }
  a.cov = in->cov;
  a.e = in->e;
  a.nsub = in->nsub;
  a.s1 = in->s1;
  a.bucket_edge = in->bucket_edge;
  a.t_table = in->t_table;
  a.t_probe = in->t_probe_us;
  a.T = cfg->T_layer_us;
  a.tau = cfg->tau;
  a.alpha = cfg->alpha;
  a.beta = cfg->beta;
  a.delta_q = cfg->delta_q;
  a.choice = out->choice;
  a.group_cand = out->group_cand;
  a.group_start = out->group_start;
  a.group_units = out->group_units;
  a.status = out->status;
  a.risk = out->risk;
  a.m_lower = out->m_lower;
  a.totals = out->totals;
  Arena ar(ws, ws_bytes);
  a.t = ar.take<double>((size_t)U * C);
  a.path = ar.take<int>((size_t)U * (C > 1 ? C - 1 : 1));
  a.rank = ar.take<int>((size_t)U * (C > 1 ? C - 1 : 1));
  a.plen = ar.take<int>((size_t)U);
  hipLaunchKernelGGL(route_kernel, dim3(1), dim3(1024), 0, st, a);
  RS_HIP(hipGetLastError());
  return RS_OK;
}

size_t routed_attn_ws_bytes(const rs_unit *units, int32_t nunits) {
  size_t items = 0;
  for (int i = 0; i < nunits; ++i) items += (size_t)tiles128(units[i]);
  Arena ar(nullptr, 0);
  ar.take<rs_unit>((size_t)nunits);
  ar.take<int>(3 * 32);
  ar.take<DevUnit>(4 * (size_t)nunits);
  ar.take<int>(4 * items);
  return ar.off + 256;
}

rs_status routed_attn_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                             const rs_candidate *grid, int32_t ncand, const rs_index_set *idx, const int32_t *choice,
                             void *o, int64_t so_h, int64_t so_t, float *lse, void *ws, size_t ws_bytes,
                             void *const *events, hipStream_t st) {
  if (nunits == 0) return RS_OK;
  if (nunits > kRouteMaxUnits) return fail(RS_ERR_UNSUPPORTED, "routed attention supports nunits <= 2048");
  const size_t need = routed_attn_ws_bytes(units, nunits);
  if (!ws || ws_bytes < need)
    return fail(RS_ERR_WORKSPACE, "routed attention workspace too small: need " + std::to_string(need) + " bytes");
  int items = 0;
  for (int i = 0; i < nunits; ++i) items += tiles128(units[i]);
  Arena ar(ws, ws_bytes);
  rs_unit *d_units = ar.take<rs_unit>((size_t)nunits);
  int *d_q = ar.take<int>(3 * 32);
  PlanArgs p{};
  p.U = nunits;
  p.C = ncand;
  p.group = qkv->hq / qkv->hkv;
  p.bm = 128;
  bool present[4] = {false, false, false, false};
  int cnt[4] = {0, 0, 0, 0};
  for (int c = 0; c < ncand; ++c) {
    p.fam[c] = grid[c].fam;
    p.cl[c] = cnt[grid[c].fam]++;
    p.ca[c] = grid[c].a;
    p.cb[c] = grid[c].b;
    present[grid[c].fam] = true;
  }
  p.units = d_units;
  p.choice = choice;
  p.dunits = ar.take<DevUnit>(4 * (size_t)nunits);
  p.order = ar.take<int>(4 * (size_t)items);
  p.max_items = items;
  p.qsize = d_q;
  p.qoff = d_q + 32;
  p.qcount = d_q + 64;
  // the unit list: from the caller's unit table, else copied into the workspace (from the
  // caller's array, which the copy reads before hipMemcpyAsync returns)
  if (qkv->tables)
    p.units = unit_tab_units(qkv->tables);
  else
    RS_HIP(hipMemcpyAsync(d_units, units, (size_t)nunits * sizeof(rs_unit), hipMemcpyHostToDevice, st));
  hipLaunchKernelGGL(plan_kernel, dim3(4), dim3(1024), 0, st, p);
  RS_HIP(hipGetLastError());
  // persistent grids: two workgroups per compute unit (the kernel's occupancy), a multiple of 8
  int dev = 0, ncu = 0;
  RS_HIP(hipGetDevice(&dev));
  RS_HIP(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
  const int nblocks = std::min(((2 * ncu + 7) / 8) * 8, ((items + 7) / 8) * 8);
  // dense first: its tiles are the longest
  const int fam_order[4] = {RS_DENSE, RS_VSLASH, RS_BSPARSE, RS_ASHAPE};
  if (events) RS_HIP(hipEventRecord((hipEvent_t)events[0], st));
  for (int k = 0; k < 4; ++k) {
    const int f = fam_order[k];
    if (present[f]) {
      const AttnQueues qs{p.qsize + 8 * f, p.qoff + 8 * f, p.qcount + 8 * f};
      rs_status s = attn_launch_list(qkv, scale, f, idx, p.dunits + (size_t)f * nunits,
                                     p.order + (size_t)f * items, &qs, nblocks, o, so_h, so_t, lse, st);
      if (s != RS_OK) return s;
    }
    if (events) RS_HIP(hipEventRecord((hipEvent_t)events[1 + k], st));
  }
  return RS_OK;
}

}  // namespace rs
