// Latency-constrained routing of one layer (Sec. 3.4, Eqs. 6-8; inference-procedure
// steps 3-6): host-only, synchronous, pure.  Compiled with floating-point contraction
// disabled so every fp64 operation happens exactly in the order written.
//
//   risk      R(c) = (1 - m_hat) + alpha * u + beta * e, u = max - min of the non-empty
//             subset means; the dense candidate has R = 0 and m_lower = 1
//   lower     m_lower = max(0, m_hat - delta_q)
//   latency   t(u, c) = t_ker(c, bucket(s1_u)) from the profiled table
//   solve     all-dense start; while t_probe + sum_u t(u, choice_u) > T_layer, switch the
//             (unit, candidate) of minimum (R(c) - R(cur)) / (t(cur) - t(c)) among
//             strictly cheaper candidates, first minimum in (unit, candidate) order
//   expand    a sparse choice with m_lower < tau takes the smallest larger budget of its
//             family with m_lower >= tau, else the cheapest sparse candidate of any family
//             with m_lower >= tau (ties: lowest index), else dense
//   group     units grouped by candidate, grid order, ascending units
#include <algorithm>
#include <string>
#include <vector>

#include "../../include/rs.h"

namespace rs {
rs_status fail(rs_status st, const std::string &msg);
}

extern "C" rs_status rs_route_layer(const rs_route_in *in, const rs_route_cfg *cfg, rs_route_out *out) {
  using rs::fail;
  if (!in || !cfg || !out) return fail(RS_ERR_INVALID_ARG, "route: NULL argument");
  const int U = in->nunits, C = in->ncand;
  if (U < 0 || C < 1 || !in->grid) return fail(RS_ERR_INVALID_ARG, "route: bad sizes");
  if (U > 0 && (!in->cov || !in->nsub || !in->s1)) return fail(RS_ERR_INVALID_ARG, "route: missing inputs");
  if (in->nbucket < 1 || !in->t_table || !in->bucket_edge) return fail(RS_ERR_INVALID_ARG, "route: missing latency table");
  if (!out->choice || !out->group_cand || !out->group_start || !out->group_units || !out->risk || !out->m_lower)
    return fail(RS_ERR_INVALID_ARG, "route: missing outputs");
  std::vector<int> fam(C), brank(C);
  int dense_c = -1;
  for (int c = 0; c < C; ++c) {
    fam[c] = in->grid[c].fam;
    if (fam[c] < RS_DENSE || fam[c] > RS_BSPARSE) return fail(RS_ERR_INVALID_ARG, "route: unknown family");
    int k = 0;
    for (int c2 = 0; c2 < c; ++c2)
      if (in->grid[c2].fam == fam[c]) ++k;
    brank[c] = k;
    if (fam[c] == RS_DENSE && dense_c < 0) dense_c = c;
  }
  if (dense_c < 0) return fail(RS_ERR_INVALID_ARG, "route: the grid must contain a dense candidate");
  for (int k = 1; k < in->nbucket; ++k)
    if (in->bucket_edge[k] < in->bucket_edge[k - 1]) return fail(RS_ERR_INVALID_ARG, "route: bucket edges must ascend");

  // latency per (unit, candidate)
  std::vector<double> t((size_t)U * C), R((size_t)U * C), ML((size_t)U * C);
  for (int u = 0; u < U; ++u) {
    int b = in->nbucket - 1;
    for (int k = 0; k < in->nbucket; ++k)
      if (in->bucket_edge[k] >= in->s1[u]) {
        b = k;
        break;
      }
    for (int c = 0; c < C; ++c) t[(size_t)u * C + c] = in->t_table[(size_t)c * in->nbucket + b];
  }
  // risk and lower mass
  for (int u = 0; u < U; ++u)
    for (int c = 0; c < C; ++c) {
      const size_t i = (size_t)u * C + c;
      if (fam[c] == RS_DENSE) {
        R[i] = 0.0;
        ML[i] = 1.0;
        continue;
      }
      const float *cv = in->cov + i * 4;
      const double mh = (double)cv[0];
      double vmax = 0.0, vmin = 0.0;
      int nv = 0;
      for (int s = 0; s < 3; ++s) {
        if (in->nsub[(size_t)u * 3 + s] <= 0) continue;
        const double x = (double)cv[1 + s];
        if (nv == 0) {
          vmax = x;
          vmin = x;
        } else {
          vmax = std::max(vmax, x);
          vmin = std::min(vmin, x);
        }
        ++nv;
      }
      const double uu = nv <= 1 ? 0.0 : vmax - vmin;
      const double e = in->e ? (double)in->e[i] : 0.0;
      R[i] = (1.0 - mh) + cfg->alpha * uu + cfg->beta * e;
      const double lm = mh - cfg->delta_q;
      ML[i] = 0.0 < lm ? lm : 0.0;
    }
  std::vector<int> choice(U, dense_c);
  auto total = [&]() {
    double tot = in->t_probe_us;
    for (int u = 0; u < U; ++u) tot = tot + t[(size_t)u * C + choice[u]];
    return tot;
  };
  // Greedy solve.  Each unit keeps its best substitution (minimum ratio, first candidate on
  // ties); a tournament tree over the units yields the global minimum with the lowest unit
  // winning ties, i.e. the first minimum of a scan in (unit, candidate) order.
  struct Move {
    double rho;
    int c;  // -1: no strictly cheaper candidate
  };
  std::vector<Move> best(U);
  auto unit_best = [&](int u) {
    Move m{0.0, -1};
    const int cur = choice[u];
    const double tc = t[(size_t)u * C + cur], rc = R[(size_t)u * C + cur];
    for (int c = 0; c < C; ++c) {
      const double tn = t[(size_t)u * C + c];
      if (!(tn < tc)) continue;
      const double rho = (R[(size_t)u * C + c] - rc) / (tc - tn);
      if (m.c < 0 || rho < m.rho) m = Move{rho, c};
    }
    return m;
  };
  int P = 1;
  while (P < U) P <<= 1;
  std::vector<int> tree(2 * (size_t)P, -1);
  auto win = [&](int l, int r) {  // l covers lower unit indices than r
    if (l < 0) return r;
    if (r < 0) return l;
    return best[r].rho < best[l].rho ? r : l;
  };
  for (int u = 0; u < U; ++u) {
    best[u] = unit_best(u);
    tree[(size_t)P + u] = best[u].c >= 0 ? u : -1;
  }
  for (int i = P - 1; i >= 1; --i) tree[i] = win(tree[2 * i], tree[2 * i + 1]);
  // The loop test is "fresh unit-order total > T_layer".  A running total is used while it
  // is farther from T_layer than its possible drift from the fresh sum (each update and each
  // term of a sum is off by at most one rounding: far below 1e-9 of the all-dense total); near
  // the budget the fresh sum decides.
  double est = total();
  const double margin = 1e-9 * (est > 0.0 ? est : -est);
  bool infeasible = false;
  for (;;) {
    if (!(est - cfg->T_layer_us > margin || cfg->T_layer_us - est > margin)) est = total();
    if (!(est > cfg->T_layer_us)) break;
    const int bu = tree[1];
    if (bu < 0) {
      infeasible = true;
      break;
    }
    const int bc = best[bu].c;
    est = (est - t[(size_t)bu * C + choice[bu]]) + t[(size_t)bu * C + bc];
    choice[bu] = bc;
    best[bu] = unit_best(bu);
    size_t i = (size_t)P + bu;
    tree[i] = best[bu].c >= 0 ? bu : -1;
    for (i >>= 1; i >= 1; i >>= 1) tree[i] = win(tree[2 * i], tree[2 * i + 1]);
  }
  // expand or fall back: larger budgets of the family first, then the cheapest passing
  // sparse candidate of any family, dense only when no sparse candidate reaches tau
  int nfb = 0;
  for (int u = 0; u < U; ++u) {
    const int c = choice[u];
    if (fam[c] == RS_DENSE || ML[(size_t)u * C + c] >= cfg->tau) continue;
    int pick = -1, pick_rank = 1 << 30;
    for (int c2 = 0; c2 < C; ++c2) {
      if (fam[c2] != fam[c] || brank[c2] <= brank[c]) continue;
      if (ML[(size_t)u * C + c2] >= cfg->tau && brank[c2] < pick_rank) {
        pick = c2;
        pick_rank = brank[c2];
      }
    }
    if (pick < 0) {
      double best_t = 0.0;
      for (int c2 = 0; c2 < C; ++c2) {
        if (fam[c2] == RS_DENSE || !(ML[(size_t)u * C + c2] >= cfg->tau)) continue;
        const double tt = t[(size_t)u * C + c2];
        if (pick < 0 || tt < best_t) {
          best_t = tt;
          pick = c2;
        }
      }
    }
    if (pick < 0) {
      pick = dense_c;
      ++nfb;
    }
    choice[u] = pick;
  }
  const double tot = total();
  double rsum = 0.0;
  for (int u = 0; u < U; ++u) rsum = rsum + R[(size_t)u * C + choice[u]];
  int ng = 0, pos = 0;
  for (int c = 0; c < C; ++c) {
    const int start = pos;
    for (int u = 0; u < U; ++u)
      if (choice[u] == c) out->group_units[pos++] = u;
    if (pos > start) {
      out->group_cand[ng] = c;
      out->group_start[ng] = start;
      ++ng;
    }
  }
  out->group_start[ng] = pos;
  for (int u = 0; u < U; ++u) out->choice[u] = choice[u];
  for (size_t i = 0; i < (size_t)U * C; ++i) {
    out->risk[i] = R[i];
    out->m_lower[i] = ML[i];
  }
  out->ngroups = ng;
  out->n_fallback = nfb;
  out->infeasible = infeasible ? 1 : 0;
  out->over_budget = (infeasible || tot > cfg->T_layer_us) ? 1 : 0;
  out->total_us = tot;
  out->total_risk = rsum;
  return out->over_budget ? RS_ERR_BUDGET_INFEASIBLE : RS_OK;
}
