// C ABI entry points of librs: argument validation and dispatch to the HIP launchers.
#include <hip/hip_runtime.h>

#include <cmath>
#include <string>
#include <vector>

#include "common.h"

namespace rs {

static thread_local std::string g_err;

void set_error(const std::string &msg) { g_err = msg; }

rs_status fail(rs_status st, const std::string &msg) {
  g_err = msg;
  return st;
}

rs_status hip_check(hipError_t e, const char *what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return RS_ERR_HIP;
}

static bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

rs_status check_qkv(const rs_qkv *qkv, float *scale) {
  if (!qkv) return fail(RS_ERR_INVALID_ARG, "qkv is NULL");
  if (!qkv->q || !qkv->k || !qkv->v) return fail(RS_ERR_INVALID_ARG, "q, k or v is NULL");
  if (qkv->n < 1 || qkv->n > kMaxN) return fail(RS_ERR_INVALID_ARG, "n must be in [1, 262144]");
  if (qkv->hq < 1 || qkv->hkv < 1 || qkv->hq % qkv->hkv != 0)
    return fail(RS_ERR_INVALID_ARG, "hq must be a positive multiple of hkv");
  if (qkv->dtype != RS_BF16 && qkv->dtype != RS_F32) return fail(RS_ERR_INVALID_ARG, "unknown dtype");
  if (qkv->d != 64 && qkv->d != 128) return fail(RS_ERR_UNSUPPORTED, "head dim must be 64 or 128");
  const int64_t vec = qkv->dtype == RS_BF16 ? 8 : 4;  // elements per 16 bytes
  const size_t esz = qkv->dtype == RS_BF16 ? 2 : 4;
  const int64_t s[6] = {qkv->sq_h, qkv->sq_t, qkv->sk_h, qkv->sk_t, qkv->sv_h, qkv->sv_t};
  for (int i = 0; i < 6; ++i)
    if (s[i] < 0 || s[i] % vec != 0)
      return fail(RS_ERR_INVALID_ARG, "strides must be non-negative multiples of 16 bytes");
  if (qkv->sq_t < qkv->d || qkv->sk_t < qkv->d || qkv->sv_t < qkv->d)
    return fail(RS_ERR_INVALID_ARG, "token stride smaller than head dim");
  if (!aligned(qkv->q, 16) || !aligned(qkv->k, 16) || !aligned(qkv->v, 16) || !aligned(qkv->vt, 16))
    return fail(RS_ERR_INVALID_ARG, "q, k, v and vt must be 16-byte aligned");
  // the attention kernels address one head's K and V rows with 32-bit byte offsets
  const uint64_t span_k = ((uint64_t)(qkv->n - 1) * (uint64_t)qkv->sk_t + (uint64_t)qkv->d) * esz;
  const uint64_t span_v = ((uint64_t)(qkv->n - 1) * (uint64_t)qkv->sv_t + (uint64_t)qkv->d) * esz;
  if (span_k > 0xffffffffull || span_v > 0xffffffffull)
    return fail(RS_ERR_UNSUPPORTED, "one head's K or V rows must span less than 4 GiB");
  if (qkv->vt && (uint64_t)qkv->d * (((uint64_t)qkv->n + 63) / 64 * 64) * 2ull > 0xffffffffull)
    return fail(RS_ERR_UNSUPPORTED, "one head's V^T rows must span less than 4 GiB");
  float sc = qkv->scale;
  if (sc == 0.f) sc = 1.f / std::sqrt((float)qkv->d);
  if (!(sc > 0.f) || !std::isfinite(sc)) return fail(RS_ERR_INVALID_ARG, "scale must be positive and finite");
  *scale = sc;
  return RS_OK;
}

rs_status check_units(const rs_qkv *qkv, const rs_unit *units, int32_t nunits) {
  if (nunits < 0) return fail(RS_ERR_INVALID_ARG, "nunits < 0");
  if (nunits > 32767) return fail(RS_ERR_INVALID_ARG, "at most 32767 units per call");
  if (nunits > 0 && !units) return fail(RS_ERR_INVALID_ARG, "units is NULL");
  for (int i = 0; i < nunits; ++i) {
    const rs_unit &u = units[i];
    if (u.head < 0 || u.head >= qkv->hq) return fail(RS_ERR_INVALID_ARG, "unit " + std::to_string(i) + ": head out of range");
    if (u.s0 < 0 || u.s1 <= u.s0 || u.s1 > qkv->n)
      return fail(RS_ERR_INVALID_ARG, "unit " + std::to_string(i) + ": need 0 <= s0 < s1 <= n");
  }
  return RS_OK;
}

static uint64_t fnv(uint64_t h, uint64_t v) {
  for (int b = 0; b < 8; ++b) {
    h ^= (v >> (8 * b)) & 0xffu;
    h *= 0x100000001b3ull;
  }
  return h;
}

uint64_t unit_list_key(const rs_qkv *qkv, const rs_unit *units, int32_t nunits) {
  uint64_t h = 0xcbf29ce484222325ull;
  h = fnv(h, (uint64_t)qkv->n);
  h = fnv(h, ((uint64_t)qkv->hq << 32) | (uint32_t)qkv->hkv);
  h = fnv(h, (uint64_t)nunits);
  for (int i = 0; i < nunits; ++i) {
    h = fnv(h, ((uint64_t)(uint32_t)units[i].head << 32) | (uint32_t)units[i].s0);
    h = fnv(h, ((uint64_t)(uint32_t)units[i].s1 << 32) | (uint32_t)units[i].slot);
  }
  return h;
}

uint64_t probe_cfg_key(const rs_probe_cfg *cfg) {
  uint64_t h = 0x84222325cbf29ce4ull;
  if (!cfg) return h;
  h = fnv(h, ((uint64_t)(uint32_t)cfg->r_rec << 32) | (uint32_t)cfg->r_uni);
  return fnv(h, (uint64_t)(uint32_t)cfg->r_bnd | (1ull << 40));
}

rs_status check_unit_table(const rs_unit_table *t, const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                           const rs_probe_cfg *cfg) {
  if (!t->dev) return fail(RS_ERR_INVALID_ARG, "unit table without device memory");
  if (t->nunits != nunits || t->n != qkv->n || t->hq != qkv->hq || t->hkv != qkv->hkv ||
      t->key_units != unit_list_key(qkv, units, nunits))
    return fail(RS_ERR_INVALID_ARG, "unit table built for another unit list");
  if (cfg && (t->key_cfg != probe_cfg_key(cfg) || t->rmax != cfg->r_rec + cfg->r_uni + cfg->r_bnd))
    return fail(RS_ERR_INVALID_ARG, "unit table built for another probe configuration");
  return RS_OK;
}

// defined in the .hip translation units
size_t attn_ws_bytes(const rs_unit *units, int32_t nunits);
rs_status attn_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits, int fam,
                      const rs_candidate *cand, int cand_local, const rs_index_set *idx, void *o, int64_t so_h,
                      int64_t so_t, float *lse, void *ws, size_t ws_bytes, hipStream_t st);
size_t unit_table_bytes(int32_t nunits, const rs_probe_cfg *cfg);
rs_status unit_table_init(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg,
                          void *dev, size_t bytes, rs_unit_table *out, hipStream_t st);
size_t probe_ws_bytes(const rs_qkv *qkv, int32_t nunits, const rs_probe_cfg *cfg);
rs_status probe_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                       const rs_probe_cfg *cfg, const rs_candidate *grid, int32_t ncand, const rs_index_set *idx,
                       void *ws, size_t ws_bytes, rs_probe_out *out, hipStream_t st);
rs_status build_indices_launch(const rs_probe_out *sc, const rs_unit *units, int32_t nunits,
                               const rs_candidate *grid, int32_t ncand, rs_index_set *out, hipStream_t st, void *ws,
                               size_t ws_bytes);

static rs_status check_grid(const rs_candidate *grid, int32_t ncand) {
  if (ncand < 1 || !grid) return fail(RS_ERR_INVALID_ARG, "empty candidate grid");
  if (ncand > 16) return fail(RS_ERR_UNSUPPORTED, "at most 16 candidates");
  int last_a[4] = {-1, -1, -1, -1}, last_b[4] = {-1, -1, -1, -1}, cnt[4] = {0, 0, 0, 0};
  for (int c = 0; c < ncand; ++c) {
    const rs_candidate &g = grid[c];
    if (g.fam < RS_DENSE || g.fam > RS_BSPARSE) return fail(RS_ERR_INVALID_ARG, "unknown family");
    if (g.a < 0 || g.b < 0) return fail(RS_ERR_INVALID_ARG, "negative budget");
    if (g.fam == RS_ASHAPE && g.b < 1) return fail(RS_ERR_INVALID_ARG, "A-shape window must be >= 1");
    if (g.fam == RS_BSPARSE && (g.b != 64 || g.a < 1 || g.a > 256))
      return fail(RS_ERR_UNSUPPORTED, "block-sparse needs block 64 and 1 <= k <= 256");
    if (g.fam == RS_VSLASH && (g.a > 2048 || g.b > 1 << 20))
      return fail(RS_ERR_UNSUPPORTED, "vertical-slash needs n_v <= 2048");
    if (g.a < last_a[g.fam] || g.b < last_b[g.fam])
      return fail(RS_ERR_INVALID_ARG, "candidates of a family must be listed in increasing budget order");
    last_a[g.fam] = g.a;
    last_b[g.fam] = g.b;
    if (++cnt[g.fam] > 8) return fail(RS_ERR_UNSUPPORTED, "at most 8 candidates per family");
  }
  return RS_OK;
}

size_t vt_bytes(const rs_qkv *qkv);
rs_status transpose_v_launch(const rs_qkv *qkv, void *vt, hipStream_t st);
size_t route_dev_ws_bytes(int32_t nunits, int32_t ncand);
rs_status route_dev_launch(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                           const int *fam, const int *brank, int dense_c, void *ws, size_t ws_bytes,
                           hipStream_t st);
rs_status route_dev_launch_noalloc(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                                   const int *fam, const int *brank, int dense_c, hipStream_t st);
rs_status error_predict_launch(const rs_probe_out *p, const rs_candidate *grid, int32_t ncand,
                               const rs_error_model *m, float *e, hipStream_t st);
size_t routed_attn_ws_bytes(const rs_unit *units, int32_t nunits);
rs_status routed_attn_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                             const rs_candidate *grid, int32_t ncand, const rs_index_set *idx, const int32_t *choice,
                             void *o, int64_t so_h, int64_t so_t, float *lse, void *ws, size_t ws_bytes,
                             void *const *events, hipStream_t st);

static int cand_local_index(const rs_candidate *grid, int c) {
  int k = 0;
  for (int i = 0; i < c; ++i)
    if (grid[i].fam == grid[c].fam) ++k;
  return k;
}

static rs_status check_out(const void *o, int64_t so_h, int64_t so_t, int d) {
  if (!o) return fail(RS_ERR_INVALID_ARG, "output is NULL");
  if (!aligned(o, 8) || so_t % 4 != 0 || so_h % 4 != 0 || so_t < d || so_h < 0)
    return fail(RS_ERR_INVALID_ARG, "output must be 8-byte aligned with strides multiple of 4 elements");
  return RS_OK;
}

}  // namespace rs

using namespace rs;

extern "C" {

const char *rs_last_error(void) { return g_err.c_str(); }
const char *rs_version(void) { return "routesparse-mi355x 0.1 (gfx950)"; }

size_t rs_attn_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits) {
  (void)qkv;
  if (nunits <= 0 || !units) return 256;
  return attn_ws_bytes(units, nunits);
}

rs_status rs_dense_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, void *o, int64_t so_h,
                                int64_t so_t, float *lse, void *ws, size_t ws_bytes, rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if ((st = check_units(qkv, units, nunits)) != RS_OK) return st;
  if ((st = check_out(o, so_h, so_t, qkv->d)) != RS_OK) return st;
  return attn_launch(qkv, scale, units, nunits, RS_DENSE, nullptr, 0, nullptr, o, so_h, so_t, lse, ws, ws_bytes,
                     (hipStream_t)stream);
}

rs_status rs_sparse_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_candidate *grid,
                                 int32_t ncand, const rs_index_set *idx, void *o, int64_t so_h, int64_t so_t,
                                 float *lse, void *ws, size_t ws_bytes, rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if ((st = check_units(qkv, units, nunits)) != RS_OK) return st;
  if ((st = check_grid(grid, ncand)) != RS_OK) return st;
  if ((st = check_out(o, so_h, so_t, qkv->d)) != RS_OK) return st;
  if (nunits == 0) return RS_OK;
  const int c = units[0].cand;
  if (c < 0 || c >= ncand) return fail(RS_ERR_INVALID_ARG, "unit candidate out of range");
  for (int i = 1; i < nunits; ++i)
    if (units[i].cand != c) return fail(RS_ERR_INVALID_ARG, "all units of one call must share a candidate");
  const rs_candidate &g = grid[c];
  const int cl = cand_local_index(grid, c);
  if (g.fam == RS_VSLASH || g.fam == RS_BSPARSE) {
    if (!idx) return fail(RS_ERR_INVALID_ARG, "index set required");
    if (idx->n != qkv->n) return fail(RS_ERR_INVALID_ARG, "index set built for another sequence length");
  }
  if (g.fam == RS_VSLASH) {
    if (!idx->vs_vsorted || !idx->vs_dsorted || !idx->vs_count || !idx->vs_vbits || !idx->vs_dbits)
      return fail(RS_ERR_INVALID_ARG, "vertical-slash arrays missing");
    if (cl >= idx->ncand_vs || idx->nwords != (qkv->n + 31) / 32 || idx->nv_max > 2048)
      return fail(RS_ERR_INVALID_ARG, "index set does not match the grid");
    for (int i = 0; i < nunits; ++i)
      if (units[i].slot < 0 || units[i].slot >= idx->nunits)
        return fail(RS_ERR_INVALID_ARG, "unit slot outside the index set");
  }
  if (g.fam == RS_BSPARSE) {
    if (!idx->bs_sorted || !idx->bs_count) return fail(RS_ERR_INVALID_ARG, "block-sparse arrays missing");
    if (cl >= idx->ncand_bs || idx->nb != (qkv->n + 63) / 64 || idx->hq != qkv->hq)
      return fail(RS_ERR_INVALID_ARG, "index set does not match the grid");
  }
  return attn_launch(qkv, scale, units, nunits, g.fam, &g, cl, idx, o, so_h, so_t, lse, ws, ws_bytes,
                     (hipStream_t)stream);
}

size_t rs_unit_table_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg) {
  (void)qkv;
  (void)units;
  if (nunits < 0) return 0;
  return unit_table_bytes(nunits, cfg);
}

rs_status rs_unit_table_init(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg,
                             void *dev, size_t bytes, rs_unit_table *out, rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if ((st = check_units(qkv, units, nunits)) != RS_OK) return st;
  if (!out) return fail(RS_ERR_INVALID_ARG, "out is NULL");
  if (cfg && (cfg->r_rec < 0 || cfg->r_uni < 0 || cfg->r_bnd < 0 || cfg->r_rec + cfg->r_uni + cfg->r_bnd > 256))
    return fail(RS_ERR_INVALID_ARG, "sampled rows must be in [0, 256]");
  if (!dev || bytes < unit_table_bytes(nunits, cfg))
    return fail(RS_ERR_WORKSPACE, "unit table memory too small: need " + std::to_string(unit_table_bytes(nunits, cfg)));
  return unit_table_init(qkv, units, nunits, cfg, dev, bytes, out, (hipStream_t)stream);
}

size_t rs_probe_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg) {
  (void)units;
  if (!qkv || !cfg || nunits < 0) return 0;
  return probe_ws_bytes(qkv, nunits, cfg);
}

rs_status rs_probe(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg,
                   const rs_candidate *grid, int32_t ncand, const rs_index_set *idx, void *ws, size_t ws_bytes,
                   rs_probe_out *out, rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if ((st = check_units(qkv, units, nunits)) != RS_OK) return st;
  if (!cfg || !out) return fail(RS_ERR_INVALID_ARG, "cfg or out is NULL");
  if (cfg->r_rec < 0 || cfg->r_uni < 0 || cfg->r_bnd < 0 || cfg->r_rec + cfg->r_uni + cfg->r_bnd > 256)
    return fail(RS_ERR_INVALID_ARG, "sampled rows must be in [0, 256]");
  if (cfg->bs_block != 64) return fail(RS_ERR_UNSUPPORTED, "block-mean block must be 64");
  if (cfg->local_w < 1) return fail(RS_ERR_INVALID_ARG, "local_w must be >= 1");
  const int rmax = cfg->r_rec + cfg->r_uni + cfg->r_bnd;
  if (out->nunits != nunits || out->rmax != rmax || out->n != qkv->n || out->nb != (qkv->n + 63) / 64 ||
      out->hq != qkv->hq)
    return fail(RS_ERR_INVALID_ARG, "probe output dimensions do not match");
  const bool need_rows = (cfg->flags & RS_PROBE_ROWS) || idx != nullptr;
  if (need_rows && rmax == 0) return fail(RS_ERR_INVALID_ARG, "sampled-row probe needs at least one row");
  if (need_rows && (!out->rows || !out->subset || !out->nsub || !out->row_max || !out->row_sum))
    return fail(RS_ERR_INVALID_ARG, "probe row arrays missing");
  if (idx == nullptr) {
    if ((cfg->flags & RS_PROBE_ROWS) && (!out->col || !out->diag || !out->entropy || !out->local))
      return fail(RS_ERR_INVALID_ARG, "probe score arrays missing");
    if ((cfg->flags & RS_PROBE_BLOCKMEAN) && !out->lbs) return fail(RS_ERR_INVALID_ARG, "lbs missing");
  } else {
    if ((st = check_grid(grid, ncand)) != RS_OK) return st;
    if (out->ncand != ncand || !out->cov_rows || !out->cov) return fail(RS_ERR_INVALID_ARG, "coverage arrays missing");
    if (idx->nunits != nunits || idx->n != qkv->n) return fail(RS_ERR_INVALID_ARG, "index set does not match");
    // the kernels index the bitmaps with the grid-local candidate index and the set's strides:
    // the set must hold every candidate of the grid with the word counts of this n
    int nvs = 0, nbs = 0;
    for (int c = 0; c < ncand; ++c) {
      nvs += grid[c].fam == RS_VSLASH;
      nbs += grid[c].fam == RS_BSPARSE;
    }
    const int nbk = (qkv->n + 63) / 64;
    if (nvs > 0) {
      if (!idx->vs_vbits || !idx->vs_dbits) return fail(RS_ERR_INVALID_ARG, "vertical-slash bitmaps missing");
      if (idx->ncand_vs < nvs || idx->nwords != (qkv->n + 31) / 32)
        return fail(RS_ERR_INVALID_ARG, "index set does not match the grid (vertical-slash candidates or nwords)");
    }
    if (nbs > 0) {
      if (!idx->bs_bits || idx->hq != qkv->hq) return fail(RS_ERR_INVALID_ARG, "block-sparse bitmaps missing");
      if (idx->ncand_bs < nbs || idx->nb != nbk || idx->nbw != (nbk + 31) / 32)
        return fail(RS_ERR_INVALID_ARG, "index set does not match the grid (block-sparse candidates, nb or nbw)");
    }
  }
  if (qkv->tables && (st = check_unit_table(qkv->tables, qkv, units, nunits, cfg)) != RS_OK) return st;
  if (nunits == 0) return RS_OK;
  return probe_launch(qkv, scale, units, nunits, cfg, grid, ncand, idx, ws, ws_bytes, out, (hipStream_t)stream);
}

size_t rs_build_indices_workspace_size(const rs_probe_out *scores, const rs_candidate *grid, int32_t ncand) {
  (void)grid;
  (void)ncand;
  if (!scores) return 0;
  return (size_t)scores->nunits * sizeof(int) + 512;
}

rs_status rs_build_indices(const rs_probe_out *scores, const rs_unit *units, int32_t nunits,
                           const rs_candidate *grid, int32_t ncand, void *ws, size_t ws_bytes, rs_index_set *out,
                           rs_stream stream) {
  g_err.clear();
  rs_status st;
  if (!scores || !out) return fail(RS_ERR_INVALID_ARG, "scores or out is NULL");
  if ((st = check_grid(grid, ncand)) != RS_OK) return st;
  if (nunits < 0 || (nunits > 0 && !units)) return fail(RS_ERR_INVALID_ARG, "bad units");
  if (scores->nunits != nunits || out->nunits != nunits) return fail(RS_ERR_INVALID_ARG, "unit count mismatch");
  const int n = scores->n;
  if (n < 1 || n > kMaxN) return fail(RS_ERR_INVALID_ARG, "bad n");
  int nvs = 0, nbs = 0, nvm = 0, nsm = 0, km = 0;
  for (int c = 0; c < ncand; ++c) {
    if (grid[c].fam == RS_VSLASH) {
      ++nvs;
      nvm = std::max(nvm, grid[c].a);
      nsm = std::max(nsm, grid[c].b);
    }
    if (grid[c].fam == RS_BSPARSE) {
      ++nbs;
      km = std::max(km, grid[c].a);
    }
  }
  const int nb = (n + 63) / 64;
  if (out->n != n || out->nb != nb || out->nwords != (n + 31) / 32 || out->nbw != (nb + 31) / 32)
    return fail(RS_ERR_INVALID_ARG, "index set dimensions do not match n");
  // a grid may leave out a family altogether (its arrays are then untouched), so that the two
  // families can be built by separate calls
  if ((nvs > 0 && out->ncand_vs != nvs) || (nbs > 0 && out->ncand_bs != nbs) || nvs + nbs == 0)
    return fail(RS_ERR_INVALID_ARG, "index set family counts");
  for (int u = 0; u < nunits; ++u)
    if (units[u].s1 < 1 || units[u].s1 > n || units[u].s0 < 0 || units[u].s0 >= units[u].s1)
      return fail(RS_ERR_INVALID_ARG, "bad unit bounds");
  if (nvs > 0) {
    if (out->nv_max < nvm || out->ns_max < nsm) return fail(RS_ERR_INVALID_ARG, "nv_max/ns_max below the grid");
    if (!scores->col || !scores->diag) return fail(RS_ERR_INVALID_ARG, "probe scores missing");
    if (!out->vs_vsorted || !out->vs_dsorted || !out->vs_count || !out->vs_vbits || !out->vs_dbits)
      return fail(RS_ERR_INVALID_ARG, "vertical-slash arrays missing");
  }
  if (nbs > 0) {
    if (out->k_max < km || out->k_max > 256) return fail(RS_ERR_INVALID_ARG, "k_max below the grid or above 256");
    if (!scores->lbs || out->hq != scores->hq) return fail(RS_ERR_INVALID_ARG, "block-mean scores missing");
    if (!out->bs_rank || !out->bs_sorted || !out->bs_count || !out->bs_bits)
      return fail(RS_ERR_INVALID_ARG, "block-sparse arrays missing");
  }
  if (scores->tables) {
    rs_qkv shape{};  // the key covers n, hq and hkv: those the table recorded
    shape.n = n;
    shape.hq = scores->tables->hq;
    shape.hkv = scores->tables->hkv;
    if ((st = check_unit_table(scores->tables, &shape, units, nunits, nullptr)) != RS_OK) return st;
  }
  if (nunits == 0 && nbs == 0) return RS_OK;
  return build_indices_launch(scores, units, nunits, grid, ncand, out, (hipStream_t)stream, ws, ws_bytes);
}

size_t rs_route_layer_device_workspace_size(int32_t nunits, int32_t ncand) {
  if (nunits < 0 || ncand < 1) return 0;
  return route_dev_ws_bytes(nunits, ncand);
}

// Validation shared by the two device-routing entry points: fills the per-candidate family,
// budget rank and the dense candidate.
static rs_status check_route_dev(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                                 int *fam, int *brank, int *dense_out) {
  if (!in || !cfg || !out) return fail(RS_ERR_INVALID_ARG, "route: NULL argument");
  const int U = in->nunits, C = in->ncand;
  if (U < 0 || C < 1 || C > 16 || !in->grid) return fail(RS_ERR_INVALID_ARG, "route: bad sizes (1 <= ncand <= 16)");
  if (U > 0 && (!in->cov || !in->nsub || !in->s1)) return fail(RS_ERR_INVALID_ARG, "route: missing inputs");
  if (in->nbucket < 1 || !in->t_table || !in->bucket_edge) return fail(RS_ERR_INVALID_ARG, "route: missing latency table");
  if (!out->choice || !out->group_cand || !out->group_start || !out->group_units || !out->risk || !out->m_lower ||
      !out->status || !out->totals)
    return fail(RS_ERR_INVALID_ARG, "route: missing outputs");
  int dense_c = -1;
  for (int c = 0; c < C; ++c) {
    fam[c] = in->grid[c].fam;
    if (fam[c] < RS_DENSE || fam[c] > RS_BSPARSE) return fail(RS_ERR_INVALID_ARG, "route: unknown family");
    brank[c] = cand_local_index(in->grid, c);
    if (fam[c] == RS_DENSE && dense_c < 0) dense_c = c;
  }
  if (dense_c < 0) return fail(RS_ERR_INVALID_ARG, "route: the grid must contain a dense candidate");
  *dense_out = dense_c;
  return RS_OK;
}

rs_status rs_route_layer_device(const rs_route_in *in, const rs_route_cfg *cfg, const rs_route_dev_out *out,
                                void *ws, size_t ws_bytes, rs_stream stream) {
  g_err.clear();
  int fam[16], brank[16], dense_c = -1;
  rs_status st = check_route_dev(in, cfg, out, fam, brank, &dense_c);
  if (st != RS_OK) return st;
  return route_dev_launch(in, cfg, out, fam, brank, dense_c, ws, ws_bytes, (hipStream_t)stream);
}

rs_status rs_route_layer_device_noalloc(const rs_route_in *in, const rs_route_cfg *cfg,
                                        const rs_route_dev_out *out, rs_stream stream) {
  g_err.clear();
  int fam[16], brank[16], dense_c = -1;
  rs_status st = check_route_dev(in, cfg, out, fam, brank, &dense_c);
  if (st != RS_OK) return st;
  return route_dev_launch_noalloc(in, cfg, out, fam, brank, dense_c, (hipStream_t)stream);
}

rs_status rs_error_predict(const rs_probe_out *probe, const rs_candidate *grid, int32_t ncand,
                           const rs_error_model *model, float *e, rs_stream stream) {
  g_err.clear();
  rs_status st;
  if (!probe || !model || !e) return fail(RS_ERR_INVALID_ARG, "probe, model or e is NULL");
  if ((st = check_grid(grid, ncand)) != RS_OK) return st;
  if (probe->ncand != ncand) return fail(RS_ERR_INVALID_ARG, "probe coverage built for another grid");
  if (probe->nunits > 0 && (!probe->cov || !probe->nsub || !probe->entropy || !probe->local))
    return fail(RS_ERR_INVALID_ARG, "probe coverage or descriptor arrays missing");
  for (int f = 0; f < 4; ++f)
    for (int k = 0; k < 4; ++k)
      if (!(model->w[f][k] >= 0.f) || !std::isfinite(model->w[f][k]))
        return fail(RS_ERR_INVALID_ARG, "error-model weights must be finite and non-negative");
  return error_predict_launch(probe, grid, ncand, model, e, (hipStream_t)stream);
}

size_t rs_routed_attn_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits) {
  (void)qkv;
  if (nunits <= 0 || !units) return 256;
  return routed_attn_ws_bytes(units, nunits);
}

rs_status rs_routed_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_candidate *grid,
                                 int32_t ncand, const rs_index_set *idx, const int32_t *choice, void *o, int64_t so_h,
                                 int64_t so_t, float *lse, void *ws, size_t ws_bytes, void *const *events,
                                 rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if ((st = check_units(qkv, units, nunits)) != RS_OK) return st;
  if ((st = check_grid(grid, ncand)) != RS_OK) return st;
  if ((st = check_out(o, so_h, so_t, qkv->d)) != RS_OK) return st;
  if (nunits == 0) return RS_OK;
  if (!choice) return fail(RS_ERR_INVALID_ARG, "choice is NULL");
  if (events)
    for (int k = 0; k < 5; ++k)
      if (!events[k]) return fail(RS_ERR_INVALID_ARG, "events must hold five events");
  bool vs = false, bs = false;
  for (int c = 0; c < ncand; ++c) {
    vs = vs || grid[c].fam == RS_VSLASH;
    bs = bs || grid[c].fam == RS_BSPARSE;
  }
  if (vs || bs) {
    if (!idx) return fail(RS_ERR_INVALID_ARG, "index set required");
    if (idx->n != qkv->n) return fail(RS_ERR_INVALID_ARG, "index set built for another sequence length");
  }
  int nvs = 0, nbs = 0;
  for (int c = 0; c < ncand; ++c) {
    nvs += grid[c].fam == RS_VSLASH;
    nbs += grid[c].fam == RS_BSPARSE;
  }
  if (vs) {
    if (!idx->vs_vsorted || !idx->vs_dsorted || !idx->vs_count || !idx->vs_vbits || !idx->vs_dbits)
      return fail(RS_ERR_INVALID_ARG, "vertical-slash arrays missing");
    if (nvs > idx->ncand_vs || idx->nwords != (qkv->n + 31) / 32 || idx->nv_max > 2048)
      return fail(RS_ERR_INVALID_ARG, "index set does not match the grid");
    for (int i = 0; i < nunits; ++i)
      if (units[i].slot < 0 || units[i].slot >= idx->nunits)
        return fail(RS_ERR_INVALID_ARG, "unit slot outside the index set");
  }
  if (bs) {
    if (!idx->bs_sorted || !idx->bs_count) return fail(RS_ERR_INVALID_ARG, "block-sparse arrays missing");
    if (nbs > idx->ncand_bs || idx->nb != (qkv->n + 63) / 64 || idx->hq != qkv->hq)
      return fail(RS_ERR_INVALID_ARG, "index set does not match the grid");
  }
  if (qkv->tables && (st = check_unit_table(qkv->tables, qkv, units, nunits, nullptr)) != RS_OK) return st;
  return routed_attn_launch(qkv, scale, units, nunits, grid, ncand, idx, choice, o, so_h, so_t, lse, ws, ws_bytes,
                            events, (hipStream_t)stream);
}

size_t rs_vt_bytes(const rs_qkv *qkv) {
  float scale;
  if (check_qkv(qkv, &scale) != RS_OK) return 0;
  return vt_bytes(qkv);
}

rs_status rs_transpose_v(const rs_qkv *qkv, void *vt, rs_stream stream) {
  g_err.clear();
  float scale;
  rs_status st;
  if ((st = check_qkv(qkv, &scale)) != RS_OK) return st;
  if (!vt || !aligned(vt, 16)) return fail(RS_ERR_INVALID_ARG, "vt must be a 16-byte aligned device pointer");
  return transpose_v_launch(qkv, vt, (hipStream_t)stream);
}

}  // extern "C"
