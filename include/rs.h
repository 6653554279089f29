/*
 * rs.h - C ABI of the routed pattern-sparse causal attention prefill library (librs.so).
 *
 * The operation (Sec. 2.1, Eq. 1): for one causal head with Q, K, V in R^{n x d},
 *   O = softmax(Q K^T / sqrt(d) + C) V,
 * and with a binary sparse mask M the logits outside M become minus infinity, so each
 * output row is a softmax over its kept key set S_i, renormalised on that set.  The
 * library computes this per (query head, prompt segment) "unit", choosing per unit one
 * candidate of the pattern library of Sec. 3.1 (A-shape, vertical-slash, block-sparse,
 * dense) with the shared probe of Sec. 3.2 (Eq. 3), the risk/certificate quantities of
 * Sec. 3.3 (Eqs. 4-5) and the latency-constrained router of Sec. 3.4 (Eqs. 6-8).
 *
 * Conventions shared by every call
 *  - Device pointers are caller-owned (e.g. allocated by torch) and must stay valid
 *    until the work queued on `stream` has finished.  Host pointers are read before the
 *    call returns.
 *  - The library allocates no device memory: calls that need scratch space take a
 *    caller-provided workspace whose size a *_workspace_size() query returns (the one
 *    exception, rs_route_layer_device_noalloc, uses a fixed static device array instead).
 *  - GPU calls are asynchronous on `stream` (a hipStream_t; NULL = the null stream).
 *    rs_route_layer is host-only, synchronous and pure.
 *  - Every call returns an rs_status; on failure nothing has been launched and
 *    rs_last_error() returns a message (thread-local, valid until the next call).
 *  - Results are deterministic: identical inputs give bitwise-identical outputs.
 *  - Layout: Q is [hq][n][d], K and V are [hkv][n][d], each with element strides
 *    (head, token) and a contiguous last dimension; query head h reads key/value head
 *    h / (hq / hkv).  O is bf16 [hq][n][d] with strides (so_h, so_t).
 *  - A unit covers query rows [s0, s1) of one query head; its rows see keys [0, s1)
 *    causally (key j visible to row i iff j <= i), as in chunked prefill.
 *  - Supported: d in {64, 128}; hq a multiple of hkv; n <= 262144; one head's K rows
 *    ((n - 1) * sk_t + d elements) and V rows span less than 4 GiB (else
 *    RS_ERR_UNSUPPORTED).
 */
#ifndef RS_H
#define RS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *rs_stream; /* hipStream_t */
struct rs_unit_table;

typedef enum {
  RS_OK = 0,
  RS_ERR_INVALID_ARG = 1,      /* bad sizes, strides, pointers or unit bounds */
  RS_ERR_UNSUPPORTED = 2,      /* valid but not implemented (e.g. d not in {64,128}) */
  RS_ERR_HIP = 3,              /* a HIP runtime call failed */
  RS_ERR_WORKSPACE = 4,        /* workspace missing or smaller than required */
  RS_ERR_BUDGET_INFEASIBLE = 5 /* rs_route_layer: route returned but over budget */
} rs_status;

typedef enum { RS_BF16 = 0, RS_F32 = 1 /* rounded to bf16 on load */ } rs_dtype;

/* Pattern families of the candidate library (Sec. 3.1). */
typedef enum { RS_DENSE = 0, RS_ASHAPE = 1, RS_VSLASH = 2, RS_BSPARSE = 3 } rs_family;

/* Q, K, V of one layer. */
typedef struct rs_qkv {
  const void *q, *k, *v;     /* device */
  int32_t dtype;             /* rs_dtype, same for q, k, v */
  int32_t n, hq, hkv, d;     /* sequence length, query heads, key/value heads, head dim */
  int32_t _pad0;
  int64_t sq_h, sq_t;        /* element strides of q (head, token) */
  int64_t sk_h, sk_t;
  int64_t sv_h, sv_t;
  float scale;               /* logit scale; 0 => 1/sqrt(d) */
  int32_t _pad1;
  const void *vt;            /* optional (device): V in the transposed layout written by
                                rs_transpose_v, or NULL.  When set, the dense, A-shape and
                                block-sparse kernels read it in place of v. */
  const struct rs_unit_table *tables; /* optional (host struct): the unit tables of the call's
                                unit list (rs_unit_table_init), or NULL; read by rs_probe and
                                rs_routed_attn_prefill in place of per-call uploads */
} rs_qkv;

/* Unit tables: everything derived from a layer's unit list alone (the list itself, each
 * unit's sampled probe rows with their subsets, the probe's unit groups), built once on the
 * host and uploaded once into caller-owned device memory by rs_unit_table_init.  Calls given
 * a table (rs_qkv.tables, rs_probe_out.tables) read it instead of rebuilding these arrays and
 * copying them to the device on every call, so a layer's calls issue no host-to-device copy.
 * The library fills the struct; the caller keeps it and its device memory unchanged while
 * calls use it.  A call whose unit list (or probe configuration) differs from the table's is
 * rejected with RS_ERR_INVALID_ARG before anything is launched. */
typedef struct rs_unit_table {
  void *dev;                 /* device memory holding the tables (caller-owned) */
  uint64_t key_units;        /* hash of n, hq, hkv and every unit's (head, s0, s1, slot) */
  uint64_t key_cfg;          /* hash of the probe configuration's sampled-row counts */
  int32_t nunits, rmax, ngroups, n, hq, hkv;
} rs_unit_table;

/* One unit: rows [s0, s1) of query head `head`; `cand` indexes the candidate grid.
 * `slot` is the unit's position in the unit list given to rs_probe / rs_build_indices,
 * i.e. its row in rs_probe_out and rs_index_set (used by vertical-slash attention;
 * those two calls ignore it and use the list position). */
typedef struct rs_unit {
  int32_t head, s0, s1, cand, slot, _pad[3];
} rs_unit;

/* One candidate (p, b) of the pattern-budget library (Sec. 3.1):
 *   RS_ASHAPE  a = sink tokens, b = window width (keys (i-b, i] plus [0, a))
 *   RS_VSLASH  a = n_v vertical columns, b = n_s slash diagonals
 *   RS_BSPARSE a = k key blocks per query block (diagonal block included), b = block (64)
 *   RS_DENSE   a = b = 0
 * Within a family, candidates must appear in the grid in increasing budget order
 * (both a and b non-decreasing); a candidate's budget rank is its position among the
 * candidates of its family.  Budgets of one family are nested prefixes of one ranking. */
typedef struct rs_candidate {
  int32_t fam, a, b, _pad;
} rs_candidate;

/* Probe configuration (Sec. 3.2).  Sampled rows of a unit [s0, s1):
 *   R  = [max(s0, s1 - r_rec), s1)                              (recent rows)
 *   U  = { s0 + floor((2t+1)(s1-s0) / (2 r_uni)) : t < r_uni } \ R  (uniform rows)
 *   Bd = { max(s0, 64) + t : t < r_bnd } within [s0, s1), \ (R u U) (boundary rows)
 * Column and diagonal scores use R; descriptors and coverage use all sampled rows. */
typedef struct rs_probe_cfg {
  int32_t r_rec, r_uni, r_bnd;
  int32_t bs_block;          /* block width of the block-mean estimator, must be 64 */
  int32_t local_w;           /* local-band width of the local-mass descriptor */
  uint32_t flags;            /* RS_PROBE_* */
} rs_probe_cfg;

#define RS_PROBE_ROWS 1u      /* sampled-row scores: stats, col, diag, descriptors */
#define RS_PROBE_BLOCKMEAN 2u /* block-mean scores L_bs of every query head */

/* Probe results, all device arrays allocated by the caller with these dimensions:
 *   nunits, rmax = r_rec + r_uni + r_bnd, n, nb = ceil(n / 64), ncand. */
typedef struct rs_probe_out {
  int32_t nunits, rmax, n, nb, ncand, hq;
  int32_t *rows;     /* [nunits][rmax] sampled rows ascending, -1 padded        (written) */
  int32_t *subset;   /* [nunits][rmax] 0 = R, 1 = U, 2 = Bd, -1 padded           (written) */
  int32_t *nsub;     /* [nunits][3] subset sizes                                 (written) */
  float *row_max;    /* [nunits][rmax] max scaled logit of the row over keys <= i (rows
                        as described under rs_probe) */
  float *row_sum;    /* [nunits][rmax] sum_j exp(l_ij - row_max)                  */
  float *col;        /* [nunits][n] col[j] = sum over R rows of a_ij (0 for j >= s1) */
  float *diag;       /* [nunits][n] diag[t] = sum over R rows of a_{i,i-t}           */
  float *entropy;    /* [nunits][rmax] 64-block entropy / log(#visible blocks) (coverage call) */
  float *local;      /* [nunits][rmax] attention mass within (i - local_w, i]  (coverage call) */
  float *lbs;        /* [hq][nb*(nb+1)/2] pooled logits, row bq at bq*(bq+1)/2, or NULL */
  float *cov_rows;   /* [nunits][ncand][rmax] m_i(c): mass of row i kept by candidate c */
  float *cov;        /* [nunits][ncand][4] m_hat, m_R, m_U, m_B (subset means; 0 if empty) */
  const struct rs_unit_table *tables; /* optional: unit tables of the probe's unit list (read
                        by rs_build_indices in place of a per-call upload), or NULL */
} rs_probe_out;

/* Index sets built from probe scores (Sec. 3.1), device arrays allocated by the caller.
 * VS arrays are per unit and per vertical-slash candidate (in grid order); BS arrays per
 * query head, per block-sparse candidate and per query block.  Sorted arrays list each
 * candidate's set in ascending order; bs_rank lists key blocks by score (diagonal block
 * first); -1 pads.  Budgets of a family are nested: each set is a prefix of one ranking. */
typedef struct rs_index_set {
  int32_t nunits, n, nb, hq;
  int32_t nv_max, ns_max, k_max, nwords; /* nwords = ceil(n/32), nbw = ceil(nb/32) */
  int32_t ncand_vs, ncand_bs, nbw, _pad;
  int32_t *vs_vsorted; /* [nunits][ncand_vs][nv_max] */
  int32_t *vs_dsorted; /* [nunits][ncand_vs][ns_max] */
  int32_t *vs_count;   /* [nunits][ncand_vs][2]  |V|, |D| (read clamped to [0, nv_max] / [0, ns_max]) */
  uint32_t *vs_vbits;  /* [nunits][ncand_vs][nwords] bit j set iff column j in V */
  uint32_t *vs_dbits;  /* [nunits][ncand_vs][nwords] bit t set iff diagonal t in D */
  int32_t *bs_rank;    /* [hq][nb][k_max]  diagonal block first */
  int32_t *bs_sorted;  /* [hq][ncand_bs][nb][k_max] */
  int32_t *bs_count;   /* [hq][ncand_bs][nb] (read clamped to [0, k_max]; entries outside the
                          causal key blocks are skipped by the attention kernel) */
  uint32_t *bs_bits;   /* [hq][ncand_bs][nb][nbw] bit bk set iff key block bk selected */
} rs_index_set;

/* Routing inputs (host arrays), [nunits][ncand] row-major unless stated. */
typedef struct rs_route_in {
  int32_t nunits, ncand;
  const rs_candidate *grid;  /* [ncand]; must contain one RS_DENSE candidate */
  const float *cov;          /* [nunits][ncand][4] as in rs_probe_out.cov */
  const int32_t *nsub;       /* [nunits][3] */
  const float *e;            /* [nunits][ncand] calibrated error predictor, or NULL (0) */
  const int32_t *s1;         /* [nunits] key length of each unit (latency bucket key) */
  /* profiled kernel latency t_ker(p, b, n) in microseconds per unit:
   * t_table[c * nbucket + k] for kv lengths up to bucket_edge[k] (ascending); a unit
   * uses the first bucket whose edge is >= s1, else the last. */
  const double *t_table;
  const int32_t *bucket_edge;
  int32_t nbucket, _pad;
  double t_probe_us;         /* probe + index + routing overhead charged to the layer */
} rs_route_in;

typedef struct rs_route_cfg {
  double T_layer_us; /* latency budget of the layer, T_l */
  double tau;        /* lower-mass threshold of the expand/fallback step */
  double alpha;      /* weight of the subset disagreement u */
  double beta;       /* weight of the error predictor e (0: training-free) */
  double delta_q;    /* calibrated residual quantile: m_lower = max(0, m_hat - delta_q) */
} rs_route_cfg;

typedef struct rs_route_out {
  int32_t *choice;      /* [nunits] chosen candidate                          (host) */
  int32_t *group_cand;  /* [ncand] candidate of group g                       (host) */
  int32_t *group_start; /* [ncand+1] group g holds units group_units[start[g]..start[g+1]) */
  int32_t *group_units; /* [nunits] unit indices, grouped, ascending within a group */
  double *risk;         /* [nunits][ncand] risk R(c) per unit (dense 0)             */
  double *m_lower;      /* [nunits][ncand] lower mass per unit (dense 1)            */
  int32_t ngroups, n_fallback, over_budget, infeasible;
  double total_us, total_risk;
} rs_route_out;

/* ---- unit tables (set-up, once per unit list) -------------------------------------------
 * rs_unit_table_size: bytes of device memory the tables of this unit list need (cfg may be
 * NULL: no probe rows).  rs_unit_table_init: builds them on the host, copies them into `dev`
 * on `stream` and synchronises the stream (a set-up call, not part of a layer); fills *out. */
size_t rs_unit_table_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg);
rs_status rs_unit_table_init(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg,
                             void *dev, size_t bytes, rs_unit_table *out, rs_stream stream);

/* ---- probe (Sec. 3.2, Eq. 3; coverage of Sec. 3.2-3.3) -------------------------------
 * Scores mode (idx == NULL): for each unit, samples rows as in rs_probe_cfg, computes
 * exact softmax statistics over keys [0, s1) of the last ceil(r_rec / 64) * 64 sampled rows
 * (the recent rows among them), the recent-row column and diagonal scores (flag
 * RS_PROBE_ROWS), and the block-mean pooled logits L_bs of every query head (flag
 * RS_PROBE_BLOCKMEAN; fp32 block means, their dot products taken as hi.hi + hi.lo + lo.hi
 * of bf16 parts hi = bf16(x), lo = bf16(x - hi): within about 2^-16 of sum_d |q_d k_d| x
 * scale of the exact product).
 * Coverage mode (idx != NULL, after a scores call on the same `out`; reads its sampled
 * rows): for each unit, candidate and sampled row, m_i(c) = sum of a_ij over the
 * candidate's key set, the subset means, the per-row descriptors (entropy, local mass) and
 * the softmax statistics (row_max, row_sum) of every sampled row, each row normalised by
 * its own running max while the keys stream past.  `grid`/`ncand` give the candidates
 * (ignored in scores mode). */
size_t rs_probe_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                               const rs_probe_cfg *cfg);
rs_status rs_probe(const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                   const rs_probe_cfg *cfg, const rs_candidate *grid, int32_t ncand,
                   const rs_index_set *idx, void *ws, size_t ws_bytes, rs_probe_out *out,
                   rs_stream stream);

/* ---- index construction (Sec. 3.1) ------------------------------------------------------
 * Total order of every selection: score descending, -0.0 after +0.0, position ascending.
 * VS per unit: V = top n_v columns of col over [0, s1); D = {0} + top (n_s - 1) diagonals
 * of diag over [1, s1).  BS per query head and query block bq (nb blocks of 64):
 * Sel(bq) = {bq} + top (k - 1) of L_bs[bq][0..bq).  Fewer candidates than the budget:
 * all are taken.  Needs the probe output of a scores call with the matching flags.  The
 * grid's vertical-slash (block-sparse) candidates must be those the index set was sized for,
 * or none: a family left out of the grid keeps its arrays untouched, so the two families may
 * be built by two calls (for instance on two streams, each after its scores). */
size_t rs_build_indices_workspace_size(const rs_probe_out *scores, const rs_candidate *grid,
                                       int32_t ncand);
rs_status rs_build_indices(const rs_probe_out *scores, const rs_unit *units, int32_t nunits,
                           const rs_candidate *grid, int32_t ncand, void *ws, size_t ws_bytes,
                           rs_index_set *out, rs_stream stream);

/* ---- routing (Sec. 3.4, Eqs. 6-8; inference-procedure steps 3-6) ------------------------
 * Host only.  Risk R = (1 - m_hat) + alpha u + beta e with u = max - min of the
 * non-empty subset means (dense: 0); greedy risk-per-microsecond substitutions from
 * all-dense until t_probe + sum t <= T_layer; then each sparse choice with
 * m_lower < tau takes the smallest larger budget of its family with m_lower >= tau, else
 * the cheapest sparse candidate of any family with m_lower >= tau, else dense; units
 * grouped by candidate.  Returns RS_ERR_BUDGET_INFEASIBLE (route still
 * filled in) when the final total exceeds T_layer. */
rs_status rs_route_layer(const rs_route_in *in, const rs_route_cfg *cfg, rs_route_out *out);

/* ---- calibrated error predictor (Sec. 3.3, the e term of Eq. 4) -------------------------
 * e(u, c) = sum_k w[fam(c)][k] x_k(u, c), a monotone regressor: the weights are
 * non-negative, so e never decreases when a feature grows.  They are fitted offline on
 * dense calibration runs.  The features use only the probe's coverage call and the
 * candidate's family:
 *   x0 = 1 - m_hat(c)            x1 = u(c), max - min of the non-empty subset means
 *   x2 = (1 - m_hat(c)) * H      x3 = (1 - m_hat(c)) * (1 - L)
 * H and L are the means, over the unit's sampled rows, of the normalised block entropy and
 * of the local-band mass.  Dense candidates get e = 0.  Sums are taken in fp64 and the
 * result is rounded to fp32.
 * e: device [nunits][ncand], written on `stream`.  Reads probe->cov, nsub, entropy and
 * local, which the coverage call of rs_probe writes. */
typedef struct rs_error_model {
  float w[4][4]; /* [family][feature], each >= 0; the RS_DENSE row is ignored */
} rs_error_model;
rs_status rs_error_predict(const rs_probe_out *probe, const rs_candidate *grid, int32_t ncand,
                           const rs_error_model *model, float *e, rs_stream stream);

/* ---- device-side routing (Sec. 3.4: routing as a fused GPU reduction) -------------------
 * Same decisions and outputs as rs_route_layer, bit for bit, computed by one workgroup on
 * `stream`.  The attention launches of the layer then follow with no host synchronisation.
 * `in` is read as by rs_route_layer, with two differences:
 *  - cov, nsub, e, s1, t_table and bucket_edge are DEVICE pointers;
 *  - grid is a host array and t_probe_us a value.
 * Outputs go to the device arrays of `out`, with the dimensions of rs_route_out.  Over
 * budget is reported in out->status; the call itself returns RS_OK.
 * Limits: nunits <= 2048 and nunits * (ncand - 1) <= 4096 (else RS_ERR_UNSUPPORTED). */
typedef struct rs_route_dev_out {
  int32_t *choice, *group_cand, *group_start, *group_units; /* as in rs_route_out */
  double *risk, *m_lower;                                   /* [nunits][ncand] */
  int32_t *status; /* [4] ngroups, n_fallback, over_budget, infeasible */
  double *totals;  /* [2] total_us, total_risk */
} rs_route_dev_out;
size_t rs_route_layer_device_workspace_size(int32_t nunits, int32_t ncand);
rs_status rs_route_layer_device(const rs_route_in *in, const rs_route_cfg *cfg,
                                const rs_route_dev_out *out, void *ws, size_t ws_bytes,
                                rs_stream stream);

/* ---- device routing without a workspace ---------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): rs_route_layer_device with the same arguments,
 * validation and results (bit for bit), except that the router's scratch lives in a fixed
 * library-owned device array of 96 KiB per GPU (one copy per device the library runs on,
 * held until the process ends) instead of a caller workspace.  The call allocates nothing.
 * Every call on one GPU shares that GPU's array, and the kernel writes every scratch element
 * before reading it, so consecutive calls need no clearing; calls that overlap on one GPU
 * (concurrent streams, several threads) race on the array and must be serialised by the
 * caller.  Limits: nunits <= 2048 and nunits * (ncand - 1) <= 4096, the largest sizes the
 * array holds; beyond them RS_ERR_UNSUPPORTED, with nothing launched. */
rs_status rs_route_layer_device_noalloc(const rs_route_in *in, const rs_route_cfg *cfg,
                                        const rs_route_dev_out *out, rs_stream stream);

/* ---- routed attention from a device route (Sec. 3.4 grouping, inference step 6) ---------
 * Runs every unit u with candidate choice[u] (device int32 [nunits], e.g.
 * rs_route_dev_out.choice): one launch per family present in the grid, each over all the
 * units routed to any budget of that family.
 *  - Work lists are built on the device by a planning kernel: query tiles bucketed by
 *    key/value head, longest first.
 *  - O and lse equal those of one rs_sparse_attn_prefill / rs_dense_attn_prefill call per
 *    (pattern, budget) group.
 *  - `units` is the layer's host unit list; `slot` is the unit's row in `idx`, and the
 *    unit's `cand` field is ignored.
 *  - Grids are sized for every unit picking the family; surplus workgroups exit at once.
 *  - A unit whose choice lies outside [0, ncand) is not computed.
 *  - `events` (optional, for measurement): five hipEvent_t.  events[0] is recorded on
 *    `stream` after the planning kernel, then events[1..4] after the launches of the
 *    dense, vertical-slash, block-sparse and A-shape families, in that order.  A family
 *    absent from the grid records its event with no launch.
 * Limit: nunits <= 2048 (else RS_ERR_UNSUPPORTED). */
size_t rs_routed_attn_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits);
rs_status rs_routed_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                                 const rs_candidate *grid, int32_t ncand,
                                 const rs_index_set *idx, const int32_t *choice, void *o,
                                 int64_t so_h, int64_t so_t, float *lse, void *ws,
                                 size_t ws_bytes, void *const *events, rs_stream stream);

/* ---- transposed V (an operand layout for the attention kernels) -------------------------
 * Writes V of the layer into `vt` (device, bf16, rs_vt_bytes(qkv) bytes) as
 * [hkv][d][npad] with npad = n rounded up to 64.  Within each group of 16 consecutive keys
 * 16g + j, position j of a row holds key 16g + perm[j], perm = {0,1,2,3, 8,9,10,11,
 * 4,5,6,7, 12,13,14,15}; keys >= n are zero.  fp32 V is rounded to bf16 (as on load).
 * Point qkv->vt at the result: the P V products then read V^T fragments with plain 16-byte
 * LDS reads instead of transposing loads.  Must be redone when V changes. */
size_t rs_vt_bytes(const rs_qkv *qkv);
rs_status rs_transpose_v(const rs_qkv *qkv, void *vt, rs_stream stream);

/* ---- attention (Sec. 2.1; kernels of Sec. 3.1) ------------------------------------------
 * Every unit of one call must use the same candidate (one (pattern, budget) group).
 * Writes rows [s0, s1) of O for each unit and, if lse != NULL, lse[head * n + i] =
 * log sum over S_i of exp(l_ij) (natural log; -inf for an empty row).  Sparse calls read
 * the index set built by rs_build_indices with the same grid (A-shape needs none and
 * accepts idx == NULL).  Units of different calls may run concurrently only if they write
 * disjoint rows. */
size_t rs_attn_workspace_size(const rs_qkv *qkv, const rs_unit *units, int32_t nunits);
rs_status rs_sparse_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                                 const rs_candidate *grid, int32_t ncand,
                                 const rs_index_set *idx, void *o, int64_t so_h, int64_t so_t,
                                 float *lse, void *ws, size_t ws_bytes, rs_stream stream);
rs_status rs_dense_attn_prefill(const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                                void *o, int64_t so_h, int64_t so_t, float *lse, void *ws,
                                size_t ws_bytes, rs_stream stream);

/* Message describing the last failure of the calling thread ("" if none). */
const char *rs_last_error(void);
/* Library version string. */
const char *rs_version(void);

#ifdef __cplusplus
}
#endif
#endif /* RS_H */
