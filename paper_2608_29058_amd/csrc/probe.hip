// Shared attention probe (Sec. 3.2, Eq. 3 with token-resolution sampled rows) and the
// block-mean estimator of the block-sparse builder (Sec. 3.1), for gfx950.
//
// For each unit (query head h, rows [s0, s1)) the sampled rows I = R u U u Bd are scored
// exactly against keys [0, s1):
//   pass 1  row statistics of the recent rows: max_j l_ij and sum_j exp(l_ij - max), j <= i;
//   pass 2  normalised a_ij of the recent rows reduced into col[j] = sum_{i in R} a_ij and
//           diag[t] = sum_{i in R} a_{i,i-t};
//   pass 3  (coverage) for every sampled row, with its own running max (online
//           normalisation): the row statistics, m_i(c) = sum_{j in S_i(c)} a_ij for every
//           candidate c, the 64-key block entropy and the local-band mass.
// Logit tiles are bf16 MFMA products, statistics fp32: S^T = K_tile x Q_rows^T (a lane per
// sampled row) in passes 1 and 3, S = Q_rows x K_tile^T (a lane per key) in pass 2, whose
// column sums are then in-lane adds.  Every cross-workgroup reduction goes through per-chunk partials
// summed in a fixed order, so results are deterministic.
//
// Block-mean estimator: qbar/kbar = means of 64-row blocks (last block over its actual
// rows), L_bs[h][bq][bk] = qbar_bq . kbar_bk * scale for bk <= bq (packed lower triangle).
#include <algorithm>
#include <cstring>
#include <vector>

#include "common.h"

namespace rs {

constexpr int kProbeMaxRows = 256;  // sampled rows per unit
constexpr int kRange = 1024;        // keys per workgroup range in the three passes
constexpr int kMaxCand = 16;
constexpr int kPrefVs = 3;   // vertical-slash candidates whose bitmap words are prefetched
constexpr int kPrefBs = 3;   // block-sparse candidates whose selection words are prefetched
constexpr int kSkew = 89;    // row stride of the skewed 16-row probability tile (79 columns + pad;
                             // rows r and r + 4, written by the two lane halves, 32 banks apart)

struct ProbeUnit {
  int head, s0, s1, nrows;  // nrows = sampled rows actually present
  int r0;                   // first recent row (R = [r0, s1)), nR = s1 - r0
  int nR, pad0, pad1;
};

struct CandDev {
  int fam, a, b, cl;  // cl = index among candidates of the same family
};

struct ProbeArgs {
  const void *q, *k;
  long long sq_h, sq_t, sk_h, sk_t;
  int n, group, rmax, nchunks;
  int lg_groups, lg_pairs;  // task grid of a range pass: unit groups x row-block pairs per range
  float c, scale;
  int local_w;
  const ProbeUnit *units;
  const int4 *groups;  // up to 4 units sharing a key/value head and a segment (-1 pads)
  const int *rows, *subset;
  float *row_max, *row_sum;
  // pass 2 partials / outputs
  float *col, *diag_part, *ent_part, *loc_part;
  float *max_part, *sum_part;  // coverage pass: per (row, range) running max and sum
  int stats_rows;              // rows (from the end of the row list) the statistics pass covers
  int diag_w;  // width of a diagonal partial row (kRange + rmax)
  // pass 3
  int ncand;
  CandDev cand[kMaxCand];
  int ncov;                  // candidates with a general kept-mass accumulator
  int cov_cand[kMaxCand];    // accumulator slot -> candidate
  int nvs_pref, vs_pref_c[kPrefVs], vs_pref_cl[kPrefVs];  // prefetched vertical-slash candidates
  int nbs_pref, bs_pref_c[kPrefBs], bs_pref_cl[kPrefBs];  // prefetched block-sparse candidates
  const uint32_t *vs_vbits, *vs_dbits;
  int nwords, ncand_vs;
  const uint32_t *bs_bits;
  int nb, nbw, ncand_bs;
  float *cov_part;
  // scores call with a unit table: the table's sampled rows are copied to the probe output
  int *rows_out, *subset_out, *nsub_out;
  const int *nsub_tab;
};

// Orders this wave's LDS writes before its following LDS reads by other lanes.  The LDS
// executes one wave's accesses in issue order, so only the compiler has to be kept from
// moving them; a memory fence here would also make it wait for the K tile copy in flight.
__device__ __forceinline__ void wave_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// cs += x[r] for every r = 0..15 (in that order) whose bit 8 (r / 4) + r % 4 of w is set:
// sign-extended bit, and, add per element, in one instruction group.  Left to the optimiser,
// bit-extract + and becomes a compare into a lane mask and a select (with a hazard wait per
// element), or all bits are extracted ahead of the sums (16 more live registers); separate
// groups per element each get a wait of their own.
__device__ __forceinline__ void masked_add16(float &cs, uint32_t w, const float (&x)[16]) {
  float t;
  asm(
      "v_bfe_i32 %1, %2, 0, 1\n\tv_and_b32 %1, %1, %3\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 1, 1\n\tv_and_b32 %1, %1, %4\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 2, 1\n\tv_and_b32 %1, %1, %5\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 3, 1\n\tv_and_b32 %1, %1, %6\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 8, 1\n\tv_and_b32 %1, %1, %7\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 9, 1\n\tv_and_b32 %1, %1, %8\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 10, 1\n\tv_and_b32 %1, %1, %9\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 11, 1\n\tv_and_b32 %1, %1, %10\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 16, 1\n\tv_and_b32 %1, %1, %11\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 17, 1\n\tv_and_b32 %1, %1, %12\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 18, 1\n\tv_and_b32 %1, %1, %13\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 19, 1\n\tv_and_b32 %1, %1, %14\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 24, 1\n\tv_and_b32 %1, %1, %15\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 25, 1\n\tv_and_b32 %1, %1, %16\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 26, 1\n\tv_and_b32 %1, %1, %17\n\tv_add_f32 %0, %0, %1\n\t"
      "v_bfe_i32 %1, %2, 27, 1\n\tv_and_b32 %1, %1, %18\n\tv_add_f32 %0, %0, %1"
      : "+v"(cs), "=&v"(t)
      : "v"(w), "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]), "v"(x[4]), "v"(x[5]), "v"(x[6]), "v"(x[7]),
        "v"(x[8]), "v"(x[9]), "v"(x[10]), "v"(x[11]), "v"(x[12]), "v"(x[13]), "v"(x[14]), "v"(x[15]));
}

// key offset within a 64-key tile of accumulator element (mb, r) for lane half hh
__device__ __forceinline__ int acc_key(int mb, int r, int hh) {
  return 32 * mb + 8 * (r >> 2) + 4 * hh + (r & 3);
}

// XOR swizzle of the 16-byte chunk index of LDS row r: with d = 128 (256-byte rows spanning
// all 64 banks) the K fragment reads of 16 consecutive rows hit distinct banks; d = 64 uses
// a 3-bit swizzle over 8 rows.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return ((r & 3) << 1) | ((r >> 2) & 1);
}

enum { M_STATS = 0, M_SCORES = 1, M_COVER = 2 };

// Three bitmap words around a bit position, loaded from clamped indices with no condition on
// the loaded values (a select right after a load makes the compiler wait for it, and with it
// for every copy issued before); win_fix zeroes the words outside the bitmap where they are used.
__device__ __forceinline__ Win3 load_win_raw(const uint32_t *bits, int nwords, int pos) {
  const int w = pos >> 5;
  const int last = nwords - 1;
  Win3 r;
  r.x0 = bits[min(max(w, 0), last)];
  r.x1 = bits[min(max(w + 1, 0), last)];
  r.x2 = bits[min(max(w + 2, 0), last)];
  return r;
}
__device__ __forceinline__ Win3 win_fix(Win3 r, int nwords, int pos) {
  const int w = pos >> 5;
  r.x0 = (w >= 0 && w < nwords) ? r.x0 : 0u;
  r.x1 = (w + 1 >= 0 && w + 1 < nwords) ? r.x1 : 0u;
  r.x2 = (w + 2 >= 0 && w + 2 < nwords) ? r.x2 : 0u;
  return r;
}

// s_waitcnt immediate (gfx9 encoding) waiting until at most n vector-memory operations are
// outstanding, with no wait on the other counters
constexpr int vm_wait_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Task of a range-pass workgroup.  The grid is one-dimensional, and workgroups are dealt to
// the 8 XCDs in turn (workgroup b on XCD b % 8).  XCD x takes the key ranges x, x + 8, ...
// and, per range, every (unit group, row-block pair) task in turn: the groups of one
// key/value head (its segments and query heads) and the pairs of a group read the same K
// range, and they then run at about the same time on one L2.  Ranges are dealt in turn so
// that the XCDs get a similar mix of early ranges (seen by every segment) and late ones.
struct RangeTask {
  int rg, gy, pz;
};
__device__ __forceinline__ RangeTask range_task(const ProbeArgs &a) {
  const int per = a.lg_groups * a.lg_pairs;
  const int b = (int)blockIdx.x, j = b >> 3;
  const int rem = j % per;
  return RangeTask{(b & 7) + 8 * (j / per), rem / a.lg_pairs, rem % a.lg_pairs};
}
// workgroups of a range pass over (ranges, groups, pairs)
static inline dim3 range_grid(int nchunks, int ngroups, int npairs) {
  return dim3((unsigned)(8 * ((nchunks + 7) / 8) * ngroups * npairs));
}

// ---- the three passes over one key range ------------------------------------------------
// tasks: (key range, unit group, row-block pair), in the XCD-aware order of range_task.  A
// group holds the units of up to 4 query heads that share a key/value head and a segment,
// hence the same sampled rows and keys; wave w computes unit w.  Sampled rows are split into
// 32-row blocks aligned at the end of the
// (ascending) row list, so the recent rows fill the last blocks, and blocks are paired from
// the end.  A workgroup streams the 64-key tiles of its range through two LDS buffers (direct
// buffer-to-LDS copies, one barrier per tile) and keeps the Q fragments of its block pair in
// registers for the whole range.  The scores pass takes every pair holding recent rows in one
// workgroup, so column sums and diagonal partials of a range have a single writer.
//   M_STATS   per (row, range): max and sum of exp over the range's visible keys
//   M_SCORES  normalised a_ij of the recent rows -> col and diagonal partials
//   M_COVER   exp(l_ij - running max of the range) -> per (row, range): max, sum, kept mass
//             per candidate, sum of B log B over the range's 64-key blocks (B the block's
//             mass) and local mass, all relative to that max
// GEN: the candidates without prefetched bitmap words (cov_cand) may include vertical-slash
// and block-sparse ones, whose words are then read inside the tile loop; without GEN they
// are all A-shape (no memory reads).
template <int D, typename InT, int MODE, int NCV, bool GEN = true>
__global__ void __launch_bounds__(256, 2) probe_range_kernel(const ProbeArgs a) {
  constexpr int KS = D / 16, CPR = D / 8, RPI = 64 / CPR, LPT = 64 / RPI / 4;
  constexpr int TE = 64 * D;
  // K fragment reads in flight ahead of the products, in a forced order; the coverage variant
  // for arbitrary grids (GEN) has no registers to spare (the reordered loop spills there) and
  // keeps the block-by-block loop
  constexpr bool kForceKpf = !(MODE == M_COVER && GEN);
  constexpr int KPF = 4;
  // K tile buffers: the next tile (and, for coverage, its bitmap words) is fetched while the
  // current one is computed.  The copy is issued once both blocks have read the current tile
  // (after the second block's products): the compiler makes every LDS read wait for the
  // LDS-bound copies in flight, so the copy overlaps the second block's softmax and coverage
  // work.  The scores pass has one buffer (a barrier after the second block's products
  // releases it), which keeps its LDS within two workgroups per compute unit.
  constexpr int NKB = MODE == M_SCORES ? 1 : 2;
  // two K buffers as arrays of their own (tile parity known at compile time): the compiler then
  // sees that the copy into one never overlaps the fragment reads of the other, and the next
  // tile's copy can be issued at the start of the current tile
  __shared__ __align__(16) bf16 sK0[TE];
  __shared__ __align__(16) bf16 sK1[NKB == 2 ? TE : 8];
  __shared__ int sRows[2][32];
  // coverage pass: per wave (unit) and prefetched vertical-slash candidate, the diagonal-bitmap
  // words that the windows of this row-block pair and key range read (staged when they fit)
  constexpr int kDCap = MODE == M_COVER ? 576 : 1;
  __shared__ uint32_t sDW[4][kPrefVs][kDCap];

  const RangeTask task = range_task(a);
  const int rg = task.rg;
  if (rg >= a.nchunks) return;
  const int4 grp = a.groups[task.gy];
  const ProbeUnit U0 = a.units[grp.x];
  const int c0 = rg * kRange;
  if (c0 >= U0.s1) return;
  const int kend = min(c0 + kRange, U0.s1);
  const int nrows = U0.nrows, nrb = (nrows + 31) / 32;
  int p_lo, p_hi;
  if constexpr (MODE == M_SCORES) {
    if (U0.nR <= 0) return;
    p_lo = 0;
    p_hi = (U0.nR - 1) / 64 + 1;
  } else {
    p_lo = task.pz;
    p_hi = p_lo + 1;
    if (2 * p_lo >= nrb) return;
  }
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hh = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int u = wave == 0 ? grp.x : wave == 1 ? grp.y : wave == 2 ? grp.z : grp.w;
  const InT *Kp = (const InT *)a.k + (long long)(U0.head / a.group) * a.sk_h;

  // K tile copies: per-lane byte offset fixed, the tile's first key as a scalar offset
  const int lrow0 = wave * RPI + lane / CPR;
  const int lchunk = (lane % CPR) ^ swz<D>(lrow0);
  const uint32_t bK = (uint32_t)(a.sk_t * sizeof(InT));
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t rK = __builtin_amdgcn_make_buffer_rsrc(
      (void *)Kp, (short)0, (int)((uint32_t)(a.n - 1) * bK + D * sizeof(InT)), 0x00020000);
  const uint32_t voK = (uint32_t)lrow0 * bK + 16u * (uint32_t)lchunk;
  auto issue_tile = [&](bf16 *dst, int k0) __attribute__((always_inline)) {
    bf16 *dK = dst + wave * RPI * D;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int rr = lrow0 + i * 4 * RPI;
      if constexpr (sizeof(InT) == 2) {
        if (k0 + 64 <= a.n) {
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rK, (__attribute__((address_space(3))) void *)(dK + i * 4 * RPI * D),
                                                   16, voK, (uint32_t)(k0 + i * 4 * RPI) * bK, 0, 0);
        } else {
          const uint32_t j = (uint32_t)min(k0 + rr, a.n - 1);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rK, (__attribute__((address_space(3))) void *)(dK + i * 4 * RPI * D),
                                                   16, j * bK + 16u * (uint32_t)lchunk, 0, 0, 0);
        }
      } else {
        const int j = min(k0 + rr, a.n - 1);
        *(u32x4 *)(dK + i * 4 * RPI * D + 8 * lane) = load8<InT>(Kp + (long long)j * a.sk_t + 8 * lchunk);
      }
    }
  };

  // scores pass: a skewed probability tile per wave, and per-unit column sums and diagonal
  // partials of this range, all in LDS
  float (*sD)[kSkew] = nullptr;
  float *sCol = nullptr, *sDg = nullptr;
  const int dw = kRange + U0.nR;                // diagonals touched by recent rows in this range
  const int dbase = U0.r0 - (c0 + kRange - 1);  // smallest such diagonal
  if constexpr (MODE == M_SCORES) {
    __shared__ float sDbuf[4][16][kSkew];
    __shared__ float sColbuf[4][kRange];
    __shared__ float sDgbuf[4][kRange + kProbeMaxRows];
    sD = sDbuf[wave];
    sCol = sColbuf[wave];
    sDg = sDgbuf[wave];
    for (int x = lane; x < kRange; x += 64) sCol[x] = 0.f;
    for (int x = lane; x < dw; x += 64) sDg[x] = 0.f;
    for (int x = lane; x < 16 * kSkew; x += 64) sD[x / kSkew][x % kSkew] = 0.f;
  }

  const int kswz = swz<D>(l32);
  const int uhead = u >= 0 ? a.units[u].head : 0;  // loaded once: no dependent load inside the tile loop
  const InT *Qp = u >= 0 ? (const InT *)a.q + (long long)uhead * a.sq_h : nullptr;
  const float c = a.c;

  for (int pr = p_lo; pr < p_hi; ++pr) {
    // ---- the pair's two blocks: rows, Q fragments, per-row constants ------------------------
    const int b1 = nrb - 1 - 2 * pr, b0 = b1 - 1;
    __syncthreads();  // previous pair done with sRows and the tile buffers
    if (tid < 64) {
      const int s = tid >> 5, b = s ? b1 : b0;
      const int x = nrows - 32 * (nrb - b) + (tid & 31);
      sRows[s][tid & 31] = (b >= 0 && x >= 0) ? a.rows[(long long)grp.x * a.rmax + x] : -1;
    }
    __syncthreads();
    const int rmax0 = sRows[0][31], rmax1 = sRows[1][31];  // rows ascending; -1: no block
    const int kstop = min(kend, rmax1 + 1);                 // keys beyond the last row are unseen
    if (kstop <= c0) continue;                              // uniform over the workgroup
    const int nt = (kstop - c0 + 63) >> 6;

    int xr[2], row[2];
    u32x4 qf[2][KS];
    // scores pass: the logit tile is S = Q K^T (a lane holds one key and the 16 rows
    // 8 (r / 4) + 4 hh + r % 4 of its accumulator), with per element the row's constant
    // -(row_max log2 e + log2 row_sum), -inf for rows that are absent or not recent
    float nmv[2][16];
    bool anyR[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int b = s ? b1 : b0;
      xr[s] = nrows - 32 * (nrb - b) + l32;
      row[s] = sRows[s][l32];
      const bool ok = u >= 0 && row[s] >= 0;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        qf[s][ks] = u32x4{0u, 0u, 0u, 0u};
        if (ok) qf[s][ks] = load8<InT>(Qp + (long long)row[s] * a.sq_t + 16 * ks + 8 * hh);
      }
      if constexpr (MODE == M_SCORES) {
        // a_ij = exp2(l_ij * c - (row_max * log2 e + log2 row_sum)); recent rows are the last
        // ones of the list, so the block holds one when its last row is recent
        const int xb = nrows - 32 * (nrb - b);
        anyR[s] = u >= 0 && b >= 0 && xb + 31 >= nrows - U0.nR;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rho = 8 * (r >> 2) + 4 * hh + (r & 3);
          const int rw = sRows[s][rho];
          float v = -INFINITY;
          if (u >= 0 && rw >= 0 && xb + rho >= nrows - U0.nR) {
            const long long o = (long long)u * a.rmax + xb + rho;
            v = -a.row_max[o] * kLog2e - __builtin_amdgcn_logf(a.row_sum[o]);
          }
          nmv[s][r] = v;
        }
      }
    }
    float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
    float ent[2] = {0.f, 0.f}, loc[2] = {0.f, 0.f};
    float cov[2][NCV], covv[2][kPrefVs], covb[2][kPrefBs];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int q = 0; q < NCV; ++q) cov[s][q] = 0.f;
#pragma unroll
      for (int k = 0; k < kPrefVs; ++k) covv[s][k] = 0.f;
#pragma unroll
      for (int k = 0; k < kPrefBs; ++k) covb[s][k] = 0.f;
    }

    // coverage pass, per range: the block-sparse selection word of each row's query block (the
    // range's 16 key blocks share one word), the range's 32 column-bitmap words (lane w holds
    // word c0 / 32 + w) and, when they fit in sDW, the diagonal-bitmap words of every window
    // the rows read here: window positions i - k0 - 63 lie in [r_lo - c0 - 1023, r_hi - c0 - 63]
    // for the pair's rows [r_lo, r_hi], and a window reads its word and the next two
    uint32_t bwr[2][kPrefBs], vmv[kPrefVs];
    int rlo = 0, dw0 = 0;
    bool stage = false;
    if constexpr (MODE == M_COVER) {
      rlo = 0x7fffffff;
#pragma unroll
      for (int s = 0; s < 2; ++s)
        if (row[s] >= 0) rlo = min(rlo, row[s]);
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) rlo = min(rlo, __shfl_xor(rlo, o));  // the last block has rows
      dw0 = (rlo - c0 - (kRange - 1)) >> 5;
      const int nspan = ((rmax1 - c0 - 63) >> 5) + 3 - dw0;
      stage = nspan <= kDCap;  // the same rows for every wave
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int k = 0; k < kPrefBs; ++k) {
          bwr[s][k] = 0u;
          if (k < a.nbs_pref && u >= 0)  // absent rows (-1) read row 0's word, unused
            bwr[s][k] = a.bs_bits[(((long long)uhead * a.ncand_bs + a.bs_pref_cl[k]) * a.nb + (max(row[s], 0) >> 6)) *
                                      a.nbw + (c0 >> 11)];
        }
#pragma unroll
      for (int k = 0; k < kPrefVs; ++k) {
        vmv[k] = 0u;
        if (k >= a.nvs_pref || u < 0) continue;
        const long long vr = ((long long)u * a.ncand_vs + a.vs_pref_cl[k]) * a.nwords;
        const int wv = (c0 >> 5) + lane;
        if (lane < 32 && wv < a.nwords) vmv[k] = a.vs_vbits[vr + wv];
        if (stage)
          for (int x = lane; x < nspan; x += 64) {
            const int w = dw0 + x;
            sDW[wave][k][x] = (w >= 0 && w < a.nwords) ? a.vs_dbits[vr + w] : 0u;
          }
      }
      wave_sync();  // sDW is written and read by the lanes of one wave
    }

    // coverage pass, when the diagonal-bitmap words are not staged: each row's windows,
    // fetched together with the K copy of the tile they serve.  Only raw words are loaded here
    // (combined where they are used, in the next tile): a use right after the loads would make
    // the compiler wait for them, and with them for the tile copy issued just before.
    struct Pref {
      Win3 wd[2][kPrefVs];  // diagonal windows when they are not staged in sDW
    };
    auto fetch = [&](int k0, Pref &f) __attribute__((always_inline)) {
      if constexpr (MODE == M_COVER) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
#pragma unroll
          for (int k = 0; k < kPrefVs; ++k) {
            f.wd[s][k] = Win3{0u, 0u, 0u};
            if (!stage && k < a.nvs_pref && u >= 0)
              f.wd[s][k] = load_win_raw(a.vs_dbits + ((long long)u * a.ncand_vs + a.vs_pref_cl[k]) * a.nwords,
                                        a.nwords, max(row[s], 0) - k0 - 63);
          }
        }
      }
    };

    // ---- one block against one tile: products, then the rest -----------------------------
    auto qk_block = [&](const bf16 *sK, int k0, int s, f32x16 (&sacc)[2]) __attribute__((always_inline)) {
      const int rmx = s ? rmax1 : rmax0;
      if (u < 0 || rmx < k0) return;  // block absent or entirely before the tile
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[mb][r] = 0.f;
      if constexpr (!kForceKpf) {  // block by block, reads as the compiler places them
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const u32x4 kf = *(const u32x4 *)&sK[(32 * mb + l32) * D + (((2 * ks + hh) ^ kswz) << 3)];
            sacc[mb] = mfma32(kf, qf[s][ks], sacc[mb]);
          }
        return;
      }
      // fragment f: 32-key block mb = f % 2, k-step ks = f / 2 (the two accumulators alternate);
      // reads run KPF fragments ahead of their products (else each product waits for its read)
      auto kread = [&](int f) __attribute__((always_inline)) -> u32x4 {
        return *(const u32x4 *)&sK[(32 * (f & 1) + l32) * D + (((2 * (f >> 1) + hh) ^ kswz) << 3)];
      };
      u32x4 kb[KPF];
#pragma unroll
      for (int f = 0; f < KPF; ++f) kb[f] = kread(f);
#pragma unroll
      for (int f = 0; f < 2 * KS; ++f) {
        if constexpr (MODE == M_SCORES)  // S = Q K^T
          sacc[f & 1] = mfma32(qf[s][f >> 1], kb[f % KPF], sacc[f & 1]);
        else  // S^T = K Q^T
          sacc[f & 1] = mfma32(kb[f % KPF], qf[s][f >> 1], sacc[f & 1]);
        if (f + KPF < 2 * KS) kb[f % KPF] = kread(f + KPF);
      }
      // keep that order: under register pressure the scheduler would otherwise put each read
      // right before its product
      __builtin_amdgcn_sched_group_barrier(0x100, KPF, 0);
#pragma unroll
      for (int f = 0; f < 2 * KS - KPF; ++f) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, KPF, 0);
    };
    auto block_tile = [&](const f32x16 (&sacc)[2], int k0, int s, const Pref &f) __attribute__((always_inline)) {
      const int rmx = s ? rmax1 : rmax0;
      if (u < 0 || rmx < k0) return;  // block absent or entirely before the tile
      if constexpr (MODE == M_SCORES) {
        if (!anyR[s]) return;
        // element (mb, r): row rho = 8 (r / 4) + 4 hh + r % 4 of the block, key k0 + 32 mb + l32
        float x[2][16];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) x[mb][r] = sacc[mb][r];
        // keys after a row: only where the block's first recent row (at least rmx - 31; recent
        // rows are consecutive and end at the block's last row) lies before the tile's end
        if (rmx - 31 < k0 + 63) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int ir = sRows[s][8 * (r >> 2) + 4 * hh + (r & 3)];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
              if (k0 + 32 * mb + l32 > ir) x[mb][r] = -INFINITY;
          }
        }
        float cA[2] = {0.f, 0.f};  // this lane's rows of key columns l32 and 32 + l32
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            x[mb][r] = __builtin_amdgcn_exp2f(fmaf(x[mb][r], c, nmv[s][r]));
            cA[mb] += x[mb][r];
          }
        // column sums: lane half 0 completes key l32, half 1 key 32 + l32, with the other
        // half's 16 rows of that key
        const float give = hh ? cA[0] : cA[1];
        const float cs = (hh ? cA[1] : cA[0]) + __shfl_xor(give, 32);
        sCol[k0 - c0 + 32 * hh + l32] += cs;
        // diagonals through the skewed tile, 16 rows at a time: row rho' = rho - 16 h, key kk
        // -> sD[rho'][kk - rho' + 15], so that a diagonal (kk - rho' constant) is a column of
        // sD; entries no key maps to stay zero.  Recent rows are consecutive and end at row
        // 31, so the last row of half h is rmx - 16 (1 - h) and column e holds diagonal
        // t = (that row - k0) - e.  Elements r in [8 h, 8 h + 8) are the lane's rows of half h.
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 8 * h; r < 8 * h + 8; ++r) {
              const int rp = 8 * ((r >> 2) & 1) + 4 * hh + (r & 3);
              sD[rp][32 * mb + l32 - rp + 15] = x[mb][r];
            }
          wave_sync();
          float d0 = 0.f, d1 = 0.f;
          const int e1 = min(64 + lane, kSkew - 1);
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) {
            d0 += sD[rr][lane];
            d1 += sD[rr][e1];
          }
          const int tb = rmx - 16 * (1 - h) - k0 - dbase;
          if (tb - lane >= 0 && tb - lane < dw) sDg[tb - lane] += d0;
          if (lane < 15 && tb - 64 - lane >= 0 && tb - 64 - lane < dw) sDg[tb - 64 - lane] += d1;
          wave_sync();
        }
        return;
      }
      const int i = row[s];
      // keys after the row: a row before the tile sees none of it; a row inside the tile
      // (some lane of the wave) masks element-wise
      const bool none = i < k0;
      const bool part = __ballot(i >= k0 && i < k0 + 63) != 0ull;
      float x[2][16];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) x[mb][r] = sacc[mb][r];
      if (part) {
        const uint64_t M = prefix_mask(i - k0 + 1) >> (4 * hh);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          const uint32_t w = (uint32_t)(M >> (32 * mb));
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const uint32_t keep = (uint32_t)__builtin_amdgcn_sbfe((int)w, 8 * (r >> 2) + (r & 3), 1);
            x[mb][r] = __builtin_bit_cast(float, (keep & __builtin_bit_cast(uint32_t, x[mb][r])) | (~keep & 0xff800000u));
          }
        }
      }
      if constexpr (MODE == M_STATS) {
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, x[mb][r]);
        if (none) mx = -INFINITY;
        const float m_new = fmaxf(m_run[s], mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float nm = none ? -INFINITY : -m_use * c;
        float ps = 0.f;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) ps += __builtin_amdgcn_exp2f(fmaf(x[mb][r], c, nm));
        l_run[s] = l_run[s] * __builtin_amdgcn_exp2f((m_run[s] - m_use) * c) + ps;
        m_run[s] = m_new;
      } else {  // M_COVER
        // online normalisation: the row's running max over this range (both halves of the
        // row see the same max); raising it rescales every accumulator of the row, and
        // S = sum B log B becomes alpha (S + log(alpha) Z) for alpha = exp(m_old - m_new)
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, x[mb][r]);
        if (none) mx = -INFINITY;
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        if (__ballot(mx > m_run[s]) != 0ull) {
          const float zt = l_run[s] + __shfl_xor(l_run[s], 32);
          if (mx > m_run[s]) {
            if (m_run[s] != -INFINITY) {  // else every accumulator is still zero
              const float la = (m_run[s] - mx) * c;  // log2 alpha
              const float al = __builtin_amdgcn_exp2f(la);
              ent[s] = al * (ent[s] + la * kLn2 * zt);
              l_run[s] *= al;
              loc[s] *= al;
#pragma unroll
              for (int q = 0; q < NCV; ++q) cov[s][q] *= al;
#pragma unroll
              for (int k = 0; k < kPrefVs; ++k) covv[s][k] *= al;
#pragma unroll
              for (int k = 0; k < kPrefBs; ++k) covb[s][k] *= al;
            }
            m_run[s] = mx;
          }
        }
        const float nm = none ? -INFINITY : -m_run[s] * c;
        float tsum = 0.f;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            x[mb][r] = __builtin_amdgcn_exp2f(fmaf(x[mb][r], c, nm));
            tsum += x[mb][r];
          }
        const float bt = tsum + __shfl_xor(tsum, 32);  // mass of the row in this 64-key block
        if (bt > 0.f) ent[s] += bt * logf(bt);
        l_run[s] += tsum;
        // kept mass of a 64-bit key mask (bits of this lane's keys after the half shift)
        auto masked = [&](uint64_t M) __attribute__((always_inline)) -> float {
          float cs = 0.f;
          masked_add16(cs, (uint32_t)M, x[0]);
          masked_add16(cs, (uint32_t)(M >> 32), x[1]);
          return cs;
        };
        // mass of the keys j >= lo: whole tile, none, or element-wise.  The element-wise sums
        // run only when some lane's boundary lies inside the tile (rows spread over a
        // segment mostly split into whole-tile and empty lanes).
        auto from = [&](int lo) __attribute__((always_inline)) -> float {
          const bool all = lo <= k0, nil = lo > k0 + 63;
          if (__ballot(!all && !nil) == 0ull) return all ? tsum : 0.f;
          const float m = masked(~prefix_mask(lo - k0) >> (4 * hh));
          return all ? tsum : nil ? 0.f : m;
        };
        loc[s] += from(i - a.local_w + 1);
        const int kt = k0 >> 6;
        const int tl = (k0 - c0) >> 5;  // column word of the tile within the range
#pragma unroll
        for (int k = 0; k < kPrefVs; ++k) {
          if (k >= a.nvs_pref) break;
          uint64_t md;
          if (stage) {  // absent rows (-1) read the first row's window, unused
            const int dpos = (i >= 0 ? i : rlo) - k0 - 63;
            const uint32_t *dw = &sDW[wave][k][(dpos >> 5) - dw0];
            md = __builtin_bitreverse64(win_bits(Win3{dw[0], dw[1], dw[2]}, dpos));
          } else {
            const int dpos = max(i, 0) - k0 - 63;
            md = __builtin_bitreverse64(win_bits(win_fix(f.wd[s][k], a.nwords, dpos), dpos));
          }
          const uint32_t mv0 = (uint32_t)__builtin_amdgcn_readlane((int)vmv[k], tl);
          const uint32_t mv1 = (uint32_t)__builtin_amdgcn_readlane((int)vmv[k], tl + 1);
          const uint64_t mv = (uint64_t)mv0 | ((uint64_t)mv1 << 32);
          const uint64_t m = (md | mv) >> (4 * hh);
          if (__ballot(m != 0ull) != 0ull) covv[s][k] += masked(m);  // wave-uniform skip
        }
#pragma unroll
        for (int k = 0; k < kPrefBs; ++k) {
          if (k >= a.nbs_pref) break;
          if ((bwr[s][k] >> (kt & 31)) & 1u) covb[s][k] += tsum;
        }
#pragma unroll
        for (int q = 0; q < NCV; ++q) {
          if (q >= a.ncov) break;
          const CandDev cd = a.cand[a.cov_cand[q]];
          if (cd.fam == RS_ASHAPE) {
            const float sink = k0 + 63 < cd.a ? tsum : k0 >= cd.a ? 0.f : masked(prefix_mask(cd.a - k0) >> (4 * hh));
            // window keys j >= i - b + 1 that are not sink keys
            cov[s][q] += sink + from(max(i - cd.b + 1, cd.a));
          } else if (!GEN) {
          } else if (cd.fam == RS_VSLASH) {
            const long long vr = ((long long)u * a.ncand_vs + cd.cl) * a.nwords;
            const uint64_t md = __builtin_bitreverse64(bits64_at(a.vs_dbits + vr, a.nwords, i - k0 - 63));
            const uint64_t mv = bits64_at(a.vs_vbits + vr, a.nwords, k0);
            cov[s][q] += masked((md | mv) >> (4 * hh));
          } else if (cd.fam == RS_BSPARSE) {
            const long long br = (((long long)uhead * a.ncand_bs + cd.cl) * a.nb + (max(i, 0) >> 6)) * a.nbw;
            if ((a.bs_bits[br + (kt >> 5)] >> (kt & 31)) & 1u) cov[s][q] += tsum;
          }
        }
      }
    };

    // ---- stream the range's tiles ---------------------------------------------------------
    // The Q fragments and row constants are waited for here, visibly to the compiler, so that
    // no wait for them lands inside the tile loop (where it would drain the tile copies).
    __builtin_amdgcn_s_waitcnt(vm_wait_imm(0));
    Pref fcur, fnext;
    issue_tile(sK0, c0);
    fetch(c0, fcur);
    if constexpr (NKB == 1) {
      for (int t = 0; t < nt; ++t) {
        __builtin_amdgcn_s_waitcnt(vm_wait_imm(0));  // tile t landed
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        const int k0 = c0 + 64 * t;
        f32x16 S[2];
        qk_block(sK0, k0, 0, S);
        block_tile(S, k0, 0, fcur);
        qk_block(sK0, k0, 1, S);
        // every wave has read the tile before it is overwritten
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        if (t + 1 < nt) issue_tile(sK0, k0 + 64);
        block_tile(S, k0, 1, fcur);
      }
    } else {
      // tile t in `cur`; after the barrier every wave is done with tile t - 1 (in `nxt`), so
      // tile t + 1 (and its bitmap words) is fetched into `nxt` before tile t's products
      auto tile = [&](int t, const bf16 *cur, bf16 *nxt) __attribute__((always_inline)) {
        __builtin_amdgcn_s_waitcnt(vm_wait_imm(0));  // tile t (and its bitmap words) landed
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        const int k0 = c0 + 64 * t;
        if (t + 1 < nt) {
          issue_tile(nxt, k0 + 64);
          fetch(k0 + 64, fnext);
        }
        f32x16 S[2];
        qk_block(cur, k0, 0, S);
        block_tile(S, k0, 0, fcur);
        qk_block(cur, k0, 1, S);
        block_tile(S, k0, 1, fcur);
        fcur = fnext;
      };
      for (int t = 0; t < nt; t += 2) {
        tile(t, sK0, sK1);
        if (t + 1 >= nt) break;
        tile(t + 1, sK1, sK0);
      }
    }

    // ---- per-row partials of this range ------------------------------------------------------
    if (u >= 0) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bool ok = row[s] >= 0 && hh == 0;
        const long long o = ((long long)u * a.rmax + xr[s]) * a.nchunks + rg;
        auto cov_out = [&](int cand, float v) {
          const float tot = v + __shfl_xor(v, 32);
          if (ok) a.cov_part[(((long long)u * a.ncand + cand) * a.rmax + xr[s]) * a.nchunks + rg] = tot;
        };
        if constexpr (MODE == M_STATS) {
          const float mo = __shfl_xor(m_run[s], 32), lo = __shfl_xor(l_run[s], 32);
          const float mm = fmaxf(m_run[s], mo);
          const float mu = mm == -INFINITY ? 0.f : mm;
          const float ll = l_run[s] * __builtin_amdgcn_exp2f((m_run[s] - mu) * c) +
                           lo * __builtin_amdgcn_exp2f((mo - mu) * c);
          if (ok) {
            a.ent_part[o] = mm;  // range max (raw dot product) in the entropy partial slot
            a.loc_part[o] = ll;  // range sum in the local-mass partial slot
          }
        } else if constexpr (MODE == M_COVER) {
          const float lt = loc[s] + __shfl_xor(loc[s], 32);
          const float zt = l_run[s] + __shfl_xor(l_run[s], 32);
          if (ok) {
            a.max_part[o] = m_run[s];  // raw dot product, as in the statistics pass
            a.sum_part[o] = zt;
            a.ent_part[o] = ent[s];
            a.loc_part[o] = lt;
          }
#pragma unroll
          for (int q = 0; q < NCV; ++q)
            if (q < a.ncov) cov_out(a.cov_cand[q], cov[s][q]);
#pragma unroll
          for (int k = 0; k < kPrefVs; ++k)
            if (k < a.nvs_pref) cov_out(a.vs_pref_c[k], covv[s][k]);
#pragma unroll
          for (int k = 0; k < kPrefBs; ++k)
            if (k < a.nbs_pref) cov_out(a.bs_pref_c[k], covb[s][k]);
        }
      }
    }
  }
  if constexpr (MODE == M_SCORES) {
    __syncthreads();
    if (u >= 0) {
      for (int x = lane; x < kRange; x += 64) {
        const int j = c0 + x;
        if (j < a.n) a.col[(long long)u * a.n + j] = (j < U0.s1) ? sCol[x] : 0.f;
      }
      for (int x = lane; x < dw; x += 64) a.diag_part[((long long)u * a.nchunks + rg) * a.diag_w + x] = sDg[x];
    }
  }
}

// ---- combination of the per-chunk partials: one wave per sampled row --------------------
// Partials of a row are contiguous over chunks; lanes stride over the chunks holding keys
// <= row in a fixed order and the wave reduces with a fixed xor-butterfly, so the result is
// deterministic.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// grid: (ceil(rmax / 4), nunits), 256 threads; wave = one sampled row
__global__ void probe_stats_combine_kernel(const ProbeArgs a) {
  const int u = blockIdx.y;
  const ProbeUnit U = a.units[u];
  const int x = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (x >= U.nrows || x < U.nrows - a.stats_rows) return;
  const int row = a.rows[(long long)u * a.rmax + x];
  const int nch = row / kRange + 1;
  const float *pm = a.ent_part + ((long long)u * a.rmax + x) * a.nchunks;
  const float *pl = a.loc_part + ((long long)u * a.rmax + x) * a.nchunks;
  float M = -INFINITY;
  for (int ch = lane; ch < nch; ch += 64) M = fmaxf(M, pm[ch]);
  M = wave_max(M);
  float L = 0.f;
  for (int ch = lane; ch < nch; ch += 64) L += pl[ch] * __builtin_amdgcn_exp2f((pm[ch] - M) * a.c);
  L = wave_sum(L);
  if (lane == 0) {
    a.row_max[(long long)u * a.rmax + x] = M * a.scale;
    a.row_sum[(long long)u * a.rmax + x] = L;
  }
}

// diagonals from their chunk partials, zero tails of col/diag: with vec, one thread per 4
// positions and 16-byte stores (n a multiple of 4, both arrays 16-byte aligned), else one
// thread per position
__global__ void probe_finish_kernel(const ProbeArgs a, float *diag, float *entropy, float *local, int vec) {
  const int u = blockIdx.y;
  const ProbeUnit U = a.units[u];
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  auto diag_at = [&](int x) -> float {
    float v = 0.f;
    if (x < U.s1 && U.nR > 0) {
      // chunks whose diagonal range [r0 - c0 - (kRange-1), r0 + nR - 1 - c0] holds t = x
      const int chi = min((U.r0 + U.nR - 1 - x) / kRange, (U.s1 - 1) / kRange);
      const int clo_num = U.r0 - (kRange - 1) - x;
      const int clo = clo_num <= 0 ? 0 : (clo_num + kRange - 1) / kRange;
      for (int ch = clo; ch <= chi; ++ch) {
        const int dbase = U.r0 - (ch * kRange + kRange - 1);
        const int xi = x - dbase;
        if (xi >= 0 && xi < kRange + U.nR) v += a.diag_part[((long long)u * a.nchunks + ch) * a.diag_w + xi];
      }
    }
    return v;
  };
  float *drow = diag + (long long)u * a.n, *crow = a.col + (long long)u * a.n;
  if (vec) {
    const int x = 4 * t;
    if (x < a.n) {
      const f32x4 v = {diag_at(x), diag_at(x + 1), diag_at(x + 2), diag_at(x + 3)};
      *(f32x4 *)(drow + x) = v;
      if (x >= U.s1) {
        *(f32x4 *)(crow + x) = f32x4{0.f, 0.f, 0.f, 0.f};
      } else {
        for (int e = max(U.s1 - x, 0); e < 4; ++e) crow[x + e] = 0.f;
      }
    }
  } else if (t < a.n) {
    drow[t] = diag_at(t);
    if (t >= U.s1) crow[t] = 0.f;
  }
  if (a.rows_out)
    for (int x = t; x < a.rmax; x += gridDim.x * blockDim.x) {
      a.rows_out[(long long)u * a.rmax + x] = a.rows[(long long)u * a.rmax + x];
      a.subset_out[(long long)u * a.rmax + x] = a.subset[(long long)u * a.rmax + x];
      if (x < 3) a.nsub_out[u * 3 + x] = a.nsub_tab[u * 3 + x];
    }
}

// coverage pass partials of each sampled row combined over its ranges:
// with M the row's max, a range's partials (relative to its own max m) are weighted by
// w = exp(m - M); Z = sum w z, m_i(c) = sum w cov(c) / Z, local mass likewise, and with
// S = sum over 64-key blocks of B log B (B relative to M) = sum w (s + log(w) z), the block
// entropy is log Z - S / Z.  Writes row_max / row_sum, the descriptors and m_i(c).
// grid (ceil(rmax / 4), nunits), 256 threads
// sixteen lanes per row (a row has at most n / 1024 ranges): four rows per wave, more loads
// in flight per lane than one row per wave; the sixteen lanes reduce with a fixed butterfly
__global__ void cover_combine_kernel(const ProbeArgs a, float *entropy, float *local, float *cov_rows) {
  const int u = blockIdx.y;
  const ProbeUnit U = a.units[u];
  const int x = blockIdx.x * 16 + (threadIdx.x >> 4), lane = threadIdx.x & 15;
  if (x >= U.nrows) return;  // the sixteen lanes of a row leave together
  const int row = a.rows[(long long)u * a.rmax + x];
  const int nch = row / kRange + 1;
  const long long base = ((long long)u * a.rmax + x) * a.nchunks;
  const float *pm = a.max_part + base, *pz = a.sum_part + base;
  const float *pe = a.ent_part + base, *pl = a.loc_part + base;
  float M = -INFINITY;
  for (int ch = lane; ch < nch; ch += 16) M = fmaxf(M, pm[ch]);
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  // a range with no visible key has z = 0 (and m = -inf): it contributes nothing
  auto lw = [&](int ch) { return pz[ch] > 0.f ? (pm[ch] - M) * a.c : -INFINITY; };  // log2 w
  // every sum of the row in one pass over its ranges, then one butterfly for all of them
  // (the same per-lane order and butterfly as a separate reduction per sum)
  float Z = 0.f, S = 0.f, L = 0.f, acc[kMaxCand];
#pragma unroll
  for (int c = 0; c < kMaxCand; ++c) acc[c] = 0.f;
  const float *pc0 = a.cov_part + ((long long)u * a.ncand * a.rmax + x) * a.nchunks;
  const long long cstride = (long long)a.rmax * a.nchunks;  // from one candidate to the next
  for (int ch = lane; ch < nch; ch += 16) {
    const float l2 = lw(ch);
    if (l2 == -INFINITY) continue;
    const float w = __builtin_amdgcn_exp2f(l2);
    Z += w * pz[ch];
    S += w * (pe[ch] + l2 * kLn2 * pz[ch]);
    L += w * pl[ch];
#pragma unroll
    for (int c = 0; c < kMaxCand; ++c)
      if (c < a.ncand && a.cand[c].fam != RS_DENSE) acc[c] += w * pc0[c * cstride + ch];
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) {
    Z += __shfl_xor(Z, o);
    S += __shfl_xor(S, o);
    L += __shfl_xor(L, o);
#pragma unroll
    for (int c = 0; c < kMaxCand; ++c)
      if (c < a.ncand) acc[c] += __shfl_xor(acc[c], o);
  }
  const float inv = Z > 0.f ? 1.f / Z : 0.f;
  if (lane == 0)
#pragma unroll
    for (int c = 0; c < kMaxCand; ++c)
      if (c < a.ncand) cov_rows[((long long)u * a.ncand + c) * a.rmax + x] = a.cand[c].fam != RS_DENSE ? acc[c] * inv : 1.f;
  if (lane == 0) {
    const long long o = (long long)u * a.rmax + x;
    a.row_max[o] = M * a.scale;
    a.row_sum[o] = Z;
    const int nvis = row / 64 + 1;
    entropy[o] = (nvis > 1 && Z > 0.f) ? (logf(Z) - S * inv) / logf((float)nvis) : 0.f;
    local[o] = L * inv;
  }
}

// subset means of the per-row coverage; grid (ncand, nunits), one wave: lane l sums rows
// l, l + 64, ... in order, then a fixed xor-butterfly combines the lanes (deterministic)
__global__ void cover_means_kernel(const ProbeArgs a, const float *cov_rows, float *cov) {
  const int u = blockIdx.y, c = blockIdx.x, lane = threadIdx.x & 63;
  const ProbeUnit U = a.units[u];
  float tot = 0.f, sub[3] = {0.f, 0.f, 0.f};
  int cnt[3] = {0, 0, 0};
  const float *m = cov_rows + ((long long)u * a.ncand + c) * a.rmax;
  for (int r = lane; r < U.nrows; r += 64) {
    const int s = a.subset[(long long)u * a.rmax + r];
    const float x = m[r];
    tot += x;
#pragma unroll
    for (int s2 = 0; s2 < 3; ++s2)
      if (s == s2) {
        sub[s2] += x;
        cnt[s2]++;
      }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    tot += __shfl_xor(tot, o);
#pragma unroll
    for (int s2 = 0; s2 < 3; ++s2) {
      sub[s2] += __shfl_xor(sub[s2], o);
      cnt[s2] += __shfl_xor(cnt[s2], o);
    }
  }
  if (lane != 0) return;
  float *o = cov + ((long long)u * a.ncand + c) * 4;
  o[0] = U.nrows ? tot / U.nrows : 0.f;
  for (int s2 = 0; s2 < 3; ++s2) o[1 + s2] = cnt[s2] ? sub[s2] / cnt[s2] : 0.f;
}

// ---- block-mean estimator ----------------------------------------------------------------
template <typename InT>
__global__ void __launch_bounds__(256) block_pool_kernel(const InT *x, long long s_h, long long s_t, int n, int d,
                                                         float *out) {
  // one 64-row block of one head: thread = (row group of 16, 8-dim chunk); 16-byte loads
  const int b = blockIdx.x, h = blockIdx.y;
  const int t = threadIdx.x;
  const int cpr = d / 8, rpp = 256 / cpr;  // chunks per row, rows per pass
  const int rg = t / cpr, cc = t % cpr;
  const int r0 = b * 64, r1 = min(n, r0 + 64);
  const InT *p = x + (long long)h * s_h + 8 * cc;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r = r0 + rg; r < r1; r += rpp) {
    const u32x4 v = load8<InT>(p + (long long)r * s_t);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      acc[2 * w] += __builtin_bit_cast(float, v[w] << 16);
      acc[2 * w + 1] += __builtin_bit_cast(float, v[w] & 0xffff0000u);
    }
  }
  __shared__ float sacc[256][9];
#pragma unroll
  for (int e = 0; e < 8; ++e) sacc[t][e] = acc[e];
  __syncthreads();
  if (t < d) {
    const int c2 = t / 8, e = t % 8;
    float s = 0.f;
    for (int g = 0; g < rpp; ++g) s += sacc[g * cpr + c2][e];  // fixed order
    out[((long long)h * gridDim.x + b) * d + t] = s / (float)(r1 - r0);
  }
}

// L[h][bq][bk] = qbar . kbar * scale for bk <= bq; 128 x 128 output tiles, each wave a 64 x 64
// quarter as 2 x 2 bf16 MFMA blocks (v_mfma_f32_32x32x16_bf16).  Each fp32 mean x is split into
// hi = bf16(x) and lo = bf16(x - hi) as it is staged in LDS, and a product takes
// hi.hi + hi.lo + lo.hi with fp32 sums: the dropped lo.lo and the rounding of lo are below
// 2^-16 of |q_d k_d|, so the result is within ~1e-5 of the fp64 dot product on logits of a few
// units, at three bf16 products per k-step instead of eight fp32 ones.  The head dimension
// goes through LDS in chunks of 32.
__global__ void __launch_bounds__(256) block_logits_kernel(const float *qbar, const float *kbar, int nb, int d,
                                                           int group, float scale, float *lbs) {
  constexpr int TB = 128, KC = 32, LD = KC + 8;  // bf16 row of a chunk, padded to 80 bytes
  const int h = blockIdx.y;
  // decode lower-triangular tile index
  int tq = 0;
  int t = blockIdx.x;
  while (t > tq) {
    t -= tq + 1;
    ++tq;
  }
  const int tk = t;
  __shared__ __align__(16) bf16 sqh[TB][LD], sql[TB][LD], skh[TB][LD], skl[TB][LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = (wave >> 1) * 64, wc = (wave & 1) * 64;  // this wave's quarter
  const int l32 = lane & 31, hh = lane >> 5;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  const float *qb = qbar + (long long)h * nb * d;
  const float *kb = kbar + (long long)(h / group) * nb * d;
  // four floats -> their hi and lo bf16 parts (two dwords each)
  auto split4 = [](f32x4 v, u32x2 &hi, u32x2 &lo) {
    hi[0] = pack_bf16x2(v[0], v[1]);
    hi[1] = pack_bf16x2(v[2], v[3]);
    f32x4 r;
    r[0] = v[0] - __builtin_bit_cast(float, hi[0] << 16);
    r[1] = v[1] - __builtin_bit_cast(float, hi[0] & 0xffff0000u);
    r[2] = v[2] - __builtin_bit_cast(float, hi[1] << 16);
    r[3] = v[3] - __builtin_bit_cast(float, hi[1] & 0xffff0000u);
    lo[0] = pack_bf16x2(r[0], r[1]);
    lo[1] = pack_bf16x2(r[2], r[3]);
  };
  // 128 rows x 32 dims of each operand per chunk: 1024 float4, 4 per thread; the next chunk is
  // loaded into registers while the current one is multiplied
  f32x4 vq[4], vk[4];
  auto load_chunk = [&](int d0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int x = 256 * e + tid, r = x / (KC / 4), c4 = x % (KC / 4);
      const int bq = tq * TB + r, bk = tk * TB + r;
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      vq[e] = bq < nb ? *(const f32x4 *)&qb[(long long)bq * d + d0 + 4 * c4] : z;
      vk[e] = bk < nb ? *(const f32x4 *)&kb[(long long)bk * d + d0 + 4 * c4] : z;
    }
  };
  static_assert(TB * KC / 4 == 4 * 256, "four float4 of each operand per thread");
  load_chunk(0);
  for (int d0 = 0; d0 < d; d0 += KC) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int x = 256 * e + tid, r = x / (KC / 4), c4 = x % (KC / 4);
      u32x2 hq, lq, hk, lk;
      split4(vq[e], hq, lq);
      split4(vk[e], hk, lk);
      *(u32x2 *)&sqh[r][4 * c4] = hq;
      *(u32x2 *)&sql[r][4 * c4] = lq;
      *(u32x2 *)&skh[r][4 * c4] = hk;
      *(u32x2 *)&skl[r][4 * c4] = lk;
    }
    __syncthreads();
    if (d0 + KC < d) load_chunk(d0 + KC);
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      u32x4 ah[2], al[2], bh[2], bl[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        ah[i] = *(const u32x4 *)&sqh[wr + 32 * i + l32][16 * ks + 8 * hh];
        al[i] = *(const u32x4 *)&sql[wr + 32 * i + l32][16 * ks + 8 * hh];
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bh[j] = *(const u32x4 *)&skh[wc + 32 * j + l32][16 * ks + 8 * hh];
        bl[j] = *(const u32x4 *)&skl[wc + 32 * j + l32][16 * ks + 8 * hh];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = mfma32(al[i], bh[j], acc[i][j]);
          acc[i][j] = mfma32(ah[i], bl[j], acc[i][j]);
          acc[i][j] = mfma32(ah[i], bh[j], acc[i][j]);
        }
    }
    __syncthreads();
  }
  // D[row][col]: col = lane % 32, row = 8 (r / 4) + 4 (lane / 32) + r % 4
  float *lh = lbs + (long long)h * ((long long)nb * (nb + 1) / 2);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int bk = tk * TB + wc + 32 * j + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int bq = tq * TB + wr + 32 * i + 8 * (r >> 2) + 4 * hh + (r & 3);
        if (bq < nb && bk <= bq) lh[(long long)bq * (bq + 1) / 2 + bk] = acc[i][j][r] * scale;
      }
    }
}

// ---- host side ---------------------------------------------------------------------------

// Sampled rows of one unit (ascending) with subset labels; see rs_probe_cfg.
static void sample_rows(int s0, int s1, const rs_probe_cfg &cfg, std::vector<int> &rows,
                        std::vector<int> &lab, int &r0) {
  std::vector<std::pair<int, int>> v;
  r0 = std::max(s0, s1 - cfg.r_rec);
  for (int i = r0; i < s1; ++i) v.push_back({i, 0});
  std::vector<int> uni;
  const long long L = s1 - s0;
  for (int t = 0; t < cfg.r_uni && L > 0; ++t) {
    const int i = s0 + (int)(((2LL * t + 1) * L) / (2LL * cfg.r_uni));
    if (i >= r0) continue;
    if (!uni.empty() && uni.back() == i) continue;
    uni.push_back(i);
  }
  for (int i : uni) v.push_back({i, 1});
  for (int t = 0; t < cfg.r_bnd; ++t) {
    const int i = std::max(s0, 64) + t;
    if (i < s0 || i >= s1 || i >= r0) continue;
    if (std::find(uni.begin(), uni.end(), i) != uni.end()) continue;
    v.push_back({i, 2});
  }
  std::sort(v.begin(), v.end());
  rows.clear();
  lab.clear();
  for (auto &p : v) {
    rows.push_back(p.first);
    lab.push_back(p.second);
  }
}

static int rmax_of(const rs_probe_cfg *cfg) { return cfg->r_rec + cfg->r_uni + cfg->r_bnd; }

// Host form of the per-unit probe tables: sampled rows, subsets and subset sizes, the units'
// ProbeUnit records and the unit groups (the query heads of one key/value head over one
// segment, up to 4).
struct ProbeHost {
  std::vector<ProbeUnit> units;
  std::vector<int4> groups;
  std::vector<int> rows, subset, nsub;
};

static void build_probe_host(const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg, int group,
                             ProbeHost &h) {
  const int rmax = rmax_of(cfg);
  h.units.assign(nunits, ProbeUnit{});
  h.rows.assign((size_t)nunits * rmax, -1);
  h.subset.assign((size_t)nunits * rmax, -1);
  h.nsub.assign((size_t)nunits * 3, 0);
  for (int u = 0; u < nunits; ++u) {
    std::vector<int> rows, lab;
    int r0;
    sample_rows(units[u].s0, units[u].s1, *cfg, rows, lab, r0);
    h.units[u] = ProbeUnit{units[u].head, units[u].s0, units[u].s1, (int)rows.size(), r0, units[u].s1 - r0, 0, 0};
    for (size_t x = 0; x < rows.size(); ++x) {
      h.rows[(size_t)u * rmax + x] = rows[x];
      h.subset[(size_t)u * rmax + x] = lab[x];
      h.nsub[(size_t)u * 3 + lab[x]]++;
    }
  }
  std::vector<std::vector<int>> open_lists;
  std::vector<long long> keys;
  for (int u = 0; u < nunits; ++u) {
    const long long key = ((long long)(units[u].head / group) * (kMaxN + 1) + units[u].s0) * (kMaxN + 1) + units[u].s1;
    int slot = -1;
    for (size_t k = 0; k < keys.size(); ++k)
      if (keys[k] == key && open_lists[k].size() < 4) {
        slot = (int)k;
        break;
      }
    if (slot < 0) {
      keys.push_back(key);
      open_lists.push_back({});
      slot = (int)keys.size() - 1;
    }
    open_lists[slot].push_back(u);
  }
  h.groups.clear();
  for (auto &l : open_lists) {
    int4 g{-1, -1, -1, -1};
    g.x = l[0];
    if (l.size() > 1) g.y = l[1];
    if (l.size() > 2) g.z = l[2];
    if (l.size() > 3) g.w = l[3];
    h.groups.push_back(g);
  }
}

// Device layout of a unit table: [rs_unit x U][s1 x U][ProbeUnit x U][int4 x U][rows][subset][nsub],
// each array 256-byte aligned; the probe arrays only with a probe configuration.
struct UnitTab {
  rs_unit *units;
  int *s1;
  ProbeUnit *punits;
  int4 *groups;
  int *rows, *subset, *nsub;
  size_t bytes;
};

static UnitTab unit_tab_layout(void *dev, int32_t nunits, int rmax, bool probe) {
  Arena ar(dev, ~size_t(0));
  UnitTab t{};
  t.units = ar.take<rs_unit>(nunits);
  t.s1 = ar.take<int>(nunits);
  if (probe) {
    t.punits = ar.take<ProbeUnit>(nunits);
    t.groups = ar.take<int4>(nunits);
    t.rows = ar.take<int>((size_t)nunits * rmax);
    t.subset = ar.take<int>((size_t)nunits * rmax);
    t.nsub = ar.take<int>((size_t)nunits * 3);
  }
  t.bytes = ar.off + 256;
  return t;
}

static UnitTab unit_tab_of(const rs_unit_table *t) {
  return unit_tab_layout(t->dev, t->nunits, t->rmax, t->key_cfg != probe_cfg_key(nullptr));
}

const rs_unit *unit_tab_units(const rs_unit_table *t) { return unit_tab_of(t).units; }
const int *unit_tab_s1(const rs_unit_table *t) { return unit_tab_of(t).s1; }

size_t unit_table_bytes(int32_t nunits, const rs_probe_cfg *cfg) {
  return unit_tab_layout(nullptr, nunits, cfg ? rmax_of(cfg) : 0, cfg != nullptr).bytes;
}

rs_status unit_table_init(const rs_qkv *qkv, const rs_unit *units, int32_t nunits, const rs_probe_cfg *cfg,
                          void *dev, size_t bytes, rs_unit_table *out, hipStream_t st) {
  const int rmax = cfg ? rmax_of(cfg) : 0;
  const UnitTab t = unit_tab_layout(dev, nunits, rmax, cfg != nullptr);
  if (bytes < t.bytes) return fail(RS_ERR_WORKSPACE, "unit table memory too small");
  // the whole table is staged in one host image and copied once
  std::vector<char> img(t.bytes, 0);
  auto at = [&](const void *p) { return img.data() + ((const char *)p - (const char *)dev); };
  std::vector<int> s1(nunits);
  for (int u = 0; u < nunits; ++u) s1[u] = units[u].s1;
  memcpy(at(t.units), units, (size_t)nunits * sizeof(rs_unit));
  memcpy(at(t.s1), s1.data(), s1.size() * sizeof(int));
  int ngroups = 0;
  if (cfg) {
    ProbeHost h;
    build_probe_host(units, nunits, cfg, qkv->hq / qkv->hkv, h);
    ngroups = (int)h.groups.size();
    memcpy(at(t.punits), h.units.data(), h.units.size() * sizeof(ProbeUnit));
    memcpy(at(t.groups), h.groups.data(), h.groups.size() * sizeof(int4));
    memcpy(at(t.rows), h.rows.data(), h.rows.size() * sizeof(int));
    memcpy(at(t.subset), h.subset.data(), h.subset.size() * sizeof(int));
    memcpy(at(t.nsub), h.nsub.data(), h.nsub.size() * sizeof(int));
  }
  RS_HIP(hipMemcpyAsync(dev, img.data(), img.size(), hipMemcpyHostToDevice, st));
  RS_HIP(hipStreamSynchronize(st));  // set-up call: the host image is released on return
  out->dev = dev;
  out->key_units = unit_list_key(qkv, units, nunits);
  out->key_cfg = probe_cfg_key(cfg);
  out->nunits = nunits;
  out->rmax = rmax;
  out->ngroups = cfg ? ngroups : 0;
  out->n = qkv->n;
  out->hq = qkv->hq;
  out->hkv = qkv->hkv;
  return RS_OK;
}

size_t probe_ws_bytes(const rs_qkv *qkv, int32_t nunits, const rs_probe_cfg *cfg) {
  const int rmax = rmax_of(cfg);
  const long long nchunks = (qkv->n + kRange - 1) / kRange;
  const int nb = (qkv->n + 63) / 64;
  Arena ar(nullptr, 0);
  ar.take<ProbeUnit>(nunits);
  ar.take<int4>(nunits);
  ar.take<float>((size_t)nunits * nchunks * (kRange + rmax));     // diag partials
  ar.take<float>((size_t)nunits * nchunks * rmax * 4);            // max / sum / entropy / local partials
  ar.take<float>((size_t)nunits * nchunks * rmax * kMaxCand);     // coverage partials
  if (cfg->flags & RS_PROBE_BLOCKMEAN) {
    ar.take<float>((size_t)qkv->hq * nb * qkv->d);
    ar.take<float>((size_t)qkv->hkv * nb * qkv->d);
  }
  return ar.off + 256;
}

template <int D, typename InT>
static hipError_t launch_rows(const ProbeArgs &pa, int nunits, int ngroups, int mode, float *diag, float *ent, float *loc,
                              float *cov_rows, float *cov, hipStream_t st) {
  const int npairs = ((pa.rmax + 31) / 32 + 1) / 2;  // row-block pairs of the fullest unit
  ProbeArgs ra = pa;  // with the task grid of each range pass
  ra.lg_groups = ngroups;
  if (mode == 0) {
    // statistics of the row pairs holding recent rows (pairs are taken from the end of the
    // ascending row list, where the recent rows are); the coverage pass normalises online
    const int spairs = std::min(npairs, pa.stats_rows / 64);
    if (spairs > 0) {
      ra.lg_pairs = spairs;
      hipLaunchKernelGGL((probe_range_kernel<D, InT, M_STATS, 1>), range_grid(pa.nchunks, ngroups, spairs), dim3(256), 0, st, ra);
      hipLaunchKernelGGL(probe_stats_combine_kernel, dim3((pa.rmax + 3) / 4, nunits), dim3(256), 0, st, pa);
    }
    ra.lg_pairs = 1;
    hipLaunchKernelGGL((probe_range_kernel<D, InT, M_SCORES, 1>), range_grid(pa.nchunks, ngroups, 1), dim3(256), 0, st, ra);
    const int vec = (pa.n & 3) == 0 && ((uintptr_t)diag & 15) == 0 && ((uintptr_t)pa.col & 15) == 0;
    const int fin_threads = vec ? pa.n / 4 : pa.n;
    hipLaunchKernelGGL(probe_finish_kernel, dim3((fin_threads + 255) / 256, nunits), dim3(256), 0, st, pa, diag, ent,
                       loc, vec);
  } else {
    bool ashape_only = true;
    for (int q = 0; q < pa.ncov; ++q) ashape_only = ashape_only && pa.cand[pa.cov_cand[q]].fam == RS_ASHAPE;
    ra.lg_pairs = npairs;
    const dim3 grid = range_grid(pa.nchunks, ngroups, npairs);
    if (ashape_only && pa.ncov <= 2)
      hipLaunchKernelGGL((probe_range_kernel<D, InT, M_COVER, 2, false>), grid, dim3(256), 0, st, ra);
    else if (pa.ncov <= 4)
      hipLaunchKernelGGL((probe_range_kernel<D, InT, M_COVER, 4>), grid, dim3(256), 0, st, ra);
    else
      hipLaunchKernelGGL((probe_range_kernel<D, InT, M_COVER, kMaxCand>), grid, dim3(256), 0, st, ra);
    hipLaunchKernelGGL(cover_combine_kernel, dim3((pa.rmax + 15) / 16, nunits), dim3(256), 0, st, pa, ent, loc, cov_rows);
    hipLaunchKernelGGL(cover_means_kernel, dim3(pa.ncand, nunits), dim3(64), 0, st, pa, cov_rows, cov);
  }
  return hipGetLastError();
}

rs_status probe_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                       const rs_probe_cfg *cfg, const rs_candidate *grid, int32_t ncand,
                       const rs_index_set *idx, void *ws, size_t ws_bytes, rs_probe_out *out, hipStream_t st) {
  const int rmax = rmax_of(cfg);
  const int nchunks = (qkv->n + kRange - 1) / kRange;
  const int nb = (qkv->n + 63) / 64;
  const size_t need = probe_ws_bytes(qkv, nunits, cfg);
  if (!ws || ws_bytes < need)
    return fail(RS_ERR_WORKSPACE, "probe workspace too small: need " + std::to_string(need));
  Arena ar(ws, ws_bytes);
  ProbeUnit *d_units = ar.take<ProbeUnit>(nunits);
  int4 *d_groups = ar.take<int4>(nunits);
  float *diag_part = ar.take<float>((size_t)nunits * nchunks * (kRange + rmax));
  float *ent_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *loc_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *max_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *sum_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *cov_part = ar.take<float>((size_t)nunits * nchunks * rmax * kMaxCand);
  float *qbar = nullptr, *kbar = nullptr;
  if (cfg->flags & RS_PROBE_BLOCKMEAN) {
    qbar = ar.take<float>((size_t)qkv->hq * nb * qkv->d);
    kbar = ar.take<float>((size_t)qkv->hkv * nb * qkv->d);
  }
  // per-unit tables: read from the caller's unit table, or built here and uploaded into the
  // workspace (sampled rows to the probe output in scores mode)
  const bool cover = idx != nullptr;
  const rs_unit_table *tab = qkv->tables;
  const ProbeUnit *pu_dev = d_units;
  const int4 *grp_dev = d_groups;
  const int *rows_dev = out->rows, *subset_dev = out->subset, *nsub_tab = nullptr;
  int ngroups = 0;
  if (tab) {
    const UnitTab t = unit_tab_of(tab);
    pu_dev = t.punits;
    grp_dev = t.groups;
    rows_dev = t.rows;
    subset_dev = t.subset;
    nsub_tab = t.nsub;
    ngroups = tab->ngroups;
  } else {
    ProbeHost h;
    build_probe_host(units, nunits, cfg, qkv->hq / qkv->hkv, h);
    ngroups = (int)h.groups.size();
    RS_HIP(hipMemcpyAsync(d_units, h.units.data(), h.units.size() * sizeof(ProbeUnit), hipMemcpyHostToDevice, st));
    RS_HIP(hipMemcpyAsync(d_groups, h.groups.data(), h.groups.size() * sizeof(int4), hipMemcpyHostToDevice, st));
    if (!cover && (cfg->flags & RS_PROBE_ROWS)) {
      RS_HIP(hipMemcpyAsync(out->rows, h.rows.data(), h.rows.size() * 4, hipMemcpyHostToDevice, st));
      RS_HIP(hipMemcpyAsync(out->subset, h.subset.data(), h.subset.size() * 4, hipMemcpyHostToDevice, st));
      RS_HIP(hipMemcpyAsync(out->nsub, h.nsub.data(), h.nsub.size() * 4, hipMemcpyHostToDevice, st));
    }
    // the pageable host vectors are copied before hipMemcpyAsync returns
  }
  ProbeArgs pa{};
  pa.q = qkv->q; pa.k = qkv->k;
  pa.sq_h = qkv->sq_h; pa.sq_t = qkv->sq_t; pa.sk_h = qkv->sk_h; pa.sk_t = qkv->sk_t;
  pa.n = qkv->n; pa.group = qkv->hq / qkv->hkv; pa.rmax = rmax; pa.nchunks = nchunks;
  pa.c = scale * kLog2e; pa.scale = scale; pa.local_w = cfg->local_w;
  pa.stats_rows = (cfg->r_rec + 63) / 64 * 64;
  pa.units = pu_dev; pa.groups = grp_dev; pa.rows = rows_dev; pa.subset = subset_dev;
  if (tab && !cover && (cfg->flags & RS_PROBE_ROWS)) {
    pa.rows_out = out->rows;
    pa.subset_out = out->subset;
    pa.nsub_out = out->nsub;
    pa.nsub_tab = nsub_tab;
  }
  pa.row_max = out->row_max; pa.row_sum = out->row_sum;
  pa.col = out->col; pa.diag_part = diag_part; pa.ent_part = ent_part; pa.loc_part = loc_part;
  pa.max_part = max_part; pa.sum_part = sum_part;
  pa.diag_w = kRange + rmax;
  pa.cov_part = cov_part;
  if (cover) {
    pa.ncand = ncand;
    int nvs = 0, nbs = 0;
    for (int c = 0; c < ncand; ++c) {
      int cl = 0;
      if (grid[c].fam == RS_VSLASH) cl = nvs++;
      if (grid[c].fam == RS_BSPARSE) cl = nbs++;
      pa.cand[c] = CandDev{grid[c].fam, grid[c].a, grid[c].b, cl};
      if (grid[c].fam == RS_VSLASH && pa.nvs_pref < kPrefVs) {
        pa.vs_pref_c[pa.nvs_pref] = c;
        pa.vs_pref_cl[pa.nvs_pref++] = cl;
      } else if (grid[c].fam == RS_BSPARSE && pa.nbs_pref < kPrefBs) {
        pa.bs_pref_c[pa.nbs_pref] = c;
        pa.bs_pref_cl[pa.nbs_pref++] = cl;
      } else if (grid[c].fam != RS_DENSE) {
        pa.cov_cand[pa.ncov++] = c;
      }
    }
    pa.vs_vbits = idx->vs_vbits; pa.vs_dbits = idx->vs_dbits; pa.nwords = idx->nwords; pa.ncand_vs = idx->ncand_vs;
    pa.bs_bits = idx->bs_bits; pa.nb = idx->nb; pa.nbw = idx->nbw; pa.ncand_bs = idx->ncand_bs;
  }
  if (cfg->flags & RS_PROBE_ROWS || cover) {
    hipError_t e;
    const int mode = cover ? 1 : 0;
    if (qkv->d == 128)
      e = qkv->dtype == RS_BF16 ? launch_rows<128, bf16>(pa, nunits, ngroups, mode, out->diag, out->entropy, out->local, out->cov_rows, out->cov, st)
                                : launch_rows<128, float>(pa, nunits, ngroups, mode, out->diag, out->entropy, out->local, out->cov_rows, out->cov, st);
    else
      e = qkv->dtype == RS_BF16 ? launch_rows<64, bf16>(pa, nunits, ngroups, mode, out->diag, out->entropy, out->local, out->cov_rows, out->cov, st)
                                : launch_rows<64, float>(pa, nunits, ngroups, mode, out->diag, out->entropy, out->local, out->cov_rows, out->cov, st);
    if (e != hipSuccess) return hip_check(e, "probe kernels");
  }
  if (!cover && (cfg->flags & RS_PROBE_BLOCKMEAN)) {
    if (qkv->dtype == RS_BF16) {
      hipLaunchKernelGGL(block_pool_kernel<bf16>, dim3(nb, qkv->hq), dim3(256), 0, st, (const bf16 *)qkv->q,
                         (long long)qkv->sq_h, (long long)qkv->sq_t, qkv->n, qkv->d, qbar);
      hipLaunchKernelGGL(block_pool_kernel<bf16>, dim3(nb, qkv->hkv), dim3(256), 0, st, (const bf16 *)qkv->k,
                         (long long)qkv->sk_h, (long long)qkv->sk_t, qkv->n, qkv->d, kbar);
    } else {
      hipLaunchKernelGGL(block_pool_kernel<float>, dim3(nb, qkv->hq), dim3(256), 0, st, (const float *)qkv->q,
                         (long long)qkv->sq_h, (long long)qkv->sq_t, qkv->n, qkv->d, qbar);
      hipLaunchKernelGGL(block_pool_kernel<float>, dim3(nb, qkv->hkv), dim3(256), 0, st, (const float *)qkv->k,
                         (long long)qkv->sk_h, (long long)qkv->sk_t, qkv->n, qkv->d, kbar);
    }
    const int nbt = (nb + 127) / 128;
    hipLaunchKernelGGL(block_logits_kernel, dim3(nbt * (nbt + 1) / 2, qkv->hq), dim3(256), 0, st, qbar, kbar, nb,
                       qkv->d, qkv->hq / qkv->hkv, scale, out->lbs);
    RS_HIP(hipGetLastError());
  }
  return RS_OK;
}

}  // namespace rs
