// Shared attention probe (Sec. 3.2, Eq. 3 with token-resolution sampled rows) and the
// block-mean estimator of the block-sparse builder (Sec. 3.1), for gfx950.
//
// For each unit (query head h, rows [s0, s1)) the sampled rows I = R u U u Bd are scored
// exactly against keys [0, s1):
//   pass 1  row statistics: max_j l_ij and sum_j exp(l_ij - max) over j <= i;
//   pass 2  normalised a_ij of the recent rows reduced into col[j] = sum_{i in R} a_ij and
//           diag[t] = sum_{i in R} a_{i,i-t};
//   pass 3  (coverage) m_i(c) = sum_{j in S_i(c)} a_ij for every candidate c, and per row
//           the 64-key block entropy and the local-band mass.
// Logit tiles are bf16 MFMA products (S^T = K_tile x Q_rows^T, one lane per sampled row),
// statistics fp32.  Every cross-workgroup reduction goes through per-chunk partials
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
constexpr int kChunk = 128;         // keys per workgroup in the three passes
constexpr int kMaxCand = 16;

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
  float c, scale;
  int local_w;
  const ProbeUnit *units;
  const int4 *groups;  // up to 4 units sharing a key/value head and a segment (-1 pads)
  const int *rows, *subset;
  float *row_max, *row_sum;
  // pass 2 partials / outputs
  float *col, *diag_part, *ent_part, *loc_part;
  int diag_w;  // width of a diagonal partial row (kChunk + rmax)
  // pass 3
  int ncand;
  CandDev cand[kMaxCand];
  const uint32_t *vs_vbits, *vs_dbits;
  int nwords, ncand_vs;
  const uint32_t *bs_bits;
  int nb, nbw, ncand_bs;
  float *cov_part;
};

// Orders this wave's LDS writes before its following LDS reads by other lanes.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// key offset within a 64-key tile of accumulator element (mb, r) for lane half hh
__device__ __forceinline__ int acc_key(int mb, int r, int hh) {
  return 32 * mb + 8 * (r >> 2) + 4 * hh + (r & 3);
}

__device__ __forceinline__ int swz(int r) { return ((r & 3) << 1) | ((r >> 2) & 1); }

// Barrier after which every wave's direct-to-LDS copies (global_load_lds, counted by
// vmcnt) and LDS accesses are complete.  The explicit vmcnt wait is required: the
// compiler's LDS release fence does not always wait for the LDS DMA.
__device__ __forceinline__ void lds_fence_barrier() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

enum { M_STATS = 0, M_SCORES = 1, M_COVER = 2 };

// ---- the three passes over one 128-key chunk --------------------------------------------
// grid: (chunk, unit group).  A group holds the units of up to 4 query heads that share a
// key/value head and a segment, hence the same sampled rows and keys: the chunk's keys are
// copied to LDS once (row-major, XOR-swizzled 16-byte chunks) and wave w handles every
// sampled-row block of the group's unit w against the chunk's 2 tiles.
//   M_STATS   per (row, chunk): max and sum of exp over the chunk's visible keys
//   M_SCORES  normalised a_ij of the recent rows -> col and diagonal partials
//   M_COVER   normalised a_ij -> per-candidate kept mass, block entropy and local mass
template <int D, typename InT, int MODE>
__global__ void __launch_bounds__(256) probe_chunk_kernel(const ProbeArgs a) {
  constexpr int CPR = D / 8, RPI = 64 / CPR;
  constexpr int NLOAD = kChunk / RPI / 4;  // 16-byte loads per thread for the chunk
  constexpr int NT = kChunk / 64;          // tiles per chunk
  const int ch = blockIdx.x;
  const int4 grp = a.groups[blockIdx.y];
  const ProbeUnit U0 = a.units[grp.x];     // shared head group, segment and sampled rows
  const int c0 = ch * kChunk;
  if (c0 >= U0.s1) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hh = lane >> 5;
  const int u = wave == 0 ? grp.x : wave == 1 ? grp.y : wave == 2 ? grp.z : grp.w;
  const InT *Kp = (const InT *)a.k + (long long)(U0.head / a.group) * a.sk_h;

  __shared__ __align__(16) bf16 sK[kChunk * D];
  __shared__ int sRows[4][32];
#pragma unroll
  for (int i = 0; i < NLOAD; ++i) {
    const int row_base = (i * 4 + wave) * RPI;
    const int row = row_base + lane / CPR;
    const int cc = (lane % CPR) ^ swz(row);
    const int j = min(c0 + row, a.n - 1);
    if constexpr (sizeof(InT) == 2) {
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)(Kp + (long long)j * a.sk_t + 8 * cc),
                                       (__attribute__((address_space(3))) void *)(sK + row_base * D), 16, 0, 0);
    } else {
      *(u32x4 *)(sK + row_base * D + 8 * lane) = load8<InT>(Kp + (long long)j * a.sk_t + 8 * cc);
    }
  }

  // pass-specific shared state (one slice per wave = per unit)
  float (*sP)[65] = nullptr;
  float *sCol = nullptr, *sDg = nullptr;
  const int dw = kChunk + U0.nR;                  // diagonals touched by R rows in this chunk
  const int dbase = U0.r0 - (c0 + kChunk - 1);    // smallest such diagonal
  if constexpr (MODE == M_SCORES) {
    __shared__ float sPbuf[4][32][65];            // per-wave probability tile [row][key]
    __shared__ float sColbuf[4][kChunk];          // per-unit column sums
    __shared__ float sDgbuf[4][kChunk + kProbeMaxRows];
    sP = sPbuf[wave];
    sCol = sColbuf[wave];
    sDg = sDgbuf[wave];
    for (int x = lane; x < kChunk; x += 64) sCol[x] = 0.f;
    for (int x = lane; x < dw; x += 64) sDg[x] = 0.f;
  }
  lds_fence_barrier();  // K chunk resident
  if (u < 0) return;    // no unit for this wave (no barrier follows)

  const ProbeUnit U = a.units[u];
  const InT *Qp = (const InT *)a.q + (long long)U.head * a.sq_h;
  const int nrb = (U.nrows + 31) / 32;
  const int kswz = swz(l32);
  // the scores pass only needs the recent rows (the last nR sampled rows)
  const int rb_first = (MODE == M_SCORES) ? (U0.nrows - U0.nR) / 32 : 0;
  for (int rb = rb_first; rb < nrb; ++rb) {
    const int ridx = 32 * rb + l32;
    const bool rvalid = ridx < U.nrows;
    const long long rofs = (long long)u * a.rmax + ridx;
    const int row = rvalid ? a.rows[rofs] : -1;
    if (hh == 0) sRows[wave][l32] = row;
    wave_sync();
    const int rbmax = sRows[wave][min(31, U.nrows - 1 - 32 * rb)];  // rows ascending
    if (rbmax < c0) {  // no row of the block sees this chunk (wave-uniform)
      wave_sync();
      continue;
    }
    u32x4 qf[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      qf[ks] = u32x4{0u, 0u, 0u, 0u};
      if (rvalid) qf[ks] = load8<InT>(Qp + (long long)row * a.sq_t + 16 * ks + 8 * hh);
    }
    float nmc = 0.f, invl = 0.f;
    int sub = -1;
    if constexpr (MODE != M_STATS) {
      nmc = rvalid ? -a.row_max[rofs] * kLog2e : 0.f;
      invl = rvalid ? 1.f / a.row_sum[rofs] : 0.f;
      sub = rvalid ? a.subset[rofs] : -1;
    }
    const bool isR = sub == 0;
    const bool blockR = (MODE == M_SCORES) && (__ballot(isR && hh == 0) != 0ull);
    const int rfirst = max(0, (U.nrows - U.nR) - 32 * rb);  // first recent row in the block
    float m_run = -INFINITY, l_run = 0.f;
    float ent = 0.f, loc = 0.f;
    float cov[kMaxCand];
#pragma unroll
    for (int c = 0; c < kMaxCand; ++c) cov[c] = 0.f;

    for (int tt = 0; tt < NT; ++tt) {
      const int k0 = c0 + 64 * tt;
      if (k0 > rbmax) break;
      f32x16 s[2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[mb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const u32x4 kf = *(const u32x4 *)&sK[(64 * tt + 32 * mb + l32) * D + (((2 * ks + hh) ^ kswz) << 3)];
          s[mb] = mfma32(kf, qf[ks], s[mb]);
        }
      }
      if constexpr (MODE == M_STATS) {
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = k0 + acc_key(mb, r, hh);
            if (j > row) s[mb][r] = -INFINITY;
            mx = fmaxf(mx, s[mb][r]);
          }
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        float ps = 0.f;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) ps += __builtin_amdgcn_exp2f((s[mb][r] - m_use) * a.c);
        l_run = l_run * __builtin_amdgcn_exp2f((m_run - m_use) * a.c) + ps;
        m_run = m_new;
        continue;
      } else {
        float p[2][16];
        float bsum = 0.f, lsum = 0.f;
        const int lo_local = row - a.local_w + 1;  // keys >= lo_local are in the local band
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = k0 + acc_key(mb, r, hh);
            const float v = (rvalid && j <= row) ? __builtin_amdgcn_exp2f(fmaf(s[mb][r], a.c, nmc)) * invl : 0.f;
            p[mb][r] = v;
            bsum += v;
            if constexpr (MODE == M_COVER) {
              if (j >= lo_local) lsum += v;
            }
          }
        if constexpr (MODE == M_SCORES) {
          if (blockR) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
              for (int r = 0; r < 16; ++r) sP[l32][acc_key(mb, r, hh)] = isR ? p[mb][r] : 0.f;
            wave_sync();
            {  // column sums: lane = key
              float cs = 0.f;
              for (int rr = 0; rr < 32; ++rr) cs += sP[rr][lane];
              sCol[64 * tt + lane] += cs;
            }
            {  // diagonal t = i - j over the block's recent rows, stored at t - dbase
              const int i_first = max(U.r0, sRows[wave][0]);
              const int i_last = rbmax;
              const int xlo = i_first - k0 - 63 - dbase;
              const int xn = i_last - i_first + 64;
              for (int xx = lane; xx < xn; xx += 64) {
                const int x = xlo + xx;
                const int t = x + dbase;
                float ds = 0.f;
                for (int i2 = i_first; i2 <= i_last; ++i2) {
                  const int kk = i2 - t - k0;
                  if (kk >= 0 && kk < 64) ds += sP[i2 - i_first + rfirst][kk];
                }
                if (x >= 0 && x < dw) sDg[x] += ds;
              }
            }
            wave_sync();
          }
        } else {  // M_COVER: kept mass of every candidate (whole-tile shortcuts first), descriptors
          const int bq = row >> 6;
          const int kt = k0 >> 6;
          const float tsum = bsum;
          {
            const float bt = bsum + __shfl_xor(bsum, 32);  // mass of the row in this 64-key block
            if (bt > 0.f) ent -= bt * logf(bt);
            loc += lsum;
          }
#pragma unroll
          for (int c = 0; c < kMaxCand; ++c) {
            if (c >= a.ncand) break;
            const CandDev cd = a.cand[c];
            if (cd.fam == RS_DENSE) continue;
            uint64_t M;
            if (cd.fam == RS_ASHAPE) {
              M = prefix_mask(cd.a - k0) | ~prefix_mask(row - cd.b + 1 - k0);
            } else if (cd.fam == RS_VSLASH) {
              const long long vr = ((long long)u * a.ncand_vs + cd.cl) * a.nwords;
              const uint64_t md = __builtin_bitreverse64(bits64_at(a.vs_dbits + vr, a.nwords, row - k0 - 63));
              const uint64_t mv = bits64_at(a.vs_vbits + vr, a.nwords, k0);
              M = md | mv;
            } else {
              const long long br = (((long long)U.head * a.ncand_bs + cd.cl) * a.nb + (rvalid ? bq : 0)) * a.nbw;
              M = (rvalid && ((a.bs_bits[br + (kt >> 5)] >> (kt & 31)) & 1u)) ? ~0ull : 0ull;
            }
            M >>= 4 * hh;
            const uint64_t sel = M & 0x0f0f0f0f0f0f0f0full;  // key slots held by this lane
            if (sel == 0x0f0f0f0f0f0f0f0full) {
              cov[c] += tsum;
            } else if (sel != 0ull) {
              float cs = 0.f;
#pragma unroll
              for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                  if ((sel >> (32 * mb + 8 * (r >> 2) + (r & 3))) & 1ull) cs += p[mb][r];
              cov[c] += cs;
            }
          }
        }
      }
    }
    if constexpr (MODE == M_STATS) {
      const float mo = __shfl_xor(m_run, 32), lo = __shfl_xor(l_run, 32);
      const float mm = fmaxf(m_run, mo);
      const float mu = mm == -INFINITY ? 0.f : mm;
      const float ll = l_run * __builtin_amdgcn_exp2f((m_run - mu) * a.c) + lo * __builtin_amdgcn_exp2f((mo - mu) * a.c);
      if (rvalid && hh == 0) {
        const long long o = ((long long)u * a.rmax + ridx) * a.nchunks + ch;
        a.ent_part[o] = mm;  // chunk max (raw dot product) in the entropy partial slot
        a.loc_part[o] = ll;  // chunk sum in the local-mass partial slot
      }
    } else if constexpr (MODE == M_COVER) {
      loc += __shfl_xor(loc, 32);
      if (rvalid && hh == 0) {
        const long long o = ((long long)u * a.rmax + ridx) * a.nchunks + ch;
        a.ent_part[o] = ent;  // the stats partials were consumed before this pass
        a.loc_part[o] = loc;
      }
      for (int c = 0; c < a.ncand; ++c) {
        const float tot = cov[c] + __shfl_xor(cov[c], 32);
        if (rvalid && hh == 0) a.cov_part[(((long long)u * a.ncand + c) * a.rmax + ridx) * a.nchunks + ch] = tot;
      }
    }
    wave_sync();
  }
  if constexpr (MODE == M_SCORES) {
    wave_sync();
    for (int x = lane; x < kChunk; x += 64) {
      const int j = c0 + x;
      if (j < a.n) a.col[(long long)u * a.n + j] = (j < U.s1) ? sCol[x] : 0.f;
    }
    for (int x = lane; x < dw; x += 64) a.diag_part[((long long)u * a.nchunks + ch) * a.diag_w + x] = sDg[x];
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
  if (x >= U.nrows) return;
  const int row = a.rows[(long long)u * a.rmax + x];
  const int nch = row / kChunk + 1;
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

// diagonals from their chunk partials, zero tails of col/diag: one thread per position
__global__ void probe_finish_kernel(const ProbeArgs a, float *diag, float *entropy, float *local) {
  const int u = blockIdx.y;
  const ProbeUnit U = a.units[u];
  const int x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x < a.n) {
    float v = 0.f;
    if (x < U.s1 && U.nR > 0) {
      // chunks whose diagonal range [r0 - c0 - (kChunk-1), r0 + nR - 1 - c0] holds t = x
      const int chi = min((U.r0 + U.nR - 1 - x) / kChunk, (U.s1 - 1) / kChunk);
      const int clo_num = U.r0 - (kChunk - 1) - x;
      const int clo = clo_num <= 0 ? 0 : (clo_num + kChunk - 1) / kChunk;
      for (int ch = clo; ch <= chi; ++ch) {
        const int dbase = U.r0 - (ch * kChunk + kChunk - 1);
        const int xi = x - dbase;
        if (xi >= 0 && xi < kChunk + U.nR) v += a.diag_part[((long long)u * a.nchunks + ch) * a.diag_w + xi];
      }
    }
    diag[(long long)u * a.n + x] = v;
    if (x >= U.s1) a.col[(long long)u * a.n + x] = 0.f;
  }
}

// descriptors: entropy and local mass of each sampled row, one wave per row
__global__ void probe_desc_kernel(const ProbeArgs a, float *entropy, float *local) {
  const int u = blockIdx.y;
  const ProbeUnit U = a.units[u];
  const int x = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (x >= U.nrows) return;
  const int row = a.rows[(long long)u * a.rmax + x];
  const int nch = row / kChunk + 1;
  const float *pe = a.ent_part + ((long long)u * a.rmax + x) * a.nchunks;
  const float *pl = a.loc_part + ((long long)u * a.rmax + x) * a.nchunks;
  float e = 0.f, l = 0.f;
  for (int ch = lane; ch < nch; ch += 64) {
    e += pe[ch];
    l += pl[ch];
  }
  e = wave_sum(e);
  l = wave_sum(l);
  if (lane == 0) {
    const int nvis = row / 64 + 1;
    entropy[(long long)u * a.rmax + x] = nvis > 1 ? e / logf((float)nvis) : 0.f;
    local[(long long)u * a.rmax + x] = l;
  }
}

// coverage per sampled row and candidate, then the subset means; grid (ncand, nunits)
__global__ void cover_finish_kernel(const ProbeArgs a, float *cov_rows, float *cov) {
  const int u = blockIdx.y, c = blockIdx.x;
  const ProbeUnit U = a.units[u];
  __shared__ float sm[kProbeMaxRows];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int x = wave; x < U.nrows; x += 4) {
    const int row = a.rows[(long long)u * a.rmax + x];
    float m;
    if (a.cand[c].fam == RS_DENSE) {
      m = 1.f;
    } else {
      const int nch = row / kChunk + 1;
      const float *pc = a.cov_part + (((long long)u * a.ncand + c) * a.rmax + x) * a.nchunks;
      float acc = 0.f;
      for (int ch = lane; ch < nch; ch += 64) acc += pc[ch];
      m = wave_sum(acc);
    }
    if (lane == 0) {
      sm[x] = m;
      cov_rows[((long long)u * a.ncand + c) * a.rmax + x] = m;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.f, sub[3] = {0.f, 0.f, 0.f};
    int cnt[3] = {0, 0, 0};
    for (int r = 0; r < U.nrows; ++r) {
      const int s = a.subset[(long long)u * a.rmax + r];
      tot += sm[r];
      if (s >= 0 && s < 3) {
        sub[s] += sm[r];
        cnt[s]++;
      }
    }
    float *o = cov + ((long long)u * a.ncand + c) * 4;
    o[0] = U.nrows ? tot / U.nrows : 0.f;
    for (int s2 = 0; s2 < 3; ++s2) o[1 + s2] = cnt[s2] ? sub[s2] / cnt[s2] : 0.f;
  }
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

// L[h][bq][bk] = qbar . kbar * scale for bk <= bq; 64 x 64 output tiles, fp32 FMA.
__global__ void __launch_bounds__(256) block_logits_kernel(const float *qbar, const float *kbar, int nb, int d,
                                                           int group, float scale, float *lbs) {
  const int h = blockIdx.y;
  // decode lower-triangular tile index
  int tq = 0;
  int t = blockIdx.x;
  while (t > tq) {
    t -= tq + 1;
    ++tq;
  }
  const int tk = t;
  const int nbt = (nb + 63) / 64;
  if (tq >= nbt) return;
  __shared__ float sq[32][65], sk[32][65];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;  // each thread: rows ty*4.., cols tx*4..
  float acc[4][4] = {};
  const float *qb = qbar + (long long)h * nb * d;
  const float *kb = kbar + (long long)(h / group) * nb * d;
  for (int d0 = 0; d0 < d; d0 += 32) {
    for (int x = tid; x < 64 * 32; x += 256) {
      const int r = x / 32, cc = x % 32;
      const int bq = tq * 64 + r, bk = tk * 64 + r;
      sq[cc][r] = bq < nb ? qb[(long long)bq * d + d0 + cc] : 0.f;
      sk[cc][r] = bk < nb ? kb[(long long)bk * d + d0 + cc] : 0.f;
    }
    __syncthreads();
    for (int cc = 0; cc < 32; ++cc) {
      float qa[4], ka[4];
      for (int i = 0; i < 4; ++i) qa[i] = sq[cc][ty * 4 + i];
      for (int j = 0; j < 4; ++j) ka[j] = sk[cc][tx * 4 + j];
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(qa[i], ka[j], acc[i][j]);
    }
    __syncthreads();
  }
  float *lh = lbs + (long long)h * ((long long)nb * (nb + 1) / 2);
  for (int i = 0; i < 4; ++i) {
    const int bq = tq * 64 + ty * 4 + i;
    if (bq >= nb) continue;
    for (int j = 0; j < 4; ++j) {
      const int bk = tk * 64 + tx * 4 + j;
      if (bk > bq) continue;
      lh[(long long)bq * (bq + 1) / 2 + bk] = acc[i][j] * scale;
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

size_t probe_ws_bytes(const rs_qkv *qkv, int32_t nunits, const rs_probe_cfg *cfg) {
  const int rmax = rmax_of(cfg);
  const long long nchunks = (qkv->n + kChunk - 1) / kChunk;
  const int nb = (qkv->n + 63) / 64;
  Arena ar(nullptr, 0);
  ar.take<ProbeUnit>(nunits);
  ar.take<int4>(nunits);
  ar.take<float>((size_t)nunits * nchunks * (kChunk + rmax));     // diag partials
  ar.take<float>((size_t)nunits * nchunks * rmax * 2);            // entropy / local partials
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
  if (mode == 0) {
    hipLaunchKernelGGL((probe_chunk_kernel<D, InT, M_STATS>), dim3(pa.nchunks, ngroups), dim3(256), 0, st, pa);
    hipLaunchKernelGGL(probe_stats_combine_kernel, dim3((pa.rmax + 3) / 4, nunits), dim3(256), 0, st, pa);
    hipLaunchKernelGGL((probe_chunk_kernel<D, InT, M_SCORES>), dim3(pa.nchunks, ngroups), dim3(256), 0, st, pa);
    hipLaunchKernelGGL(probe_finish_kernel, dim3((pa.n + 255) / 256, nunits), dim3(256), 0, st, pa, diag, ent, loc);
  } else {
    hipLaunchKernelGGL((probe_chunk_kernel<D, InT, M_COVER>), dim3(pa.nchunks, ngroups), dim3(256), 0, st, pa);
    hipLaunchKernelGGL(cover_finish_kernel, dim3(pa.ncand, nunits), dim3(256), 0, st, pa, cov_rows, cov);
    hipLaunchKernelGGL(probe_desc_kernel, dim3((pa.rmax + 3) / 4, nunits), dim3(256), 0, st, pa, ent, loc);
  }
  return hipGetLastError();
}

rs_status probe_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                       const rs_probe_cfg *cfg, const rs_candidate *grid, int32_t ncand,
                       const rs_index_set *idx, void *ws, size_t ws_bytes, rs_probe_out *out, hipStream_t st) {
  const int rmax = rmax_of(cfg);
  const int nchunks = (qkv->n + kChunk - 1) / kChunk;
  const int nb = (qkv->n + 63) / 64;
  const size_t need = probe_ws_bytes(qkv, nunits, cfg);
  if (!ws || ws_bytes < need)
    return fail(RS_ERR_WORKSPACE, "probe workspace too small: need " + std::to_string(need));
  Arena ar(ws, ws_bytes);
  ProbeUnit *d_units = ar.take<ProbeUnit>(nunits);
  int4 *d_groups = ar.take<int4>(nunits);
  float *diag_part = ar.take<float>((size_t)nunits * nchunks * (kChunk + rmax));
  float *ent_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *loc_part = ar.take<float>((size_t)nunits * nchunks * rmax);
  float *cov_part = ar.take<float>((size_t)nunits * nchunks * rmax * kMaxCand);
  float *qbar = nullptr, *kbar = nullptr;
  if (cfg->flags & RS_PROBE_BLOCKMEAN) {
    qbar = ar.take<float>((size_t)qkv->hq * nb * qkv->d);
    kbar = ar.take<float>((size_t)qkv->hkv * nb * qkv->d);
  }
  // sampled rows are computed here and uploaded (scores mode), or re-derived (coverage)
  std::vector<ProbeUnit> hu(nunits);
  std::vector<int> hrows((size_t)nunits * rmax, -1), hsub((size_t)nunits * rmax, -1), hn((size_t)nunits * 3, 0);
  for (int u = 0; u < nunits; ++u) {
    std::vector<int> rows, lab;
    int r0;
    sample_rows(units[u].s0, units[u].s1, *cfg, rows, lab, r0);
    hu[u] = ProbeUnit{units[u].head, units[u].s0, units[u].s1, (int)rows.size(), r0, units[u].s1 - r0, 0, 0};
    for (size_t x = 0; x < rows.size(); ++x) {
      hrows[(size_t)u * rmax + x] = rows[x];
      hsub[(size_t)u * rmax + x] = lab[x];
      hn[(size_t)u * 3 + lab[x]]++;
    }
  }
  RS_HIP(hipMemcpyAsync(d_units, hu.data(), hu.size() * sizeof(ProbeUnit), hipMemcpyHostToDevice, st));
  // unit groups: the query heads of one key/value head over the same segment, up to 4
  std::vector<int4> hg;
  {
    const int G = qkv->hq / qkv->hkv;
    std::vector<std::vector<int>> open_lists;
    std::vector<long long> keys;
    for (int u = 0; u < nunits; ++u) {
      const long long key = ((long long)(units[u].head / G) * (kMaxN + 1) + units[u].s0) * (kMaxN + 1) + units[u].s1;
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
    for (auto &l : open_lists) {
      int4 g{-1, -1, -1, -1};
      g.x = l[0];
      if (l.size() > 1) g.y = l[1];
      if (l.size() > 2) g.z = l[2];
      if (l.size() > 3) g.w = l[3];
      hg.push_back(g);
    }
  }
  const int ngroups = (int)hg.size();
  RS_HIP(hipMemcpyAsync(d_groups, hg.data(), hg.size() * sizeof(int4), hipMemcpyHostToDevice, st));
  const bool cover = idx != nullptr;
  if (!cover && (cfg->flags & RS_PROBE_ROWS)) {
    RS_HIP(hipMemcpyAsync(out->rows, hrows.data(), hrows.size() * 4, hipMemcpyHostToDevice, st));
    RS_HIP(hipMemcpyAsync(out->subset, hsub.data(), hsub.size() * 4, hipMemcpyHostToDevice, st));
    RS_HIP(hipMemcpyAsync(out->nsub, hn.data(), hn.size() * 4, hipMemcpyHostToDevice, st));
  }
  ProbeArgs pa{};
  pa.q = qkv->q; pa.k = qkv->k;
  pa.sq_h = qkv->sq_h; pa.sq_t = qkv->sq_t; pa.sk_h = qkv->sk_h; pa.sk_t = qkv->sk_t;
  pa.n = qkv->n; pa.group = qkv->hq / qkv->hkv; pa.rmax = rmax; pa.nchunks = nchunks;
  pa.c = scale * kLog2e; pa.scale = scale; pa.local_w = cfg->local_w;
  pa.units = d_units; pa.groups = d_groups; pa.rows = out->rows; pa.subset = out->subset;
  pa.row_max = out->row_max; pa.row_sum = out->row_sum;
  pa.col = out->col; pa.diag_part = diag_part; pa.ent_part = ent_part; pa.loc_part = loc_part;
  pa.diag_w = kChunk + rmax;
  pa.cov_part = cov_part;
  if (cover) {
    pa.ncand = ncand;
    int nvs = 0, nbs = 0;
    for (int c = 0; c < ncand; ++c) {
      int cl = 0;
      if (grid[c].fam == RS_VSLASH) cl = nvs++;
      if (grid[c].fam == RS_BSPARSE) cl = nbs++;
      pa.cand[c] = CandDev{grid[c].fam, grid[c].a, grid[c].b, cl};
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
    const int nbt = (nb + 63) / 64;
    hipLaunchKernelGGL(block_logits_kernel, dim3(nbt * (nbt + 1) / 2, qkv->hq), dim3(256), 0, st, qbar, kbar, nb,
                       qkv->d, qkv->hq / qkv->hkv, scale, out->lbs);
    RS_HIP(hipGetLastError());
  }
  return RS_OK;
}

}  // namespace rs
