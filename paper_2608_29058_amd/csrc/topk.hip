// Candidate index construction (Sec. 3.1) for gfx950: deterministic top-k selection.
//
// Every selection uses one total order: score descending (scores mapped to
// order-preserving 32-bit keys, so -0.0 ranks below +0.0), then position ascending.
// The k-th key is found by a 4-pass radix select over 8-bit digits (LDS histograms with
// integer atomics); elements above it are taken, and among elements equal to it the
// lowest positions are taken through an ordered block scan.  Sets are emitted as bitmaps
// and as ascending lists.
//
//   vertical-slash, per unit and candidate (n_v, n_s):
//     V = top n_v columns of col[0, s1);  D = {0} + top (n_s - 1) diagonals of diag[1, s1)
//   block-sparse, per query head and query block bq:
//     ranking {bq} + blocks [0, bq) by pooled score; Sel_k(bq) = first k of the ranking
#include <algorithm>
#include <vector>

#include "common.h"

namespace rs {

constexpr int kMaxCandFam = 8;

// The helpers below run over a group of NT threads: the whole workgroup, or with NT = 64 one
// wave of it (each wave then works on its own data and LDS, synchronising only itself).
template <int NT>
__device__ __forceinline__ void gsync() {
  if constexpr (NT == 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}
template <int NT>
__device__ __forceinline__ int gtid() {
  return NT == 64 ? (int)(threadIdx.x & 63u) : (int)threadIdx.x;
}

// inclusive prefix sum of v over the group; returns it, total in *tot
template <int NT>
__device__ int block_incl_scan(int v, int *sWave, int *tot) {
  constexpr int NWV = NT / 64;
  const int lane = threadIdx.x & 63, wave = gtid<NT>() >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if constexpr (NWV == 1) {
    *tot = __shfl(x, 63);
    return x;
  }
  if (lane == 63) sWave[wave] = x;
  gsync<NT>();
  int off = 0, all = 0;
  for (int w = 0; w < NWV; ++w) {
    const int t = sWave[w];
    if (w < wave) off += t;
    all += t;
  }
  gsync<NT>();
  *tot = all;
  return x + off;
}

// Radix select over keys of vals[0, len): finds the key T of rank K (1-based, descending),
// how many elements equal to T are taken and how many there are.  Requires len > K >= 1.
// sHist holds one 256-bin histogram per wave of the group (values of similar magnitude share
// their leading digits: one histogram for all waves would serialise their atomics).
// Returns true when it stopped early instead: the elements above the digit bin holding the
// K-th key and that bin together number at most cap, and T is then the bin's leading digits
// with zero lower digits (they are exactly the keys >= T).
template <int NT>
__device__ bool radix_select(const float *vals, int len, int K, int cap, uint32_t *T_out, int *take_out,
                             int *eq_out, int *sHist, int *sBcast) {
  constexpr int NWV = NT / 64;
  uint32_t prefix = 0, maskhi = 0;
  int krem = K;
  int *myHist = sHist + 256 * (gtid<NT>() >> 6);
  for (int byte = 3; byte >= 0; --byte) {
    for (int b = gtid<NT>(); b < 256 * NWV; b += NT) sHist[b] = 0;
    gsync<NT>();
    // eight loads in flight per thread before their histogram updates (counts do not depend
    // on the order of the adds)
    int i = gtid<NT>();
    for (; i + 7 * NT < len; i += 8 * NT) {
      uint32_t k8[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) k8[j] = float_key(vals[i + j * NT]);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if ((k8[j] & maskhi) == prefix) atomicAdd(&myHist[(k8[j] >> (8 * byte)) & 255u], 1);
    }
    for (; i < len; i += NT) {
      const uint32_t key = float_key(vals[i]);
      if ((key & maskhi) == prefix) atomicAdd(&myHist[(key >> (8 * byte)) & 255u], 1);
    }
    gsync<NT>();
    if (gtid<NT>() < 64) {
      // lane l owns bins 255-4l .. 252-4l (descending); wave-wide inclusive scan of counts
      const int l = gtid<NT>();
      int c4[4], own = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c4[q] = 0;
        for (int w = 0; w < NWV; ++w) c4[q] += sHist[256 * w + 255 - 4 * l - q];
        own += c4[q];
      }
      int incl = own;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (l >= o) incl += y;
      }
      const int excl = incl - own;
      // the selected bin lies in the first lane whose inclusive count reaches krem
      if (excl < krem && incl >= krem) {
        int cum = excl, sel = 255 - 4 * l, cnt = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (cum + c4[q] >= krem) {
            sel = 255 - 4 * l - q;
            cnt = c4[q];
            break;
          }
          cum += c4[q];
        }
        sBcast[0] = sel;
        sBcast[1] = krem - cum;
        sBcast[2] = cnt;  // after the last digit: the number of keys equal to T
      }
    }
    gsync<NT>();
    prefix |= (uint32_t)sBcast[0] << (8 * byte);
    maskhi |= 0xffu << (8 * byte);
    krem = sBcast[1];
    *eq_out = sBcast[2];
    gsync<NT>();
    if (byte > 0 && K - krem + *eq_out <= cap) {
      *T_out = prefix;
      *take_out = krem;
      return true;
    }
  }
  *T_out = prefix;
  *take_out = krem;
  return false;
}

// Calls emit(i) for each selected element index of vals[0, len) (top K in the total order).
// With cap > K the radix passes may stop early: emit is then called for every element whose
// key shares the leading digits of the K-th key or is above them (at most cap elements, the
// top K among them), and the caller selects the top K from those.
template <int NT, typename F>
__device__ void select_top(const float *vals, int len, int K, int *sHist, int *sBcast, int *sWave, F emit,
                           int cap = 0) {
  if (K <= 0) return;
  if (len <= K) {
    for (int i = gtid<NT>(); i < len; i += NT) emit(i);
    return;
  }
  uint32_t T;
  int take, neq;
  if (radix_select<NT>(vals, len, K, max(cap, K), &T, &take, &neq, sHist, sBcast)) {
    int ie = gtid<NT>();
    for (; ie + 7 * NT < len; ie += 8 * NT) {
      uint32_t k8[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) k8[j] = float_key(vals[ie + j * NT]);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (k8[j] >= T) emit(ie + j * NT);
    }
    for (; ie < len; ie += NT)
      if (float_key(vals[ie]) >= T) emit(ie);
    return;
  }
  // every key equal to T is taken when there are no more of them than needed (the usual case)
  const bool all_eq = take == neq;
  int ie = gtid<NT>();
  for (; ie + 7 * NT < len; ie += 8 * NT) {
    uint32_t k8[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) k8[j] = float_key(vals[ie + j * NT]);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k8[j] > T || (all_eq && k8[j] == T)) emit(ie + j * NT);
  }
  for (; ie < len; ie += NT) {
    const uint32_t key = float_key(vals[ie]);
    if (key > T || (all_eq && key == T)) emit(ie);
  }
  if (all_eq) return;
  // equal keys: lowest positions first
  int seen = 0;
  for (int i0 = 0; i0 < len && seen < take; i0 += NT) {
    const int i = i0 + gtid<NT>();
    const int f = (i < len && float_key(vals[i]) == T) ? 1 : 0;
    int tot;
    const int incl = block_incl_scan<NT>(f, sWave, &tot);
    if (f && seen + incl - 1 < take) emit(i);
    seen += tot;
  }
}

// ascending list of set bits of bits[0, nwords) -> out, padded with -1 to cap; returns count
template <int NT>
__device__ int bits_to_list(const uint32_t *bits, int nwords, int *out, int cap, int *sWave) {
  constexpr int WPT_MAX = 16;
  const int wpt = (nwords + NT - 1) / NT;  // contiguous words per thread
  const int w0 = gtid<NT>() * wpt;
  int cnt = 0;
  for (int w = w0; w < min(nwords, w0 + wpt); ++w) cnt += __builtin_popcount(bits[w]);
  int tot;
  const int incl = block_incl_scan<NT>(cnt, sWave, &tot);
  int p = incl - cnt;
  for (int w = w0; w < min(nwords, w0 + wpt); ++w) {
    uint32_t b = bits[w];
    while (b) {
      const int bit = __builtin_ctz(b);
      b &= b - 1;
      if (p < cap) out[p] = w * 32 + bit;
      ++p;
    }
  }
  (void)WPT_MAX;
  for (int x = tot + gtid<NT>(); x < cap; x += NT) out[x] = -1;
  return tot;
}

struct VsArgs {
  const float *col, *diag;
  int n, nunits, ncand_vs;
  const int *s1;  // [nunits]
  int nv[kMaxCandFam], ns[kMaxCandFam];
  int nv_max, ns_max, nwords;
  int gcap;  // capacity of the LDS gather of the largest set
  int *vsorted, *dsorted, *count;
  uint32_t *vbits, *dbits;
};

// grid: (2, nunits); blockIdx.x = array (0: V from col, 1: D from diag).  Budgets of the family
// are nested prefixes of one ranking: a superset of the largest set is taken from the whole
// array (the radix passes stop once the keys sharing the leading digits of its last key fit
// the gather, usually after two of the four passes), gathered in ascending position into LDS,
// and every budget is selected from it.
constexpr int kVsGather = 8192;  // elements kept in LDS, at most
// Dynamic LDS: [nwords bitmap words][gcap values][gcap positions], gcap = twice the largest
// budget selected from the whole array (at most kVsGather): the LDS of a workgroup is then
// sized for the grid's budgets (two workgroups share a compute unit for budgets up to about
// 3K at n = 128K, where the bitmap takes 16 KB).
__global__ void __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8, 8))) vs_select_kernel(const VsArgs a) {
  constexpr int NT = 1024;
  extern __shared__ uint32_t sDyn[];
  uint32_t *sBits = sDyn;
  float *sVal = (float *)(sDyn + a.nwords);
  int *sPos = (int *)(sVal + a.gcap);
  __shared__ int sHist[256 * (NT / 64)], sBcast[3], sWave[NT / 64];
  const int arr = blockIdx.x;
  const int u = blockIdx.y;
  const int s1 = a.s1[u];
  // the array and its offset: D selects diagonals [1, s1) and forces diagonal 0
  const float *vals = arr == 0 ? a.col + (long long)u * a.n : a.diag + (long long)u * a.n + 1;
  const int len = arr == 0 ? s1 : s1 - 1, off = arr == 0 ? 0 : 1;
  auto budget = [&](int c) { return arr == 0 ? a.nv[c] : a.ns[c] - 1; };  // selected from vals
  int cmax = 0;
  for (int c = 1; c < a.ncand_vs; ++c)
    if (budget(c) > budget(cmax)) cmax = c;
  const int kmax = budget(cmax);
  // a superset of the largest set (at most gcap elements): bitmap, then its members in
  // ascending position with their values (when the largest set fits in LDS; otherwise every
  // budget is selected from the whole array)
  const bool gather = kmax <= a.gcap;
  int nmax = 0;
  if (gather) {
    for (int w = threadIdx.x; w < a.nwords; w += NT) sBits[w] = 0u;
    __syncthreads();
    select_top<NT>(
        vals, len, kmax, sHist, sBcast, sWave, [&](int i) { atomicOr(&sBits[(i + off) >> 5], 1u << ((i + off) & 31)); },
        a.gcap);
    __syncthreads();
    nmax = bits_to_list<NT>(sBits, a.nwords, sPos, a.gcap, sWave);
    __syncthreads();
    for (int x = threadIdx.x; x < nmax; x += NT) sVal[x] = vals[sPos[x] - off];
    __syncthreads();
  }
  for (int c = 0; c < a.ncand_vs; ++c) {
    const long long row = (long long)u * a.ncand_vs + c;
    for (int w = threadIdx.x; w < a.nwords; w += NT) sBits[w] = 0u;
    __syncthreads();
    if (!gather) {
      select_top<NT>(vals, len, budget(c), sHist, sBcast, sWave,
                     [&](int i) { atomicOr(&sBits[(i + off) >> 5], 1u << ((i + off) & 31)); });
    } else if (nmax <= budget(c)) {  // the whole gathered set (the largest set itself)
      for (int x = threadIdx.x; x < nmax; x += NT) atomicOr(&sBits[sPos[x] >> 5], 1u << (sPos[x] & 31));
    } else {
      select_top<NT>(sVal, nmax, budget(c), sHist, sBcast, sWave, [&](int x) {
        const int t = sPos[x];
        atomicOr(&sBits[t >> 5], 1u << (t & 31));
      });
    }
    __syncthreads();
    if (arr == 1 && a.ns[c] >= 1 && threadIdx.x == 0) atomicOr(&sBits[0], 1u);  // diagonal 0
    __syncthreads();
    uint32_t *gb = (arr == 0 ? a.vbits : a.dbits) + row * a.nwords;
    for (int w = threadIdx.x; w < a.nwords; w += NT) gb[w] = sBits[w];
    int *list = arr == 0 ? a.vsorted + row * a.nv_max : a.dsorted + row * a.ns_max;
    const int cnt = bits_to_list<NT>(sBits, a.nwords, list, arr == 0 ? a.nv_max : a.ns_max, sWave);
    if (threadIdx.x == 0) a.count[row * 2 + arr] = cnt;
    __syncthreads();
  }
}

// select_top for one wave whose elements are held in registers: key[c] is the key of element
// c * 64 + lane (elements >= len are ignored).  emit(c, take) is called by the whole wave, once
// per register c and step (take: this lane's element c * 64 + lane is selected there), so that
// it can place the selected elements with a ballot instead of an LDS counter.  Radix
// select over 8-bit digits with one 256-bin histogram, then the lowest positions among keys
// equal to the threshold.  With cap > K the caller orders what it gets and keeps the first K:
// the passes then stop as soon as the elements above the digit bin holding the K-th key and
// that bin together number at most cap, and every one of them is emitted (the top K and the
// rest of that bin; at most cap taken).  With cap = K it takes exactly the top K.
template <int NV, typename F>
__device__ void select_top_regs(const uint32_t (&key)[NV], int len, int K, int cap, int *sHist, int *sBcast,
                                F emit) {
  const int l = (int)(threadIdx.x & 63u);
  if (K <= 0) return;
  if (len <= K) {
#pragma unroll
    for (int c = 0; c < NV; ++c) emit(c, c * 64 + l < len);
    return;
  }
  uint32_t prefix = 0, maskhi = 0;
  int krem = K, neq = 0;
  for (int byte = 3; byte >= 0; --byte) {
    for (int b = l; b < 256; b += 64) sHist[b] = 0;
    gsync<64>();
#pragma unroll
    for (int c = 0; c < NV; ++c)
      if (c * 64 + l < len && (key[c] & maskhi) == prefix) atomicAdd(&sHist[(key[c] >> (8 * byte)) & 255u], 1);
    gsync<64>();
    // lane l owns bins 255-4l .. 252-4l (descending); inclusive scan of the counts
    int c4[4], own = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c4[q] = sHist[255 - 4 * l - q];
      own += c4[q];
    }
    int incl = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (l >= o) incl += y;
    }
    const int excl = incl - own;
    if (excl < krem && incl >= krem) {
      int cum = excl, sel = 255 - 4 * l, cnt = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (cum + c4[q] >= krem) {
          sel = 255 - 4 * l - q;
          cnt = c4[q];
          break;
        }
        cum += c4[q];
      }
      sBcast[0] = sel;
      sBcast[1] = krem - cum;
      sBcast[2] = cnt;
    }
    gsync<64>();
    prefix |= (uint32_t)sBcast[0] << (8 * byte);
    maskhi |= 0xffu << (8 * byte);
    krem = sBcast[1];
    neq = sBcast[2];
    gsync<64>();
    // K - krem elements lie in higher bins, neq in the bin of the K-th key: when they fit in
    // cap, they are all the keys whose leading digits are at least prefix's (key >= prefix,
    // the lower digits of prefix being zero)
    if (byte > 0 && K - krem + neq <= cap) {
#pragma unroll
      for (int c = 0; c < NV; ++c) emit(c, c * 64 + l < len && key[c] >= prefix);
      return;
    }
  }
  const uint32_t T = prefix;
  const int take = krem;
  const bool all_eq = take == neq;
#pragma unroll
  for (int c = 0; c < NV; ++c) emit(c, c * 64 + l < len && (key[c] > T || (all_eq && key[c] == T)));
  if (all_eq) return;
  int seen = 0;
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    if (c * 64 >= len || seen >= take) break;
    const int f = (c * 64 + l < len && key[c] == T) ? 1 : 0;
    int tot;
    const int in = block_incl_scan<64>(f, nullptr, &tot);
    emit(c, f && seen + in - 1 < take);
    seen += tot;
  }
}

struct BsArgs {
  const float *lbs;
  int nb, hq, ncand_bs, k_max, nbw;
  int k[kMaxCandFam];
  int *rank, *sorted, *count;
  uint32_t *bits;
};

// grid: (ceil(nb / 4), hq), 256 threads; one query block per wave (waves synchronise only
// themselves: each has its own LDS).  The wave's pooled scores are read once into registers
// (NV per lane, NV * 64 >= nb - 1).
template <int NV>
__global__ void __launch_bounds__(256) bs_select_kernel(const BsArgs a) {
  constexpr int NT = 64;
  constexpr int SP = 256;  // sort capacity (k_max <= 256)
  constexpr int NBW = kMaxN / 64 / 32;
  __shared__ int sHistA[4][256], sBcastA[4][3];
  __shared__ unsigned long long sKeyA[4][SP];
  __shared__ uint32_t sBA[4][NBW];
  const int w = (int)(threadIdx.x >> 6), l = (int)(threadIdx.x & 63u);
  const int bq = (int)blockIdx.x * 4 + w, h = blockIdx.y;
  if (bq >= a.nb) return;  // this wave has no query block; the others never wait for it
  int *sHist = sHistA[w], *sBcast = sBcastA[w];
  unsigned long long *sKey = sKeyA[w];
  uint32_t *sB = sBA[w];
  const float *vals = a.lbs + (long long)h * ((long long)a.nb * (a.nb + 1) / 2) + (long long)bq * (bq + 1) / 2;
  for (int x = l; x < SP; x += NT) sKey[x] = 0ull;
  gsync<NT>();
  const int K = a.k_max - 1;
  uint32_t key[NV];
#pragma unroll
  for (int c = 0; c < NV; ++c) key[c] = c * 64 + l < bq ? float_key(vals[c * 64 + l]) : 0u;
  // up to SP candidates are taken, in slots given by a ballot (nsel, the same in every lane,
  // counts the slots used); the sort below orders them and the first K are kept
  int nsel_t = 0;
  select_top_regs<NV>(key, bq, K, SP, sHist, sBcast, [&](int c, bool take) {
    const uint64_t m = __ballot(take);
    if (take) {
      const int p = nsel_t + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      sKey[p] = ((unsigned long long)key[c] << 32) | (unsigned long long)(0xffffffffu - (uint32_t)(c * 64 + l));
    }
    nsel_t += __popcll(m);
  });
  gsync<NT>();
  // bitonic sort, descending, in registers: element e = 4 l + j is key kr[j] of lane l; pairs
  // at a distance of 4 or more meet across lanes (lane l ^ stride / 4), closer ones within a
  // lane.  The keys are distinct (block index in the low word; empty slots are 0), so the
  // order is the unique descending one.
  static_assert(SP == 4 * NT, "four keys per lane");
  unsigned long long kr[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) kr[j] = sKey[4 * l + j];
#pragma unroll
  for (int size = 2; size <= SP; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= 4) {
        const int lx = stride >> 2;
        const bool lo = (l & lx) == 0, desc = ((4 * l) & size) == 0;  // size >= 8: j drops out
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t plo = (uint32_t)__shfl_xor((int)(uint32_t)kr[j], lx);
          const uint32_t phi = (uint32_t)__shfl_xor((int)(uint32_t)(kr[j] >> 32), lx);
          const unsigned long long p = ((unsigned long long)phi << 32) | plo;
          const bool keep_max = lo == desc;  // the lower element keeps the larger key when descending
          kr[j] = keep_max ? (kr[j] > p ? kr[j] : p) : (kr[j] < p ? kr[j] : p);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (j & stride) continue;
          const bool desc = ((4 * l + j) & size) == 0;
          const unsigned long long A = kr[j], B = kr[j | stride];
          if ((A < B) == desc) {
            kr[j] = B;
            kr[j | stride] = A;
          }
        }
      }
    }
#pragma unroll
  for (int j = 0; j < 4; ++j) sKey[4 * l + j] = kr[j];
  gsync<NT>();
  const int nsel = min(K, bq);
  int *rk = a.rank + ((long long)h * a.nb + bq) * a.k_max;
  for (int x = l; x < a.k_max; x += NT) {
    int v = -1;
    if (x == 0) v = bq;
    else if (x - 1 < nsel) v = (int)(0xffffffffu - (uint32_t)(sKey[x - 1] & 0xffffffffull));
    rk[x] = v;
  }
  for (int c = 0; c < a.ncand_bs; ++c) {
    for (int x = l; x < a.nbw; x += NT) sB[x] = 0u;
    gsync<NT>();
    const int take = min(a.k[c], bq + 1);
    for (int x = l; x < take; x += NT) {
      const int blk = x == 0 ? bq : (int)(0xffffffffu - (uint32_t)(sKey[x - 1] & 0xffffffffull));
      atomicOr(&sB[blk >> 5], 1u << (blk & 31));
    }
    gsync<NT>();
    const long long crow = ((long long)h * a.ncand_bs + c) * a.nb + bq;
    for (int x = l; x < a.nbw; x += NT) a.bits[crow * a.nbw + x] = sB[x];
    const int cnt = bits_to_list<NT>(sB, a.nbw, a.sorted + crow * a.k_max, a.k_max, nullptr);
    if (l == 0) a.count[crow] = cnt;
    gsync<NT>();
  }
}

rs_status build_indices_launch(const rs_probe_out *sc, const rs_unit *units, int32_t nunits,
                               const rs_candidate *grid, int32_t ncand, rs_index_set *out, hipStream_t st,
                               void *ws, size_t ws_bytes) {
  int nvs = 0, nbs = 0;
  VsArgs va{};
  BsArgs ba{};
  for (int c = 0; c < ncand; ++c) {
    if (grid[c].fam == RS_VSLASH) {
      va.nv[nvs] = grid[c].a;
      va.ns[nvs] = grid[c].b;
      ++nvs;
    } else if (grid[c].fam == RS_BSPARSE) {
      ba.k[nbs++] = grid[c].a;
    }
  }
  if (nvs > 0) {
    // unit key lengths: from the probe's unit table, else uploaded into the workspace
    const int *d_s1 = nullptr;
    if (sc->tables) {
      d_s1 = unit_tab_s1(sc->tables);
    } else {
      Arena ar(ws, ws_bytes);
      int *w_s1 = ar.take<int>(nunits);
      if (!ws || !ar.ok()) return fail(RS_ERR_WORKSPACE, "index workspace too small");
      std::vector<int> hs1(nunits);
      for (int u = 0; u < nunits; ++u) hs1[u] = units[u].s1;
      // the pageable host vector is copied before hipMemcpyAsync returns
      RS_HIP(hipMemcpyAsync(w_s1, hs1.data(), nunits * sizeof(int), hipMemcpyHostToDevice, st));
      d_s1 = w_s1;
    }
    va.col = sc->col; va.diag = sc->diag; va.n = sc->n; va.nunits = nunits; va.ncand_vs = nvs;
    va.s1 = d_s1; va.nv_max = out->nv_max; va.ns_max = out->ns_max; va.nwords = out->nwords;
    va.vsorted = out->vs_vsorted; va.dsorted = out->vs_dsorted; va.count = out->vs_count;
    va.vbits = out->vs_vbits; va.dbits = out->vs_dbits;
    int kbig = 0;  // the largest budget selected from a whole array (columns: n_v, diagonals: n_s - 1)
    for (int c = 0; c < nvs; ++c) kbig = std::max(kbig, std::max(va.nv[c], va.ns[c] - 1));
    va.gcap = std::min(kVsGather, 2 * std::max(kbig, 1));
    const size_t lds = (size_t)out->nwords * sizeof(uint32_t) + (size_t)va.gcap * (sizeof(float) + sizeof(int));
    hipLaunchKernelGGL(vs_select_kernel, dim3(2, nunits), dim3(1024), lds, st, va);
    RS_HIP(hipGetLastError());
  }
  if (nbs > 0) {
    ba.lbs = sc->lbs; ba.nb = out->nb; ba.hq = out->hq; ba.ncand_bs = nbs; ba.k_max = out->k_max; ba.nbw = out->nbw;
    ba.rank = out->bs_rank; ba.sorted = out->bs_sorted; ba.count = out->bs_count; ba.bits = out->bs_bits;
    if (out->nb - 1 <= 32 * 64)
      hipLaunchKernelGGL(bs_select_kernel<32>, dim3((out->nb + 3) / 4, out->hq), dim3(256), 0, st, ba);
    else
      hipLaunchKernelGGL(bs_select_kernel<kMaxN / 64 / 64>, dim3((out->nb + 3) / 4, out->hq), dim3(256), 0, st, ba);
    RS_HIP(hipGetLastError());
  }
  return RS_OK;
}

}  // namespace rs
