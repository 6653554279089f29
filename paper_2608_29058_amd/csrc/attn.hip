// Causal dense and pattern-sparse attention prefill for gfx950 (bf16 MFMA, fp32 softmax).
//
// Computes, for each unit (query head, rows [s0, s1)), O_i = sum_{j in S_i} softmax(l_i.)_j v_j
// over the kept key set S_i of the unit's pattern (Sec. 2.1: masked logits are minus
// infinity, rows renormalise on their kept set).  The sets are token-exact:
//   dense      S_i = {j <= i}
//   A-shape    S_i = {j <= i : j < sink or j > i - window}
//   block      S_i = {j <= i : j / 64 in Sel(i / 64)}
//   vert-slash S_i = {j in V, j <= i} u {i - t : t in D, t <= i}
//
// Work decomposition: one workgroup = one 128-row query tile of one unit, 4 waves of 32
// rows each; two workgroups share a CU (<= 256 VGPRs, 64 KB LDS each), so one's softmax
// overlaps the other's matrix work.  Keys stream through two LDS buffers in tiles of 64
// (contiguous keys, or gathered vertical columns for vertical-slash): the next tile is
// copied global -> LDS directly (global_load_lds_dwordx4, no registers) while the current
// one is computed, with one barrier per tile.  K and V tiles are row-major with an XOR
// swizzle of the 16-byte chunks.  Per wave and key tile:
//   S^T[64 keys x 32 rows] = K_tile (A operand) x Q^T (B operand, registers)
// with v_mfma_f32_32x32x16_bf16, so each lane holds one query row and 32 of its keys:
// row max / row sum are in-lane plus one exchange with the other lane half.  Then
//   O^T[d x 32 rows] += V^T (A operand, read transposed with ds_read_b64_tr_b16) x P^T
// (B operand: the probabilities straight from the S^T accumulators, packed to bf16).
// Online softmax in the exp2 domain (logit * scale * log2 e), fp32 statistics; the running
// max is raised only when it grows by more than 2^8, so the O rescale is rare.
// Block-sparse: the workgroup's two 64-row query blocks walk the union of their block
// lists from the diagonal block down; each pair of waves computes only the blocks its own
// query block selected.  The two blocks are the same rows of two heads that read one
// key/value head when both heads' units are block-sparse (their selections overlap far more
// than two consecutive blocks of one head do), else consecutive blocks of one head.
// Vertical-slash takes its diagonal-band tiles from the diagonal down as well, then the
// gathered columns.  (Items that start together share their blocks near the diagonal; taken
// first, those are still in L2 when the neighbours reach them.)
#include <algorithm>
#include <cstring>
#include <map>
#include <tuple>
#include <vector>

#include "common.h"

namespace rs {

enum { P_DENSE = 0, P_ASHAPE = 1, P_VS = 2, P_BS = 3 };

struct AttnArgs {
  const void *q, *k, *v;
  long long sq_h, sq_t, sk_h, sk_t, sv_h, sv_t;
  bf16 *o;
  long long so_h, so_t;
  float *lse;
  int n, group;
  float c, scale;
  const DevUnit *units;
  const int *order;   // items; with queues, bucket b's at order[qoff[b] .. qoff[b] + qsize[b])
  const int *qsize;   // [8] items per key/value bucket (device), or NULL: one item per workgroup
  const int *qoff;    // [8]
  int *qcount;        // [8] items taken per bucket (device counters, start at 0)
  const bf16 *vt;  // V^T layout of rs_transpose_v (used by the VT instantiations)
  int npad;
  const int *vs_vsorted, *vs_dsorted, *vs_count;
  const uint32_t *vs_vbits, *vs_dbits;
  int nv_max, ns_max, nwords, ncand_vs;
  const int *bs_sorted, *bs_count;
  int k_max, nb, ncand_bs;
};

constexpr int kMaxTiles = kMaxN / 64;  // key tiles of the longest supported sequence
constexpr int kMaxGather = 2048;       // vertical columns gathered per query tile

// XOR swizzle of the 16-byte chunk index of LDS row r.  With d = 128 a 256-byte row spans all
// 64 LDS banks; rows 0-15 then give K fragment reads (16 rows, one chunk column per 16
// lanes) and transposed V reads (4 rows x 4 adjacent chunks per 32 lanes) distinct banks.
// With d = 64 (128-byte rows) a 3-bit swizzle over 8 rows does the same.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return ((r & 3) << 1) | ((r >> 2) & 1);
}

typedef short v4i16 __attribute__((ext_vector_type(4)));

// Barrier after which every wave's direct-to-LDS copies (global_load_lds, counted by
// vmcnt) and LDS accesses are complete.  The explicit vmcnt wait is required: the
// compiler's LDS release fence does not always wait for the LDS DMA.
__device__ __forceinline__ void lds_fence_barrier() {
  // vmcnt(0) through the builtin, which the compiler's wait insertion knows about (it then
  // treats every earlier load as complete, instead of waiting for them again later)
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Per-tile description produced ahead of its use (the next tile is issued while the
// current one is computed).
struct TileRef {
  int key0;  // first key of a contiguous tile, or -(1 + gather offset)
  int tag;   // bit 0: rows of waves 0-1 use it, bit 1: rows of waves 2-3 (block-sparse)
  Win3 wd;   // vertical-slash: diagonal-bitmap words of this lane's row (prefetched)
  Win3 wv;   // vertical-slash: column-bitmap words of the tile (prefetched)
  int hm;    // 32-key halves of the tile that are copied and may be kept (bit 0: keys 0-31)
};

// bit 2m of the result: either of bits 2m, 2m + 1 of w (64-key tile m of a word of 32-key halves)
__device__ __forceinline__ uint32_t tile_bits(uint32_t w) { return (w | (w >> 1)) & 0x55555555u; }

// One work item: query tile `item & 0xffff` of unit `item >> 16` of the launch's unit list.
// VT: V is read from the transposed copy (tiles of D rows x 64 keys), else from V itself.
template <int D, int PAT, typename InT, bool VT>
__device__ __forceinline__ void attn_item(const AttnArgs &a, const int item) {
  constexpr int NW = 4, NT = 256, BM = 128;
  constexpr int KS = D / 16;             // k-steps of the QK^T contraction
  constexpr int DB = D / 32;             // 32-row blocks of O^T
  constexpr int CPR = D / 8;             // 16-byte chunks per K/V row
  constexpr int RPI = 64 / CPR;          // rows covered by one wave-wide 16-byte load
  constexpr int LPT = 64 / RPI / NW;     // loads per thread per K (or V) tile
  constexpr int TE = 64 * D;             // elements of one K or V tile
  static_assert(LPT % 2 == 0 && LPT <= 4 && LPT * NW * RPI == 64, "K/V copies: two halves of LPT / 2 loads");
  // fragment reads in flight ahead of the products (K for QK^T, V for P V); vertical-slash
  // keeps two (its tile bookkeeping leaves fewer registers; more spill)
  constexpr int KPF = PAT == P_VS ? 2 : 4;
  constexpr int VPF = PAT == P_VS ? 2 : 3;
  // the products of the tile-skipping families sit under a branch, where the compiler puts
  // each K read right before its product unless the order is forced (scheduling groups)
  constexpr bool kForceOrder = PAT == P_VS || PAT == P_BS;

  // K and V tiles are double-buffered separately (K runs one tile ahead of V), row-major and
  // swizzled.  Four distinct arrays, addressed with a parity known at compile time, let the
  // compiler see that a copy in flight never overlaps the tiles being read.
  __shared__ __align__(16) bf16 sK0[TE];
  __shared__ __align__(16) bf16 sK1[TE];
  __shared__ __align__(16) bf16 sV0[TE];
  __shared__ __align__(16) bf16 sV1[TE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;

  const DevUnit U = a.units[item >> 16];
  const int qt = item & 0xffff;
  const int head = U.head, s0 = U.s0, s1 = U.s1;
  const int kvh = head / a.group;
  // A block-sparse unit with a mate runs 64-row items: waves 0-1 take its rows of query block
  // qt, waves 2-3 the same rows of the mate head (same key/value head, so the key blocks the
  // two selections share are copied once); otherwise an item is a 128-row query tile.
  const bool paired = PAT == P_BS && U.mate > 0;
  const int IM = paired ? 64 : BM;  // rows of an item
  const int base = (s0 / IM + qt) * IM;
  const int r_lo = max(s0, base), r_hi = min(s1, base + IM);  // valid rows [r_lo, r_hi)
  const int wbase = base + 32 * (paired ? (wave & 1) : wave);
  const int whead = paired && wave >= 2 ? U.mate - 1 : head;  // this wave's query head
  const int w_lo = max(r_lo, wbase), w_hi = min(r_hi, wbase + 32) - 1;
  const bool wave_active = w_lo <= w_hi;
  const int my_row = wbase + l32;
  const int last_tile = (r_hi - 1) >> 6;

  const InT *Qp = (const InT *)a.q + (long long)whead * a.sq_h;
  const InT *Kp = (const InT *)a.k + (long long)kvh * a.sk_h;
  const InT *Vp = (const InT *)a.v + (long long)kvh * a.sv_h;

  // ---- tile enumeration state ----------------------------------------------------------
  int ntiles = 0;
  int st0 = 0, st1 = 0;  // pattern cursors
  // block-sparse: key blocks selected by query block bq (sBA) and bq + 1 (sBB) as bitmaps;
  // words for key blocks 0 .. bq + 1, where bq + 1 reaches kMaxTiles for the last 64-row item
  // of a sequence of the maximum length
  __shared__ uint32_t sBA[PAT == P_BS ? kMaxTiles / 32 + 1 : 1], sBB[PAT == P_BS ? kMaxTiles / 32 + 1 : 1];
  const uint32_t *vbits = nullptr, *dbits = nullptr;
  int n_contig = 0, n_gather = 0;
  // vertical-slash: sTB, one bit per 32-key half of the key range the block's diagonals touch
  // (a 64-key tile is in the list when either of its halves is, and only those halves are
  // copied); sG, the gathered vertical columns.  Arrays of their own, not pointers, so that
  // the compiler sees them apart from the tiles being copied.
  __shared__ uint32_t sTB[PAT == P_VS ? kMaxTiles / 16 : 1];
  __shared__ int sG[PAT == P_VS ? kMaxGather : 1];

  if constexpr (PAT == P_VS) {
    __shared__ int sScan[NW + 1];
    const long long vsrow = (long long)U.slot * a.ncand_vs + U.cl;
    const int *vsorted = a.vs_vsorted + vsrow * a.nv_max;
    const int *dsorted = a.vs_dsorted + vsrow * a.ns_max;
    // counts are read within [0, nv_max] / [0, ns_max]: a malformed set never reads past its row
    const int nvc = min(max(a.vs_count[vsrow * 2 + 0], 0), a.nv_max);
    const int ndc = min(max(a.vs_count[vsrow * 2 + 1], 0), a.ns_max);
    vbits = a.vs_vbits + vsrow * a.nwords;
    dbits = a.vs_dbits + vsrow * a.nwords;
    const int nwt = ((2 * last_tile + 1) >> 5) + 1;
    for (int w = tid; w < nwt; w += NT) sTB[w] = 0u;
    __syncthreads();
    // diagonal t covers keys [r_lo - t, r_hi - 1 - t] of this tile's rows
    for (int x = tid; x < ndc; x += NT) {
      const int t = dsorted[x];
      if (t < 0 || t > r_hi - 1) continue;
      const int lo = max(0, r_lo - t) >> 5, hi = (r_hi - 1 - t) >> 5;
      for (int kh = lo; kh <= hi; ++kh) atomicOr(&sTB[kh >> 5], 1u << (kh & 31));
    }
    __syncthreads();
    {
      int cnt = 0;
      for (int w = 0; w < nwt; ++w) cnt += __builtin_popcount(tile_bits(sTB[w]));
      n_contig = cnt;
    }
    // vertical columns outside the diagonal tiles are gathered, ascending
    int total = 0;
    for (int x0 = 0; x0 < nvc; x0 += NT) {
      const int x = x0 + tid;
      const int j = (x < nvc) ? vsorted[x] : 0x7fffffff;
      bool f = false;
      if (x < nvc && j >= 0 && j <= r_hi - 1) {
        const int kh = j >> 5;
        f = !((sTB[kh >> 5] >> (kh & 31)) & 1u);
      }
      const uint64_t bal = __ballot(f);
      const int before = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) sScan[wave] = __popcll(bal);
      __syncthreads();
      int woff = total, blk = 0;
      for (int w = 0; w < NW; ++w) {
        if (w < wave) woff += sScan[w];
        blk += sScan[w];
      }
      if (f && woff + before < kMaxGather) sG[woff + before] = j;
      total += blk;
      __syncthreads();
      if (x0 + NT <= nvc && vsorted[x0 + NT - 1] > r_hi - 1) break;  // sorted: rest is beyond
    }
    n_gather = min(total, kMaxGather);
    __syncthreads();
    ntiles = n_contig + (n_gather + 63) / 64;
    // contiguous tiles are taken from the diagonal down (descending keys)
    st0 = nwt - 1;                                                            // bitmap word of the next contiguous tile
    st1 = __builtin_amdgcn_readfirstlane((int)tile_bits(sTB[st0]));           // remaining tiles (even bits)
  } else if constexpr (PAT == P_DENSE) {
    ntiles = last_tile + 1;
  } else if constexpr (PAT == P_ASHAPE) {
    const int ns = min((U.sink + 63) >> 6, last_tile + 1);
    const int wlo = max(0, r_lo - U.window + 1) >> 6;
    st0 = ns;
    st1 = max(wlo, ns);
    ntiles = ns + max(0, last_tile - st1 + 1);
  } else {  // P_BS: query blocks bq = base/64 (waves 0-1) and bq + 1 (waves 2-3), or block bq
    // of this head (waves 0-1) and of the mate head (waves 2-3)
    // the two sorted selections are loaded in parallel into key-block bitmaps; the tiles are
    // their union, walked from the highest key block down (a tile's tag says which selection
    // holds it)
    const int bq = base >> 6;
    const long long brow = ((long long)head * a.ncand_bs + U.cl) * a.nb + bq;
    const long long brow2 = paired ? ((long long)(U.mate - 1) * a.ncand_bs + U.mate_cl) * a.nb + bq : brow + 1;
    // counts within [0, k_max]; entries outside key blocks [0, bq + 1] (pads, malformed sets)
    // are skipped, so the bitmaps are never written out of range
    const int na = r_lo < base + 64 ? min(max(a.bs_count[brow], 0), a.k_max) : 0;
    const int nb2 = (paired || (r_hi > base + 64 && bq + 1 < a.nb)) ? min(max(a.bs_count[brow2], 0), a.k_max) : 0;
    const int nwb = ((bq + 1) >> 5) + 1;  // words holding key blocks 0 .. bq + 1
    for (int w = tid; w < nwb; w += NT) {
      sBA[w] = 0u;
      sBB[w] = 0u;
    }
    __syncthreads();
    for (int x = tid; x < na + nb2; x += NT) {
      const int v = x < na ? a.bs_sorted[brow * a.k_max + x] : a.bs_sorted[brow2 * a.k_max + x - na];
      if (v < 0 || v > bq + 1) continue;
      atomicOr(x < na ? &sBA[v >> 5] : &sBB[v >> 5], 1u << (v & 31));
    }
    __syncthreads();
    int cnt = 0;  // every wave sums the same words (no further barrier)
    for (int w = lane; w < nwb; w += 64) cnt += __builtin_popcount(sBA[w] | sBB[w]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o);
    ntiles = cnt;
    // the union is walked from the diagonal block down (descending key blocks)
    st0 = nwb - 1;                                                      // bitmap word of the next tile
    st1 = __builtin_amdgcn_readfirstlane((int)(sBA[st0] | sBB[st0]));  // remaining blocks of that word
  }

  // next tile in order (t increases by one per call)
  int t_next = 0;
  auto next_tile = [&]() -> TileRef {
    const int t = t_next++;
    if constexpr (PAT == P_DENSE) {
      return TileRef{t * 64, 3, {0u, 0u, 0u}, {0u, 0u, 0u}, 3};
    } else if constexpr (PAT == P_ASHAPE) {
      return TileRef{(t < st0 ? t : st1 + (t - st0)) * 64, 3, {0u, 0u, 0u}, {0u, 0u, 0u}, 3};
    } else if constexpr (PAT == P_BS) {
      // the words are the same for every lane: kept in scalar registers
      while (st1 == 0) {
        --st0;
        st1 = __builtin_amdgcn_readfirstlane((int)(sBA[st0] | sBB[st0]));
      }
      const int bit = 31 - __builtin_clz((uint32_t)st1);
      st1 &= ~(1u << bit);
      const int wa = __builtin_amdgcn_readfirstlane((int)sBA[st0]), wb = __builtin_amdgcn_readfirstlane((int)sBB[st0]);
      const int tag = ((wa >> bit) & 1) | (((wb >> bit) & 1) << 1);
      return TileRef{(st0 * 32 + bit) * 64, tag, {0u, 0u, 0u}, {0u, 0u, 0u}, 3};
    } else {
      if (t < n_contig) {
        // the bitmap words are the same for every lane: kept in scalar registers
        while (st1 == 0) st1 = __builtin_amdgcn_readfirstlane((int)tile_bits(sTB[--st0]));
        const int bit = 31 - __builtin_clz((uint32_t)st1);
        st1 &= ~(1u << bit);
        const int key0 = (st0 * 16 + (bit >> 1)) * 64;
        const int hm = (__builtin_amdgcn_readfirstlane((int)sTB[st0]) >> bit) & 3;
        TileRef tr{key0, 3, {0u, 0u, 0u}, {0u, 0u, 0u}, hm};
        // bitmap words of the element mask, fetched with the tile so that their latency
        // hides behind the previous tile's compute
        tr.wd = load_win(dbits, a.nwords, my_row - key0 - 63);
        tr.wv = load_win(vbits, a.nwords, key0);
        return tr;
      }
      return TileRef{-(1 + (t - n_contig) * 64), 3, {0u, 0u, 0u}, {0u, 0u, 0u}, 3};
    }
  };

  // ---- Q fragment in registers (B operand of QK^T) ---------------------------------------
  u32x4 qf[KS];
  {
    const bool ok = wave_active && my_row < a.n;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qf[ks] = u32x4{0u, 0u, 0u, 0u};
      if (ok) qf[ks] = load8<InT>(Qp + (long long)my_row * a.sq_t + 16 * ks + 8 * hh);
    }
  }

  // ---- tile loads: global -> LDS (direct for bf16, through registers for fp32) ----------
  auto key_of_row = [&](int key0, int row) -> int {
    if constexpr (PAT == P_VS) {
      if (key0 < 0) {
        const int g = -key0 - 1 + row;
        return sG[g < n_gather ? g : -key0 - 1];
      }
    }
    return min(key0 + row, a.n - 1);
  };
  // bf16 tiles are copied with buffer loads whose per-lane byte offset is the same for every
  // tile (row within the tile and swizzled chunk); the tile's first key enters as a scalar
  // offset.  One head's K (V) rows span less than 4 GiB (checked by the host).
  const int lrow0 = wave * RPI + lane / CPR;          // tile row of load 0; load i adds i*NW*RPI
  const int lchunk = (lane % CPR) ^ swz<D>(lrow0);    // swz sees only row & 15: same for all i
  const uint32_t bK = (uint32_t)(a.sk_t * sizeof(InT)), bV = (uint32_t)(a.sv_t * sizeof(InT));
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t rK = __builtin_amdgcn_make_buffer_rsrc(
      (void *)Kp, (short)0, (int)((uint32_t)(a.n - 1) * bK + D * sizeof(InT)), 0x00020000);
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t rV = __builtin_amdgcn_make_buffer_rsrc(
      (void *)Vp, (short)0, (int)((uint32_t)(a.n - 1) * bV + D * sizeof(InT)), 0x00020000);
  [[maybe_unused]] const uint32_t voK = (uint32_t)lrow0 * bK + 16u * (uint32_t)lchunk;
  [[maybe_unused]] const uint32_t voV = (uint32_t)lrow0 * bV + 16u * (uint32_t)lchunk;
  // V^T tile: D rows (dims) of 64 keys (128 bytes); a wave instruction copies 8 rows, lane l
  // landing at row l / 8, chunk l % 8, which holds global chunk (l % 8) ^ ((row / 2) % 8) (the
  // read-side swizzle).  Rows of load i are 8 (i NW + wave) + l / 8, so the swizzle is the same
  // for every i.
  const uint32_t bVT = (uint32_t)a.npad * 2u;
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t rVT = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.vt + (long long)kvh * D * a.npad), (short)0, (int)((uint32_t)D * bVT), 0x00020000);
  [[maybe_unused]] const uint32_t voVT =
      (uint32_t)(8 * wave + lane / 8) * bVT + 16u * (uint32_t)((lane % 8) ^ ((4 * (wave & 1) + (lane >> 4)) & 7));
  // one K or V tile (64 key rows) into dst
  auto issue = [&](bf16 *dst, int key0, bool isV, int hm) {
    if constexpr (VT) {
      if (isV) {
        constexpr int LPV = D / 8 / NW;  // 8-row groups per wave
        static_assert(LPV == LPT && NW % 2 == 0, "V^T tile: same load count as a row tile");
        bf16 *dw = dst + wave * 8 * 64;
#pragma unroll
        for (int i = 0; i < LPV; ++i)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rVT, (__attribute__((address_space(3))) void *)(dw + i * NW * 8 * 64),
                                                   16, voVT, (uint32_t)key0 * 2u + (uint32_t)(i * NW * 8) * bVT, 0, 0);
        return;
      }
    }
    const InT *src = isV ? Vp : Kp;
    const long long st = isV ? a.sv_t : a.sk_t;
    if constexpr (sizeof(InT) == 2) {
      const __amdgpu_buffer_rsrc_t rs = isV ? rV : rK;
      const uint32_t b = isV ? bV : bK, vo = isV ? voV : voK;
      bf16 *dw = dst + wave * RPI * D;
      // load i copies tile rows [i NW RPI, (i + 1) NW RPI), inside 32-row half (i NW RPI) / 32
      // loads [h LPT / 2, (h + 1) LPT / 2) fill 32-key half h (one test of hm per half)
      if (key0 >= 0 && key0 + 64 <= a.n) {  // contiguous rows: offsets are scalar
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (!((hm >> h) & 1)) continue;
#pragma unroll
          for (int i = h * LPT / 2; i < (h + 1) * LPT / 2; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)(dw + i * NW * RPI * D),
                                                     16, vo, (uint32_t)(key0 + i * NW * RPI) * b, 0, 0);
        }
      } else {  // gathered rows, or the last tile (rows clamped to the sequence)
        uint32_t jr[4];  // (LPT <= 4) every row index first: one LDS round trip for a gathered tile
#pragma unroll
        for (int i = 0; i < LPT; ++i) jr[i] = (uint32_t)key_of_row(key0, lrow0 + i * NW * RPI);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (!((hm >> h) & 1)) continue;
#pragma unroll
          for (int i = h * LPT / 2; i < (h + 1) * LPT / 2; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)(dw + i * NW * RPI * D),
                                                     16, jr[i] * b + 16u * (uint32_t)lchunk, 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < LPT; ++i) {
        if (!((hm >> ((i * NW * RPI) >> 5)) & 1)) continue;
        const int row_base = (i * NW + wave) * RPI;
        const int row = row_base + lane / CPR;
        const int cc = (lane % CPR) ^ swz<D>(row);
        const int j = key_of_row(key0, row);
        *(u32x4 *)(dst + row_base * D + 8 * lane) = load8<InT>(src + (long long)j * st + 8 * cc);
      }
    }
  };

  // ---- per-lane LDS fragment offsets -----------------------------------------------------
  const int kswz = swz<D>(l32);                 // K rows 32 mb + l32
  const int g16 = lane >> 4, i16 = lane & 15;
  const int esrc = i16 >> 2, qv = i16 & 3;   // transposed V read: source row / dd quad
  const int vrow = 4 * hh + esrc;            // + 32 mb + 16 s + 8 half
  // swz<D>(vrow + 8 half + 16 s + 32 mb) depends on the half only
  const int vsw0 = swz<D>(vrow), vsw1 = swz<D>(vrow + 8);
  int voff[DB], voff1[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int dd0 = 32 * db + 16 * (g16 & 1) + 4 * qv;
    voff[db] = vrow * D + (((dd0 >> 3) ^ vsw0) << 3) + (dd0 & 7);
    voff1[db] = (vrow + 8) * D + (((dd0 >> 3) ^ vsw1) << 3) + (dd0 & 7);
  }

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.c;
  const int my_rows_tag = wave < 2 ? 1 : 2;
  const bf16x2 ones = {(bf16)1.f, (bf16)1.f};

  // Dense and A-shape compute every tile of the list for every wave (a tile outside a
  // wave's rows is fully masked), so that the softmax of one tile and the products of the
  // next form one branch-free block the scheduler interleaves.
  constexpr bool kOverlap = PAT == P_DENSE || PAT == P_ASHAPE;

  // ---- per-tile plan of this wave: participation, mask need, active 32-key halves ---------
  struct Plan {
    bool on, need_mask, do0, do1;
    uint64_t Mvs;  // vertical-slash contiguous tile: this lane's kept keys (after half shift)
    int g0, g_cnt; // vertical-slash gathered tile: first column slot, column count
  };
  auto plan_of = [&](const TileRef &tr, bool valid) -> Plan {
    Plan p{false, true, true, true, 0ull, 0, 0};
    if (!valid) return p;
    const int key0 = tr.key0;
    if constexpr (kOverlap) {
      p.on = true;
      if constexpr (PAT == P_ASHAPE)
        p.need_mask = !(key0 + 63 <= w_lo && (key0 + 63 < U.sink || key0 > w_hi - U.window));
      else
        p.need_mask = key0 + 63 > w_lo;
      return p;
    }
    if (!wave_active || !(tr.tag & my_rows_tag)) return p;
    if constexpr (PAT == P_VS) {
      if (key0 < 0) {
        p.g0 = -key0 - 1;
        p.g_cnt = min(64, n_gather - p.g0);
        p.on = sG[p.g0] <= w_hi;
        p.do1 = p.g_cnt > 32;
      } else if (key0 <= w_hi) {
        // the lane's kept keys are known before any product: a 32-key half no row of the
        // wave keeps skips both of its products
        const int i = my_row;
        const uint64_t md = __builtin_bitreverse64(win_bits(tr.wd, i - key0 - 63));
        const uint64_t mv = win_bits(tr.wv, key0);
        const uint64_t halves = (tr.hm & 1 ? 0xffffffffull : 0ull) | (tr.hm & 2 ? 0xffffffff00000000ull : 0ull);
        p.Mvs = ((md | mv) & prefix_mask(i - key0 + 1) & halves) >> (4 * hh);
        p.do0 = __ballot(((uint32_t)p.Mvs & 0x0f0f0f0fu) != 0u) != 0ull;
        p.do1 = __ballot(((uint32_t)(p.Mvs >> 32) & 0x0f0f0f0fu) != 0u) != 0ull;
        p.on = p.do0 || p.do1;
      }
    } else {  // block-sparse
      p.on = key0 <= w_hi;
      p.need_mask = key0 + 63 > w_lo;
    }
    return p;
  };

  // ---- S^T[64 keys x 32 rows] = K_tile x Q^T ---------------------------------------------
  auto qk = [&](f32x16 (&s)[2], const bf16 *sKt, const Plan &p) {
    if constexpr (PAT != P_VS) {
      // fragment f: 32-key block mb = f % 2, k-step ks = f / 2 (the two accumulators
      // alternate); reads run KPF fragments ahead of their products
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[mb][r] = 0.f;
      auto kread = [&](int f) -> u32x4 {
        return *(const u32x4 *)&sKt[(32 * (f & 1) + l32) * D + (((2 * (f >> 1) + hh) ^ kswz) << 3)];
      };
      u32x4 kb[KPF];
#pragma unroll
      for (int f = 0; f < KPF; ++f) kb[f] = kread(f);
#pragma unroll
      for (int f = 0; f < 2 * KS; ++f) {
        s[f & 1] = mfma32(kb[f % KPF], qf[f >> 1], s[f & 1]);
        if (f + KPF < 2 * KS) kb[f % KPF] = kread(f + KPF);
      }
      if constexpr (kForceOrder) {
        __builtin_amdgcn_sched_group_barrier(0x100, KPF, 0);
#pragma unroll
        for (int f = 0; f < 2 * KS - KPF; ++f) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, KPF, 0);
      }
      return;
    }
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const bool dm = mb ? p.do1 : p.do0;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[mb][r] = 0.f;
      if (!dm) continue;
      auto kread = [&](int ks) -> u32x4 {
        return *(const u32x4 *)&sKt[(32 * mb + l32) * D + (((2 * ks + hh) ^ kswz) << 3)];
      };
      u32x4 kb[KPF];
#pragma unroll
      for (int ks = 0; ks < KPF; ++ks) kb[ks] = kread(ks);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s[mb] = mfma32(kb[ks % KPF], qf[ks], s[mb]);
        if (ks + KPF < KS) kb[ks % KPF] = kread(ks + KPF);
      }
      if constexpr (kForceOrder) {
        __builtin_amdgcn_sched_group_barrier(0x100, KPF, 0);
#pragma unroll
        for (int ks = 0; ks < KS - KPF; ++ks) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, KPF, 0);
      }
    }
  };

  // ---- masks: this lane's keys are bits 0-3 of every byte of M (after the half shift); a
  // kept key keeps its logit, a dropped one (or a skipped half) becomes -inf ---------------
  auto apply_mask = [&](f32x16 (&s)[2], const TileRef &tr, const Plan &p) -> bool {
    const int key0 = tr.key0, i = my_row;
    uint64_t M;
    if constexpr (PAT == P_VS) {
      if (key0 < 0) {
        int lo = 0, hi = p.g_cnt;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (sG[p.g0 + mid] <= i) lo = mid + 1;
          else hi = mid;
        }
        M = prefix_mask(lo) >> (4 * hh);
      } else {
        M = p.Mvs;
      }
      if (!p.do0) M &= ~0xffffffffull;
      if (!p.do1) M &= 0xffffffffull;
    } else if constexpr (PAT == P_ASHAPE) {
      const uint64_t keep = prefix_mask(U.sink - key0) | ~prefix_mask(i - U.window + 1 - key0);
      M = (keep & prefix_mask(i - key0 + 1)) >> (4 * hh);
    } else {
      M = prefix_mask(i - key0 + 1) >> (4 * hh);
    }
    const uint32_t Mw[2] = {(uint32_t)M, (uint32_t)(M >> 32)};
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t keep = (uint32_t)__builtin_amdgcn_sbfe((int)Mw[mb], 8 * (r >> 2) + (r & 3), 1);
        // the element goes through a scalar: bit_cast of a vector element in place reads
        // element 0 with this compiler
        const float x = s[mb][r];
        s[mb][r] = __builtin_bit_cast(float, (keep & __builtin_bit_cast(uint32_t, x)) | (~keep & 0xff800000u));
      }
    return (M & 0x0F0F0F0F0F0F0F0Full) != 0ull;
  };

  // ---- online softmax in the exp2 domain with a lazily raised running max ------------------
  // P is formed against the current m_run; only if some lane's probability sum exceeds 2^8
  // (so every probability stays <= 2^8 otherwise), or a row sees its first kept key, is the
  // exact tile max taken, m_run raised, O rescaled and P formed again.  Row sums are taken
  // over the bf16-rounded probabilities that also multiply V.
  u32x4 pb[2][2];
  auto form_p = [&](const f32x16 (&s)[2], float nmc) -> float {
    float ps = 0.f;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[mb][8 * h + 2 * w], c, nmc));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(s[mb][8 * h + 2 * w + 1], c, nmc));
          const bf16x2 pk = cvt_bf16x2(p0, p1);
          pb[mb][h][w] = __builtin_bit_cast(uint32_t, pk);
          ps = __builtin_amdgcn_fdot2_f32_bf16(pk, ones, ps, false);
        }
    return ps;
  };

  // ---- O^T[d x 32 rows] += V^T x P^T (V read transposed from its row-major tile, or, with
  // VT, 8 consecutive keys of a V^T row per lane: the tile's keys are stored in the order in
  // which the S^T accumulator hands them to P) ----------------------------------------------
  [[maybe_unused]] const int vts = (l32 >> 1) & 7;
  auto pv = [&](const bf16 *sVt, const Plan &p) {
    if constexpr (VT) {
      // fragment f: 16-key group g = f / DB (g = 2 mb + h), 32-dim block db = f % DB, so that
      // consecutive products accumulate into different blocks; reads run PF fragments ahead
      constexpr int NF = 4 * DB, PF = 4;
      auto vread = [&](int f) -> u32x4 {
        const int g = f / DB, db = f % DB;
        return *(const u32x4 *)(sVt + (32 * db + l32) * 64 + (((2 * g + hh) ^ vts) << 3));
      };
      u32x4 vb[PF];
#pragma unroll
      for (int f = 0; f < PF; ++f) vb[f] = vread(f);
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const int g = f / DB, db = f % DB;
        oacc[db] = mfma32(vb[f % PF], pb[g >> 1][g & 1], oacc[db]);
        if (f + PF < NF) vb[f % PF] = vread(f + PF);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, PF, 0);
#pragma unroll
      for (int f = 0; f < NF - PF; ++f) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, PF, 0);
      return;
    }
    // per 32-key half mb (skipped by vertical-slash when no row of the wave keeps a key of
    // it): fragment f = (h, db) = (f / DB, f % DB), consecutive products into different
    // blocks, reads VPF fragments ahead
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      if constexpr (PAT == P_VS)
        if (!(mb ? p.do1 : p.do0)) continue;
      auto vread = [&](int f) -> u32x4 {
        const int h = f / DB, db = f % DB;
        const bf16 *vp = sVt + voff[db] + (32 * mb + 16 * h) * D;
        const bf16 *vq = sVt + voff1[db] + (32 * mb + 16 * h) * D;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(vp));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(vq));
        const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
        return u32x4{l2[0], l2[1], h2[0], h2[1]};
      };
      u32x4 vb[VPF];
#pragma unroll
      for (int f = 0; f < VPF; ++f) vb[f] = vread(f);
#pragma unroll
      for (int f = 0; f < 2 * DB; ++f) {
        oacc[f % DB] = mfma32(vb[f % VPF], pb[mb][f / DB], oacc[f % DB]);
        if (f + VPF < 2 * DB) vb[f % VPF] = vread(f + VPF);
      }
      if constexpr (kForceOrder) {  // two transposing reads per fragment
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * VPF, 0);
#pragma unroll
        for (int f = 0; f < 2 * DB - VPF; ++f) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, VPF, 0);
      }
    }
  };

  // ---- one pipeline step: tile t's softmax and P V, tile t+1's products -------------------
  // On entry sc holds S^T of tile t; K of tile t+1 (in kn) and V of tile t (in vc) are resident
  // after the barrier.  The step copies K of tile t+2 into kc (released by tile t's products)
  // and V of tile t+1 into vn (released by tile t-1's P V).
  TileRef Tc{0, 0, {0u, 0u, 0u}, {0u, 0u, 0u}, 3}, Tn = Tc;
  Plan Pc = plan_of(Tc, false), Pn = Pc;
  auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2], bf16 *kc, bf16 *kn, bf16 *vc, bf16 *vn) {
    // the next tile is taken after the barrier: the barrier waits for every load in flight,
    // and the vertical-slash mask words that next_tile fetches are only needed a step later
    lds_fence_barrier();
    TileRef T2{0, 0, {0u, 0u, 0u}, {0u, 0u, 0u}, 3};
    if (t + 2 < ntiles) T2 = next_tile();
    if (t + 2 < ntiles) issue(kc, T2.key0, false, T2.hm);
    if (t + 1 < ntiles) issue(vn, Tn.key0, true, Tn.hm);
    Pn = plan_of(Tn, t + 1 < ntiles);
    bool has_key = true;
    if (kOverlap || Pc.on)
      if (PAT == P_VS || Pc.need_mask) has_key = apply_mask(sc, Tc, Pc);
    // tile t+1's products, then tile t's softmax: the two waves of a SIMD tend to alternate
    // between product bursts and softmax bursts, so that one's products overlap the other's
    // vector work (interleaving them within a wave was measured slower)
    // (vertical-slash, dense and block-sparse take tile t+1's products after tile t's P V
    // instead: the two S tiles are then never live together, which leaves registers for
    // fragment read-ahead; 1-2% faster for dense and for block-sparse with mates, not for
    // A-shape, whose short items keep the early products)
    constexpr bool kLateQK = PAT == P_VS || PAT == P_DENSE || PAT == P_BS;
    if constexpr (!kLateQK)
      if (kOverlap || Pn.on) qk(sn, kn, Pn);
    if (kOverlap || Pc.on) {
      float psum = form_p(sc, (m_run == -INFINITY) ? 0.f : -m_run * c);
      const uint64_t want = __ballot(!(psum <= 256.f) || (m_run == -INFINITY && has_key));
      if (want != 0ull) {
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[mb][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        // both lanes of a row take the same decision
        if (((want >> l32) | (want >> (l32 + 32))) & 1ull) {
          const float m_new = fmaxf(m_run, mx);
          if (m_new > m_run) {
            const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);  // 0 for m_run = -inf
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
              for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
            m_run = m_new;
          }
        }
        psum = form_p(sc, (m_run == -INFINITY) ? 0.f : -m_run * c);
      }
      l_run += psum;
      pv(vc, Pc);
    }
    if constexpr (kLateQK)
      if (Pn.on) qk(sn, kn, Pn);
    Tc = Tn;
    Tn = T2;
    Pc = Pn;
  };

  // ---- main loop ---------------------------------------------------------------------------
  f32x16 sA[2], sB[2];
  if (ntiles > 0) {
    Tc = next_tile();
    issue(sK0, Tc.key0, false, Tc.hm);
    issue(sV0, Tc.key0, true, Tc.hm);
    if (ntiles > 1) {
      Tn = next_tile();
      issue(sK1, Tn.key0, false, Tn.hm);
    }
    lds_fence_barrier();
    Pc = plan_of(Tc, true);
    if (kOverlap || Pc.on) qk(sA, sK0, Pc);
  }
  for (int t = 0; t < ntiles; t += 2) {
    step(t, sA, sB, sK0, sK1, sV0, sV1);
    if (t + 1 >= ntiles) break;
    step(t + 1, sB, sA, sK1, sK0, sV1, sV0);
  }

  // ---- epilogue --------------------------------------------------------------------------
  if (!wave_active) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const int i = my_row;
  if (i < r_lo || i >= r_hi) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  bf16 *op = a.o + (long long)whead * a.so_h + (long long)i * a.so_t;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      u32x2 w;
      w[0] = pack_bf16x2(oacc[db][4 * ii + 0] * inv, oacc[db][4 * ii + 1] * inv);
      w[1] = pack_bf16x2(oacc[db][4 * ii + 2] * inv, oacc[db][4 * ii + 3] * inv);
      *(u32x2 *)(op + 32 * db + 8 * ii + 4 * hh) = w;
    }
  if (a.lse && hh == 0)
    a.lse[(long long)whead * a.n + i] = l_tot > 0.f ? m_run * a.scale + logf(l_tot) : -INFINITY;
}

// attn_fwd_kernel: workgroup b runs item order[b].  attn_fwd_queue_kernel: the grid is
// persistent; workgroup b (on XCD b % 8 under round-robin dispatch) takes the next item of the
// queue of key/value bucket b % 8 (items there are longest first), then of the other buckets
// once its own is empty, until every queue is drained.  Each queue counter starts at 0 (the
// planner writes it) and is only ever incremented, so every workgroup reaches the exit.
template <int D, int PAT, typename InT, bool VT>
__global__ void __launch_bounds__(256, 2) attn_fwd_kernel(const AttnArgs a) {
  attn_item<D, PAT, InT, VT>(a, a.order[blockIdx.x]);
}

template <int D, int PAT, typename InT, bool VT>
__global__ void __launch_bounds__(256, 2) attn_fwd_queue_kernel(const AttnArgs a) {
  __shared__ int sItem;
  const int x = (int)(blockIdx.x & 7u);
  for (;;) {
    __syncthreads();  // the previous item is done with the tile buffers and sItem
    if (threadIdx.x == 0) {
      int got = -1;
      for (int k = 0; k < 8 && got < 0; ++k) {
        const int b = (x + k) & 7;
        if (__hip_atomic_load(&a.qcount[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= a.qsize[b]) continue;
        const int r = atomicAdd(&a.qcount[b], 1);
        if (r < a.qsize[b]) got = a.order[a.qoff[b] + r];
      }
      sItem = got;
    }
    __syncthreads();
    const int it = sItem;
    if (it < 0) break;
    attn_item<D, PAT, InT, VT>(a, it);
  }
}

// ---- V^T: [hkv][d][npad] bf16, keys permuted within groups of 16 ---------------------------
// Position j of a 16-key group holds key perm[j]: in the P V product a lane of half hh supplies
// the keys {4 hh .. 4 hh + 3, 8 + 4 hh .. 8 + 4 hh + 3} of each group of 16 (the order in which
// the S^T accumulator hands them to P), which are then 8 consecutive positions.
__device__ __forceinline__ int vt_perm(int j) { return (j & 3) | ((j & 4) << 1) | ((j & 8) >> 1); }

// grid (npad / 64, hkv), 256 threads: 64 keys of one key/value head through LDS
template <int D, typename InT>
__global__ void __launch_bounds__(256) transpose_v_kernel(const InT *v, long long sv_h, long long sv_t, int n,
                                                          int npad, bf16 *vt) {
  constexpr int LD = D + 8;
  __shared__ __align__(16) bf16 sT[64][LD];
  const int k0 = blockIdx.x * 64, g = blockIdx.y, tid = threadIdx.x;
  const InT *vp = v + (long long)g * sv_h;
  // 64 rows x D, 8 elements per 16-byte chunk of the bf16 tile
  for (int x = tid; x < 64 * (D / 8); x += 256) {
    const int r = x / (D / 8), c = x % (D / 8), key = k0 + r;
    u32x4 w = {0u, 0u, 0u, 0u};
    if (key < n) w = load8<InT>(vp + (long long)key * sv_t + 8 * c);
    *(u32x4 *)&sT[r][8 * c] = w;
  }
  __syncthreads();
  bf16 *out = vt + (long long)g * D * npad + k0;
  for (int x = tid; x < D * 8; x += 256) {
    const int dd = x / 8, c = x % 8;  // row dd of V^T, positions 8c .. 8c + 7 of the 64 keys
    bf16 e[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int p = 8 * c + j;
      e[j] = sT[(p & ~15) + vt_perm(p & 15)][dd];
    }
    *(u32x4 *)(out + (long long)dd * npad + 8 * c) = __builtin_bit_cast(u32x4, e);
  }
}

size_t vt_bytes(const rs_qkv *qkv) {
  const long long npad = ((long long)qkv->n + 63) / 64 * 64;
  return (size_t)qkv->hkv * qkv->d * npad * sizeof(bf16);
}

rs_status transpose_v_launch(const rs_qkv *qkv, void *vt, hipStream_t st) {
  const int npad = (qkv->n + 63) / 64 * 64;
  const dim3 grid(npad / 64, qkv->hkv);
  if (qkv->d == 128) {
    if (qkv->dtype == RS_BF16)
      hipLaunchKernelGGL((transpose_v_kernel<128, bf16>), grid, dim3(256), 0, st, (const bf16 *)qkv->v,
                         (long long)qkv->sv_h, (long long)qkv->sv_t, qkv->n, npad, (bf16 *)vt);
    else
      hipLaunchKernelGGL((transpose_v_kernel<128, float>), grid, dim3(256), 0, st, (const float *)qkv->v,
                         (long long)qkv->sv_h, (long long)qkv->sv_t, qkv->n, npad, (bf16 *)vt);
  } else {
    if (qkv->dtype == RS_BF16)
      hipLaunchKernelGGL((transpose_v_kernel<64, bf16>), grid, dim3(256), 0, st, (const bf16 *)qkv->v,
                         (long long)qkv->sv_h, (long long)qkv->sv_t, qkv->n, npad, (bf16 *)vt);
    else
      hipLaunchKernelGGL((transpose_v_kernel<64, float>), grid, dim3(256), 0, st, (const float *)qkv->v,
                         (long long)qkv->sv_h, (long long)qkv->sv_t, qkv->n, npad, (bf16 *)vt);
  }
  RS_HIP(hipGetLastError());
  return RS_OK;
}

// ---- host side ---------------------------------------------------------------------------

static int family_bm(int) { return 128; }

static int tiles_of(const rs_unit &u, int bm) { return (u.s1 - 1) / bm - u.s0 / bm + 1; }

// (a unit with a mate has at most twice its 128-row tiles in 64-row blocks, and its mate none)
size_t attn_ws_bytes(const rs_unit *units, int32_t nunits) {
  size_t items = 0;
  for (int i = 0; i < nunits; ++i) items += (size_t)tiles_of(units[i], 128);
  Arena ar(nullptr, 0);
  ar.take<DevUnit>((size_t)nunits);
  ar.take<int>(items);
  return ar.off + 256;
}

// Block-sparse mates: a unit of an even head takes along the unit of the next head with the
// same rows when both heads read the same key/value head (their items then run the two
// heads' selections of one 64-row query block side by side).  mate[u]: the unit taken along
// by u, -2 for a unit taken along, -1 otherwise.
static void pair_units(const rs_unit *units, int nunits, int group, std::vector<int> &mate) {
  mate.assign(nunits, -1);
  std::map<std::tuple<int, int, int>, int> at;  // (head, s0, s1) -> first unit
  for (int u = 0; u < nunits; ++u) at.emplace(std::make_tuple(units[u].head, units[u].s0, units[u].s1), u);
  for (int u = 0; u < nunits; ++u) {
    const int h = units[u].head;
    if ((h & 1) || mate[u] != -1 || (h + 1) / group != h / group) continue;
    const auto it = at.find(std::make_tuple(h + 1, units[u].s0, units[u].s1));
    if (it == at.end() || mate[it->second] != -1) continue;
    mate[u] = it->second;
    mate[it->second] = -2;
  }
}

// Build the dispatch order: items bucketed by key/value head (round-robin workgroup
// dispatch places workgroup b on XCD b % 8, so the query heads sharing one K/V stream
// share one XCD's L2), longest query tiles first within a bucket.  Items of a unit with a
// mate are 64-row query blocks, others bm-row query tiles (bm = 128); units taken along by a
// mate have none.
static void build_order(const rs_unit *units, int nunits, int group, int bm, const std::vector<int> &mate,
                        std::vector<int> &order) {
  std::vector<std::vector<std::pair<int, int>>> buckets(8);  // (-first row / 64, item)
  for (int u = 0; u < nunits; ++u) {
    if (mate[u] == -2) continue;
    const int im = mate[u] >= 0 ? 64 : bm;
    const int t0 = units[u].s0 / im, nt = tiles_of(units[u], im);
    const int b = (units[u].head / group) & 7;
    for (int t = 0; t < nt; ++t) buckets[b].push_back({-((t0 + t) * (im / 64)), (u << 16) | t});
  }
  size_t mx = 0;
  for (auto &b : buckets) {
    std::stable_sort(b.begin(), b.end(),
                     [](const std::pair<int, int> &x, const std::pair<int, int> &y) { return x.first < y.first; });
    mx = std::max(mx, b.size());
  }
  order.clear();
  for (size_t i = 0; i < mx; ++i)
    for (int b = 0; b < 8; ++b)
      if (i < buckets[b].size()) order.push_back(buckets[b][i].second);
}

template <int D, int PAT>
static hipError_t launch_pat(int dtype, const AttnArgs &a, int nitems, hipStream_t st) {
  if (a.vt) {
    if constexpr (PAT != P_VS) {  // vertical-slash gathers V rows: it keeps the row-major V
      if (a.qsize) {
        if (dtype == RS_BF16)
          hipLaunchKernelGGL((attn_fwd_queue_kernel<D, PAT, bf16, true>), dim3(nitems), dim3(256), 0, st, a);
        else
          hipLaunchKernelGGL((attn_fwd_queue_kernel<D, PAT, float, true>), dim3(nitems), dim3(256), 0, st, a);
      } else {
        if (dtype == RS_BF16)
          hipLaunchKernelGGL((attn_fwd_kernel<D, PAT, bf16, true>), dim3(nitems), dim3(256), 0, st, a);
        else
          hipLaunchKernelGGL((attn_fwd_kernel<D, PAT, float, true>), dim3(nitems), dim3(256), 0, st, a);
      }
      return hipGetLastError();
    }
  }
  if (a.qsize) {
    if (dtype == RS_BF16)
      hipLaunchKernelGGL((attn_fwd_queue_kernel<D, PAT, bf16, false>), dim3(nitems), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_queue_kernel<D, PAT, float, false>), dim3(nitems), dim3(256), 0, st, a);
  } else {
    if (dtype == RS_BF16)
      hipLaunchKernelGGL((attn_fwd_kernel<D, PAT, bf16, false>), dim3(nitems), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<D, PAT, float, false>), dim3(nitems), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

template <int D>
static hipError_t launch_d(int fam, int dtype, const AttnArgs &a, int nitems, hipStream_t st) {
  switch (fam) {
    case RS_DENSE: return launch_pat<D, P_DENSE>(dtype, a, nitems, st);
    case RS_ASHAPE: return launch_pat<D, P_ASHAPE>(dtype, a, nitems, st);
    case RS_VSLASH: return launch_pat<D, P_VS>(dtype, a, nitems, st);
    default: return launch_pat<D, P_BS>(dtype, a, nitems, st);
  }
}

// One launch of a family's kernel over a device work list: `d_units` and `d_order` as built
// by attn_launch (host; one workgroup per item, `nblocks` items) or by the device planner
// (device routing; `queues` set, `nblocks` persistent workgroups drain the bucket queues).
rs_status attn_launch_list(const rs_qkv *qkv, float scale, int fam, const rs_index_set *idx,
                           const DevUnit *d_units, const int *d_order, const AttnQueues *queues, int nblocks,
                           void *o, int64_t so_h, int64_t so_t, float *lse, hipStream_t st) {
  if (nblocks <= 0) return RS_OK;
  AttnArgs a{};
  a.q = qkv->q; a.k = qkv->k; a.v = qkv->v;
  a.sq_h = qkv->sq_h; a.sq_t = qkv->sq_t; a.sk_h = qkv->sk_h; a.sk_t = qkv->sk_t;
  a.sv_h = qkv->sv_h; a.sv_t = qkv->sv_t;
  a.o = (bf16 *)o; a.so_h = so_h; a.so_t = so_t; a.lse = lse;
  a.n = qkv->n; a.group = qkv->hq / qkv->hkv; a.scale = scale; a.c = scale * kLog2e;
  a.units = d_units; a.order = d_order;
  a.vt = (const bf16 *)qkv->vt; a.npad = (qkv->n + 63) / 64 * 64;
  if (queues) { a.qsize = queues->size; a.qoff = queues->off; a.qcount = queues->count; }
  if (fam == RS_VSLASH) {
    a.vs_vsorted = idx->vs_vsorted; a.vs_dsorted = idx->vs_dsorted; a.vs_count = idx->vs_count;
    a.vs_vbits = idx->vs_vbits; a.vs_dbits = idx->vs_dbits;
    a.nv_max = idx->nv_max; a.ns_max = idx->ns_max; a.nwords = idx->nwords; a.ncand_vs = idx->ncand_vs;
  }
  if (fam == RS_BSPARSE) {
    a.bs_sorted = idx->bs_sorted; a.bs_count = idx->bs_count;
    a.k_max = idx->k_max; a.nb = idx->nb; a.ncand_bs = idx->ncand_bs;
  }
  hipError_t e = qkv->d == 128 ? launch_d<128>(fam, qkv->dtype, a, nblocks, st)
                               : launch_d<64>(fam, qkv->dtype, a, nblocks, st);
  if (e != hipSuccess) return hip_check(e, "attention kernel launch");
  return RS_OK;
}

// Shared entry of the dense and sparse calls (arguments validated by the caller).
rs_status attn_launch(const rs_qkv *qkv, float scale, const rs_unit *units, int32_t nunits,
                      int fam, const rs_candidate *cand, int cand_local,
                      const rs_index_set *idx, void *o, int64_t so_h, int64_t so_t, float *lse,
                      void *ws, size_t ws_bytes, hipStream_t st) {
  if (nunits == 0) return RS_OK;
  const int bm = family_bm(fam);
  const int group = qkv->hq / qkv->hkv;
  std::vector<int> mate(nunits, -1), order;
  if (fam == RS_BSPARSE) pair_units(units, nunits, group, mate);
  build_order(units, nunits, group, bm, mate, order);
  const size_t need = attn_ws_bytes(units, nunits);
  if (!ws || ws_bytes < need)
    return fail(RS_ERR_WORKSPACE, "attention workspace too small: need " + std::to_string(need) +
                                      " bytes, got " + std::to_string(ws_bytes));
  // host staging: [DevUnit x nunits][order]
  Arena ar(ws, ws_bytes);
  DevUnit *d_units = ar.take<DevUnit>((size_t)nunits);
  int *d_order = ar.take<int>(order.size());
  const size_t off_order = (char *)d_order - (char *)ws;
  std::vector<char> stage(off_order + order.size() * sizeof(int));
  DevUnit *h_units = (DevUnit *)stage.data();
  for (int u = 0; u < nunits; ++u) {
    h_units[u] = DevUnit{units[u].head, units[u].s0, units[u].s1, cand_local, units[u].slot,
                         fam == RS_ASHAPE ? cand->a : 0, fam == RS_ASHAPE ? cand->b : 0,
                         mate[u] >= 0 ? units[mate[u]].head + 1 : 0, cand_local};
  }
  memcpy(stage.data() + off_order, order.data(), order.size() * sizeof(int));
  RS_HIP(hipMemcpyAsync(ws, stage.data(), stage.size(), hipMemcpyHostToDevice, st));

  return attn_launch_list(qkv, scale, fam, idx, d_units, d_order, nullptr, (int)order.size(), o, so_h, so_t, lse,
                          st);
}

}  // namespace rs
