// Internal helpers shared by the HIP kernels and host code of librs (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/rs.h"

namespace rs {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxN = 262144;

// ---- error reporting (host) -------------------------------------------------------------
void set_error(const std::string &msg);
rs_status fail(rs_status st, const std::string &msg);
rs_status hip_check(hipError_t e, const char *what);

#define RS_HIP(call)                                                   \
  do {                                                                 \
    hipError_t _e = (call);                                            \
    if (_e != hipSuccess) return ::rs::hip_check(_e, #call);           \
  } while (0)

// Keys of a unit table (FNV-1a over the fields that define it).
uint64_t unit_list_key(const rs_qkv *qkv, const rs_unit *units, int32_t nunits);
uint64_t probe_cfg_key(const rs_probe_cfg *cfg);
// Device arrays of a unit table (probe.hip lays the table out).
const rs_unit *unit_tab_units(const rs_unit_table *t);
const int *unit_tab_s1(const rs_unit_table *t);
// Checks that `t` was built for this unit list (and, with cfg, this probe configuration).
rs_status check_unit_table(const rs_unit_table *t, const rs_qkv *qkv, const rs_unit *units, int32_t nunits,
                           const rs_probe_cfg *cfg);

// Validate rs_qkv; fills scale.  Returns RS_OK or an error (message set).
rs_status check_qkv(const rs_qkv *qkv, float *scale);
rs_status check_units(const rs_qkv *qkv, const rs_unit *units, int32_t nunits);

// Unit descriptor read by the attention kernels (work lists built on the host or on the device).
struct DevUnit {
  int head, s0, s1, cl, slot;  // cl: index of the unit's candidate among its family's
  int sink, window;            // A-shape candidate of the unit
  // block-sparse: head + 1 of a second unit (same rows, same key/value head) whose query
  // blocks this unit's items also run, and that unit's cl; 0: none (items of 128 rows)
  int mate, mate_cl;
};

// Device work queues of a persistent attention launch: per key/value bucket b (8), the items
// order[off[b] .. off[b] + size[b]) and a counter of items taken (starts at 0).
struct AttnQueues {
  const int *size, *off;
  int *count;
};

// One launch of a family's attention kernel over a device work list (attn.hip).
rs_status attn_launch_list(const rs_qkv *qkv, float scale, int fam, const rs_index_set *idx,
                           const DevUnit *d_units, const int *d_order, const AttnQueues *queues, int nblocks,
                           void *o, int64_t so_h, int64_t so_t, float *lse, hipStream_t st);

// bump allocator over a caller workspace
struct Arena {
  char *base;
  size_t cap, off;
  explicit Arena(void *b, size_t c) : base((char *)b), cap(c), off(0) {}
  template <typename T>
  T *take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T *p = (T *)(base ? base + off : nullptr);
    off += count * sizeof(T);
    return p;
  }
  bool ok() const { return off <= cap; }
};

// ---- device helpers ----------------------------------------------------------------------
#if defined(__HIP_DEVICE_COMPILE__) || defined(__HIPCC__)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats rounded to nearest-even bf16 and packed (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x2 cvt_bf16x2(float lo, float hi) {
  return __builtin_convertvector(f32x2{lo, hi}, bf16x2);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, cvt_bf16x2(lo, hi));
}

// 8 consecutive elements as 8 bf16 packed in 4 dwords (fp32 input is rounded to bf16).
template <typename T>
__device__ __forceinline__ u32x4 load8(const T *p);
template <>
__device__ __forceinline__ u32x4 load8<bf16>(const bf16 *p) {
  return *(const u32x4 *)p;
}
template <>
__device__ __forceinline__ u32x4 load8<float>(const float *p) {
  f32x4 a = *(const f32x4 *)p, b = *(const f32x4 *)(p + 4);
  u32x4 r;
  r[0] = pack_bf16x2(a[0], a[1]);
  r[1] = pack_bf16x2(a[2], a[3]);
  r[2] = pack_bf16x2(b[0], b[1]);
  r[3] = pack_bf16x2(b[2], b[3]);
  return r;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// 64-bit mask with bits [0, c) set (c clamped to [0, 64]).
__device__ __forceinline__ uint64_t prefix_mask(int c) {
  return c <= 0 ? 0ull : (c >= 64 ? ~0ull : ((1ull << c) - 1ull));
}

// 64 bits of a bitmap starting at bit position pos (may be negative); bits outside
// [0, 32*nwords) read as 0.
__device__ __forceinline__ uint64_t bits64_at(const uint32_t *bits, int nwords, int pos) {
  int w = pos >> 5;             // floor division (arithmetic shift)
  int sh = pos & 31;
  uint32_t x0 = (w >= 0 && w < nwords) ? bits[w] : 0u;
  uint32_t x1 = (w + 1 >= 0 && w + 1 < nwords) ? bits[w + 1] : 0u;
  uint32_t x2 = (w + 2 >= 0 && w + 2 < nwords) ? bits[w + 2] : 0u;
  uint64_t lo = (uint64_t)x0 | ((uint64_t)x1 << 32);
  uint64_t r = lo >> sh;
  if (sh) r |= (uint64_t)x2 << (64 - sh);
  return r;
}

// Three consecutive bitmap words around a bit position (loaded ahead of their use).
struct Win3 {
  uint32_t x0, x1, x2;
};

__device__ __forceinline__ Win3 load_win(const uint32_t *bits, int nwords, int pos) {
  const int w = pos >> 5;
  Win3 r;
  r.x0 = (w >= 0 && w < nwords) ? bits[w] : 0u;
  r.x1 = (w + 1 >= 0 && w + 1 < nwords) ? bits[w + 1] : 0u;
  r.x2 = (w + 2 >= 0 && w + 2 < nwords) ? bits[w + 2] : 0u;
  return r;
}

// load_win for a position that is the same in every lane, through the scalar cache (the
// bitmap is read-only while the kernel runs)
__device__ __forceinline__ Win3 load_win_uniform(const uint32_t *bits, int nwords, int pos) {
  typedef const __attribute__((address_space(4))) uint32_t cu32;
  cu32 *cb = (cu32 *)bits;
  const int w = pos >> 5;
  Win3 r;
  r.x0 = (w >= 0 && w < nwords) ? cb[w] : 0u;
  r.x1 = (w + 1 >= 0 && w + 1 < nwords) ? cb[w + 1] : 0u;
  r.x2 = (w + 2 >= 0 && w + 2 < nwords) ? cb[w + 2] : 0u;
  return r;
}

// the 64 bits starting at `pos` from a window loaded with load_win(.., pos)
__device__ __forceinline__ uint64_t win_bits(const Win3 &r, int pos) {
  const int sh = pos & 31;
  uint64_t v = ((uint64_t)r.x0 | ((uint64_t)r.x1 << 32)) >> sh;
  if (sh) v |= (uint64_t)r.x2 << (64 - sh);
  return v;
}


// order-preserving map of a float to uint32 (larger value => larger key; -0.0 < +0.0)
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

#endif

}  // namespace rs
