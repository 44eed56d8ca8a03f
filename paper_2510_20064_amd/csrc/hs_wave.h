// Wave64 building blocks of the evaluation kernels: DPP reductions and the 64-bit words
// through which workgroups exchange results.
#pragma once

#include <climits>

#include "hs_internal.h"

namespace hs {

// ---- words shared between workgroups ------------------------------------------------------
// A word is written once per call with one relaxed 64-bit agent-scope store: the value in the
// high half, a tag naming the call in the low half. A reader that sees the current tag has
// the whole value (the store is single-copy atomic), so no fence is needed.

__device__ inline void put_word(uint64_t* w, uint64_t v) {
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t get_word(const uint64_t* w) {
  return __hip_atomic_load(const_cast<uint64_t*>(w), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t word_of(float x, uint32_t tag) {
  return ((uint64_t)__float_as_uint(x) << 32) | tag;
}
__device__ inline uint64_t word_of(int x, uint32_t tag) {
  return ((uint64_t)(uint32_t)x << 32) | tag;
}
__device__ inline float word_f(uint64_t w) { return __uint_as_float((uint32_t)(w >> 32)); }
__device__ inline int word_i(uint64_t w) { return (int)(uint32_t)(w >> 32); }
// Tags are 31-bit. Bit 31 of a word's tag half marks a value computed from a word that was
// lost (a wait that gave up): the mark travels with the data, so whoever consumes the value,
// directly or through later words, knows it without any ordering between different words.
constexpr uint32_t kTaint = 0x80000000u;
__device__ inline uint32_t tag_of(uint64_t w) { return (uint32_t)w & ~kTaint; }
__device__ inline bool tainted(uint64_t w) { return ((uint32_t)w & kTaint) != 0; }
__device__ inline uint32_t taint_bits(bool t) { return t ? kTaint : 0u; }

// ---- wave reductions on the DPP network ----------------------------------------------------
// Pairs and quads by quad_perm, 8- and 16-lane groups by the half-row and row mirrors, then
// the four row results are combined in a fixed order; every lane gets the same value. All
// 64 lanes must be active.

// These patterns read only existing lanes of the row, so bound_ctrl changes no value; with it
// set the compiler may fold the move into the consuming instruction (v_add_f32_dpp ...).
template <int CTRL>
__device__ inline float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ inline int dpp_i(int x) {
  return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
}
// Order-preserving map of a non-NaN float to a signed int (and back): negative values have
// their magnitude bits flipped. Integer max needs no NaN canonicalisation, unlike fmaxf.
__device__ inline int fkey(float x) {
  const int b = __float_as_int(x);
  return b ^ ((b >> 31) & 0x7FFFFFFF);
}
__device__ inline float fkey_inv(int k) { return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF)); }
__device__ inline float lane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ inline float wave_sum_f(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}

template <int CTRL>
__device__ inline void argmax_step(float& m, int& idx) {
  const float m2 = dpp_f<CTRL>(m);
  const int i2 = dpp_i<CTRL>(idx);
  argmax_combine(m, idx, m2, i2);
}
// Wave max of m (not NaN); with NEED_ARG also the lowest index attaining it.
template <bool NEED_ARG>
__device__ inline void wave_max(float& m, int& idx) {
  if (NEED_ARG) {
    argmax_step<0xB1>(m, idx);
    argmax_step<0x4E>(m, idx);
    argmax_step<0x141>(m, idx);
    argmax_step<0x140>(m, idx);
    float r = lane_f(m, 0);
    int ri = __builtin_amdgcn_readlane(idx, 0);
#pragma unroll
    for (int l = 16; l < 64; l += 16)
      argmax_combine(r, ri, lane_f(m, l), __builtin_amdgcn_readlane(idx, l));
    m = r;
    idx = ri;
  } else {  // m not NaN
    int k = fkey(m);
    k = max(k, dpp_i<0xB1>(k));
    k = max(k, dpp_i<0x4E>(k));
    k = max(k, dpp_i<0x141>(k));
    k = max(k, dpp_i<0x140>(k));
    k = max(max(__builtin_amdgcn_readlane(k, 0), __builtin_amdgcn_readlane(k, 16)),
            max(__builtin_amdgcn_readlane(k, 32), __builtin_amdgcn_readlane(k, 48)));
    m = fkey_inv(k);
  }
}

// ---- reductions within a DPP row: 16-lane groups ---------------------------------------------
// Pairs, quads, half-rows, then the row; afterwards every lane of the group holds the result
// (each step combines a lane with its mirror, so all lanes form bitwise the same value). All
// 16 lanes of the group must be active.
__device__ inline float row16_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  return v;
}
__device__ inline int row16_max(int k) {
  k = max(k, dpp_i<0xB1>(k));
  k = max(k, dpp_i<0x4E>(k));
  k = max(k, dpp_i<0x141>(k));
  return max(k, dpp_i<0x140>(k));
}
__device__ inline void row16_argmax(float& m, int& idx) {
  argmax_step<0xB1>(m, idx);
  argmax_step<0x4E>(m, idx);
  argmax_step<0x141>(m, idx);
  argmax_step<0x140>(m, idx);
}

// Lane j of a 16-lane group reads the values 64 i + 4 j + k (i, k = 0..3) of an LDS row of
// 256: one 16-byte read per i, consecutive lanes on consecutive 16 bytes (no bank conflict).
template <typename T>
__device__ inline void group_read(const T* row, int j, T (&v)[16]) {
  typedef T T4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const T4 x = *reinterpret_cast<const T4*>(row + 64 * i + 4 * j);
#pragma unroll
    for (int k = 0; k < 4; ++k) v[4 * i + k] = x[k];
  }
}
// Sum of 16 values in a fixed pairwise order.
__device__ inline float sum16(const float (&v)[16]) {
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = v[2 * i] + v[2 * i + 1];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = a[2 * i] + a[2 * i + 1];
  return (a[0] + a[1]) + (a[2] + a[3]);
}

template <int CTRL>
__device__ inline void lse_step(float& o, float& s) {
  const float o2 = dpp_f<CTRL>(o);
  const float s2 = dpp_f<CTRL>(s);
  lse2_combine(o, s, o2, s2);
}
// Wave combine of (offset, exp2 sum) pairs.
__device__ inline void wave_lse(float& o, float& s) {
  lse_step<0xB1>(o, s);
  lse_step<0x4E>(o, s);
  lse_step<0x141>(o, s);
  lse_step<0x140>(o, s);
  float ro = lane_f(o, 0), rs = lane_f(s, 0);
#pragma unroll
  for (int l = 16; l < 64; l += 16) lse2_combine(ro, rs, lane_f(o, l), lane_f(s, l));
  o = ro;
  s = rs;
}

}  // namespace hs
