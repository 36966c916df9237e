// Device helpers shared by the two-level sparse decode kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tls {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Element types.  Inputs are fp32 or bf16; all arithmetic is fp32.
// ---------------------------------------------------------------------------
struct F32 {
  using T = float;
  static constexpr int kVec = 4;  // elements per 16-byte load
  static constexpr bool kIsBf16 = false;
  __device__ static inline float to_f(T x) { return x; }
};

struct BF16 {
  using T = uint16_t;
  static constexpr int kVec = 8;
  static constexpr bool kIsBf16 = true;
  __device__ static inline float to_f(T x) { return __uint_as_float(uint32_t(x) << 16); }
};

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even float -> bf16 bits (NaN kept quiet).
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t(0x7fc0u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

template <class E>
__device__ inline void store_out(typename E::T* p, float v);
template <>
__device__ inline void store_out<F32>(float* p, float v) { *p = v; }
template <>
__device__ inline void store_out<BF16>(uint16_t* p, float v) { *p = f32_to_bf16(v); }

// Unpack one 16-byte vector into fp32 lanes.
template <class E>
__device__ inline void unpack16(const uint4& v, float* out);
template <>
__device__ inline void unpack16<F32>(const uint4& v, float* out) {
  out[0] = __uint_as_float(v.x);
  out[1] = __uint_as_float(v.y);
  out[2] = __uint_as_float(v.z);
  out[3] = __uint_as_float(v.w);
}
template <>
__device__ inline void unpack16<BF16>(const uint4& v, float* out) {
  out[0] = bf16_lo(v.x); out[1] = bf16_hi(v.x);
  out[2] = bf16_lo(v.y); out[3] = bf16_hi(v.y);
  out[4] = bf16_lo(v.z); out[5] = bf16_hi(v.z);
  out[6] = bf16_lo(v.w); out[7] = bf16_hi(v.w);
}

__device__ inline uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// Non-temporal 16-byte load for data touched once per step (gathered K/V,
// index rows): keeps them from displacing reusable lines in L2.
__device__ inline uint4 ld16_stream(const void* p) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
  uint4 r;
  r.x = __builtin_nontemporal_load(&q->x);
  r.y = __builtin_nontemporal_load(&q->y);
  r.z = __builtin_nontemporal_load(&q->z);
  r.w = __builtin_nontemporal_load(&q->w);
  return r;
}

// ---------------------------------------------------------------------------
// Wave reductions (xor butterflies over `width` lanes, width a power of two)
// ---------------------------------------------------------------------------
template <int W>
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
template <int W>
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ inline int lane_id() { return __lane_id(); }

// Number of set bits of `mask` in lanes below the calling lane.
__device__ inline int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(mask >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(mask), 0));
}

// ---------------------------------------------------------------------------
// Whole-wave reductions on DPP lane moves (VALU latency) plus four lane
// reads, instead of LDS-routed shuffles.  Every lane of the wave must be
// active.  The result is wave-uniform.
//   quad_perm [1,0,3,2] / [2,3,0,1]: xor 1 / xor 2 inside a quad
//   row_half_mirror / row_mirror: the other quad of 8 / the other 8 of 16
// Each of these moves reads a valid lane of the same row for every lane, so
// the move's "old" operand is never used; passing 0 there lets the compiler
// fold the move into the integer or float-add instruction that consumes it
// (one v_*_dpp instruction per step).
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ inline int dpp_perm(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

template <class Op>
__device__ inline uint32_t wave_reduce_bits(uint32_t x, Op op) {
  int v = int(x);
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0xB1>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x4E>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x141>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x140>(v))));
  const uint32_t r0 = uint32_t(__builtin_amdgcn_readlane(v, 0)), r1 = uint32_t(__builtin_amdgcn_readlane(v, 16));
  const uint32_t r2 = uint32_t(__builtin_amdgcn_readlane(v, 32)), r3 = uint32_t(__builtin_amdgcn_readlane(v, 48));
  return op(op(r0, r1), op(r2, r3));
}

__device__ inline uint32_t wave_max_u32(uint32_t x) {
  return wave_reduce_bits(x, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}
__device__ inline uint32_t wave_min_u32(uint32_t x) {
  return wave_reduce_bits(x, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}
// Order-preserving map of a float to a signed int (an involution on the
// bits: non-negative floats keep their bits, negative ones flip the
// magnitude bits), so float maxima reduce as integer maxima, which fold into
// DPP instructions.  A NaN enters as -inf, so that, as with fmaxf, it is
// ignored unless every value is NaN or -inf (the result is then -inf).
__device__ inline int f32_ord(float f) {
  const int b = f == f ? __float_as_int(f) : int(0xff800000u);
  return b ^ ((b >> 31) & 0x7fffffff);
}
__device__ inline float ord_f32(int o) { return __int_as_float(o ^ ((o >> 31) & 0x7fffffff)); }

// Wave maximum as an order-preserving int (f32_ord form), for callers that
// keep combining it as an integer.
__device__ inline int wave_max_ord(float x) {
  return int(wave_reduce_bits(uint32_t(f32_ord(x)), [](uint32_t a, uint32_t b) { return uint32_t(max(int(a), int(b))); }));
}

__device__ inline float wave_max_f32(float x) {
  return ord_f32(int(wave_reduce_bits(uint32_t(f32_ord(x)), [](uint32_t a, uint32_t b) {
    return uint32_t(max(int(a), int(b)));
  })));
}
__device__ inline float wave_sum_f32(float x) {
  return __uint_as_float(wave_reduce_bits(__float_as_uint(x), [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}

// Reduction inside each 16-lane row on DPP lane moves (xor 1, xor 2, the
// other quad of 8, the other 8 of 16): afterwards every lane of a row holds
// the row's result.  Used to combine one value per wave (at most 16 waves),
// read from LDS into lanes 0-15 of every row, with four instructions instead
// of a read of every lane.  Every lane must be active.
template <class Op>
__device__ inline uint32_t row16_reduce_bits(uint32_t x, Op op) {
  int v = int(x);
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0xB1>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x4E>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x141>(v))));
  v = int(op(uint32_t(v), uint32_t(dpp_perm<0x140>(v))));
  return uint32_t(v);
}

// Combines one value per wave, w_0..w_{nw-1} (nw <= 16): `mine` is lane l's
// copy of w_{l mod 16} (the operation's identity where l mod 16 >= nw).  The
// result is wave-uniform.
template <class Op>
__device__ inline uint32_t combine_waves_bits(uint32_t mine, Op op) {
  return uint32_t(__builtin_amdgcn_readfirstlane(int(row16_reduce_bits(mine, op))));
}
__device__ inline float combine_waves_max_f32(float mine) {
  return ord_f32(int(combine_waves_bits(uint32_t(f32_ord(mine)), [](uint32_t a, uint32_t b) {
    return uint32_t(max(int(a), int(b)));
  })));
}
__device__ inline float combine_waves_sum_f32(float mine) {
  return __uint_as_float(combine_waves_bits(__float_as_uint(mine), [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}
__device__ inline int combine_waves_max_i32(int mine) {
  return int(combine_waves_bits(uint32_t(mine), [](uint32_t a, uint32_t b) { return uint32_t(max(int(a), int(b))); }));
}
__device__ inline uint32_t combine_waves_sum_u32(uint32_t mine) {
  return combine_waves_bits(mine, [](uint32_t a, uint32_t b) { return a + b; });
}
__device__ inline uint32_t combine_waves_max_u32(uint32_t mine) {
  return combine_waves_bits(mine, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}
__device__ inline uint32_t combine_waves_min_u32(uint32_t mine) {
  return combine_waves_bits(mine, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}

// Inclusive prefix sum over the wave on DPP lane moves: a Hillis-Steele scan
// inside each 16-lane row (row_shr 1, 2, 4, 8), then row 0's total into row 1
// and row 2's into row 3 (row_bcast:15), then rows 0-1 into rows 2-3
// (row_bcast:31).  Lanes without a source add 0.  Every lane must be active.
__device__ inline uint32_t wave_incl_scan_u32(uint32_t v) {
  int x = int(v);
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
  return uint32_t(x);
}

// Inclusive prefix sum over the wave of small non-negative integers
// (v < 2^BITS), one ballot per bit; *total receives the wave sum.
template <int BITS>
__device__ inline uint32_t wave_incl_scan_small(uint32_t v, uint32_t* total) {
  uint32_t incl = 0, tot = 0;
#pragma unroll
  for (int b = 0; b < BITS; ++b) {
    const uint32_t bit = (v >> b) & 1u;
    const uint64_t m = __ballot(bit != 0);
    incl += (uint32_t(lanes_below(m)) + bit) << b;
    tot += uint32_t(__popcll(m)) << b;
  }
  *total = tot;
  return incl;
}

// ---------------------------------------------------------------------------
// Orderable keys: larger float -> larger uint32.  -0.0 == +0.0; NaN ranks
// just above key 0, which marks an empty / invalid slot.
// ---------------------------------------------------------------------------
constexpr uint32_t kInvalidKey = 0u;

__device__ inline uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 1u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float key_float(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

// Block of a token position (or candidate slot) t >= 0 and its offset inside
// the block, for the power-of-two block size B (the library supports B = 64):
// a shift and a mask instead of an integer division by a runtime value.
__device__ inline int tok_block(int t, int B) { return t >> __builtin_ctz(unsigned(B)); }
__device__ inline int tok_offset(int t, int B) { return t & (B - 1); }

// Device error word (first 4 bytes of the workspace).
__device__ inline void set_error(uint32_t* err, uint32_t bit) {
  if (err) atomicOr(err, bit);
}

}  // namespace tls

// Work-group top-k selection (keys in registers, LDS histograms).
#include "topk.hpp"
