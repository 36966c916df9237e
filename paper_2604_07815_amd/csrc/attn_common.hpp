// Helpers shared by the attention kernels.
#pragma once

#include "kernels.hpp"

namespace tls {

// Address of token `tok`'s row in the direct layout [units][T][d] or, with a
// slot map, in the block pool [units][n_slots][B][d].  *ok turns false when
// the token's block is not resident.
template <class S>
__device__ inline const S* kv_row(const S* base, const int32_t* slot_map, int64_t n_slots, size_t unit, int T,
                                  int B, int m_max, int d, int tok, bool* ok) {
  if (!slot_map) return base + (unit * size_t(T) + size_t(tok)) * d;
  const int slot = slot_map[unit * size_t(m_max) + tok_block(tok, B)];
  if (slot < 0 || slot >= n_slots) {
    *ok = false;
    return base;
  }
  return base + ((unit * size_t(n_slots) + size_t(slot)) * B + tok_offset(tok, B)) * d;
}

// Token of entry p of a unit's work list (-1: empty).  *bad turns true for
// an explicit id at or past ctx_len n (the caller flags it and skips it).
__device__ inline int list_token(const TokenList& L, size_t unit, int p, int n, bool* bad) {
  if (L.kind == kListIds) {
    const int t = L.ids[unit * size_t(L.stride) + p];
    if (t >= n) {
      *bad = true;
      return -1;
    }
    return t < 0 ? -1 : t;
  }
  if (L.kind == kListBlocks) {
    const int blk = L.ids[unit * size_t(L.stride) + tok_block(p, L.B)];
    const int t = blk * L.B + tok_offset(p, L.B);
    return blk < 0 || t >= n ? -1 : t;
  }
  return p < n ? p : -1;
}

__device__ inline float exp_or_zero(float x) { return x == -INFINITY ? 0.f : expf(x); }

// Transposing butterfly all-reduce over the MASK*2 lanes of a lane group:
// while more than one value is left, each xor step sends half of the values
// to the partner lane and keeps the other half, so NV values are reduced with
// NV - 1 shuffles instead of NV*log2(W).  On return v[j] holds the fully
// reduced value of original index xreduce_index<NV, W>(lane, j), for
// j < max(1, NV / W).
template <int NV, int MASK>
struct XReduce {
  __device__ static inline void run(float* v, int lane) {
    if constexpr (MASK == 0) {
      return;
    } else if constexpr (NV > 1) {
      constexpr int H = NV / 2;
      const bool upper = (lane & MASK) != 0;
#pragma unroll
      for (int j = 0; j < H; ++j) {
        const float send = upper ? v[j] : v[j + H];
        const float keep = upper ? v[j + H] : v[j];
        v[j] = keep + __shfl_xor(send, MASK, 64);
      }
      XReduce<H, MASK / 2>::run(v, lane);
    } else {
      v[0] += __shfl_xor(v[0], MASK, 64);
      XReduce<1, MASK / 2>::run(v, lane);
    }
  }
};

// The same transposing reduction with the partner lane chosen by DPP mirror
// patterns inside 16-lane rows (row_mirror, row_half_mirror, quad reverse,
// quad swap): a VALU lane move instead of an LDS-routed shuffle.  Within a
// group of W lanes the mirror partner has the opposite W/2 bit and the same
// higher bits, so the kept halves and the resulting index map are those of
// XReduce.  A 32-lane first step (W = 32) uses one xor-16 shuffle.
template <int CTRL>
__device__ inline float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int W>
__device__ inline float mirror_partner(float v) {
  if constexpr (W == 32) return __shfl_xor(v, 16, 64);
  else if constexpr (W == 16) return dpp_mov<0x140>(v);  // row_mirror
  else if constexpr (W == 8) return dpp_mov<0x141>(v);   // row_half_mirror
  else if constexpr (W == 4) return dpp_mov<0x1B>(v);    // quad_perm [3,2,1,0]
  else return dpp_mov<0xB1>(v);                          // quad_perm [1,0,3,2]
}

template <int NV, int W>
struct XReduceDpp {
  __device__ static inline void run(float* v, int lane) {
    if constexpr (W < 2) {
      return;
    } else if constexpr (NV > 1) {
      constexpr int H = NV / 2;
      const bool upper = (lane & (W / 2)) != 0;
#pragma unroll
      for (int j = 0; j < H; ++j) {
        const float send = upper ? v[j] : v[j + H];
        const float keep = upper ? v[j + H] : v[j];
        v[j] = keep + mirror_partner<W>(send);
      }
      XReduceDpp<H, W / 2>::run(v, lane);
    } else {
      v[0] += mirror_partner<W>(v[0]);
      XReduceDpp<1, W / 2>::run(v, lane);
    }
  }
};

template <int NV, int W>
__device__ inline int xreduce_index(int lane, int j) {
  int idx = j, cur = NV;
#pragma unroll
  for (int mask = W / 2; mask > 0; mask >>= 1) {
    if (cur > 1) {
      cur >>= 1;
      if (lane & mask) idx += cur;
    }
  }
  return idx;
}

}  // namespace tls
