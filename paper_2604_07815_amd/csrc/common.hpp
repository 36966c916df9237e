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
  __device__ static inline float to_f(T x) { return x; }
};

struct BF16 {
  using T = uint16_t;
  static constexpr int kVec = 8;
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

// ---------------------------------------------------------------------------
// Work-group top-k over keys held in LDS.
//
// Selects the k largest keys among keys[0, n) (kInvalidKey entries never
// count), ties resolved toward the lower position, and writes
// map(position) for the selected positions in ascending position order to
// out[0, k'), k' = min(k, #valid), then -1 up to out_cap.  If out_scores is
// non-null it receives key_float of each selected key.
//
// Method: MSB-first radix select (4 passes of 8 bits, histograms in LDS)
// finds the k'-th largest key T and how many keys equal to T are taken
// (the lowest positions first); an ordered compaction then emits, in
// position order, every key > T plus the first r keys == T.  No sort is
// needed because the output is ordered by position.
//
// Scratch: `hist` holds 256 + 32 uint32; `NT` is the work-group size.
// ---------------------------------------------------------------------------
template <int NT, class Map>
__device__ void wg_topk_ascending(const uint32_t* keys, int n, int k, int32_t* out, int out_cap,
                                  float* out_scores, Map map, uint32_t* hist) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid / kWave;
  uint32_t* wsum = hist + 256;  // per-wave partials (NW <= 16) + broadcast slots

  // count valid keys
  int cnt = 0;
  for (int i = tid; i < n; i += NT) cnt += keys[i] != kInvalidKey;
  for (int o = kWave / 2; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, kWave);
  if (lane == 0) wsum[wid] = cnt;
  __syncthreads();
  int n_valid = 0;
  for (int w = 0; w < NW; ++w) n_valid += wsum[w];
  const int kk = min(k, n_valid);
  __syncthreads();

  uint32_t prefix = 0, pmask = 0;
  int remaining = kk;
  if (kk > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += NT) hist[i] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += NT) {
        uint32_t key = keys[i];
        if (key != kInvalidKey && (key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wid == 0) {
        // lane L owns digits 255-4L .. 252-4L (descending); suffix-scan from the top
        uint32_t c[4];
        uint32_t local = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) { c[j] = hist[255 - 4 * lane - j]; local += c[j]; }
        uint32_t incl = local;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          uint32_t t = __shfl_up(incl, o, kWave);
          if (lane >= o) incl += t;
        }
        uint32_t above = incl - local;  // keys with larger digits than this lane's range
        // find the digit where the cumulative count first reaches `remaining`
        uint32_t run = above;
        int found = -1;
        uint32_t found_above = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (found < 0 && run + c[j] >= uint32_t(remaining)) { found = 255 - 4 * lane - j; found_above = run; }
          run += c[j];
        }
        uint64_t hit = __ballot(found >= 0);
        int src = __ffsll((unsigned long long)hit) - 1;  // the first (highest-digit) lane that hits
        int dig = __shfl(found, src, kWave);
        uint32_t ab = __shfl(found_above, src, kWave);
        if (lane == 0) { wsum[16] = uint32_t(dig); wsum[17] = ab; }
      }
      __syncthreads();
      uint32_t dig = wsum[16];
      remaining -= int(wsum[17]);
      prefix |= dig << shift;
      pmask |= 255u << shift;
      __syncthreads();
    }
  }
  const uint32_t T = prefix;
  const int r = remaining;  // number of keys equal to T to take (lowest positions)

  // ordered compaction, one tile of NT positions at a time
  int gt_base = 0, eq_base = 0;
  if (kk > 0) {
    for (int base = 0; base < n; base += NT) {
      int i = base + tid;
      uint32_t key = i < n ? keys[i] : kInvalidKey;
      bool gt = key != kInvalidKey && key > T;
      bool eq = key != kInvalidKey && key == T;
      uint64_t bg = __ballot(gt), be = __ballot(eq);
      if (lane == 0) { wsum[wid] = __popcll(bg); wsum[NW + wid] = __popcll(be); }
      __syncthreads();
      int gb = gt_base, eb = eq_base, gtot = 0, etot = 0;
      for (int w = 0; w < NW; ++w) {
        int g = wsum[w], e = wsum[NW + w];
        if (w < wid) { gb += g; eb += e; }
        gtot += g; etot += e;
      }
      gb += lanes_below(bg);
      eb += lanes_below(be);
      if (gt || (eq && eb < r)) {
        int pos = gb + min(eb, r);
        out[pos] = map(i);
        if (out_scores) out_scores[pos] = key_float(key);
      }
      gt_base += gtot;
      eq_base += etot;
      __syncthreads();
    }
  }
  for (int i = kk + tid; i < out_cap; i += NT) {
    out[i] = -1;
    if (out_scores) out_scores[i] = 0.0f;
  }
}

// Device error word (first 4 bytes of the workspace).
__device__ inline void set_error(uint32_t* err, uint32_t bit) {
  if (err) atomicOr(err, bit);
}

}  // namespace tls
