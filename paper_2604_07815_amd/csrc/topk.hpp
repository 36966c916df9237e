// Work-group top-k selection with lowest-position tie-breaking.
#pragma once

#include "common.hpp"

namespace tls {

constexpr int kTopkMaxEPT = 16;  // keys per thread: n <= NT * kTopkMaxEPT

// LDS words the selection needs: four 256-bin histograms (one per radix
// pass, cleared once up front) and two sets of broadcast slots.
__host__ __device__ constexpr int topk_scratch_words(int /*nt*/) { return 4 * 256 + 64 + 32; }

__device__ inline uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// Selects the k largest keys among keys[0, n) (LDS; kInvalidKey entries never
// count), ties resolved toward the lower position, and writes map(position)
// of the selected positions in ascending position order to out[0, k'),
// k' = min(k, #valid keys), then -1 up to out_cap.  out_scores (nullable)
// receives key_float of each selected key.  `stage` (LDS, out_cap ints) and
// `stage_sc` (LDS, out_cap floats, when scores are wanted) hold the result
// until one final copy, because a work-group barrier waits for outstanding
// global stores.  Every thread of the work-group must call it.
//
// Method: each thread keeps the keys of positions [tid*ept, tid*ept + ept)
// in registers.  An MSB-first radix select over the bits where the valid keys
// differ (8-bit digits, LDS histograms) finds the k'-th largest key T and the
// number r of keys equal to T to take; an ordered compaction (one prefix sum
// of per-thread counts) then emits every key > T and the first r keys == T.
// The output is ordered by position, so no sort is needed.
template <int NT, class Map>
__device__ void wg_topk_ascending(const uint32_t* keys, int n, int k, int32_t* out, int out_cap,
                                  float* out_scores, Map map, uint32_t* scratch, int32_t* stage,
                                  float* stage_sc) {
  constexpr int NW = NT / 64;
  static_assert(NW >= 1 && NW <= 16, "work-group of 64..1024 threads");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  uint32_t* hist = scratch;           // [4][256]
  uint32_t* misc = scratch + 1024;    // [64] count / radix broadcast slots
  uint32_t* comp = misc + 64;         // [16] compaction wave totals
  const int ept = (n + NT - 1) / NT;
  const int p0 = tid * ept;

  uint32_t kr[kTopkMaxEPT];
  int cnt = 0;
  uint32_t kmx = 0u, kmn = 0xffffffffu;
#pragma unroll
  for (int j = 0; j < kTopkMaxEPT; ++j) {
    const int p = p0 + j;
    const uint32_t key = (j < ept && p < n) ? keys[p] : kInvalidKey;
    kr[j] = key;
    if (key != kInvalidKey) {
      ++cnt;
      kmx = max(kmx, key);
      kmn = min(kmn, key);
    }
  }
  for (int i = tid; i < 1024; i += NT) hist[i] = 0u;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    cnt += __shfl_xor(cnt, o, 64);
    kmx = max(kmx, (uint32_t)__shfl_xor((int)kmx, o, 64));
    kmn = min(kmn, (uint32_t)__shfl_xor((int)kmn, o, 64));
  }
  if (lane == 0) {
    misc[wid] = uint32_t(cnt);
    misc[16 + wid] = kmx;
    misc[32 + wid] = kmn;
  }
  __syncthreads();
  {
    const int w = lane & 15;
    const bool in = w < NW;
    cnt = in ? int(misc[w]) : 0;
    kmx = in ? misc[16 + w] : 0u;
    kmn = in ? misc[32 + w] : 0xffffffffu;
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      cnt += __shfl_xor(cnt, o, 64);
      kmx = max(kmx, (uint32_t)__shfl_xor((int)kmx, o, 64));
      kmn = min(kmn, (uint32_t)__shfl_xor((int)kmn, o, 64));
    }
  }
  const int kk = min(k, cnt);

  uint32_t prefix = 0u, pmask = 0u;
  int remaining = kk;
  int bits_left = 0;
  if (kk > 0) {
    const uint32_t diff = kmx ^ kmn;
    bits_left = diff ? 32 - __clz(diff) : 0;
    pmask = bits_left >= 32 ? 0u : ~((1u << bits_left) - 1u);
    prefix = kmx & pmask;
  }
  for (int pass = 0; bits_left > 0; ++pass) {
    const int nb = bits_left < 8 ? bits_left : 8;
    const int shift = bits_left - nb;
    const uint32_t dmask = (1u << nb) - 1u;
    uint32_t* h = hist + 256 * pass;
#pragma unroll
    for (int j = 0; j < kTopkMaxEPT; ++j) {
      const uint32_t key = kr[j];
      if (key != kInvalidKey && (key & pmask) == prefix) atomicAdd(&h[(key >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (wid == 0) {
      // lane L owns digits 255-4L .. 252-4L (descending); scan from the top
      uint32_t c[4];
      uint32_t local = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = h[255 - 4 * lane - j];
        local += c[j];
      }
      const uint32_t incl = wave_incl_scan(local);
      uint32_t run = incl - local;
      int found = -1;
      uint32_t found_above = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (found < 0 && run + c[j] >= uint32_t(remaining)) {
          found = 255 - 4 * lane - j;
          found_above = run;
        }
        run += c[j];
      }
      const uint64_t hit = __ballot(found >= 0);
      const int src = __ffsll((unsigned long long)hit) - 1;
      const int dig = __shfl(found, src, 64);
      const uint32_t ab = __shfl(found_above, src, 64);
      if (lane == 0) {
        misc[48] = uint32_t(dig);
        misc[49] = ab;
      }
    }
    __syncthreads();
    prefix |= misc[48] << shift;
    remaining -= int(misc[49]);
    pmask |= dmask << shift;
    bits_left -= nb;
  }
  const uint32_t T = prefix;
  const int r = remaining;  // keys equal to T still to take, lowest positions first

  if (kk > 0) {
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int j = 0; j < kTopkMaxEPT; ++j) {
      const uint32_t key = kr[j];
      gt += (key != kInvalidKey && key > T) ? 1u : 0u;
      eq += (key != kInvalidKey && key == T) ? 1u : 0u;
    }
    const uint32_t v = (gt << 16) | eq;  // both counts < 2^16
    const uint32_t incl = wave_incl_scan(v);
    if (lane == 63) comp[wid] = incl;
    __syncthreads();
    const uint32_t wsc = wave_incl_scan(lane < NW ? comp[lane] : 0u);
    const uint32_t before = wid > 0 ? __shfl(wsc, wid - 1, 64) : 0u;
    const uint32_t excl = before + incl - v;
    int gb = int(excl >> 16), eb = int(excl & 0xffffu);
#pragma unroll
    for (int j = 0; j < kTopkMaxEPT; ++j) {
      const uint32_t key = kr[j];
      const bool g = key != kInvalidKey && key > T;
      const bool e = key != kInvalidKey && key == T;
      if (g || (e && eb < r)) {
        const int pos = gb + min(eb, r);
        stage[pos] = map(p0 + j);
        if (out_scores) stage_sc[pos] = key_float(key);
      }
      gb += g ? 1 : 0;
      eb += e ? 1 : 0;
    }
    __syncthreads();
  }
  for (int i = tid; i < out_cap; i += NT) {
    out[i] = i < kk ? stage[i] : -1;
    if (out_scores) out_scores[i] = i < kk ? stage_sc[i] : 0.0f;
  }
}

}  // namespace tls
