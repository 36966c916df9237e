// Work-group top-k selection with lowest-position tie-breaking.
#pragma once

#include "common.hpp"

namespace tls {

constexpr int kTopkMaxEPT = 16;  // keys per thread: n <= NT * kTopkMaxEPT

// LDS words the selection needs: four 256-bin histograms (one per radix
// pass, cleared once up front) and broadcast slots.
__host__ __device__ constexpr int topk_scratch_words(int /*nt*/) { return 4 * 256 + 64 + 32; }

// Round a count of 32-bit LDS words up to a multiple of 4 (16 bytes), so the
// region that follows can be read with 16-byte accesses.
__host__ __device__ constexpr int align4w(int words) { return (words + 3) & ~3; }

// Selects the k largest keys among keys[0, n) (LDS; kInvalidKey entries never
// count), ties resolved toward the lower position, and writes map(position)
// of the selected positions in ascending position order to out[0, k'),
// k' = min(k, #valid keys), then -1 up to out_cap.  out_scores (nullable)
// receives key_float of each selected key.  `stage` (LDS, out_cap ints) and
// `stage_sc` (LDS, out_cap floats, when scores are wanted) hold the result
// until one final copy, because a work-group barrier waits for outstanding
// global stores.  Every thread of the work-group must call it, with n and k
// uniform.
//
// Method: each thread keeps the keys of positions [tid*ept, tid*ept + ept)
// in registers.  An MSB-first radix select over the bits where the valid keys
// differ (8-bit digits, LDS histograms) finds the k'-th largest key T and the
// number r of keys equal to T to take; an ordered compaction (one prefix sum
// of per-thread counts) then emits every key > T and the first r keys == T.
// The output is ordered by position, so no sort is needed.  Wave-level
// reductions and scans use DPP moves, ballots and lane reads; cross-wave
// values go through one LDS word per wave.
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
  if ((ept & 3) == 0 && (reinterpret_cast<uintptr_t>(keys) & 15u) == 0) {
    // 16-byte reads; p0 is a multiple of 4, so they are aligned
#pragma unroll
    for (int v = 0; v < kTopkMaxEPT / 4; ++v) {
      uint4 w = make_uint4(kInvalidKey, kInvalidKey, kInvalidKey, kInvalidKey);
      if (4 * v < ept && p0 + 4 * v + 3 < n) {
        w = *reinterpret_cast<const uint4*>(keys + p0 + 4 * v);
      } else if (4 * v < ept) {
        if (p0 + 4 * v < n) w.x = keys[p0 + 4 * v];
        if (p0 + 4 * v + 1 < n) w.y = keys[p0 + 4 * v + 1];
        if (p0 + 4 * v + 2 < n) w.z = keys[p0 + 4 * v + 2];
      }
      kr[4 * v] = w.x;
      kr[4 * v + 1] = w.y;
      kr[4 * v + 2] = w.z;
      kr[4 * v + 3] = w.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTopkMaxEPT; ++j) kr[j] = (j < ept && p0 + j < n) ? keys[p0 + j] : kInvalidKey;
  }
  for (int i = tid; i < 1024; i += NT) hist[i] = 0u;

  // valid count, max and min valid key over the work-group
  uint32_t cnt = 0, kmx = 0u, kmn = 0xffffffffu;
#pragma unroll
  for (int j = 0; j < kTopkMaxEPT; ++j) {
    const uint32_t key = kr[j];
    cnt += uint32_t(__popcll(__ballot(key != kInvalidKey)));
    if (key != kInvalidKey) {
      kmx = max(kmx, key);
      kmn = min(kmn, key);
    }
  }
  kmx = wave_max_u32(kmx);
  kmn = wave_min_u32(kmn);
  if (lane == 0) {
    misc[wid] = cnt;
    misc[16 + wid] = kmx;
    misc[32 + wid] = kmn;
  }
  __syncthreads();
  {
    const uint32_t a = misc[lane & 15], b = misc[16 + (lane & 15)], c = misc[32 + (lane & 15)];
    cnt = 0;
    kmx = 0u;
    kmn = 0xffffffffu;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      cnt += uint32_t(__builtin_amdgcn_readlane(int(a), w));
      kmx = max(kmx, uint32_t(__builtin_amdgcn_readlane(int(b), w)));
      kmn = min(kmn, uint32_t(__builtin_amdgcn_readlane(int(c), w)));
    }
  }
  const int kk = min(k, int(cnt));

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
      uint32_t tot;
      const uint32_t incl = wave_incl_scan_small<15>(local, &tot);
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
      if (lane == src) {
        misc[48] = uint32_t(found);
        misc[49] = found_above;
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
    uint32_t gtot, etot;
    const uint32_t gin = wave_incl_scan_small<5>(gt, &gtot);
    const uint32_t ein = wave_incl_scan_small<5>(eq, &etot);
    if (lane == 0) comp[wid] = (gtot << 16) | etot;  // totals < 2^16
    __syncthreads();
    const uint32_t cw = comp[lane & 15];
    uint32_t gb0 = 0, eb0 = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t t = uint32_t(__builtin_amdgcn_readlane(int(cw), w));
      if (w < wid) {
        gb0 += t >> 16;
        eb0 += t & 0xffffu;
      }
    }
    int gb = int(gb0 + gin - gt), eb = int(eb0 + ein - eq);
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
