// Work-group top-k selection with lowest-position tie-breaking.
#pragma once

#include "common.hpp"

namespace tls {

__host__ __device__ constexpr int align4w_c(int words) { return (words + 3) & ~3; }

constexpr int kTopkMaxEPT = 16;  // keys per thread: n <= NT * kTopkMaxEPT
constexpr int kTopkMaxNW = 16;   // waves per work-group

// Each radix pass counts into kTopkHistCopies interleaved copies of a 256-bin
// histogram (lane l uses copy l % kTopkHistCopies; copies kTopkHistStride
// words apart so equal digits land in different LDS banks): keys of one
// instruction that share a digit then collide only within their copy.
constexpr int kTopkHistCopies = 4;
constexpr int kTopkHistStride = 257;
constexpr int kTopkHistWords = kTopkHistCopies * kTopkHistStride;  // per pass
constexpr int kTopkPasses = 5;  // histograms: a spread first pass plus up to four 8-bit passes

// LDS words of the scratch area: the passes' histograms (cleared on
// entry), broadcast slots, and the per-(key slot, wave) counts of the ordered
// compaction.
__host__ __device__ constexpr int topk_scratch_words(int /*nt*/) {
  return align4w_c(kTopkPasses * kTopkHistWords) + 64 + 2 * kTopkMaxEPT * kTopkMaxNW;
}

// Round a count of 32-bit LDS words up to a multiple of 4 (16 bytes), so the
// region that follows can be read with 16-byte accesses.
__host__ __device__ constexpr int align4w(int words) { return (words + 3) & ~3; }

// Selects the k largest of the keys held in registers, ties resolved toward
// the lower position, and writes map(position) of the selected positions in
// ascending position order to out[0, k'), k' = min(k, #valid keys), then -1
// up to out_cap.  Thread t holds the keys of positions t + j*NT, j < EPT
// (kInvalidKey marks an empty position, never selected).  out_scores
// (nullable) receives key_float of each selected key.  Each thread writes its
// own selected positions straight to `out` (global memory, or LDS that the
// caller reads after a barrier): no staging and no trailing barrier.  Every
// thread of the work-group must call it, with k uniform.
//
// Method: an MSB-first radix select over the bits where the valid keys
// differ (8-bit digits, LDS histograms) finds the k'-th largest key T and the
// number r of keys equal to T to take.  Every pass counts the keys still in
// play straight from the registers (a key is only compared with the prefix
// found so far, so later passes cost a few compares per key), into a
// histogram of its own; after the pass's one barrier every wave scans that
// histogram itself, so no broadcast and no second barrier follow.  An ordered
// compaction then emits every key > T and the first r keys == T: per (key
// slot j, wave) counts in position order (j-major, then wave, then lane) give
// every key its output index with one barrier, so the output is ordered by
// position without a sort.  When all keys equal to T are taken (r equals
// their count, the usual case) the compaction selects the keys > T - 1 and
// needs one count per key.  SPREAD (with known bounds) replaces the first
// pass by the spread pass described at kTopkSpreadShift.
// The digit of one radix pass: the digit holding the remaining-th largest key
// in play, the number of keys in play in higher digits, and its own count.
struct TopkDigit {
  uint32_t digit, above, cnt;
};

// Run by a whole wave after a pass's histogram is complete: scans the digits
// from the top and returns the pass's digit, the same in every lane.  Lane L
// reads digits 255 - (64 j + L), j < 4 (summed over the histogram copies), so
// the lanes of one read touch consecutive words (no bank conflicts); a wave
// prefix sum per quarter, from the top quarter down, locates the digit.
// Every wave that runs it on the same histogram gets the same answer, so no
// broadcast (and no barrier after it) is needed.
__device__ inline TopkDigit topk_scan_wave(const uint32_t* h, int remaining) {
  const int lane = __lane_id();
  TopkDigit r{255u, 0u, 0u};  // stands in if the histogram held fewer keys than `remaining`
  uint32_t before = 0;        // keys in play in the quarters above (uniform)
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int dgt = 255 - 64 * j - lane;
    uint32_t c = 0;
#pragma unroll
    for (int cp = 0; cp < kTopkHistCopies; ++cp) c += h[cp * kTopkHistStride + dgt];
    const uint32_t incl = wave_incl_scan_u32(c);
    const uint32_t tot = uint32_t(__builtin_amdgcn_readlane(int(incl), 63));
    if (before + tot >= uint32_t(remaining)) {
      // the first lane whose running count reaches `remaining` holds the digit
      const uint64_t hit = __ballot(before + incl >= uint32_t(remaining));
      const int src = __ffsll((unsigned long long)hit) - 1;
      r.digit = uint32_t(255 - 64 * j - src);
      r.above = before + uint32_t(__builtin_amdgcn_readlane(int(incl - c), src));
      r.cnt = uint32_t(__builtin_amdgcn_readlane(int(c), src));
      break;
    }
    before += tot;
  }
  return r;
}

// topk_scan_wave run by one wave, publishing misc[48] = digit, misc[49] =
// keys in higher digits, misc[51] = 1 when the digit's keys are all taken,
// misc[52] = its key count (for the other waves, after a barrier).
__device__ inline void topk_scan_pass(const uint32_t* h, int remaining, uint32_t* misc) {
  const TopkDigit r = topk_scan_wave(h, remaining);
  if (__lane_id() == 0) {
    misc[48] = r.digit;
    misc[49] = r.above;
    misc[51] = r.cnt == uint32_t(remaining) - r.above ? 1u : 0u;
    misc[52] = r.cnt;
  }
}

// Ordered compaction of one tile of keys held in registers (slot j of thread
// t at tile position t + j*NT, position order = j-major, then wave, then
// lane): writes every key > T and, in position order, the keys == T while
// fewer than r ties have been taken, at out[#earlier keys > T + min(#earlier
// ties, r)] (map(j, tile position) gives the value written).  gbase / ebase
// count the keys > T and == T of earlier tiles (uniform); the return value
// holds this tile's counts (x: keys > T, y: keys == T, 0 when r == 0).  One
// work-group barrier inside; cg / ce (LDS) must not be rewritten before every
// thread has returned.
// r == 0 (no key equal to T is taken, the usual case, see wg_topk_regs)
// needs one count per (slot, wave) and one prefix sum.
template <int NT, int EPT, bool TIES, class Map>
__device__ __forceinline__ int2 topk_compact_impl(const uint32_t (&kr)[EPT], uint32_t T, int r, int gbase,
                                                  int ebase, int32_t* out, float* out_scores, Map map,
                                                  uint32_t* cg, uint32_t* ce) {
  constexpr int NW = NT / 64;
  static_assert(NW % ((EPT * NW + 63) / 64) == 0, "keys per thread must keep NW a multiple of PER");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // scalar: the lane reads below take it directly
  constexpr bool ties = TIES;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const uint32_t key = kr[j];
    const uint64_t bg = __ballot(key != kInvalidKey && key > T);
    const uint64_t be = ties ? __ballot(key != kInvalidKey && key == T) : 0ull;
    if (lane == 0) {
      cg[j * NW + wid] = uint32_t(__popcll(bg));
      ce[j * NW + wid] = uint32_t(__popcll(be));
    }
  }
  __syncthreads();
  // exclusive prefix of the (slot, wave) counts in position order; lane L
  // holds entries L*PER .. L*PER+PER-1
  constexpr int NE = EPT * NW;
  constexpr int PER = (NE + 63) / 64;
  uint32_t xg[PER], xe[PER];
  uint32_t sg = 0, se = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int t = lane * PER + q;
    xg[q] = sg;
    xe[q] = se;
    if (t < NE) {
      sg += cg[t];
      if (ties) se += ce[t];
    }
  }
  const uint32_t ig = wave_incl_scan_u32(sg);
  const uint32_t ie = ties ? wave_incl_scan_u32(se) : 0u;
  const int tot_g = __builtin_amdgcn_readlane(int(ig), 63);
  const int tot_e = ties ? __builtin_amdgcn_readlane(int(ie), 63) : 0;
  // entry (j, wid) sits at t = j*NW + wid: lane t / PER, slot t % PER = wid % PER
  uint32_t pg = xg[0], pe = xe[0];
#pragma unroll
  for (int q = 1; q < PER; ++q) {
    if ((wid % PER) == q) {
      pg = xg[q];
      pe = xe[q];
    }
  }
  pg += ig - sg;
  pe += ie - se;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int src = (j * NW + wid) / PER;
    const uint32_t key = kr[j];
    const bool g = key != kInvalidKey && key > T;
    const bool e = ties && key != kInvalidKey && key == T;
    const uint64_t bg = __ballot(g);
    const int gb = gbase + __builtin_amdgcn_readlane(int(pg), src) + lanes_below(bg);
    int eb = 0;
    if (ties) {
      const uint64_t be = __ballot(e);
      eb = ebase + __builtin_amdgcn_readlane(int(pe), src) + lanes_below(be);
    }
    if (g || (e && eb < r)) {
      // (a 32-bit byte offset from the uniform base: pos >= 0)
      const uint32_t off = uint32_t(gb + min(eb, r)) * 4u;
      *reinterpret_cast<int32_t*>(reinterpret_cast<char*>(out) + off) = map(j, tid + j * NT);
      if (out_scores) *reinterpret_cast<float*>(reinterpret_cast<char*>(out_scores) + off) = key_float(key);
    }
  }
  return make_int2(tot_g, tot_e);
}

// Two instances, so that the usual r == 0 case carries none of the tie
// bookkeeping (r is uniform).
template <int NT, int EPT, class Map>
__device__ __forceinline__ int2 topk_compact_tile(const uint32_t (&kr)[EPT], uint32_t T, int r, int gbase,
                                                  int ebase, int32_t* out, float* out_scores, Map map,
                                                  uint32_t* cg, uint32_t* ce) {
  if (r > 0) return topk_compact_impl<NT, EPT, true>(kr, T, r, gbase, ebase, out, out_scores, map, cg, ce);
  return topk_compact_impl<NT, EPT, false>(kr, T, r, gbase, ebase, out, out_scores, map, cg, ce);
}

// Counts the caller already knows about its keys: the number of valid keys
// and bounds lo <= key <= hi of every valid key.  With them the selection
// skips its own statistics pass and barrier; the caller must then have run
// topk_prepare on the scratch area before a work-group barrier.
struct TopkKnown {
  uint32_t cnt, hi, lo;
};

// Spread first pass (wg_topk_regs<..., true>): bucket b of the first pass
// holds the keys with key >> kTopkSpreadShift == base + b, base =
// (hi >> kTopkSpreadShift) - 254, bucket 0 also every key below.  The
// caller's hi bounds every key up to rounding (a sum of products of
// exponentials <= 1, in the bound's own operation order); the bucket of
// headroom above it (an eighth of an octave) keeps a key a few ulps above hi
// in a bucket whose keys the next passes count, so the counts stay
// consistent and the compaction never writes past the k-th output; for the
// keys of non-negative floats (float_key) that is an eighth of an octave
// per bucket over the 32 octaves below the upper bound, where the top-k of
// softmax-like scores spreads over many buckets instead of the few that the
// leading bits of the key span (fewer colliding histogram updates, and
// usually one pass fewer).  Bucket 0 is refined by ordinary passes with the
// keys above its range excluded.
constexpr int kTopkSpreadShift = 20;

template <int NT>
__device__ inline void topk_prepare(uint32_t* scratch) {
  constexpr int kHistAll = align4w_c(kTopkPasses * kTopkHistWords);
  for (int i = threadIdx.x; i < kHistAll; i += NT) scratch[i] = 0u;
}

template <int NT, int EPT, bool SPREAD = false, class Map>
__device__ void wg_topk_regs(const uint32_t (&kr)[EPT], int k, int32_t* out, int out_cap, float* out_scores,
                             Map map, uint32_t* scratch, const TopkKnown* known = nullptr) {
  constexpr int NW = NT / 64;
  static_assert(NW >= 1 && NW <= kTopkMaxNW && EPT >= 1 && EPT <= kTopkMaxEPT, "work-group shape");
  // the ordered compaction gives lane L the (slot, wave) entries L*PER ..
  // L*PER + PER - 1 and finds wave w's entry of every slot at index w % PER,
  // which needs NW to be a multiple of PER
  static_assert(NW % ((EPT * NW + 63) / 64) == 0, "keys per thread must keep NW a multiple of PER");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int kHistAll = align4w_c(kTopkPasses * kTopkHistWords);
  uint32_t* hist = scratch;             // [4 passes][copies][stride]
  uint32_t* misc = scratch + kHistAll;  // [64]: 0..47 wave partials
  uint32_t* cg = misc + 64;             // [EPT][NW] keys > T per (slot, wave)
  uint32_t* ce = cg + kTopkMaxEPT * kTopkMaxNW;  // [EPT][NW] keys == T

  uint32_t cnt = 0, kmx = 0u, kmn = 0xffffffffu;
  if (known) {
    cnt = known->cnt;
    kmx = known->hi;
    kmn = known->lo;
  } else {
    // valid count, max and min valid key over the work-group
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const uint32_t key = kr[j];
      cnt += uint32_t(__popcll(__ballot(key != kInvalidKey)));
      if (key != kInvalidKey) {
        kmx = max(kmx, key);
        kmn = min(kmn, key);
      }
    }
    kmx = wave_max_u32(kmx);
    kmn = wave_min_u32(kmn);
    for (int i = tid; i < kHistAll; i += NT) hist[i] = 0u;
    if (lane == 0) {
      misc[wid] = cnt;
      misc[16 + wid] = kmx;
      misc[32 + wid] = kmn;
    }
    __syncthreads();
    {
      const int w = lane & 15;
      const bool ok = w < NW;
      cnt = combine_waves_sum_u32(ok ? misc[w] : 0u);
      kmx = combine_waves_max_u32(ok ? misc[16 + w] : 0u);
      kmn = combine_waves_min_u32(ok ? misc[32 + w] : 0xffffffffu);
    }
  }
  const int kk = min(k, int(cnt));

  uint32_t prefix = 0u, pmask = 0u;
  int remaining = kk;
  int bits_left = 0;
  // keys equal to the running prefix's bucket: after the last pass, the
  // number of keys equal to T (all valid keys when they are all equal)
  uint32_t cnt_T = cnt;
  uint32_t cap = 0xffffffffu;  // keys above cap are out of play (spread pass, bucket 0)
  int pass = 0;
  if (kk > 0) {
    const uint32_t diff = kmx ^ kmn;
    bits_left = diff ? 32 - __clz(diff) : 0;
    pmask = bits_left >= 32 ? 0u : ~((1u << bits_left) - 1u);
    prefix = kmx & pmask;
  }
  if (SPREAD && kk > 0 && int(kmx >> kTopkSpreadShift) - int(kmn >> kTopkSpreadShift) > 254) {
    constexpr int fs = kTopkSpreadShift;
    const int base = int(kmx >> fs) - 254;  // above kmn's bucket: bucket 0 is clamped
    uint32_t* h = hist;
    uint32_t* hc = h + (lane % kTopkHistCopies) * kTopkHistStride;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const uint32_t key = kr[j];
      // (clamped to the 256 buckets also if a key exceeded the stated bound)
      if (key != kInvalidKey) atomicAdd(&hc[min(max(int(key >> fs) - base, 0), 255)], 1u);
    }
    __syncthreads();
    const TopkDigit dg = topk_scan_wave(h, remaining);
    remaining -= int(dg.above);
    cnt_T = dg.cnt;
    pass = 1;
    uint32_t lowest;  // the smallest key the bucket can hold
    if (dg.digit > 0) {
      lowest = uint32_t(base + int(dg.digit)) << fs;
      prefix = lowest;
      pmask = ~((1u << fs) - 1u);
      bits_left = fs;
    } else {
      lowest = kmn;
      cap = (uint32_t(base + 1) << fs) - 1u;
      bits_left = 32 - __clz(kmn ^ cap);
      pmask = bits_left >= 32 ? 0u : ~((1u << bits_left) - 1u);
      prefix = cap & pmask;
    }
    if (dg.cnt == uint32_t(remaining)) {
      // the bucket is taken whole (lowest >= 1: valid keys are >= 1)
      prefix = lowest - 1u;
      remaining = 0;
      bits_left = 0;
    }
  }
  // 8-bit passes, each on its own histogram: a wave still scanning pass p's
  // histogram never sees pass p+1's counts
  for (; bits_left > 0; ++pass) {
    const int nb = bits_left < 8 ? bits_left : 8;
    const int shift = bits_left - nb;
    const uint32_t dmask = (1u << nb) - 1u;
    uint32_t* h = hist + kTopkHistWords * pass;
    uint32_t* hc = h + (lane % kTopkHistCopies) * kTopkHistStride;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const uint32_t key = kr[j];
      // the digit as the 8 bits at `shift`: in a last pass narrower than 8
      // bits (shift 0) the upper bits are prefix bits that every key in play
      // shares, so the buckets keep their order and OR-ing the found digit
      // into the prefix below changes nothing else (one v_bfe_u32 with an
      // inline width)
      if (key != kInvalidKey && (key & pmask) == prefix && (!SPREAD || key <= cap))
        atomicAdd(&hc[__builtin_amdgcn_ubfe(key, uint32_t(shift), 8u)], 1u);
    }
    __syncthreads();
    const TopkDigit dg = topk_scan_wave(h, remaining);
    prefix |= dg.digit << shift;
    remaining -= int(dg.above);
    pmask |= dmask << shift;
    bits_left -= nb;
    cnt_T = dg.cnt;
    if (dg.cnt == uint32_t(remaining) && bits_left > 0 && prefix != 0u) {
      // the threshold's bucket is taken whole: every key >= prefix is
      // selected, i.e. T = prefix - 1 with no equal keys to take
      prefix -= 1u;
      remaining = 0;
      bits_left = 0;
    }
  }
  uint32_t T = prefix;
  int r = remaining;  // keys equal to T still to take, lowest positions first
  if (r > 0 && uint32_t(r) == cnt_T) {
    // every key equal to T is taken: select the keys > T - 1 instead, which
    // the compaction handles with one count per key (valid keys are >= 1)
    T -= 1u;
    r = 0;
  }

  if (kk > 0) topk_compact_tile<NT, EPT>(kr, T, r, 0, 0, out, out_scores, map, cg, ce);
  for (int i = kk + tid; i < out_cap; i += NT) {
    out[i] = -1;
    if (out_scores) out_scores[i] = 0.0f;
  }
}

// The same selection over keys[0, n) in global memory, for more keys than
// the registers hold (token-level selection over a whole context): every
// pass streams the keys in tiles of NT*16; after the first pass the keys
// still in play are gathered into `list` (LDS, list_cap words) when they fit,
// so later passes read only those; the ordered compaction then walks the
// tiles in position order with running counts.  Writes the selected
// positions ascending to out[0, k'), then -1 up to out_cap.
template <int NT>
__device__ void wg_topk_global(const uint32_t* __restrict__ keys, int n, int k, int32_t* out, int out_cap,
                               uint32_t* scratch, uint32_t* list, int list_cap) {
  constexpr int NW = NT / 64;
  constexpr int EPT = kTopkMaxEPT;
  constexpr int TILE = NT * EPT;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int kHistAll = align4w_c(kTopkPasses * kTopkHistWords);
  uint32_t* hist = scratch;
  uint32_t* misc = scratch + kHistAll;
  uint32_t* cg = misc + 64;
  uint32_t* ce = cg + kTopkMaxEPT * kTopkMaxNW;
  const int ntiles = (n + TILE - 1) / TILE;
  auto load_tile = [&](int t, uint32_t (&kr)[EPT]) {
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const int p = t * TILE + tid + j * NT;
      kr[j] = p < n ? keys[p] : kInvalidKey;
    }
  };

  uint32_t cnt = 0, kmx = 0u, kmn = 0xffffffffu;
  for (int t = 0; t < ntiles; ++t) {
    uint32_t kr[EPT];
    load_tile(t, kr);
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const uint32_t key = kr[j];
      cnt += uint32_t(__popcll(__ballot(key != kInvalidKey)));
      if (key != kInvalidKey) {
        kmx = max(kmx, key);
        kmn = min(kmn, key);
      }
    }
  }
  kmx = wave_max_u32(kmx);
  kmn = wave_min_u32(kmn);
  for (int i = tid; i < kHistAll; i += NT) hist[i] = 0u;
  if (lane == 0) {
    misc[wid] = cnt;
    misc[16 + wid] = kmx;
    misc[32 + wid] = kmn;
  }
  if (tid == 0) misc[50] = 0u;
  __syncthreads();
  {
    const int w = lane & 15;
    const bool ok = w < NW;
    cnt = combine_waves_sum_u32(ok ? misc[w] : 0u);
    kmx = combine_waves_max_u32(ok ? misc[16 + w] : 0u);
    kmn = combine_waves_min_u32(ok ? misc[32 + w] : 0xffffffffu);
  }
  const int kk = min(k, int(cnt));
  uint32_t prefix = 0u, pmask = 0u;
  int remaining = kk, bits_left = 0;
  if (kk > 0) {
    const uint32_t diff = kmx ^ kmn;
    bits_left = diff ? 32 - __clz(diff) : 0;
    pmask = bits_left >= 32 ? 0u : ~((1u << bits_left) - 1u);
    prefix = kmx & pmask;
  }
  int list_n = -1;  // < 0: the keys in play are read from global memory
  uint32_t cnt_T = cnt;  // as in wg_topk_regs
  for (int pass = 0; bits_left > 0; ++pass) {
    const int nb = bits_left < 8 ? bits_left : 8;
    const int shift = bits_left - nb;
    const uint32_t dmask = (1u << nb) - 1u;
    uint32_t* h = hist + kTopkHistWords * pass;
    uint32_t* hc = h + (lane % kTopkHistCopies) * kTopkHistStride;
    if (list_n < 0) {
      for (int t = 0; t < ntiles; ++t) {
        uint32_t kr[EPT];
        load_tile(t, kr);
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
          const uint32_t key = kr[j];
          if (key != kInvalidKey && (key & pmask) == prefix)
            atomicAdd(&hc[__builtin_amdgcn_ubfe(key, uint32_t(shift), 8u)], 1u);  // as in wg_topk_regs
        }
      }
    } else {
      for (int i = tid; i < list_n; i += NT) {
        const uint32_t key = list[i];
        if ((key & pmask) == prefix) atomicAdd(&hc[__builtin_amdgcn_ubfe(key, uint32_t(shift), 8u)], 1u);
      }
    }
    __syncthreads();
    if (wid == 0) topk_scan_pass(h, remaining, misc);
    __syncthreads();
    prefix |= misc[48] << shift;
    remaining -= int(misc[49]);
    pmask |= dmask << shift;
    bits_left -= nb;
    cnt_T = misc[52];
    if (misc[51] && bits_left > 0 && prefix != 0u) {
      prefix -= 1u;
      remaining = 0;
      bits_left = 0;
    }
    if (list_n < 0 && bits_left > 0 && int(misc[52]) <= list_cap) {
      for (int t = 0; t < ntiles; ++t) {
        uint32_t kr[EPT];
        load_tile(t, kr);
        uint32_t wcount = 0;
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
          const uint32_t key = kr[j];
          wcount += uint32_t(__popcll(__ballot(key != kInvalidKey && (key & pmask) == prefix)));
        }
        uint32_t base = 0;
        if (lane == 0 && wcount) base = atomicAdd(&misc[50], wcount);
        base = uint32_t(__builtin_amdgcn_readfirstlane(int(base)));
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
          const uint32_t key = kr[j];
          const bool in = key != kInvalidKey && (key & pmask) == prefix;
          const uint64_t bal = __ballot(in);
          if (in) list[base + lanes_below(bal)] = key;
          base += uint32_t(__popcll(bal));
        }
      }
      __syncthreads();
      list_n = int(misc[50]);
    }
  }
  uint32_t T = prefix;
  int r = remaining;
  if (r > 0 && uint32_t(r) == cnt_T) {
    T -= 1u;
    r = 0;
  }
  if (kk > 0) {
    int gbase = 0, ebase = 0;
    for (int t = 0; t < ntiles; ++t) {
      uint32_t kr[EPT];
      load_tile(t, kr);
      const int2 c = topk_compact_tile<NT, EPT>(kr, T, r, gbase, ebase, out, nullptr,
                                                [=](int, int p) { return int32_t(t * TILE + p); }, cg, ce);
      gbase += c.x;
      ebase += c.y;
      __syncthreads();  // cg / ce are rewritten by the next tile
    }
  }
  for (int i = kk + tid; i < out_cap; i += NT) out[i] = -1;
}

}  // namespace tls
