// The fused two-level selection body for grouped-query layouts (launched by
// token_select_mfma_kernel).
#pragma once

#include "token_common.hpp"

namespace tls {

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

constexpr int kSelNT = 1024;
constexpr int kSelNW = kSelNT / 64;
constexpr int kSelSPT = 8;  // candidate slots per thread
constexpr int kSelMaxSlots = kSelNT * kSelSPT;
constexpr int kSelBPT = 2;  // block scores per thread
constexpr int kSelMaxBlocks = kSelNT * kSelBPT;
constexpr int kSelMaxG = 4;
constexpr size_t kSelMaxLds = 160 * 1024;
constexpr uint32_t kBf16Base = 0x43434343u;  // high byte of bf16(128 + c), c < 16

// Element order of one 4-channel k-slice: within the 8 channels of code dword
// w, slice 2w holds channels (0, 2, 1, 3) and slice 2w+1 channels (4, 6, 5, 7)
// (offsets from 8w): the low nibbles of two bytes, then their high nibbles.
// slice_chan(j) = {0, 2, 1, 3, 4, 6, 5, 7}[j], computed (a table would be one
// more dependent memory request in the prologue).
__device__ inline int slice_chan(int j) { return (j & 4) | ((j & 1) << 1) | ((j >> 1) & 1); }

// LDS words: top-k scratch | block list | q~ table (4 heads x 32 channels of
// bf16, in slice order) | the heads' q~ sums (4) | per-wave partials.
inline size_t mfma_select_lds_bytes(int K_b) {
  return (size_t(topk_scratch_words(kSelNT)) + size_t(align4w(K_b)) + 64 + 4 + kSelNW * 12) * sizeof(uint32_t);
}

// The fused selection of one unit by a 1024-thread work-group, on LDS
// `smem` (mfma_select_lds_bytes).  WB: B >= 64 (whole blocks per wave).
template <int G, bool WB>
__device__ inline void token_select_mfma_body(
    uint32_t* smem, const uint16_t* __restrict__ q, const uint8_t* __restrict__ codes,
    const float* __restrict__ qparams, const int32_t* __restrict__ channels, const float* __restrict__ block_scores,
    const int32_t* __restrict__ block_ids_in, int32_t* __restrict__ block_ids_out,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int d, int B, int T, int m_max, int K_b, int K_t,
    float sigma, int32_t* __restrict__ token_ids, float* __restrict__ token_scores, uint32_t* err, const int unit) {
  constexpr int NT = kSelNT, NW = kSelNW;
  uint32_t* scratch = smem;
  int32_t* s_bl = reinterpret_cast<int32_t*>(smem + topk_scratch_words(NT));
  uint16_t* s_qt = reinterpret_cast<uint16_t*>(s_bl + align4w(K_b));  // [4][32] (64 words)
  float* s_qsum = reinterpret_cast<float*>(s_qt + 128);                   // [4]
  float* s_red = s_qsum + 4;                                              // [NW][12]
  const int S = K_b * B;

  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (tid == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int m = (n + B - 1) / B;
  const int lgB = __builtin_ctz(unsigned(B));  // B is a power of two here
  const float sigma2 = sigma * 1.4426950408889634f;  // logits in base 2

  // block scores (requested first: the longest dependency); every lane loads
  // from a clamped index, so that both requests leave before either is used
  float bsv[kSelBPT] = {};
  if (block_scores) {
    const float* sc = block_scores + size_t(unit) * m_max;
#pragma unroll
    for (int j = 0; j < kSelBPT; ++j) bsv[j] = sc[min(tid + j * NT, m_max - 1)];
  }
  // q~ entries in slice order: entry (h, 4k + e) = q[h][C[8(k/2) + slice_chan(4(k%2) + e)]]
  // (channel id, then the query element: two dependent requests; the
  // element is written to LDS only after the block top-k, which hides it)
  const bool qt_lane = tid < 4 * 32 && (tid >> 5) < G;
  int ch = 0;
  if (qt_lane) {
    const int x = tid & 31, k = x >> 2, e = x & 3;
    ch = channels[g * 32 + 8 * (k >> 1) + slice_chan(4 * (k & 1) + e)];
    if (ch < 0 || ch >= d) {
      set_error(err, 32u);
      ch = 0;
    }
  }
  if (block_ids_in) {
    // the candidate blocks are given (with block scores too: the lagged
    // operator, whose new block selection goes to block_ids_out)
    for (int i = tid; i < K_b; i += NT) {
      int b = block_ids_in[size_t(unit) * K_b + i];
      if (b >= m) {
        set_error(err, 2u);
        b = -1;
      }
      s_bl[i] = b < 0 ? -1 : b;
    }
  }
  // the scores are consumed here on every path (not only inside the branches
  // below), so that no later wait has to cover their loads
#pragma unroll
  for (int j = 0; j < kSelBPT; ++j) asm volatile("" : : "v"(bsv[j]));
  uint32_t bk[kSelBPT];
  if (block_scores) {
#pragma unroll
    for (int j = 0; j < kSelBPT; ++j) bk[j] = tid + j * NT < m ? float_key(bsv[j]) : kInvalidKey;
  }
  // the query elements are requested only now: every earlier request is
  // consumed above, so no wait before the block top-k covers these
  __builtin_amdgcn_sched_barrier(0);
  uint16_t qv = 0;
  if (qt_lane) qv = q[(size_t(s) * H_q + size_t(g) * G + (tid >> 5)) * d + ch];
  if (block_scores) {
    int32_t* dst = block_ids_in ? block_ids_out + size_t(unit) * K_b : s_bl;
    wg_topk_regs<NT, kSelBPT>(bk, K_b, dst, K_b, nullptr, [](int, int i) { return int32_t(i); }, scratch);
  }
  if (tid < 4 * 32) {
    s_qt[tid] = qv;
    // the head's q~ sum, over the 32 lanes holding its channels
    float sum = __uint_as_float(uint32_t(qv) << 16);
#pragma unroll
    for (int m = 16; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 32);
    if ((tid & 31) == 0) s_qsum[tid >> 5] = sum;
  }
  __syncthreads();

  // A operands (row = head lane%4, slice k: four bf16 channels, as they lie
  // in the table) and the per-head q~ sums
  i16x4_t qa[8];
  float qsum[4];
  {
    const uint2* row = reinterpret_cast<const uint2*>(s_qt + (lane & 3) * 32);
#pragma unroll
    for (int k = 0; k < 8; ++k) qa[k] = __builtin_bit_cast(i16x4_t, row[k]);
    const float4 qs = *reinterpret_cast<const float4*>(s_qsum);
    qsum[0] = qs.x;
    qsum[1] = qs.y;
    qsum[2] = qs.z;
    qsum[3] = qs.w;
  }

  // 1. index rows of the owned slots
  uint4 cw[kSelSPT];
  float2 qp[kSelSPT];
  int32_t tokpos[kSelSPT];  // token position of each owned slot (for the output)
  uint32_t vmask = 0;
  if constexpr (WB) {
    // B >= 64: the 64 slots a wave owns for one i lie in one block, so the
    // block id and the row base are wave-uniform (scalar).  Every lane loads
    // unconditionally from a row inside the unit's index (row 0 for an empty
    // list entry, at most T - 1 past the context); vmask drops those slots.
    const int wv = __builtin_amdgcn_readfirstlane(wid);
    // lane j < 8 reads the wave's block-list entry for slot group j (one LDS
    // round trip for all eight)
    const int blv = s_bl[min((wv * 64 + (lane & 7) * NT) >> lgB, K_b - 1)];
    // (32-bit byte offsets from the unit's base: T is far below 2^28 rows)
    const uint8_t* ucodes = codes + size_t(unit) * T * 16;
    const uint8_t* uqp = reinterpret_cast<const uint8_t*>(qparams + size_t(unit) * T * 2);
#pragma unroll
    for (int i = 0; i < kSelSPT; ++i) {
      const int s0 = wv * 64 + i * NT;  // the wave's first slot (uniform)
      const int blk = s0 < S ? __builtin_amdgcn_readlane(blv, i) : -1;
      const int tok = blk * B + (s0 & (B - 1)) + lane;
      tokpos[i] = tok;
      const bool ok = blk >= 0 && tok < n;
      const uint32_t rr = blk < 0 ? 0u : uint32_t(min(tok, T - 1));
      cw[i] = ld16_stream(ucodes + (rr << 4));
      const float* pr = reinterpret_cast<const float*>(uqp + (rr << 3));
      qp[i] = make_float2(__builtin_nontemporal_load(pr), __builtin_nontemporal_load(pr + 1));
      vmask |= ok ? 1u << i : 0u;
    }
    // every row request leaves before the first use waits on them
    __builtin_amdgcn_sched_barrier(0);
  } else {
#pragma unroll
    for (int i = 0; i < kSelSPT; ++i) {
      const int slot = tid + i * NT;
      const int e = slot >> lgB, o = slot & (B - 1);
      cw[i] = make_uint4(0, 0, 0, 0);
      qp[i] = make_float2(0.f, 0.f);
      tokpos[i] = -1;
      if (slot < S) {
        const int blk = s_bl[e];
        const int tok = blk * B + o;
        tokpos[i] = tok;
        if (blk >= 0 && tok < n) {
          const size_t r = size_t(unit) * T + tok;
          cw[i] = ld16_stream(codes + r * 16);
          const float* pr = qparams + r * 2;
          qp[i] = make_float2(__builtin_nontemporal_load(pr), __builtin_nontemporal_load(pr + 1));
          vmask |= 1u << i;
        }
      }
    }
  }

  // 2. dots on the matrix cores, logits, per-head max
  float qs2[G];
#pragma unroll
  for (int h = 0; h < G; ++h) qs2[h] = sigma2 * qsum[h];
  float lg[kSelSPT][G];
  float mx[G];
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = -INFINITY;
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i) {
    const uint32_t wd[4] = {cw[i].x, cw[i].y, cw[i].z, cw[i].w};
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t lo = wd[w] & 0x0f0f0f0fu, hi = (wd[w] >> 4) & 0x0f0f0f0fu;
      const u32x2_t b0 = {__builtin_amdgcn_perm(kBf16Base, lo, 0x04010400u),
                          __builtin_amdgcn_perm(kBf16Base, hi, 0x04010400u)};
      const u32x2_t b1 = {__builtin_amdgcn_perm(kBf16Base, lo, 0x04030402u),
                          __builtin_amdgcn_perm(kBf16Base, hi, 0x04030402u)};
      acc = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(qa[2 * w], __builtin_bit_cast(i16x4_t, b0), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(qa[2 * w + 1], __builtin_bit_cast(i16x4_t, b1), acc, 0, 0, 0);
    }
    const bool valid = (vmask >> i) & 1u;
    // sigma (base 2) folded into the slot's scale and the heads' q~ sums
    const float sc = sigma2 * qp[i].x, off = qp[i].y - 128.0f * qp[i].x;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      lg[i][h] = valid ? fmaf(sc, acc[h], off * qs2[h]) : -INFINITY;
      mx[h] = fmaxf(mx[h], lg[i][h]);
    }
  }
  const uint32_t wcnt = wave_reduce_bits(uint32_t(__popc(vmask)), [](uint32_t a, uint32_t b) { return a + b; });
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const int w = wave_max_ord(mx[h]);  // order-preserving int form
    if (lane == 0) s_red[wid * 12 + h] = __int_as_float(w);
  }
  if (lane == 0) s_red[wid * 12 + 8] = __uint_as_float(wcnt);
  __syncthreads();
  static_assert(NW == 16, "one wave value per lane of a 16-lane row");
#pragma unroll
  for (int h = 0; h < G; ++h) {
    mx[h] = ord_f32(combine_waves_max_i32(__float_as_int(s_red[(lane & 15) * 12 + h])));
    if (mx[h] == -INFINITY) mx[h] = 0.f;  // no candidate: every logit is -inf, every exponential 0
  }
  const uint32_t n_valid = combine_waves_sum_u32(__float_as_uint(s_red[(lane & 15) * 12 + 8]));
  // 3. exponentials (base 2: the logits carry log2(e)) and their per-head sums
  float sum[G];
#pragma unroll
  for (int h = 0; h < G; ++h) sum[h] = 0.f;
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float e = __builtin_amdgcn_exp2f(lg[i][h] - mx[h]);  // 0 for an empty slot (logit -inf)
      lg[i][h] = e;
      sum[h] += e;
    }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float w = wave_sum_f32(sum[h]);
    if (lane == 0) s_red[wid * 12 + 4 + h] = w;
  }
  topk_prepare<NT>(scratch);  // the token top-k's histograms, cleared before the barrier below
  __syncthreads();
  float iz[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float Z = combine_waves_sum_f32(s_red[(lane & 15) * 12 + 4 + h]);
    iz[h] = Z > 0.f ? __builtin_amdgcn_rcpf(Z) : 0.f;
  }
  // 4. alpha keys in registers, top-K_t
  // Every alpha lies in [0, bound] with bound = (1/G) sum_h 1/Z_h, evaluated in
  // the same operation order (each exponential is <= 1 and rounding is
  // monotone), so the top-k needs no statistics pass of its own.  A NaN alpha
  // (NaN inputs only; arithmetic NaNs are quiet) ranks as 0: fmaxf(alpha, 0)
  // is then 0, and for alpha >= +0 the key bits | 2^31 equal float_key.
  const float invG = 1.0f / float(G);
  float bsum = 0.f;
#pragma unroll
  for (int h = 0; h < G; ++h) bsum = fmaf(1.0f, iz[h], bsum);
  uint32_t keys[kSelSPT];
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i) {
    float a = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h) a = fmaf(lg[i][h], iz[h], a);
    const float av = fmaxf(a * invG, 0.f);
    keys[i] = ((vmask >> i) & 1u) ? (__float_as_uint(av) | 0x80000000u) : kInvalidKey;
  }
  const TopkKnown known{n_valid, float_key(bsum * invG), float_key(0.f)};
  wg_topk_regs<NT, kSelSPT, true>(keys, K_t, token_ids + size_t(unit) * K_t, K_t,
                            token_scores ? token_scores + size_t(unit) * K_t : nullptr,
                            [&](int j, int) { return tokpos[j]; }, scratch, &known);
  if (block_scores && !block_ids_in && block_ids_out)
    for (int i = tid; i < K_b; i += NT) block_ids_out[size_t(unit) * K_b + i] = s_bl[i];
}

}  // namespace tls
