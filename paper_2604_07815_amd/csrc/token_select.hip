// Fine token selection inside the selected blocks (AsyncTLS Sec. 4.1).
//
// Candidate slots of a unit: slot = i*B + o for the i-th entry of its block
// list and offset o; the slot is a valid candidate when that entry is a
// block id >= 0 and token id*B + o < ctx_len.  With an ascending block list,
// slot order is token order, so lowest-slot tie-breaking is lowest-position
// tie-breaking.
//
// token_score_kernel: per slot and head, l = sigma * q~_h . dequant(code_j).
//   With dequant = min + code*scale per 32-channel group this is
//   sigma * sum_grp (min_grp * sum_c q~_hc + scale_grp * sum_c q~_hc code_c):
//   the integer codes enter the dot product directly.  Also emits each
//   work-group's per-head (max, sum exp) of its slots.
// token_alpha_kernel: per-head normalisers over all candidates, then
//   alpha_j = (1/G) sum_h exp(l_hj - m_h) / Z_h as an orderable key.
// token_topk_kernel: the K_t largest alpha, ascending token positions.
#include "token_common.hpp"

namespace tls {

constexpr int kMaxG = 32;
constexpr int kMaxGroups = 8;  // d_c <= 256

template <class E>
__global__ __launch_bounds__(256) void token_score_kernel(
    const typename E::T* __restrict__ q, const uint8_t* __restrict__ codes, const float* __restrict__ qparams,
    const int32_t* __restrict__ channels, const int32_t* __restrict__ block_ids, int K_b,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int G, int d, int d_c, int B, int T, float sigma,
    float* __restrict__ logits, float* __restrict__ stats, uint32_t* err) {
  __shared__ float s_qt[kMaxG * 256];
  __shared__ float s_qsum[kMaxG * kMaxGroups];
  __shared__ float s_red[4 * kMaxG];
  __shared__ int s_ch[kMaxGroups * 32];
  const int unit = blockIdx.y, chunk = blockIdx.x;
  const int s = unit / H_kv, g = unit % H_kv;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  const int ngr = d_c / 32;
  const int S = K_b * B;
  const typename E::T* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
  // the group's channel ids once (every head uses the same), then the q~ gather
  if (threadIdx.x < d_c) {
    int ch = channels[g * d_c + threadIdx.x];
    if (ch < 0 || ch >= d) {  // caller-supplied channel id out of range
      set_error(err, 32u);
      ch = 0;
    }
    s_ch[threadIdx.x] = ch;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < G * d_c; i += 256) {
    const int h = i / d_c, c = i % d_c;
    s_qt[i] = E::to_f(qg[size_t(h) * d + s_ch[c]]);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < G * ngr; i += 256) {
    const int h = i / ngr, gr = i % ngr;
    float acc = 0.f;
    for (int c = 0; c < 32; ++c) acc += s_qt[h * d_c + gr * 32 + c];
    s_qsum[i] = acc;
  }
  __syncthreads();

  const int slot = chunk * kTokenSlotsPerWG + threadIdx.x;
  const int32_t* bl = block_ids + size_t(unit) * K_b;
  int tok = 0;
  const bool valid = slot < S && slot_token(bl, K_b, B, m, n, slot, &tok, err);
  float acc[kMaxG];
#pragma unroll
  for (int h = 0; h < kMaxG; ++h) acc[h] = 0.f;
  if (valid) {
    const size_t row = size_t(unit) * T + tok;
    const uint8_t* crow = codes + row * (d_c / 2);
    const float* prow = qparams + row * ngr * 2;
    for (int gr = 0; gr < ngr; ++gr) {
      const uint4 cw = ld16_stream(crow + gr * 16);
      const float scale = prow[gr * 2 + 0], mn = prow[gr * 2 + 1];
      float cf[32];
      unpack_nibbles8(cw.x, cf + 0);
      unpack_nibbles8(cw.y, cf + 8);
      unpack_nibbles8(cw.z, cf + 16);
      unpack_nibbles8(cw.w, cf + 24);
#pragma unroll
      for (int h = 0; h < kMaxG; ++h) {
        if (h < G) {
          const float* qt = s_qt + h * d_c + gr * 32;
          float dot = 0.f;
#pragma unroll
          for (int c = 0; c < 32; ++c) dot = fmaf(qt[c], cf[c], dot);
          acc[h] += mn * s_qsum[h * ngr + gr] + scale * dot;
        }
      }
    }
  }
  // logits and this work-group's per-head softmax statistics
  float* lg = logits + size_t(unit) * G * S;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int h = 0; h < kMaxG; ++h) {
    if (h < G) {
      const float l = valid ? sigma * acc[h] : -INFINITY;
      acc[h] = l;
      if (slot < S) lg[size_t(h) * S + slot] = l;
      const float wm = wave_max<64>(l);
      if (lane == 0) s_red[wid * kMaxG + h] = wm;
    }
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < kMaxG; ++h) {
    if (h < G) {
      const float M = fmaxf(fmaxf(s_red[h], s_red[kMaxG + h]), fmaxf(s_red[2 * kMaxG + h], s_red[3 * kMaxG + h]));
      acc[h] = (valid && M != -INFINITY) ? __expf(acc[h] - M) : 0.f;
    }
  }
  __syncthreads();
  __shared__ float s_sum[4 * kMaxG];
#pragma unroll
  for (int h = 0; h < kMaxG; ++h) {
    if (h < G) {
      const float ws = wave_sum<64>(acc[h]);
      if (lane == 0) s_sum[wid * kMaxG + h] = ws;
    }
  }
  __syncthreads();
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    const float M = fmaxf(fmaxf(s_red[h], s_red[kMaxG + h]), fmaxf(s_red[2 * kMaxG + h], s_red[3 * kMaxG + h]));
    const float Z = ((s_sum[h] + s_sum[kMaxG + h]) + s_sum[2 * kMaxG + h]) + s_sum[3 * kMaxG + h];
    float* st = stats + ((size_t(unit) * gridDim.x + chunk) * G + h) * 2;
    st[0] = M;
    st[1] = Z;
  }
}

// The same logits and statistics with the code contraction on the matrix
// cores, for bf16 with G a multiple of 16 (the absorbed MLA layout: 32 heads
// over d_c = 128 channels).  A work-group (4 waves) takes 256 slots; each
// wave takes four 16-slot tiles.  Per tile and 32-channel group,
// v_mfma_f32_16x16x32_bf16 with A = q~ (16 heads x 32 channels, exact in
// bf16) and B = the tile's codes, entering as the bf16 number 128 + c (one
// byte permute per two codes; exact) gives dot'_hj = dot_hj + 128 sum_c q~_hc,
// so per group l gains sigma (scale_j dot'_hj + (min_j - 128 scale_j) qsum_h).
// Lane (g, i) of the result holds slot i of the tile for heads 4g..4g+3.
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 ts_bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float ts_f32x4_t;
typedef uint32_t ts_u32x4_t __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ inline float dpp_row_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int HT, int NGR>
__global__ __launch_bounds__(256) void token_score_mfma_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ codes, const float* __restrict__ qparams,
    const int32_t* __restrict__ channels, const int32_t* __restrict__ block_ids, int K_b,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int d, int B, int T, float sigma,
    float* __restrict__ logits, float* __restrict__ stats, uint32_t* err) {
  constexpr int G = 16 * HT, DC = 32 * NGR;
  constexpr uint32_t kBase = 0x43434343u;  // high byte of bf16(128 + c), c < 16
  // q~ in operand order: [head][group][lane group g][8], channel g*8 + {0,2,4,6,1,3,5,7}
  __shared__ __attribute__((aligned(16))) uint16_t s_qt[G * DC];
  __shared__ float s_qs[G * NGR];
  __shared__ float s_red[4][G][2];
  const int unit = blockIdx.y, chunk = blockIdx.x;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int t16 = lane & 15, lg = lane >> 4;
  const int S = K_b * B;
  const uint16_t* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
  const int32_t* bl = block_ids + size_t(unit) * K_b;
  // Two rounds of requests, each with every load in flight at once (loads
  // are unconditional at clamped addresses, so that none is sunk into a
  // branch and waited for alone):
  // 1. the context length, the block-list entries of the four tiles' slots
  //    and the channel id of this thread's q~ position;
  // 2. the q~ elements, then the tiles' index rows (so that the wait for q~
  //    does not cover the rows).
  // Thread t holds q~ entries t + 256 j: with 256 a multiple of DC they all
  // lie at operand position x = t % DC, of heads j (256 / DC) + t / DC.
  static_assert(256 % DC == 0 && G * DC % 256 == 0, "q~ entries per thread");
  constexpr int PER = G * DC / 256;
  const int x = tid % DC;
  int n = ctx_lens[s];
  int blk[4];
#pragma unroll
  for (int tl = 0; tl < 4; ++tl) {
    const int slot = chunk * kTokenSlotsPerWG + w * 64 + tl * 16 + t16;
    blk[tl] = bl[min(tok_block(min(slot, S - 1), B), K_b - 1)];
  }
  int ch;
  {
    const int e = x & 7;
    ch = channels[g * DC + (x & ~7) + ((e & 3) << 1) + (e >> 2)];  // channel index of position x
  }
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  if (ch < 0 || ch >= d) {
    set_error(err, 32u);
    ch = 0;
  }
  uint16_t qv[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) qv[j] = qg[size_t(j * (256 / DC) + tid / DC) * d + ch];
  __builtin_amdgcn_sched_barrier(0);
  bool valid[4];
  uint32_t cx[4][NGR];
  float2 pqv[4][NGR];
#pragma unroll
  for (int tl = 0; tl < 4; ++tl) {
    const int slot = chunk * kTokenSlotsPerWG + w * 64 + tl * 16 + t16;
    const int b = blk[tl];
    if (slot < S && b >= m) set_error(err, 2u);
    const int tok = b * B + tok_offset(slot, B);
    valid[tl] = slot < S && b >= 0 && b < m && tok < n;
    const size_t row = size_t(unit) * T + (valid[tl] ? tok : 0);
#pragma unroll
    for (int grp = 0; grp < NGR; ++grp) {
      cx[tl][grp] = *reinterpret_cast<const uint32_t*>(codes + row * (DC / 2) + grp * 16 + lg * 4);
      pqv[tl][grp] = *reinterpret_cast<const float2*>(qparams + (row * NGR + grp) * 2);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  // q~ to LDS in operand order, and each (head, 32-channel group) sum over
  // the 32 lanes that hold its positions (a 32-lane aligned half-wave): DPP
  // sums inside each 16-lane row, then the two rows' sums exchanged
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    s_qt[tid + j * 256] = qv[j];
    const uint32_t r16 = row16_reduce_bits(uint32_t(qv[j]) << 16, [](uint32_t u, uint32_t v) {
      return __float_as_uint(__uint_as_float(u) + __uint_as_float(v));
    });
    const auto sw = __builtin_amdgcn_permlane16_swap(r16, r16, false, false);
    if ((tid & 31) == 0)
      s_qs[(j * (256 / DC) + tid / DC) * NGR + x / 32] = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  __syncthreads();
  // A operands: head ht*16 + t16, channels of group grp at lane group lg
  ts_bf16x8_t qa[HT][NGR];
#pragma unroll
  for (int ht = 0; ht < HT; ++ht)
#pragma unroll
    for (int grp = 0; grp < NGR; ++grp)
      qa[ht][grp] = *reinterpret_cast<const ts_bf16x8_t*>(&s_qt[(ht * 16 + t16) * DC + grp * 32 + lg * 8]);
  float qs[HT][4][NGR];  // heads ht*16 + 4lg + r
#pragma unroll
  for (int ht = 0; ht < HT; ++ht)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int grp = 0; grp < NGR; ++grp) qs[ht][r][grp] = s_qs[(ht * 16 + lg * 4 + r) * NGR + grp];

  float lgt[4][HT][4];  // [tile][ht][r]
#pragma unroll
  for (int tl = 0; tl < 4; ++tl) {
    const int slot = chunk * kTokenSlotsPerWG + w * 64 + tl * 16 + t16;
    ts_f32x4_t acc[HT][NGR];
#pragma unroll
    for (int ht = 0; ht < HT; ++ht)
#pragma unroll
      for (int grp = 0; grp < NGR; ++grp) acc[ht][grp] = ts_f32x4_t{0.f, 0.f, 0.f, 0.f};
    float sc[NGR], off[NGR];
#pragma unroll
    for (int grp = 0; grp < NGR; ++grp) {
      const uint32_t x = cx[tl][grp];
      sc[grp] = pqv[tl][grp].x;
      off[grp] = pqv[tl][grp].y - 128.0f * pqv[tl][grp].x;
      const uint32_t lo = x & 0x0f0f0f0fu, hi = (x >> 4) & 0x0f0f0f0fu;
      const ts_u32x4_t bw = {__builtin_amdgcn_perm(kBase, lo, 0x04010400u), __builtin_amdgcn_perm(kBase, lo, 0x04030402u),
                             __builtin_amdgcn_perm(kBase, hi, 0x04010400u), __builtin_amdgcn_perm(kBase, hi, 0x04030402u)};
      const ts_bf16x8_t b = __builtin_bit_cast(ts_bf16x8_t, bw);
#pragma unroll
      for (int ht = 0; ht < HT; ++ht)
        acc[ht][grp] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[ht][grp], b, acc[ht][grp], 0, 0, 0);
    }
    // validity of slot t16 for the result lanes (lane (lg, t16) holds slot t16)
#pragma unroll
    for (int ht = 0; ht < HT; ++ht)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = 0.f;
#pragma unroll
        for (int grp = 0; grp < NGR; ++grp) v += fmaf(sc[grp], acc[ht][grp][r], off[grp] * qs[ht][r][grp]);
        lgt[tl][ht][r] = valid[tl] ? sigma * v : -INFINITY;
      }
    if (slot < S) {
      float* lg_out = logits + size_t(unit) * G * S + slot;
#pragma unroll
      for (int ht = 0; ht < HT; ++ht)
#pragma unroll
        for (int r = 0; r < 4; ++r) lg_out[size_t(ht * 16 + lg * 4 + r) * S] = lgt[tl][ht][r];
    }
  }
  // this work-group's per-head max and sum of exponentials (a DPP row holds
  // the 16 slots of one head)
  auto row16 = [](float v, bool is_max) {
    float o = dpp_row_move<0xB1>(v);
    v = is_max ? fmaxf(v, o) : v + o;
    o = dpp_row_move<0x4E>(v);
    v = is_max ? fmaxf(v, o) : v + o;
    o = dpp_row_move<0x141>(v);
    v = is_max ? fmaxf(v, o) : v + o;
    o = dpp_row_move<0x140>(v);
    return is_max ? fmaxf(v, o) : v + o;
  };
#pragma unroll
  for (int ht = 0; ht < HT; ++ht)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float mx = fmaxf(fmaxf(lgt[0][ht][r], lgt[1][ht][r]), fmaxf(lgt[2][ht][r], lgt[3][ht][r]));
      mx = row16(mx, true);
      float sm = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int tl = 0; tl < 4; ++tl) sm += lgt[tl][ht][r] == -INFINITY ? 0.f : __expf(lgt[tl][ht][r] - mx);
      }
      sm = row16(sm, false);
      if (t16 == 0) {
        s_red[w][ht * 16 + lg * 4 + r][0] = mx;
        s_red[w][ht * 16 + lg * 4 + r][1] = sm;
      }
    }
  __syncthreads();
  if (tid < G) {
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < 4; ++v) M = fmaxf(M, s_red[v][tid][0]);
    float Z = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (s_red[v][tid][0] != -INFINITY) Z += s_red[v][tid][1] * __expf(s_red[v][tid][0] - M);
    }
    float* st = stats + ((size_t(unit) * gridDim.x + chunk) * G + tid) * 2;
    st[0] = M;
    st[1] = Z;
  }
}

// Work-group 0 of a unit's alpha kernel also writes the unit's number of
// valid candidate slots and the key of a bound on every alpha key: with each
// exponential <= 1, the alpha of a slot is at most (1/G) sum_h 1/Z_h summed
// in the key loop's order (rounding is monotone), so the top-K_t kernel needs
// no statistics pass of its own.  All 256 threads call it; b_first is the
// list entry bl[threadIdx.x] (any value where threadIdx.x >= K_b), requested
// by the caller with its other loads.
__device__ inline void write_unit_info(const int32_t* bl, int b_first, int K_b, int B, int m, int n,
                                       const float* s_iz, int G, float invG, uint32_t* kinfo, int unit,
                                       uint32_t* s_cnt) {
  uint32_t c = 0;
  for (int i = threadIdx.x; i < K_b; i += 256) {
    const int b = i == int(threadIdx.x) ? b_first : bl[i];
    if (b >= 0 && b < m) c += uint32_t(min(B, n - b * B));
  }
  c = wave_reduce_bits(c, [](uint32_t a, uint32_t b) { return a + b; });
  if ((threadIdx.x & 63) == 0) s_cnt[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    float bsum = 0.f;
    for (int h = 0; h < G; ++h) bsum = fmaf(1.0f, s_iz[h], bsum);
    kinfo[2 * size_t(unit)] = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    kinfo[2 * size_t(unit) + 1] = __float_as_uint(fmaxf(bsum * invG, 0.f)) | 0x80000000u;
  }
}

// The alpha key of a candidate: alpha >= +0 has the key bits | 2^31 (as
// float_key); a NaN alpha (NaN inputs only) ranks as 0.
__device__ inline uint32_t alpha_key(float a) { return __float_as_uint(fmaxf(a, 0.f)) | 0x80000000u; }

__global__ __launch_bounds__(256) void token_alpha_kernel(
    const float* __restrict__ logits, const float* __restrict__ stats, int n_tchunks,
    const int32_t* __restrict__ block_ids, int K_b, const int32_t* __restrict__ ctx_lens, int H_kv, int G,
    int B, int T, uint32_t* __restrict__ keys, uint32_t* __restrict__ kinfo) {
  __shared__ float s_m[kMaxG], s_iz[kMaxG];
  __shared__ uint32_t s_cnt[4];
  const int unit = blockIdx.y;
  const int s = unit / H_kv;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  const int S = K_b * B;
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    const float* st = stats + size_t(unit) * n_tchunks * G * 2;
    float M = -INFINITY;
    for (int c = 0; c < n_tchunks; ++c) M = fmaxf(M, st[(c * G + h) * 2]);
    float Z = 0.f;
    if (M != -INFINITY)
      for (int c = 0; c < n_tchunks; ++c) {
        const float mc = st[(c * G + h) * 2], zc = st[(c * G + h) * 2 + 1];
        if (mc != -INFINITY) Z += zc * __expf(mc - M);
      }
    s_m[h] = M;
    s_iz[h] = Z > 0.f ? 1.0f / Z : 0.f;
  }
  __syncthreads();
  const float invG = 1.0f / float(G);
  const int32_t* bl = block_ids + size_t(unit) * K_b;
  if (blockIdx.x == 0)
    write_unit_info(bl, threadIdx.x < K_b ? bl[threadIdx.x] : -1, K_b, B, m, n, s_iz, G, invG, kinfo, unit, s_cnt);
  const float* lg = logits + size_t(unit) * G * S;
  for (int slot = blockIdx.x * 256 + threadIdx.x; slot < S; slot += gridDim.x * 256) {
    int tok;
    uint32_t key = kInvalidKey;
    if (slot_token(bl, K_b, B, m, n, slot, &tok, nullptr)) {
      float a = 0.f;
      for (int h = 0; h < G; ++h) a += __expf(lg[size_t(h) * S + slot] - s_m[h]) * s_iz[h];
      key = alpha_key(a * invG);
    }
    keys[size_t(unit) * S + slot] = key;
  }
}

// token_alpha_kernel with the head count fixed at compile time, for a grid
// of one slot per thread: 256/G lanes combine each head's work-group
// statistics, and every request of a work-group leaves at once before the
// first is used (its lanes' statistics, the block-list entries of its slots
// and of the unit information, the slots' G logits; unconditional loads at
// clamped addresses), so the kernel waits for one memory round trip.
template <int G>
__global__ __launch_bounds__(256) void token_alpha_kernel_g(
    const float* __restrict__ logits, const float* __restrict__ stats, int n_tchunks,
    const int32_t* __restrict__ block_ids, int K_b, const int32_t* __restrict__ ctx_lens, int H_kv, int B, int T,
    uint32_t* __restrict__ keys, uint32_t* __restrict__ kinfo) {
  constexpr int TPH = 256 / G;  // lanes per head (a power of two)
  constexpr int kC = 8;         // statistics chunks per lane requested together
  __shared__ float s_m[G], s_iz[G];
  __shared__ uint32_t s_cnt[4];
  const int unit = blockIdx.y, tid = threadIdx.x;
  const int s = unit / H_kv;
  const int S = K_b * B;
  const int h = tid / TPH, j = tid % TPH;
  const float2* st = reinterpret_cast<const float2*>(stats) + size_t(unit) * n_tchunks * G;
  const int32_t* bl = block_ids + size_t(unit) * K_b;
  const float* lg = logits + size_t(unit) * G * S;
  const int slot = blockIdx.x * 256 + tid, sl = min(slot, S - 1);
  float2 sv[kC];
#pragma unroll
  for (int c = 0; c < kC; ++c) sv[c] = st[size_t(min(j + c * TPH, n_tchunks - 1)) * G + h];
  __builtin_amdgcn_sched_barrier(0);
  const int b_slot = bl[tok_block(sl, B)];
  const int b_first = bl[min(tid, K_b - 1)];
  float v[G];
#pragma unroll
  for (int hh = 0; hh < G; ++hh) v[hh] = lg[size_t(hh) * S + sl];
  __builtin_amdgcn_sched_barrier(0);
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  {
    // chunks j, j + TPH, ... in ascending order, then the lanes' tree (the
    // requested entries are used through selects, not branches, so that
    // no load is sunk into a branch; adding +0 leaves Z >= +0 unchanged)
    float M = -INFINITY;
#pragma unroll
    for (int c = 0; c < kC; ++c) M = fmaxf(M, j + c * TPH < n_tchunks ? sv[c].x : -INFINITY);
    for (int c = j + kC * TPH; c < n_tchunks; c += TPH) M = fmaxf(M, st[size_t(c) * G + h].x);
#pragma unroll
    for (int o = TPH / 2; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
    float Z = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int c = 0; c < kC; ++c) {
        const bool ok = j + c * TPH < n_tchunks && sv[c].x != -INFINITY;
        Z += ok ? sv[c].y * __expf(sv[c].x - M) : 0.f;
      }
      for (int c = j + kC * TPH; c < n_tchunks; c += TPH) {
        const float2 e = st[size_t(c) * G + h];
        if (e.x != -INFINITY) Z += e.y * __expf(e.x - M);
      }
    }
#pragma unroll
    for (int o = TPH / 2; o > 0; o >>= 1) Z += __shfl_xor(Z, o, 64);
    if (j == 0) {
      s_m[h] = M;
      s_iz[h] = Z > 0.f ? 1.0f / Z : 0.f;
    }
  }
  __syncthreads();
  const float invG = 1.0f / float(G);
  if (blockIdx.x == 0) write_unit_info(bl, b_first, K_b, B, m, n, s_iz, G, invG, kinfo, unit, s_cnt);
  if (slot < S) {
    const int t = b_slot * B + tok_offset(slot, B);
    uint32_t key = kInvalidKey;
    if (b_slot >= 0 && b_slot < m && t < n) {
      float a = 0.f;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) a += __expf(v[hh] - s_m[hh]) * s_iz[hh];
      key = alpha_key(a * invG);
    }
    keys[size_t(unit) * S + slot] = key;
  }
}

// Top-K_t of the alpha keys of each unit, one work-group per unit.  Thread t
// holds the keys of slots t + 1024 j (j < EPT), requested together straight
// into registers.
template <int EPT>
__global__ __launch_bounds__(1024) void token_topk_kernel(const uint32_t* __restrict__ keys,
                                                           const uint32_t* __restrict__ kinfo,
                                                           const int32_t* __restrict__ block_ids, int K_b,
                                                           int B, int K_t, int32_t* __restrict__ token_ids,
                                                           float* __restrict__ token_scores) {
  extern __shared__ uint32_t smem[];
  uint32_t* scratch = smem;
  int32_t* s_bl = reinterpret_cast<int32_t*>(smem + topk_scratch_words(1024));
  const int S = K_b * B;
  const int unit = blockIdx.x;
  uint32_t kr[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int p = threadIdx.x + j * 1024;
    kr[j] = p < S ? keys[size_t(unit) * S + p] : kInvalidKey;
  }
  // the valid count and the key bound from the alpha kernel; every valid key
  // is >= the key of +0
  const TopkKnown known{kinfo[2 * size_t(unit)], kinfo[2 * size_t(unit) + 1], 0x80000000u};
  for (int i = threadIdx.x; i < K_b; i += 1024) s_bl[i] = block_ids[size_t(unit) * K_b + i];
  topk_prepare<1024>(scratch);
  __syncthreads();
  wg_topk_regs<1024, EPT, true>(kr, K_t, token_ids + size_t(unit) * K_t, K_t,
                                token_scores ? token_scores + size_t(unit) * K_t : nullptr,
                                [=](int, int slot) { return int32_t(s_bl[tok_block(slot, B)] * B + tok_offset(slot, B)); }, scratch,
                                &known);
}

template <int HT, int NGR>
static void launch_score_mfma(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                              const int32_t* channels, const int32_t* block_ids, int K_b, const int32_t* ctx_lens,
                              float* logits, float* stats, int n_tchunks, uint32_t* err, hipStream_t st) {
  token_score_mfma_kernel<HT, NGR><<<dim3(n_tchunks, P.units), 256, 0, st>>>(
      (const uint16_t*)q, codes, qparams, channels, block_ids, K_b, ctx_lens, P.H_q, P.H_kv, P.d_qk, P.B, P.T,
      P.sigma, logits, stats, err);
}

hipError_t launch_token_score(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                              const int32_t* channels, const int32_t* block_ids, int K_b,
                              const int32_t* ctx_lens, float* logits, float* stats, int n_tchunks,
                              uint32_t* err, hipStream_t st) {
  if (P.dtype == 1 && (P.G == 16 || P.G == 32) && (P.d_c == 64 || P.d_c == 128)) {
    if (P.G == 32 && P.d_c == 128) launch_score_mfma<2, 4>(P, q, codes, qparams, channels, block_ids, K_b, ctx_lens, logits, stats, n_tchunks, err, st);
    else if (P.G == 32) launch_score_mfma<2, 2>(P, q, codes, qparams, channels, block_ids, K_b, ctx_lens, logits, stats, n_tchunks, err, st);
    else if (P.d_c == 128) launch_score_mfma<1, 4>(P, q, codes, qparams, channels, block_ids, K_b, ctx_lens, logits, stats, n_tchunks, err, st);
    else launch_score_mfma<1, 2>(P, q, codes, qparams, channels, block_ids, K_b, ctx_lens, logits, stats, n_tchunks, err, st);
    return hipGetLastError();
  }
  dim3 grid(n_tchunks, P.units);
  if (P.dtype == 1)
    token_score_kernel<BF16><<<grid, 256, 0, st>>>((const uint16_t*)q, codes, qparams, channels, block_ids,
                                                   K_b, ctx_lens, P.H_q, P.H_kv, P.G, P.d_qk, P.d_c, P.B,
                                                   P.T, P.sigma, logits, stats, err);
  else
    token_score_kernel<F32><<<grid, 256, 0, st>>>((const float*)q, codes, qparams, channels, block_ids, K_b,
                                                  ctx_lens, P.H_q, P.H_kv, P.G, P.d_qk, P.d_c, P.B, P.T,
                                                  P.sigma, logits, stats, err);
  return hipGetLastError();
}

hipError_t launch_token_alpha(const Problem& P, const float* logits, const float* stats, int n_tchunks,
                              const int32_t* block_ids, int K_b, const int32_t* ctx_lens, uint32_t* keys,
                              uint32_t* kinfo, hipStream_t st) {
  const int S = K_b * P.B;
  dim3 grid((S + 255) / 256, P.units);
  switch (P.G) {
    case 4: token_alpha_kernel_g<4><<<grid, 256, 0, st>>>(logits, stats, n_tchunks, block_ids, K_b, ctx_lens, P.H_kv, P.B, P.T, keys, kinfo); break;
    case 8: token_alpha_kernel_g<8><<<grid, 256, 0, st>>>(logits, stats, n_tchunks, block_ids, K_b, ctx_lens, P.H_kv, P.B, P.T, keys, kinfo); break;
    case 16: token_alpha_kernel_g<16><<<grid, 256, 0, st>>>(logits, stats, n_tchunks, block_ids, K_b, ctx_lens, P.H_kv, P.B, P.T, keys, kinfo); break;
    case 32: token_alpha_kernel_g<32><<<grid, 256, 0, st>>>(logits, stats, n_tchunks, block_ids, K_b, ctx_lens, P.H_kv, P.B, P.T, keys, kinfo); break;
    default:
      token_alpha_kernel<<<grid, 256, 0, st>>>(logits, stats, n_tchunks, block_ids, K_b, ctx_lens, P.H_kv, P.G,
                                               P.B, P.T, keys, kinfo);
  }
  return hipGetLastError();
}

hipError_t launch_token_topk(const Problem& P, const uint32_t* keys, const uint32_t* kinfo, const int32_t* block_ids,
                             int K_b, int K_t, int32_t* token_ids, float* token_scores, hipStream_t st) {
  const int S = K_b * P.B;
  const size_t lds = (topk_scratch_words(1024) + size_t(align4w(K_b))) * sizeof(uint32_t);
  const int ept = (S + 1023) / 1024;
  auto go = [&](auto kern) {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), lds);
    if (e != hipSuccess) return e;
    kern<<<P.units, 1024, lds, st>>>(keys, kinfo, block_ids, K_b, P.B, K_t, token_ids, token_scores);
    return hipGetLastError();
  };
  if (ept <= 1) return go(token_topk_kernel<1>);
  if (ept <= 2) return go(token_topk_kernel<2>);
  if (ept <= 4) return go(token_topk_kernel<4>);
  if (ept <= 8) return go(token_topk_kernel<8>);
  return go(token_topk_kernel<16>);
}

}  // namespace tls
