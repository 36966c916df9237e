// Fused two-level selection for grouped-query layouts (AsyncTLS Sec. 4.1):
// one 1024-thread work-group per (sequence, KV head) unit runs, on chip,
//   1. top-K_b over the unit's block scores (or takes a given block list);
//   2. the approximate logits of every candidate token,
//        l_hj = sigma * q~_h . dequant(k~_j)
//             = sigma * (min_j * sum_c q~_hc + scale_j * sum_c q~_hc code_jc),
//      where the integer-code contraction runs on MFMA
//      (v_mfma_f32_16x16x32_bf16: A = q~, G heads padded to 16 rows x 32
//      channels, exact in bf16; B = the codes of 16 slots, exact small
//      integers; fp32 accumulation);
//   3. per-head max and sum of exponentials over all candidates and
//      alpha_j = (1/G) sum_h exp(l_hj - m_h) / Z_h;
//   4. top-K_t of alpha (ties to the lower position), ascending positions.
//
// Data movement: every thread owns slots t, t+1024, ...; all candidates'
// index rows (16 B codes + 8 B params per slot) are requested at once with
// wide coalesced loads (one 64-slot block per wave instruction), the codes
// are staged in LDS, each wave turns 16-slot tiles of them into raw dot
// products written back in place (16 B per slot either way), and the owning
// threads finish the logits in registers.
#include "token_common.hpp"

namespace tls {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;

constexpr int kSelNT = 1024;
constexpr int kSelNW = kSelNT / 64;
constexpr int kSelSPT = 8;  // slots per thread
constexpr int kSelMaxSlots = kSelNT * kSelSPT;
constexpr int kSelMaxG = 4;
constexpr size_t kSelMaxLds = 160 * 1024;

// Channel order of the eight codes of one packed dword as they enter the
// MFMA k-slice: low nibbles (channels 0,2,4,6) then high nibbles (1,3,5,7).
// The contraction is order-free, so A uses the same order.
__device__ constexpr int kSlicePerm[8] = {0, 2, 4, 6, 1, 3, 5, 7};

// bf16 bit pattern of a small non-negative integer (exact).
__device__ inline uint32_t int_bf16(uint32_t c) { return __float_as_uint(float(c)) >> 16; }

__device__ inline bf16x8_t codes_operand(uint32_t w) {
  const uint32_t lo = w & 0x0f0f0f0fu, hi = (w >> 4) & 0x0f0f0f0fu;
  u32x4_t p;
  p[0] = int_bf16(lo & 0xffu) | (int_bf16((lo >> 8) & 0xffu) << 16);
  p[1] = int_bf16((lo >> 16) & 0xffu) | (int_bf16(lo >> 24) << 16);
  p[2] = int_bf16(hi & 0xffu) | (int_bf16((hi >> 8) & 0xffu) << 16);
  p[3] = int_bf16((hi >> 16) & 0xffu) | (int_bf16(hi >> 24) << 16);
  return __builtin_bit_cast(bf16x8_t, p);
}

// LDS words: top-k scratch | block list | block-list stage | q sums | reduce
// slots | region R.  R holds the block keys, then the codes / raw dots
// (4 words per slot), then the alpha keys and the top-K_t stage.
static size_t region_words(int S, int K_t, int m_max) {
  size_t r = size_t(4) * S;
  if (size_t(m_max) > r) r = m_max;
  if (size_t(S) + 2 * size_t(K_t) > r) r = size_t(S) + 2 * size_t(K_t);
  return r;
}

size_t mfma_select_lds_bytes(int S, int K_b, int K_t, int m_max) {
  return (size_t(topk_scratch_words(kSelNT)) + size_t(align4w(2 * K_b)) + 4 + kSelNW * 4 +
          region_words(S, K_t, m_max)) *
         sizeof(uint32_t);
}

template <int G>
__global__ __launch_bounds__(kSelNT) void token_select_mfma_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ codes, const float* __restrict__ qparams,
    const int32_t* __restrict__ channels, const float* __restrict__ block_scores,
    const int32_t* __restrict__ block_ids_in, int32_t* __restrict__ block_ids_out,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int d, int B, int T, int m_max, int K_b, int K_t,
    float sigma, int32_t* __restrict__ token_ids, float* __restrict__ token_scores, uint32_t* err) {
  constexpr int NT = kSelNT, NW = kSelNW;
  extern __shared__ uint32_t smem[];
  uint32_t* scratch = smem;
  int32_t* s_bl = reinterpret_cast<int32_t*>(smem + topk_scratch_words(NT));
  int32_t* s_bstage = s_bl + K_b;
  float* s_qs = reinterpret_cast<float*>(s_bl + align4w(2 * K_b));  // [4]
  float* s_red = s_qs + 4;                                 // [NW][4]
  uint32_t* R = reinterpret_cast<uint32_t*>(s_red + NW * 4);

  const int unit = blockIdx.x;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (tid == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int m = (n + B - 1) / B;
  const int S = K_b * B;
  const uint16_t* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
  const int32_t* chs = channels + g * 32;

  // A operand: row = head (lane % 16; zero rows past G), k-slice lane / 16
  bf16x8_t a_op;
  {
    const int h = lane & 15, ks = lane >> 4;
    u32x4_t pa;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      uint32_t v[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        int ch = chs[8 * ks + kSlicePerm[2 * e2 + t]];
        if (ch < 0 || ch >= d) {
          set_error(err, 32u);
          ch = 0;
        }
        v[t] = h < G ? qg[size_t(h) * d + ch] : 0u;
      }
      pa[e2] = v[0] | (v[1] << 16);
    }
    a_op = __builtin_bit_cast(bf16x8_t, pa);
  }
  if (tid < G) {
    float a = 0.f;
    for (int c = 0; c < 32; ++c) {
      int ch = chs[c];
      ch = (ch < 0 || ch >= d) ? 0 : ch;
      a += BF16::to_f(qg[size_t(tid) * d + ch]);
    }
    s_qs[tid] = a;
  }
  // block list
  if (block_scores) {
    const float* sc = block_scores + size_t(unit) * m_max;
    for (int i = tid; i < m; i += NT) R[i] = float_key(sc[i]);
    __syncthreads();
    wg_topk_ascending<NT>(R, m, K_b, s_bl, K_b, nullptr, [](int i) { return int32_t(i); }, scratch, s_bstage,
                          nullptr);
  } else {
    for (int i = tid; i < K_b; i += NT) s_bl[i] = block_ids_in[size_t(unit) * K_b + i];
  }
  __syncthreads();

  // 1. request every index row of this thread's slots, stage codes in LDS
  float2 qp[kSelSPT];
  uint32_t vmask = 0;
  {
    uint4 cw[kSelSPT];
#pragma unroll
    for (int i = 0; i < kSelSPT; ++i) {
      const int slot = tid + i * NT;
      int tok = 0;
      const bool valid = slot < S && slot_token(s_bl, K_b, B, m, n, slot, &tok, err);
      cw[i] = make_uint4(0, 0, 0, 0);
      qp[i] = make_float2(0.f, 0.f);
      if (valid) {
        const size_t row = size_t(unit) * T + tok;
        cw[i] = ld16_stream(codes + row * 16);
        qp[i] = *reinterpret_cast<const float2*>(qparams + row * 2);
        vmask |= 1u << i;
      }
    }
#pragma unroll
    for (int i = 0; i < kSelSPT; ++i) {
      const int slot = tid + i * NT;
      if (slot < S) *reinterpret_cast<uint4*>(R + size_t(slot) * 4) = cw[i];
    }
  }
  __syncthreads();

  // 2. raw dots on MFMA, 16-slot tiles, written back over their own codes
  {
    const int ntiles = S / 16;
    const int r16 = lane & 15, ks = lane >> 4;
    for (int t0 = wid; t0 < ntiles; t0 += NW * 4) {
      uint32_t w4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int tile = t0 + u * NW;
        w4[u] = tile < ntiles ? R[(tile * 16 + r16) * 4 + ks] : 0u;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int tile = t0 + u * NW;
        if (tile >= ntiles) break;
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_op, codes_operand(w4[u]), acc, 0, 0, 0);
        if (lane < 16) {
          // rows 0..3 of the result are heads 0..3 of slot tile*16 + lane
          uint4 o;
          o.x = __float_as_uint(acc[0]);
          o.y = __float_as_uint(acc[1]);
          o.z = __float_as_uint(acc[2]);
          o.w = __float_as_uint(acc[3]);
          *reinterpret_cast<uint4*>(R + size_t(tile * 16 + lane) * 4) = o;
        }
      }
    }
  }
  __syncthreads();

  // 3. logits of the owned slots, per-head max over the work-group
  float lg[kSelSPT][G];
  float mx[G];
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = -INFINITY;
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i) {
    const int slot = tid + i * NT;
    const bool valid = (vmask >> i) & 1u;
    float raw[4] = {0.f, 0.f, 0.f, 0.f};
    if (slot < S) {
      const uint4 o = *reinterpret_cast<const uint4*>(R + size_t(slot) * 4);
      raw[0] = __uint_as_float(o.x);
      raw[1] = __uint_as_float(o.y);
      raw[2] = __uint_as_float(o.z);
      raw[3] = __uint_as_float(o.w);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      lg[i][h] = valid ? sigma * (qp[i].y * s_qs[h] + qp[i].x * raw[h]) : -INFINITY;
      mx[h] = fmaxf(mx[h], lg[i][h]);
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float w = wave_max_f32(mx[h]);
    if (lane == 0) s_red[wid * 4 + h] = w;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float v = s_red[(lane & 15) * 4 + h];
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, __uint_as_float(__builtin_amdgcn_readlane(__float_as_int(v), w)));
    mx[h] = M;
  }
  __syncthreads();
  // exponentials and their per-head sums
  float sum[G];
#pragma unroll
  for (int h = 0; h < G; ++h) sum[h] = 0.f;
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float e = ((vmask >> i) & 1u) ? __expf(lg[i][h] - mx[h]) : 0.f;
      lg[i][h] = e;
      sum[h] += e;
    }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float w = wave_sum_f32(sum[h]);
    if (lane == 0) s_red[wid * 4 + h] = w;
  }
  __syncthreads();
  float iz[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float v = s_red[(lane & 15) * 4 + h];
    float Z = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) Z += __uint_as_float(__builtin_amdgcn_readlane(__float_as_int(v), w));
    iz[h] = Z > 0.f ? 1.0f / Z : 0.f;
  }
  // 4. alpha keys over R[0, S), top-K_t
  const float invG = 1.0f / float(G);
#pragma unroll
  for (int i = 0; i < kSelSPT; ++i) {
    const int slot = tid + i * NT;
    if (slot < S) {
      float a = 0.f;
#pragma unroll
      for (int h = 0; h < G; ++h) a += lg[i][h] * iz[h];
      R[slot] = ((vmask >> i) & 1u) ? float_key(a * invG) : kInvalidKey;
    }
  }
  __syncthreads();
  int32_t* stage = reinterpret_cast<int32_t*>(R + S);
  float* stage_sc = reinterpret_cast<float*>(R + S + K_t);
  wg_topk_ascending<NT>(R, S, K_t, token_ids + size_t(unit) * K_t, K_t,
                        token_scores ? token_scores + size_t(unit) * K_t : nullptr,
                        [=](int slot) { return int32_t(s_bl[slot / B] * B + slot % B); }, scratch, stage,
                        stage_sc);
  if (block_scores && block_ids_out)
    for (int i = tid; i < K_b; i += NT) block_ids_out[size_t(unit) * K_b + i] = s_bl[i];
}

bool fused_token_select_ok(const Problem& P, int K_b, int K_t) {
  const int S = K_b * P.B;
  return P.dtype == 1 && P.G >= 1 && P.G <= kSelMaxG && P.d_c == 32 && S <= kSelMaxSlots && S % 16 == 0 &&
         mfma_select_lds_bytes(S, K_b, K_t, P.m_max) <= kSelMaxLds;
}

template <int G>
static hipError_t launch_g(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                           const int32_t* channels, const float* block_scores, const int32_t* block_ids_in,
                           int32_t* block_ids_out, const int32_t* ctx_lens, int K_b, int K_t, int32_t* token_ids,
                           float* token_scores, uint32_t* err, hipStream_t st) {
  const size_t lds = mfma_select_lds_bytes(K_b * P.B, K_b, K_t, P.m_max);
  auto kern = token_select_mfma_kernel<G>;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  kern<<<P.units, kSelNT, lds, st>>>((const uint16_t*)q, codes, qparams, channels, block_scores, block_ids_in,
                                     block_ids_out, ctx_lens, P.H_q, P.H_kv, P.d_qk, P.B, P.T, P.m_max, K_b, K_t,
                                     P.sigma, token_ids, token_scores, err);
  return hipGetLastError();
}

hipError_t launch_token_select_fused(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                                     const int32_t* channels, const float* block_scores,
                                     const int32_t* block_ids_in, int32_t* block_ids_out, const int32_t* ctx_lens,
                                     int K_b, int K_t, int32_t* token_ids, float* token_scores, uint32_t* err,
                                     hipStream_t st) {
  switch (P.G) {
    case 1: return launch_g<1>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                               K_b, K_t, token_ids, token_scores, err, st);
    case 2: return launch_g<2>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                               K_b, K_t, token_ids, token_scores, err, st);
    case 3: return launch_g<3>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                               K_b, K_t, token_ids, token_scores, err, st);
    default: return launch_g<4>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                                K_b, K_t, token_ids, token_scores, err, st);
  }
}

}  // namespace tls
