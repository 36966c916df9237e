// Fused two-level selection for grouped-query layouts (AsyncTLS Sec. 4.1):
// one 1024-thread work-group per (sequence, KV head) unit runs, on chip,
//   1. top-K_b over the unit's block scores (or takes a given block list;
//      with both, the lagged operator of Sec. 4.2: the new top-K_b goes to
//      the output list and the tokens are chosen from the given blocks);
//   2. the approximate logits of every candidate token,
//        l_hj = sigma * q~_h . dequant(k~_j)
//             = sigma * (min_j * sum_c q~_hc + scale_j * sum_c q~_hc code_jc);
//   3. per-head max and sum of exponentials over all candidates and
//      alpha_j = (1/G) sum_h exp(l_hj - m_h) / Z_h;
//   4. top-K_t of alpha (ties to the lower position), ascending positions.
//
// Everything a thread computes stays in its registers: thread t owns the
// candidate slots t + 1024 i (i < 8), so each wave reads 64 consecutive
// tokens' index rows (coalesced 16-byte code and 8-byte parameter loads) and
// hands its alpha keys straight to the register top-k, whose ordered
// compaction works on exactly this strided ownership.
//
// The code contraction runs on v_mfma_f32_4x4x4_16b_bf16: sixteen 4x4x4
// blocks per instruction, block b = lanes 4b..4b+3, A = the (up to) four
// heads' q~ on 4 channels (the same in every block), B = 4 channels of the
// four slots of the block, so lane l receives the four heads' dots of its own
// slot.  Eight instructions cover the 32 channels of one index group.  A code
// c enters as the bf16 number 128 + c (bit pattern 0x4300 | c, built with one
// byte permute per two codes), so the product gives sum_c q~_c (128 + c_c);
// the 128 sum_c q~_c part is folded into the offset term:
//   l_hj = sigma * (scale_j * dot_hj + (min_j - 128 scale_j) * sum_c q~_hc).
// All products are exact in fp32; accumulation is fp32.
#include "token_select_mfma.hpp"

namespace tls {

template <int G, bool WB>
__global__ __launch_bounds__(kSelNT) void token_select_mfma_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ codes, const float* __restrict__ qparams,
    const int32_t* __restrict__ channels, const float* __restrict__ block_scores,
    const int32_t* __restrict__ block_ids_in, int32_t* __restrict__ block_ids_out,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int d, int B, int T, int m_max, int K_b, int K_t,
    float sigma, int32_t* __restrict__ token_ids, float* __restrict__ token_scores, uint32_t* err) {
  extern __shared__ uint32_t smem[];
  token_select_mfma_body<G, WB>(smem, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                            H_q, H_kv, d, B, T, m_max, K_b, K_t, sigma, token_ids, token_scores, err, blockIdx.x);
}

bool fused_token_select_ok(const Problem& P, int K_b, int K_t) {
  const int S = K_b * P.B;
  return P.dtype == 1 && P.G >= 1 && P.G <= kSelMaxG && P.d_c == 32 && (P.B & (P.B - 1)) == 0 && S <= kSelMaxSlots &&
         P.m_max <= kSelMaxBlocks && mfma_select_lds_bytes(K_b) <= kSelMaxLds;
}

template <int G, bool WB>
static hipError_t launch_gw(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                           const int32_t* channels, const float* block_scores, const int32_t* block_ids_in,
                           int32_t* block_ids_out, const int32_t* ctx_lens, int K_b, int K_t, int32_t* token_ids,
                           float* token_scores, uint32_t* err, hipStream_t st) {
  const size_t lds = mfma_select_lds_bytes(K_b);
  auto kern = token_select_mfma_kernel<G, WB>;
  const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), lds);
  if (e != hipSuccess) return e;
  kern<<<P.units, kSelNT, lds, st>>>((const uint16_t*)q, codes, qparams, channels, block_scores, block_ids_in,
                                     block_ids_out, ctx_lens, P.H_q, P.H_kv, P.d_qk, P.B, P.T, P.m_max, K_b, K_t,
                                     P.sigma, token_ids, token_scores, err);
  return hipGetLastError();
}

template <int G>
static hipError_t launch_g(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                           const int32_t* channels, const float* block_scores, const int32_t* block_ids_in,
                           int32_t* block_ids_out, const int32_t* ctx_lens, int K_b, int K_t, int32_t* token_ids,
                           float* token_scores, uint32_t* err, hipStream_t st) {
  if (P.B >= 64)
    return launch_gw<G, true>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                              K_b, K_t, token_ids, token_scores, err, st);
  return launch_gw<G, false>(P, q, codes, qparams, channels, block_scores, block_ids_in, block_ids_out, ctx_lens,
                             K_b, K_t, token_ids, token_scores, err, st);
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
