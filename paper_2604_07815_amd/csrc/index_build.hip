// Index construction at prefill (AsyncTLS Sec. 4.1):
//  * block_index_kernel - per-channel max/min key of every block of B tokens
//    (the Quest block representation), tail block over its valid tokens;
//  * token_index_kernel - keys projected on the channel set C and quantised
//    to asymmetric uint4 per group of 32 channels (INT4 per Sec. 5 setup),
//    computed with an exact float32 op sequence so the codes are
//    reproducible bit for bit.
#include "kernels.hpp"

namespace tls {

// One thread per (block, 16-byte channel chunk); rows streamed top to bottom.
template <class E>
__global__ __launch_bounds__(256) void block_index_kernel(
    const typename E::T* __restrict__ K, const int32_t* __restrict__ ctx_lens, int H_kv, int T, int d,
    int B, int m_max, int tok_begin, int tok_end, typename E::T* __restrict__ kmax,
    typename E::T* __restrict__ kmin, uint32_t* err) {
  using S = typename E::T;
  constexpr int V = E::kVec;
  const int s = blockIdx.z, g = blockIdx.y;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (threadIdx.x == 0 && blockIdx.x == 0 && g == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int hi = min(tok_end, n);
  if (tok_begin >= hi) return;
  const int b0 = tok_begin / B, b1 = (hi + B - 1) / B;  // blocks overlapping [tok_begin, hi)
  const int cpb = d / V;                                 // chunks per block row
  const size_t unit = size_t(s) * H_kv + g;
  const S* Ku = K + unit * size_t(T) * d;
  const int items = (b1 - b0) * cpb;
  for (int it = blockIdx.x * blockDim.x + threadIdx.x; it < items; it += gridDim.x * blockDim.x) {
    const int i = b0 + it / cpb, c = it % cpb;
    const int r0 = i * B, r1 = min(r0 + B, n);
    float mx[V], mn[V];
    {
      float x[V];
      unpack16<E>(ld16(Ku + size_t(r0) * d + c * V), x);
#pragma unroll
      for (int e = 0; e < V; ++e) mx[e] = mn[e] = x[e];
    }
    for (int r = r0 + 1; r < r1; ++r) {
      float x[V];
      unpack16<E>(ld16(Ku + size_t(r) * d + c * V), x);
#pragma unroll
      for (int e = 0; e < V; ++e) {
        mx[e] = fmaxf(mx[e], x[e]);
        mn[e] = fminf(mn[e], x[e]);
      }
    }
    S* pmax = kmax + (unit * m_max + i) * d + c * V;
    S* pmin = kmin + (unit * m_max + i) * d + c * V;
#pragma unroll
    for (int e = 0; e < V; ++e) {
      // values are exact copies of inputs; +0.0f turns -0.0 into +0.0
      store_out<E>(pmax + e, mx[e] + 0.0f);
      store_out<E>(pmin + e, mn[e] + 0.0f);
    }
  }
}

// 32 lanes per (token, channel group); a wave covers two (token, group) pairs.
template <class E>
__global__ __launch_bounds__(256) void token_index_kernel(
    const typename E::T* __restrict__ K, const int32_t* __restrict__ ctx_lens,
    const int32_t* __restrict__ channels, int H_kv, int T, int d, int d_c, int tok_begin, int tok_end,
    uint8_t* __restrict__ codes, float* __restrict__ qparams, uint32_t* err) {
#pragma clang fp contract(off)
  const int s = blockIdx.z, g = blockIdx.y;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (threadIdx.x == 0 && blockIdx.x == 0 && g == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int hi = min(tok_end, n);
  if (tok_begin >= hi) return;
  const int ngroups = d_c / 32;
  const int lane = threadIdx.x & 63;
  const int c = lane & 31;
  const int half = (blockIdx.x * blockDim.x + threadIdx.x) >> 5;  // global half-wave id
  const int nhalves = (gridDim.x * blockDim.x) >> 5;
  const size_t unit = size_t(s) * H_kv + g;
  const typename E::T* Ku = K + unit * size_t(T) * d;
  const int items = (hi - tok_begin) * ngroups;
  for (int it = half; it < items; it += nhalves) {
    const int j = tok_begin + it / ngroups, grp = it % ngroups;
    int ch = channels[g * d_c + grp * 32 + c];
    if (ch < 0 || ch >= d) {  // caller-supplied channel id out of range
      set_error(err, 32u);
      ch = 0;
    }
    const float x = E::to_f(Ku[size_t(j) * d + ch]);
    float mn = x, mx = x;
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) {
      mn = fminf(mn, __shfl_xor(mn, o, 64));
      mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    }
    const float scale = (mx - mn) / 15.0f;  // IEEE float32 subtract and divide
    uint32_t code = 0;
    if (scale != 0.0f) {
      float v = __builtin_rintf((x - mn) / scale);  // round half to even
      v = fminf(fmaxf(v, 0.0f), 15.0f);
      code = uint32_t(v);
    }
    const uint32_t nxt = __shfl_down(code, 1, 64);
    const size_t row = unit * size_t(T) + j;
    if ((c & 1) == 0) codes[row * (d_c / 2) + grp * 16 + (c >> 1)] = uint8_t(code | (nxt << 4));
    if (c == 0) {
      qparams[(row * ngroups + grp) * 2 + 0] = scale;
      qparams[(row * ngroups + grp) * 2 + 1] = mn + 0.0f;
    }
  }
}

hipError_t launch_block_index(const Problem& P, const void* K, const int32_t* ctx_lens, int tok_begin,
                              int tok_end, void* kmax, void* kmin, uint32_t* err, hipStream_t st) {
  const int B = P.B, d = P.d_qk;
  const int span_blocks = (tok_end - tok_begin + B - 1) / B + 1;
  const int cpb = d / (P.dtype == 1 ? 8 : 4);
  int gx = (span_blocks * cpb + 255) / 256;
  gx = gx < 1 ? 1 : (gx > 4096 ? 4096 : gx);
  dim3 grid(gx, P.H_kv, P.b);
  if (P.dtype == 1)
    block_index_kernel<BF16><<<grid, 256, 0, st>>>((const uint16_t*)K, ctx_lens, P.H_kv, P.T, d, B,
                                                   P.m_max, tok_begin, tok_end, (uint16_t*)kmax,
                                                   (uint16_t*)kmin, err);
  else
    block_index_kernel<F32><<<grid, 256, 0, st>>>((const float*)K, ctx_lens, P.H_kv, P.T, d, B, P.m_max,
                                                  tok_begin, tok_end, (float*)kmax, (float*)kmin, err);
  return hipGetLastError();
}

hipError_t launch_token_index(const Problem& P, const void* K, const int32_t* ctx_lens,
                              const int32_t* channels, int tok_begin, int tok_end, uint8_t* codes,
                              float* qparams, uint32_t* err, hipStream_t st) {
  const int ngroups = P.d_c / 32;
  const long items = long(tok_end - tok_begin) * ngroups;  // half-waves of work
  long gx = (items + 7) / 8;                                // 8 half-waves per 256-thread group
  gx = gx < 1 ? 1 : (gx > 8192 ? 8192 : gx);
  dim3 grid(unsigned(gx), P.H_kv, P.b);
  if (P.dtype == 1)
    token_index_kernel<BF16><<<grid, 256, 0, st>>>((const uint16_t*)K, ctx_lens, channels, P.H_kv, P.T,
                                                   P.d_qk, P.d_c, tok_begin, tok_end, codes, qparams, err);
  else
    token_index_kernel<F32><<<grid, 256, 0, st>>>((const float*)K, ctx_lens, channels, P.H_kv, P.T,
                                                  P.d_qk, P.d_c, tok_begin, tok_end, codes, qparams, err);
  return hipGetLastError();
}

}  // namespace tls
