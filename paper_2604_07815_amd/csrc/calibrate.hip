// Channel set of the token index (AsyncTLS Sec. 4.1, fine-grained token
// selection): over a held-out calibration set, the importance of channel i
// for the KV group g is
//   s_i = (1/G) sum_{h in g} max|q_h[i]| * max|k_g[i]|,
// and the group keeps the d_c channels of highest importance.
//  * calib_absmax_kernel: running max |x| per (head, channel) over
//    token-major activation rows [N][H][d].  One work-group per (chunk of
//    rows, head) folds its rows in registers with 16-byte loads, combines its
//    row lanes in LDS and merges into the output with an integer atomic max:
//    |x| as bits orders like its value, so the result is exact and does not
//    depend on the order of the work-groups.
//  * calib_select_kernel: one work-group per KV head computes the scores,
//    each channel's rank among all channels (ties to the lower channel) and
//    an ascending compaction of the d_c best.
#include "kernels.hpp"

namespace tls {

constexpr int kCalThreads = 256;
constexpr int kCalRows = 256;        // calibration rows per work-group
constexpr int kCalSelThreads = 1024;  // >= d

template <class E>
__device__ inline void fold_absmax(const uint4& v, uint32_t* m);
template <>
__device__ inline void fold_absmax<F32>(const uint4& v, uint32_t* m) {
  m[0] = max(m[0], v.x & 0x7fffffffu);
  m[1] = max(m[1], v.y & 0x7fffffffu);
  m[2] = max(m[2], v.z & 0x7fffffffu);
  m[3] = max(m[3], v.w & 0x7fffffffu);
}
template <>
__device__ inline void fold_absmax<BF16>(const uint4& v, uint32_t* m) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {  // |x| of each bf16 half as the bits of its fp32 value
    m[2 * k] = max(m[2 * k], (w[k] & 0x7fffu) << 16);
    m[2 * k + 1] = max(m[2 * k + 1], w[k] & 0x7fff0000u);
  }
}

template <class E>
__global__ __launch_bounds__(kCalThreads) void calib_absmax_kernel(const typename E::T* __restrict__ x, int n, int H,
                                                                   int d, uint32_t* __restrict__ out) {
  constexpr int V = E::kVec;
  __shared__ uint32_t s_part[kCalThreads * V];  // [row lane][channel]
  const int h = blockIdx.y, tid = threadIdx.x;
  const int cpr = d / V;           // 16-byte chunks per row (<= 256)
  const int nrl = kCalThreads / cpr;  // row lanes
  const int rl = tid / cpr, c = tid % cpr;
  const int r0 = blockIdx.x * kCalRows, r1 = min(r0 + kCalRows, n);
  uint32_t m[V];
#pragma unroll
  for (int e = 0; e < V; ++e) m[e] = 0u;
  if (rl < nrl) {
    const size_t stride = size_t(H) * d;  // elements between consecutive rows of one head
    const typename E::T* p = x + size_t(h) * d + c * V;
    int r = r0 + rl;
    for (; r + 3 * nrl < r1; r += 4 * nrl) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = ld16_stream(p + size_t(r + u * nrl) * stride);
#pragma unroll
      for (int u = 0; u < 4; ++u) fold_absmax<E>(v[u], m);
    }
    for (; r < r1; r += nrl) fold_absmax<E>(ld16_stream(p + size_t(r) * stride), m);
#pragma unroll
    for (int e = 0; e < V; ++e) s_part[rl * d + c * V + e] = m[e];
  }
  __syncthreads();
  for (int i = tid; i < d; i += kCalThreads) {
    uint32_t best = 0u;
    for (int q = 0; q < nrl; ++q) best = max(best, s_part[q * d + i]);
    if (best) atomicMax(&out[size_t(h) * d + i], best);
  }
}

__global__ __launch_bounds__(kCalSelThreads) void calib_select_kernel(const float* __restrict__ qa,
                                                                      const float* __restrict__ ka, int G, int d,
                                                                      int d_c, int32_t* __restrict__ channels,
                                                                      float* __restrict__ scores) {
  __shared__ uint32_t s_key[kCalSelThreads];
  __shared__ uint32_t s_wcnt[kCalSelThreads / kWave];
  const int g = blockIdx.x, i = threadIdx.x;
  uint32_t key = 0u;
  if (i < d) {
    const float kv = ka[size_t(g) * d + i];
    float acc = 0.0f;
    for (int h = 0; h < G; ++h) acc += qa[(size_t(g) * G + h) * d + i] * kv;  // heads in order
    const float sc = acc / float(G);
    key = float_key(sc);
    s_key[i] = key;
    if (scores) scores[size_t(g) * d + i] = sc;
  }
  __syncthreads();
  // rank = channels ahead of i: higher score, or equal score and lower id
  int rank = 0;
  if (i < d) {
#pragma unroll 8
    for (int j = 0; j < d; ++j) {
      const uint32_t kj = s_key[j];
      rank += (kj > key || (kj == key && j < i)) ? 1 : 0;
    }
  }
  const bool sel = i < d && rank < d_c;
  const uint64_t bal = __ballot(sel);
  const int lane = i & (kWave - 1), w = i / kWave;
  if (lane == 0) s_wcnt[w] = uint32_t(__popcll(bal));
  __syncthreads();
  if (sel) {
    int pos = lanes_below(bal);
    for (int v = 0; v < w; ++v) pos += int(s_wcnt[v]);
    channels[size_t(g) * d_c + pos] = i;
  }
}

hipError_t launch_calib_absmax(const Problem& P, const void* x, int n, int H, float* out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  dim3 grid(unsigned((n + kCalRows - 1) / kCalRows), unsigned(H));
  if (P.dtype == 1)
    calib_absmax_kernel<BF16><<<grid, kCalThreads, 0, st>>>((const uint16_t*)x, n, H, P.d_qk, (uint32_t*)out);
  else
    calib_absmax_kernel<F32><<<grid, kCalThreads, 0, st>>>((const float*)x, n, H, P.d_qk, (uint32_t*)out);
  return hipGetLastError();
}

hipError_t launch_calib_select(const Problem& P, const float* q_absmax, const float* k_absmax, int32_t* channels,
                               float* scores, hipStream_t st) {
  calib_select_kernel<<<P.H_kv, kCalSelThreads, 0, st>>>(q_absmax, k_absmax, P.G, P.d_qk, P.d_c, channels, scores);
  return hipGetLastError();
}

}  // namespace tls
