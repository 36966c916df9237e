// Token-level selection over a whole context: the token-only operator of the
// paper's kernel study (Sec. 5; Double Sparsity), i.e. the token stage of
// Sec. 4.1 with every block of the unit as candidates.  For every valid token
// j of a unit:
//   l_hj = sigma * q~_h . dequant(k~_j)        (INT4 index on the channels C)
//   alpha_j = (1/G) sum_h exp(l_hj - m_h) / Z_h,  m_h, Z_h over all valid j
// then the K_t largest alpha (ties to the lower position), ascending.
//
//   ds_score_kernel pass 0: per chunk of tokens, each head's maximum logit
//                           and sum of exponentials;
//   ds_score_kernel pass 1: the unit's m_h, Z_h from every chunk, then the
//                           alpha keys of the chunk's tokens (recomputing the
//                           logits costs one more read of the index rows,
//                           less than writing and reading them back);
//   ds_topk_kernel:         top-K_t of the unit's keys (wg_topk_global).
// The dot products run on the vector units: per token and channel one code
// extraction and G multiply-adds, the queries broadcast from LDS.
#include "token_common.hpp"

namespace tls {

constexpr int kDsThreads = 256;
constexpr int kDsNW = kDsThreads / 64;
constexpr int kDsMaxDc = 256;
constexpr int kDsTopkThreads = 1024;
constexpr int kDsListCap = 16384;  // keys in play kept in LDS after the first radix pass

template <int G>
__host__ __device__ constexpr int ds_tpt() { return G <= 8 ? 4 : 1; }  // tokens per thread
template <int G>
__host__ __device__ constexpr int ds_chunk() { return kDsThreads * ds_tpt<G>(); }

template <class E, int G>
__global__ __launch_bounds__(kDsThreads) void ds_score_kernel(
    const typename E::T* __restrict__ q, const uint8_t* __restrict__ codes, const float* __restrict__ qparams,
    const int32_t* __restrict__ channels, const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int d, int d_c,
    int T, float sigma, int pass, int nchunks, float* __restrict__ stats, uint32_t* __restrict__ keys,
    uint32_t* err) {
  constexpr int TPT = ds_tpt<G>();
  constexpr int CH = ds_chunk<G>();
  __shared__ __attribute__((aligned(16))) float s_q[kDsMaxDc * G];  // [channel][head]
  __shared__ float s_qs[(kDsMaxDc / 32) * G];                       // [group][head]: sum of q~ over the group
  __shared__ float s_red[kDsNW][G][2];
  __shared__ float s_mz[G][2];
  __shared__ float s_tmp[kDsThreads];
  __shared__ int s_ch[kDsMaxDc];
  const int chunk = blockIdx.x, unit = blockIdx.y;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (tid == 0 && chunk == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int j0 = chunk * CH;
  if (pass == 1 && j0 >= n) return;
  const int ngr = d_c / 32;
  // the group's channel ids once (every head uses the same), then the q~ gather
  for (int c = tid; c < d_c; c += kDsThreads) {
    int ch = channels[g * d_c + c];
    if (ch < 0 || ch >= d) {
      set_error(err, 32u);
      ch = 0;
    }
    s_ch[c] = ch;
  }
  __syncthreads();
  for (int i = tid; i < G * d_c; i += kDsThreads) {
    const int h = i / d_c, c = i % d_c;
    s_q[c * G + h] = E::to_f(q[(size_t(s) * H_q + size_t(g) * G + h) * d + s_ch[c]]);
  }
  __syncthreads();
  for (int i = tid; i < G * ngr; i += kDsThreads) {
    const int gr = i / G, h = i % G;
    float a = 0.f;
    for (int c = 0; c < 32; ++c) a += s_q[(gr * 32 + c) * G + h];
    s_qs[gr * G + h] = a;
  }
  // the unit's normalisers from every chunk (pass 1): thread t folds chunks
  // t / G, t / G + 256 / G, ... of head t % G, then the partials of each head
  // are combined in a fixed order
  if (pass == 1) {
    const int h = tid % G, ks = kDsThreads / G;
    const float* st = stats + size_t(unit) * nchunks * G * 2;
    float M = -INFINITY;
#pragma unroll 4
    for (int c = tid / G; c < nchunks; c += ks) M = fmaxf(M, st[(c * G + h) * 2]);
    s_tmp[tid] = M;
    __syncthreads();
    if (tid < G) {
      float m = -INFINITY;
      for (int k = 0; k < ks; ++k) m = fmaxf(m, s_tmp[k * G + tid]);
      s_mz[tid][0] = m;
    }
    __syncthreads();
    M = s_mz[h][0];
    float Z = 0.f;
    if (M != -INFINITY) {
#pragma unroll 4
      for (int c = tid / G; c < nchunks; c += ks) {
        const float mc = st[(c * G + h) * 2], zc = st[(c * G + h) * 2 + 1];
        if (mc != -INFINITY) Z += zc * __builtin_amdgcn_exp2f(mc - M);
      }
    }
    s_tmp[tid] = Z;
    __syncthreads();
    if (tid < G) {
      float z = 0.f;
      for (int k = 0; k < ks; ++k) z += s_tmp[k * G + tid];
      s_mz[tid][1] = z > 0.f ? 1.0f / z : 0.f;
    }
  }
  __syncthreads();

  // base-2 logits of this thread's tokens j0 + tid + t*256 (-inf when invalid)
  const float sigma2 = sigma * 1.4426950408889634f;
  const size_t ubase = size_t(unit) * T;
  const int rowb = d_c / 2;
  float lg[TPT][G];
  bool ok[TPT];
#pragma unroll
  for (int t = 0; t < TPT; ++t) {
    ok[t] = j0 + tid + t * kDsThreads < n;
#pragma unroll
    for (int h = 0; h < G; ++h) lg[t][h] = 0.f;
  }
  for (int gr = 0; gr < ngr; ++gr) {
    uint4 cw[TPT];
    float2 pr[TPT];
#pragma unroll
    for (int t = 0; t < TPT; ++t) {
      const size_t row = ubase + size_t(ok[t] ? j0 + tid + t * kDsThreads : 0);
      cw[t] = ld16_stream(codes + row * rowb + gr * 16);
      pr[t] = *reinterpret_cast<const float2*>(qparams + (row * ngr + gr) * 2);
    }
    float dot[TPT][G];
#pragma unroll
    for (int t = 0; t < TPT; ++t)
#pragma unroll
      for (int h = 0; h < G; ++h) dot[t][h] = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // byte b of the dword holds channels 2b (low nibble) and 2b + 1
        const int c = gr * 32 + w * 8 + e;
        const int sh = (e >> 1) * 8 + (e & 1) * 4;
        float qv[G];
        if constexpr (G % 4 == 0) {
#pragma unroll
          for (int h = 0; h < G; h += 4) {  // 16-byte aligned: G is a multiple of 4
            const float4 v = *reinterpret_cast<const float4*>(&s_q[c * G + h]);
            qv[h] = v.x;
            qv[h + 1] = v.y;
            qv[h + 2] = v.z;
            qv[h + 3] = v.w;
          }
        } else {
#pragma unroll
          for (int h = 0; h < G; ++h) qv[h] = s_q[c * G + h];
        }
#pragma unroll
        for (int t = 0; t < TPT; ++t) {
          const uint32_t wd = w == 0 ? cw[t].x : (w == 1 ? cw[t].y : (w == 2 ? cw[t].z : cw[t].w));
          const float code = float((wd >> sh) & 15u);
#pragma unroll
          for (int h = 0; h < G; ++h) dot[t][h] = fmaf(qv[h], code, dot[t][h]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < TPT; ++t)
#pragma unroll
      for (int h = 0; h < G; ++h) lg[t][h] += fmaf(pr[t].y, s_qs[gr * G + h], pr[t].x * dot[t][h]);
  }
#pragma unroll
  for (int t = 0; t < TPT; ++t)
#pragma unroll
    for (int h = 0; h < G; ++h) lg[t][h] = ok[t] ? sigma2 * lg[t][h] : -INFINITY;

  if (pass == 0) {
    // this chunk's maximum and sum of exponentials per head
    float mx[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float m = -INFINITY;
#pragma unroll
      for (int t = 0; t < TPT; ++t) m = fmaxf(m, lg[t][h]);
      mx[h] = wave_max_f32(m);
      if (lane == 0) s_red[wid][h][0] = mx[h];
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float m = s_red[0][h][0];
#pragma unroll
      for (int w = 1; w < kDsNW; ++w) m = fmaxf(m, s_red[w][h][0]);
      mx[h] = m;
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float z = 0.f;
      if (mx[h] != -INFINITY)
#pragma unroll
        for (int t = 0; t < TPT; ++t) z += __builtin_amdgcn_exp2f(lg[t][h] - mx[h]);
      z = wave_sum_f32(z);
      if (lane == 0) s_red[wid][h][1] = z;
    }
    __syncthreads();
    if (tid < G) {
      float m = s_red[0][tid][0], z = 0.f;
      for (int w = 1; w < kDsNW; ++w) m = fmaxf(m, s_red[w][tid][0]);
      for (int w = 0; w < kDsNW; ++w) z += s_red[w][tid][1];
      float* st = stats + ((size_t(unit) * nchunks + chunk) * G + tid) * 2;
      st[0] = m;
      st[1] = z;
    }
    return;
  }
  // pass 1: alpha keys (a NaN alpha, from NaN inputs, ranks as 0)
  const float invG = 1.0f / float(G);
#pragma unroll
  for (int t = 0; t < TPT; ++t) {
    const int j = j0 + tid + t * kDsThreads;
    if (j >= n) continue;
    float a = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h) a = fmaf(__builtin_amdgcn_exp2f(lg[t][h] - s_mz[h][0]), s_mz[h][1], a);
    const float av = a * invG;
    keys[ubase + j] = av == av ? float_key(av) : float_key(0.f);
  }
}

__global__ __launch_bounds__(kDsTopkThreads) void ds_topk_kernel(const uint32_t* __restrict__ keys,
                                                                  const int32_t* __restrict__ ctx_lens, int H_kv,
                                                                  int T, int K_t, int32_t* __restrict__ token_ids) {
  extern __shared__ uint32_t smem[];
  uint32_t* scratch = smem;
  uint32_t* list = smem + topk_scratch_words(kDsTopkThreads);
  const int unit = blockIdx.x;
  int n = ctx_lens[unit / H_kv];
  n = n < 0 ? 0 : (n > T ? T : n);
  wg_topk_global<kDsTopkThreads>(keys + size_t(unit) * T, n, K_t, token_ids + size_t(unit) * K_t, K_t, scratch,
                                 list, kDsListCap);
}

size_t ds_stats_floats(const Problem& P) {
  const int ch = P.G <= 8 ? ds_chunk<8>() : ds_chunk<16>();
  return size_t(P.units) * ((P.T + ch - 1) / ch) * P.G * 2;
}

bool ds_supported(const Problem& P) {
  return (P.G == 1 || P.G == 2 || P.G == 4 || P.G == 8 || P.G == 16 || P.G == 32) && P.d_c <= kDsMaxDc;
}

template <class E, int G>
static hipError_t launch_ds_g(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                              const int32_t* channels, const int32_t* ctx_lens, float* stats, uint32_t* keys,
                              uint32_t* err, hipStream_t st) {
  using S = typename E::T;
  const int nchunks = (P.T + ds_chunk<G>() - 1) / ds_chunk<G>();
  const dim3 grid(nchunks, P.units);
  for (int pass = 0; pass < 2; ++pass) {
    ds_score_kernel<E, G><<<grid, kDsThreads, 0, st>>>((const S*)q, codes, qparams, channels, ctx_lens, P.H_q,
                                                       P.H_kv, P.d_qk, P.d_c, P.T, P.sigma, pass, nchunks, stats,
                                                       keys, err);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <class E>
static hipError_t launch_ds_e(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                              const int32_t* channels, const int32_t* ctx_lens, float* stats, uint32_t* keys,
                              uint32_t* err, hipStream_t st) {
  switch (P.G) {
    case 1: return launch_ds_g<E, 1>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    case 2: return launch_ds_g<E, 2>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    case 4: return launch_ds_g<E, 4>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    case 8: return launch_ds_g<E, 8>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    case 16: return launch_ds_g<E, 16>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    case 32: return launch_ds_g<E, 32>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_token_select_dense(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                                     const int32_t* channels, const int32_t* ctx_lens, int K_t, float* stats,
                                     uint32_t* keys, int32_t* token_ids, uint32_t* err, hipStream_t st) {
  if (!ds_supported(P)) return hipErrorInvalidValue;
  const hipError_t e = P.dtype == 1 ? launch_ds_e<BF16>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st)
                                    : launch_ds_e<F32>(P, q, codes, qparams, channels, ctx_lens, stats, keys, err, st);
  if (e != hipSuccess) return e;
  const size_t lds = (size_t(topk_scratch_words(kDsTopkThreads)) + kDsListCap) * sizeof(uint32_t);
  const hipError_t a = allow_dynamic_lds(reinterpret_cast<const void*>(ds_topk_kernel), lds);
  if (a != hipSuccess) return a;
  ds_topk_kernel<<<P.units, kDsTopkThreads, lds, st>>>(keys, ctx_lens, P.H_kv, P.T, K_t, token_ids);
  return hipGetLastError();
}

}  // namespace tls
