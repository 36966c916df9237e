// Exact attention over the selected tokens (AsyncTLS Sec. 4.1, final step;
// sparse attention as defined in Sec. 3):
//   o_h = softmax(sigma q_h K_S^T) V_S,   lse_h = log sum_j exp(sigma q_h . k_j).
//
// Split-K: the K_t token ids of a unit are cut into `nsplit` contiguous
// ranges; each work-group gathers its rows, keeps an online softmax per head
// and writes a normalised partial output plus its log-sum-exp; merge_kernel
// combines the partials exactly: o = sum_s e^{lse_s - M} o_s / sum_s e^{lse_s - M}.
#include "attn_common.hpp"

namespace tls {

// ---------------------------------------------------------------------------
// Absorbed MLA (one shared latent row per token; V = K[:, :d_v]), bf16.
// A split of up to 32 tokens: rows and queries staged in LDS, scores by
// head x token pairs, local softmax, then P.V with two output columns per
// thread for all heads.
// ---------------------------------------------------------------------------
constexpr int kMlaCt = 32;
constexpr int kMlaMaxG = 32;
constexpr int kMlaMaxD = 576;
constexpr int kMlaRow = kMlaMaxD + 8;  // padded row (elements) against bank conflicts

__global__ __launch_bounds__(256) void attn_mla_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp, const int32_t* __restrict__ slot_map,
    int64_t n_slots, const TokenList tl, const int32_t* __restrict__ ctx_lens, int H_q,
    int H_kv, int G, int d, int d_v, int T, int B, int m_max, int K_t, int ct, float sigma,
    float* __restrict__ po, float* __restrict__ plse, uint32_t* err) {
  __shared__ uint16_t s_q[kMlaMaxG * kMlaRow];
  __shared__ uint16_t s_k[kMlaCt * kMlaRow];
  __shared__ float s_p[kMlaMaxG][kMlaCt];
  __shared__ float s_ml[kMlaMaxG][2];
  __shared__ int s_ok[kMlaCt];
  __shared__ int s_tok[kMlaCt];
  const int unit = blockIdx.y, split = blockIdx.x, nsplit = gridDim.x;
  const int s = unit / H_kv, g = unit % H_kv;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int p0 = split * ct, p1 = min(K_t, p0 + ct);
  const int cnt = max(0, p1 - p0);
  const int nch = d / 8;
  const uint16_t* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
  for (int i = threadIdx.x; i < G * nch; i += 256) {
    const int h = i / nch, c = i % nch;
    *reinterpret_cast<uint4*>(s_q + h * kMlaRow + c * 8) = ld16(qg + size_t(h) * d + c * 8);
  }
  if (threadIdx.x < kMlaCt) {
    int okv = 0, tok = -1;
    const int p = p0 + threadIdx.x;
    if (threadIdx.x < cnt) {
      bool bad = false;
      tok = list_token(tl, unit, p, n, &bad);
      if (bad) {
        set_error(err, 4u);
      } else if (tok >= 0) {
        bool good = true;
        kv_row(Kp, slot_map, n_slots, unit, T, B, m_max, d, tok, &good);
        if (good) okv = 1;
        else set_error(err, 8u);
      }
    }
    s_ok[threadIdx.x] = okv;
    s_tok[threadIdx.x] = tok;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kMlaCt * nch; i += 256) {
    const int t = i / nch, c = i % nch;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (s_ok[t]) {
      bool good = true;
      const int tok = s_tok[t];
      const uint16_t* kr = kv_row(Kp, slot_map, n_slots, unit, T, B, m_max, d, tok, &good);
      v = ld16_stream(kr + c * 8);
    }
    *reinterpret_cast<uint4*>(s_k + t * kMlaRow + c * 8) = v;
  }
  __syncthreads();
  // scores: thread -> token t, heads h0, h0+8, h0+16, h0+24
  {
    const int t = threadIdx.x % kMlaCt, h0 = threadIdx.x / kMlaCt;
    float z[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nch; ++c) {
      float kf[8];
      unpack16<BF16>(*reinterpret_cast<const uint4*>(s_k + t * kMlaRow + c * 8), kf);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int h = h0 + 8 * j;
        if (h < G) {
          float qf[8];
          unpack16<BF16>(*reinterpret_cast<const uint4*>(s_q + h * kMlaRow + c * 8), qf);
#pragma unroll
          for (int e = 0; e < 8; ++e) z[j] = fmaf(qf[e], kf[e], z[j]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int h = h0 + 8 * j;
      if (h < G) s_p[h][t] = s_ok[t] ? z[j] * sigma : -INFINITY;
    }
  }
  __syncthreads();
  // per-head max and sum over the split's tokens: 8 lanes per head
  {
    const int h = threadIdx.x / 8, sub = threadIdx.x % 8;
    float zz[4], mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      zz[j] = h < G ? s_p[h][sub * 4 + j] : -INFINITY;
      mx = fmaxf(mx, zz[j]);
    }
    mx = wave_max<8>(mx);
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      zz[j] = exp_or_zero(zz[j] - (mx == -INFINITY ? 0.f : mx));
      sum += zz[j];
    }
    sum = wave_sum<8>(sum);
    __syncthreads();
    if (h < G) {
#pragma unroll
      for (int j = 0; j < 4; ++j) s_p[h][sub * 4 + j] = zz[j];
      if (sub == 0) {
        s_ml[h][0] = mx;
        s_ml[h][1] = sum;
      }
    }
  }
  __syncthreads();
  // P.V: thread owns output columns 2*tid, 2*tid+1 (d_v <= 512)
  const size_t pbase = (size_t(unit) * nsplit + split) * G;
  const int v0 = 2 * threadIdx.x;
  if (v0 < d_v) {
    float o[kMlaMaxG][2];
#pragma unroll
    for (int h = 0; h < kMlaMaxG; ++h) o[h][0] = o[h][1] = 0.f;
    for (int t = 0; t < kMlaCt; ++t) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(s_k + t * kMlaRow + v0);
      const float a = bf16_lo(w), b = bf16_hi(w);
#pragma unroll
      for (int h = 0; h < kMlaMaxG; ++h) {
        if (h < G) {
          const float p = s_p[h][t];
          o[h][0] = fmaf(p, a, o[h][0]);
          o[h][1] = fmaf(p, b, o[h][1]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < kMlaMaxG; ++h) {
      if (h < G) {
        const float L = s_ml[h][1];
        po[(pbase + h) * d_v + v0] = L > 0.f ? o[h][0] / L : 0.f;
        po[(pbase + h) * d_v + v0 + 1] = L > 0.f ? o[h][1] / L : 0.f;
      }
    }
  }
  if (threadIdx.x < G) {
    const float L = s_ml[threadIdx.x][1];
    plse[pbase + threadIdx.x] = L > 0.f ? s_ml[threadIdx.x][0] + logf(L) : -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// Split merge: one work-group per (unit, head).
// ---------------------------------------------------------------------------
template <class E>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ po, const float* __restrict__ plse,
                                                    int nsplit, int G, int d_v, int H_q, int H_kv,
                                                    typename E::T* __restrict__ out, float* __restrict__ lse) {
  __shared__ float s_w[kMaxSplits];
  __shared__ float s_lse;
  const int unit = blockIdx.x / G, h = blockIdx.x % G;
  const int s = unit / H_kv, g = unit % H_kv;
  const float* ls = plse + size_t(unit) * nsplit * G + h;
  if (threadIdx.x < 64) {  // split weights e^{lse_i - M} / sum_j e^{lse_j - M}; lane l holds splits l, l + 64, ...
    constexpr int PER = kMaxSplits / 64;
    static_assert(PER * 64 == kMaxSplits, "splits per lane");
    float l[PER], e[PER];
    float lm = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = int(threadIdx.x) + 64 * j;
      l[j] = i < nsplit ? ls[size_t(i) * G] : -INFINITY;
      lm = fmaxf(lm, l[j]);
    }
    const float M = wave_max_f32(lm);
    float es = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      e[j] = (M == -INFINITY) ? 0.f : exp_or_zero(l[j] - M);
      es += e[j];
    }
    const float W = wave_sum_f32(es);
#pragma unroll
    for (int j = 0; j < PER; ++j) s_w[threadIdx.x + 64 * j] = W > 0.f ? e[j] / W : 0.f;
    if (threadIdx.x == 0) s_lse = W > 0.f ? M + logf(W) : -INFINITY;
  }
  __syncthreads();
  const size_t orow = size_t(s) * H_q + size_t(g) * G + h;
  const float* base = po + (size_t(unit) * nsplit * G + h) * d_v;
  const size_t stride = size_t(G) * d_v;  // between splits
  if (d_v % 4 == 0 && nsplit >= 8) {
    // many splits: thread (r, c) takes float4 column c of splits r, r + rows,
    // ...; every load is requested before the first use, then the rows are
    // summed in order
    __shared__ float4 s_part[256];
    const int ncol = d_v / 4;  // <= 256 = blockDim.x
    const int rows = int(blockDim.x) / ncol;
    const int c = threadIdx.x % ncol, r = threadIdx.x / ncol;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < rows) {
      constexpr int U = 8;
      for (int i0 = r; i0 < nsplit; i0 += U * rows) {
        float4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int i = i0 + u * rows;
          v[u] = i < nsplit ? reinterpret_cast<const float4*>(base + size_t(i) * stride)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int i = i0 + u * rows;
          const float w = i < nsplit ? s_w[i] : 0.f;
          acc.x = fmaf(w, v[u].x, acc.x);
          acc.y = fmaf(w, v[u].y, acc.y);
          acc.z = fmaf(w, v[u].z, acc.z);
          acc.w = fmaf(w, v[u].w, acc.w);
        }
      }
      s_part[threadIdx.x] = acc;
    }
    __syncthreads();
    if (r == 0) {
      for (int q = 1; q < rows; ++q) {
        const float4 p = s_part[q * ncol + c];
        acc.x += p.x;
        acc.y += p.y;
        acc.z += p.z;
        acc.w += p.w;
      }
      typename E::T* o = out + orow * d_v + 4 * c;
      store_out<E>(o + 0, acc.x);
      store_out<E>(o + 1, acc.y);
      store_out<E>(o + 2, acc.z);
      store_out<E>(o + 3, acc.w);
    }
  } else {
    for (int dd = threadIdx.x; dd < d_v; dd += blockDim.x) {
      float o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;
      int i = 0;
      for (; i + 4 <= nsplit; i += 4) {
        o0 = fmaf(s_w[i], base[size_t(i) * stride + dd], o0);
        o1 = fmaf(s_w[i + 1], base[size_t(i + 1) * stride + dd], o1);
        o2 = fmaf(s_w[i + 2], base[size_t(i + 2) * stride + dd], o2);
        o3 = fmaf(s_w[i + 3], base[size_t(i + 3) * stride + dd], o3);
      }
      for (; i < nsplit; ++i) o0 = fmaf(s_w[i], base[size_t(i) * stride + dd], o0);
      store_out<E>(out + orow * d_v + dd, (o0 + o1) + (o2 + o3));
    }
  }
  if (threadIdx.x == 0 && lse) lse[orow] = s_lse;
}

__global__ void fill_u32_kernel(uint32_t* p, uint32_t v, size_t n) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  fill_u32_kernel<<<unsigned(blocks), 256, 0, st>>>(p, v, n);
  return hipGetLastError();
}

int gqa_tokens_per_split(const Problem& P);
int gqa_auto_splits(const Problem& P, int K_t);
bool mla_mfma_ok(const Problem& P);
int mla_mfma_tokens_per_split();
int mla_mfma_splits(const Problem& P, int K_t);
hipError_t launch_attention_mla_mfma(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                                     uint32_t* err, hipStream_t st);
hipError_t launch_attention_gqa(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                                uint32_t* err, hipStream_t st);

int attn_tokens_per_split(const Problem& P) {
  if (P.mla) return mla_mfma_ok(P) ? mla_mfma_tokens_per_split() : kMlaCt;
  return gqa_tokens_per_split(P);
}

int attn_splits_for(const Problem& P, int K_t, int requested) {
  const int cap = attn_tokens_per_split(P);
  const int need = (K_t + cap - 1) / cap;  // fewest splits the work-group capacity allows
  int ns = requested > 0 ? requested : need;
  const int tuned = requested > 0 ? 0 : (P.mla ? (mla_mfma_ok(P) ? mla_mfma_splits(P, K_t) : 0)
                                                : gqa_auto_splits(P, K_t));
  if (tuned > 0) {
    ns = tuned;
  } else if (requested <= 0) {
    // small batches: more, shorter splits so the launch fills the chip
    while (ns * 2 <= kMaxSplits && long(P.units) * ns < 1024 && K_t / (ns * 2) >= 32) ns *= 2;
  }
  if (ns <= 1 && gqa_whole_ok(P, K_t)) return 1;  // one work-group per unit takes every token
  if (ns < need) ns = need;
  if (ns > K_t) ns = K_t;
  return ns < 1 ? 1 : ns;
}

hipError_t launch_attention(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                            const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                            uint32_t* err, hipStream_t st) {
  if (P.mla && mla_mfma_ok(P))
    return launch_attention_mla_mfma(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
  if (P.mla) {
    dim3 grid(nsplit, P.units);
    const int ct = (K_t + nsplit - 1) / nsplit;
    attn_mla_kernel<<<grid, 256, 0, st>>>((const uint16_t*)q, (const uint16_t*)kv.k, kv.slot_map, kv.n_slots,
                                          tl, ctx_lens, P.H_q, P.H_kv, P.G, P.d_qk, P.d_v, P.T, P.B,
                                          P.m_max, K_t, ct, P.sigma, po, plse, err);
    return hipGetLastError();
  }
  return launch_attention_gqa(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
}

hipError_t launch_merge(const Problem& P, const float* po, const float* plse, int nsplit, void* out, float* lse,
                        hipStream_t st) {
  const int threads = 256;  // the float4 path assigns splits to rows of 256 / (d_v / 4) threads
  if (P.dtype == 1)
    merge_kernel<BF16><<<P.units * P.G, threads, 0, st>>>(po, plse, nsplit, P.G, P.d_v, P.H_q, P.H_kv,
                                                          (uint16_t*)out, lse);
  else
    merge_kernel<F32><<<P.units * P.G, threads, 0, st>>>(po, plse, nsplit, P.G, P.d_v, P.H_q, P.H_kv,
                                                         (float*)out, lse);
  return hipGetLastError();
}

}  // namespace tls
