// Exact attention over the selected tokens for grouped-query layouts
// (AsyncTLS Sec. 4.1 final step; sparse attention as defined in Sec. 3):
//   o_h = softmax(sigma q_h K_S^T) V_S,   lse_h = log sum_j exp(sigma q_h . k_j)
// for the G query heads of each (sequence, KV head) unit.
//
// One work-group handles CT consecutive entries of a unit's token list.
// A row group of LPR = D/VEC lanes owns one token row at a time (VEC channels
// per lane, 16-byte loads), and owns TPR = 8 tokens.  Every K and V row of the
// work-group is requested before any arithmetic, so each work-group waits on
// memory once.  Scores are reduced across the row group with a transposing
// butterfly, normalised once per (head, token) in LDS against the
// work-group's per-head max, and P.V is accumulated in registers.  The
// work-group writes its normalised partial output and log-sum-exp; the merge
// kernel combines the splits.  HBM-bound: (d_qk + d_v) * sizeof(elem) bytes
// per token.
#include "attn_common.hpp"

namespace tls {

constexpr int kGqaTPR = 8;

template <class E, int D>
constexpr int gqa_ct() {
  return (256 / (D / E::kVec)) * kGqaTPR;
}

template <class E, int D, int G>
__global__ __launch_bounds__(256) void attn_gqa_kernel(
    const typename E::T* __restrict__ q, const typename E::T* __restrict__ Kp,
    const typename E::T* __restrict__ Vp, const int32_t* __restrict__ slot_map, int64_t n_slots,
    const int32_t* __restrict__ token_ids, const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int T,
    int B, int m_max, int K_t, int ct, float sigma, float* __restrict__ po, float* __restrict__ plse,
    uint32_t* err) {
  using S = typename E::T;
  constexpr int V = E::kVec;
  constexpr int LPR = D / V;          // lanes per token row
  constexpr int RG = 256 / LPR;       // row groups per work-group
  constexpr int RPW = 64 / LPR;       // row groups per wave
  constexpr int TPR = kGqaTPR;        // tokens per row group
  constexpr int CT = RG * TPR;        // token capacity of a work-group
  constexpr int NZ = TPR * G;         // (token, head) scores per row group
  constexpr int NRES = NZ / LPR > 0 ? NZ / LPR : 1;
  __shared__ float s_z[G][CT];
  __shared__ float s_m[G], s_l[G];
  __shared__ float s_acc[4][G * D];

  const int unit = blockIdx.y, split = blockIdx.x, nsplit = gridDim.x;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, li = tid % LPR, rg = tid / LPR, lane = tid & 63, wid = tid >> 6;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int p0 = split * ct, p1 = min(K_t, p0 + ct);
  const int32_t* ids = token_ids + size_t(unit) * K_t;

  // token rows of this row group, then every K/V load
  uint4 kv[TPR], vv[TPR];
  uint32_t okmask = 0;
#pragma unroll
  for (int i = 0; i < TPR; ++i) {
    const int p = p0 + rg + RG * i;
    kv[i] = vv[i] = make_uint4(0, 0, 0, 0);
    const int tok = p < p1 ? ids[p] : -1;
    if (tok >= 0) {
      if (tok >= n) {
        if (li == 0) set_error(err, 4u);
      } else {
        bool good = true;
        const S* kr = kv_row(Kp, slot_map, n_slots, unit, T, B, m_max, D, tok, &good);
        const S* vr = kv_row(Vp, slot_map, n_slots, unit, T, B, m_max, D, tok, &good);
        if (good) {
          kv[i] = ld16_stream(kr + li * V);
          vv[i] = ld16_stream(vr + li * V);
          okmask |= 1u << i;
        } else if (li == 0) {
          set_error(err, 8u);
        }
      }
    }
  }
  float qr[G][V];
  {
    const S* qg = q + (size_t(s) * H_q + size_t(g) * G) * D;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      unpack16<E>(ld16(qg + size_t(h) * D + li * V), qr[h]);
#pragma unroll
      for (int e = 0; e < V; ++e) qr[h][e] *= sigma;
    }
  }
  // partial dot products, reduced across the row group
  float z[NZ];
#pragma unroll
  for (int i = 0; i < TPR; ++i) {
    float kf[V];
    unpack16<E>(kv[i], kf);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < V; ++e) dot = fmaf(qr[h][e], kf[e], dot);
      z[i * G + h] = dot;
    }
  }
  XReduce<NZ, LPR / 2>::run(z, li);
#pragma unroll
  for (int j = 0; j < NRES; ++j) {
    const int idx = xreduce_index<NZ, LPR>(li, j);
    const int i = idx / G, h = idx % G;
    s_z[h][rg + RG * i] = ((okmask >> i) & 1u) ? z[j] : -INFINITY;
  }
  __syncthreads();
  // per-head max and exponentials over the work-group's tokens
  for (int h = wid; h < G; h += 4) {
    float mx = -INFINITY;
    for (int t = lane; t < CT; t += 64) mx = fmaxf(mx, s_z[h][t]);
    mx = wave_max<64>(mx);
    float sum = 0.f;
    for (int t = lane; t < CT; t += 64) {
      const float p = mx == -INFINITY ? 0.f : exp_or_zero(s_z[h][t] - mx);
      s_z[h][t] = p;
      sum += p;
    }
    sum = wave_sum<64>(sum);
    if (lane == 0) {
      s_m[h] = mx;
      s_l[h] = sum;
    }
  }
  __syncthreads();
  // P.V for this row group's tokens
  float acc[G][V];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int i = 0; i < TPR; ++i) {
    float vf[V];
    unpack16<E>(vv[i], vf);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float p = s_z[h][rg + RG * i];
#pragma unroll
      for (int e = 0; e < V; ++e) acc[h][e] = fmaf(p, vf[e], acc[h][e]);
    }
  }
#pragma unroll
  for (int mask = LPR; mask < 64; mask <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[h][e] += __shfl_xor(acc[h][e], mask, 64);
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < V; ++e) s_acc[wid][h * D + li * V + e] = acc[h][e];
  }
  __syncthreads();
  const size_t pbase = (size_t(unit) * nsplit + split) * G;
  for (int idx = tid; idx < G * D; idx += 256) {
    const int h = idx / D;
    const float o = (s_acc[0][idx] + s_acc[1][idx]) + (s_acc[2][idx] + s_acc[3][idx]);
    const float L = s_l[h];
    po[pbase * D + idx] = L > 0.f ? o / L : 0.f;
    if (idx % D == 0) plse[pbase + h] = L > 0.f ? s_m[h] + logf(L) : -INFINITY;
  }
  (void)RPW;
}

int gqa_tokens_per_split(const Problem& P) {
  const int V = P.dtype == 1 ? 8 : 4;
  return (256 / (P.d_qk / V)) * kGqaTPR;
}

template <class E, int D, int G>
static void launch_t(const Problem& P, const void* q, const KvView& kv, const int32_t* token_ids,
                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse, uint32_t* err,
                     hipStream_t st) {
  using S = typename E::T;
  const int ct = (K_t + nsplit - 1) / nsplit;
  dim3 grid(nsplit, P.units);
  attn_gqa_kernel<E, D, G><<<grid, 256, 0, st>>>((const S*)q, (const S*)kv.k, (const S*)kv.v, kv.slot_map,
                                                 kv.n_slots, token_ids, ctx_lens, P.H_q, P.H_kv, P.T, P.B,
                                                 P.m_max, K_t, ct, P.sigma, po, plse, err);
}

template <class E, int D>
static bool launch_d(const Problem& P, const void* q, const KvView& kv, const int32_t* token_ids,
                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse, uint32_t* err,
                     hipStream_t st) {
  switch (P.G) {
    case 1: launch_t<E, D, 1>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 2: launch_t<E, D, 2>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 4: launch_t<E, D, 4>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 8: launch_t<E, D, 8>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    default: return false;
  }
}

hipError_t launch_attention_gqa(const Problem& P, const void* q, const KvView& kv, const int32_t* token_ids,
                                const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                                uint32_t* err, hipStream_t st) {
  bool ok = false;
  if (P.dtype == 1) {
    if (P.d_qk == 128) ok = launch_d<BF16, 128>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st);
    else if (P.d_qk == 64) ok = launch_d<BF16, 64>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st);
  } else {
    if (P.d_qk == 128) ok = launch_d<F32, 128>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st);
    else if (P.d_qk == 64) ok = launch_d<F32, 64>(P, q, kv, token_ids, ctx_lens, K_t, nsplit, po, plse, err, st);
  }
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tls
