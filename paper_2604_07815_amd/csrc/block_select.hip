// Coarse block selection (AsyncTLS Sec. 4.1).
//
// block_score_kernel: the Quest block score in the paper's GEMM form,
//   s_i = sum_h (max(q_h,0) . kmax_i + min(q_h,0) . kmin_i).
// Because the sum over the G heads of a group is linear, it is taken first:
// Q+ = sum_h max(q_h,0), Q- = sum_h min(q_h,0) (fp32, heads in ascending
// order), leaving one 2*d dot product per block - a GEMV that streams the
// block summaries once.  HBM-bound: 2*d*sizeof(elem) bytes per block.
//
// block_topk_kernel: top-K_b block ids per unit, ties to the lower id,
// ascending, -1 padded.
#include "kernels.hpp"

namespace tls {

constexpr int kBlkUnroll = 4;  // blocks in flight per lane group

// Q+ and Q- of every unit, once, for wide groups (the absorbed MLA layout:
// 32 heads x 576 dims), so the scoring work-groups do not each re-reduce
// the group's queries.  qpn: [units][2][d] fp32; the heads are summed in a
// fixed order (each quarter sequentially, then the quarters pairwise).
template <class E>
__global__ __launch_bounds__(256) void qsum_kernel(const typename E::T* __restrict__ q, int H_q, int H_kv, int G,
                                                   int d, float* __restrict__ qpn) {
  // work-group (channel chunk of 64, unit); thread (quarter, channel): the
  // heads quarter, quarter + 4, ... of one channel, then a 4-way LDS sum
  __shared__ float s_p[4][64], s_n[4][64];
  const int unit = blockIdx.y, c = blockIdx.x * 64 + (threadIdx.x & 63), qt = threadIdx.x >> 6;
  const int s = unit / H_kv, g = unit % H_kv;
  const typename E::T* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
  float p = 0.f, ng = 0.f;
  if (c < d) {
    float x[8];
    int h = qt;
    for (; h + 28 < G; h += 32) {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = E::to_f(qg[size_t(h + 4 * j) * d + c]);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        p += fmaxf(x[j], 0.f);
        ng += fminf(x[j], 0.f);
      }
    }
    for (; h < G; h += 4) {
      const float v = E::to_f(qg[size_t(h) * d + c]);
      p += fmaxf(v, 0.f);
      ng += fminf(v, 0.f);
    }
  }
  s_p[qt][threadIdx.x & 63] = p;
  s_n[qt][threadIdx.x & 63] = ng;
  __syncthreads();
  if (qt == 0 && c < d) {
    const int i = threadIdx.x;
    qpn[(size_t(unit) * 2) * d + c] = (s_p[0][i] + s_p[1][i]) + (s_p[2][i] + s_p[3][i]);
    qpn[(size_t(unit) * 2 + 1) * d + c] = (s_n[0][i] + s_n[1][i]) + (s_n[2][i] + s_n[3][i]);
  }
}

template <class E, int LPB, int CPL>
__global__ __launch_bounds__(256) void block_score_kernel(
    const typename E::T* __restrict__ q, const float* __restrict__ qpn, const typename E::T* __restrict__ kmax,
    const typename E::T* __restrict__ kmin, const int32_t* __restrict__ ctx_lens, int H_q, int H_kv,
    int G, int d, int B, int T, int m_max, int bpw, float* __restrict__ scores, uint32_t* err) {
  using S = typename E::T;
  constexpr int V = E::kVec;
  constexpr int NG = 256 / LPB;  // lane groups per work-group
  const int unit = blockIdx.y;
  const int s = unit / H_kv, g = unit % H_kv;
  const int li = threadIdx.x % LPB, grp = threadIdx.x / LPB;
  const int nch = d / V;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (threadIdx.x == 0 && blockIdx.x == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int m = (n + B - 1) / B;
  const int c0 = blockIdx.x * bpw, c1 = min(c0 + bpw, m_max);
  float* out = scores + size_t(unit) * m_max;
  if (c0 >= m) {
    for (int i = c0 + threadIdx.x; i < c1; i += 256) out[i] = -INFINITY;
    return;
  }
  const size_t ubase = size_t(unit) * m_max;
  // Loads are unconditional at clamped rows so that, with no branch around
  // each load, all of them stay in flight together: a block past the
  // work-group's last valid one re-reads that block (its result is replaced
  // by -inf below), a lane past d reads channel 0 (its partial is dropped).
  // Every row read is a written summary of the unit.
  const int blk_hi = min(c1, m) - 1;  // >= c0 here
  uint4 vmax[kBlkUnroll][CPL], vmin[kBlkUnroll][CPL];
  auto request = [&](int b0) {
#pragma unroll
    for (int u = 0; u < kBlkUnroll; ++u) {
      const int blk = b0 + u * NG;
      const int rb = blk < blk_hi ? blk : blk_hi;
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const int c = li + k * LPB;
        const int rc = c < nch ? c : 0;
        vmax[u][k] = ld16_stream(kmax + (ubase + rb) * d + rc * V);
        vmin[u][k] = ld16_stream(kmin + (ubase + rb) * d + rc * V);
      }
    }
  };
  // Q+ / Q- of this lane's channels.  Narrow groups sum the heads here, in
  // ascending order (one channel per thread, through LDS), before the first
  // batch of summaries is requested; wide groups read the per-unit sums
  // straight into registers after requesting it, so those reads overlap.
  float qp[CPL][V], qn[CPL][V];
  int b0 = c0 + grp;
  if (qpn) {
    request(b0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int c = li + k * LPB;
      const float* pp = qpn + (size_t(unit) * 2) * d + (c < nch ? c : 0) * V;
#pragma unroll
      for (int e = 0; e < V; ++e) {
        qp[k][e] = pp[e];
        qn[k][e] = pp[d + e];
      }
    }
  } else {
    __shared__ float s_qp[1024], s_qn[1024];
    const S* qg = q + (size_t(s) * H_q + size_t(g) * G) * d;
    for (int c = threadIdx.x; c < d; c += 256) {
      float p = 0.f, ng = 0.f;
      // four heads' values requested together (one memory latency, not four)
      for (int h0 = 0; h0 < G; h0 += 4) {
        S x[4];
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) x[hh] = qg[size_t(h0 + hh < G ? h0 + hh : G - 1) * d + c];
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          if (h0 + hh < G) {
            const float v = E::to_f(x[hh]);
            p += fmaxf(v, 0.f);
            ng += fminf(v, 0.f);
          }
        }
      }
      s_qp[c] = p;
      s_qn[c] = ng;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int c = li + k * LPB;
#pragma unroll
      for (int e = 0; e < V; ++e) {
        qp[k][e] = c < nch ? s_qp[c * V + e] : 0.f;
        qn[k][e] = c < nch ? s_qn[c * V + e] : 0.f;
      }
    }
    request(b0);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (;;) {
#pragma unroll
    for (int u = 0; u < kBlkUnroll; ++u) {
      const int blk = b0 + u * NG;
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        float a[V], b[V];
        unpack16<E>(vmax[u][k], a);
        unpack16<E>(vmin[u][k], b);
        float part = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) part = fmaf(qp[k][e], a[e], fmaf(qn[k][e], b[e], part));
        acc += li + k * LPB < nch ? part : 0.f;  // a lane past d read channel 0: drop it
      }
      acc = wave_sum<LPB>(acc);
      if (li == 0 && blk < c1) out[blk] = blk < m ? acc : -INFINITY;
    }
    b0 += NG * kBlkUnroll;
    if (b0 >= c1) break;
    request(b0);
    __builtin_amdgcn_sched_barrier(0);  // every load of the batch is issued before the first use
  }
}

// One work-group per unit: the unit's scores as keys in registers (thread t
// holds blocks t + 1024 j, requested together), then the work-group top-k.
template <int EPT>
__global__ __launch_bounds__(1024) void block_topk_kernel(const float* __restrict__ scores,
                                                          const int32_t* __restrict__ ctx_lens, int H_kv,
                                                          int T, int B, int m_max, int K_b,
                                                          int32_t* __restrict__ block_ids) {
  extern __shared__ uint32_t smem[];
  uint32_t* scratch = smem;
  const int unit = blockIdx.x;
  const int s = unit / H_kv;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  const float* sc = scores + size_t(unit) * m_max;
  uint32_t kr[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int i = threadIdx.x + j * 1024;
    kr[j] = i < m ? float_key(sc[i]) : kInvalidKey;
  }
  wg_topk_regs<1024, EPT>(kr, K_b, block_ids + size_t(unit) * K_b, K_b, nullptr, [](int, int i) { return int32_t(i); },
                          scratch);
}

template <class E, int LPB, int CPL>
static void launch_score_t(const Problem& P, const void* q, const void* kmax, const void* kmin,
                           const int32_t* ctx_lens, float* qpn, float* scores, uint32_t* err, hipStream_t st) {
  using S = typename E::T;
  int bpw = 64;
  if (long(P.units) * ((P.m_max + 63) / 64) < 1024) bpw = 16;
  dim3 grid((P.m_max + bpw - 1) / bpw, P.units);
  // wide groups: reduce the queries once per unit instead of in every work-group
  const bool pre = qpn && long(P.G) * P.d_qk > 2048;
  if (pre)
    qsum_kernel<E><<<dim3((P.d_qk + 63) / 64, P.units), 256, 0, st>>>((const S*)q, P.H_q, P.H_kv, P.G, P.d_qk, qpn);
  block_score_kernel<E, LPB, CPL><<<grid, 256, 0, st>>>((const S*)q, pre ? qpn : nullptr, (const S*)kmax,
                                                        (const S*)kmin, ctx_lens, P.H_q, P.H_kv, P.G, P.d_qk, P.B,
                                                        P.T, P.m_max, bpw, scores, err);
}

hipError_t launch_block_score(const Problem& P, const void* q, const void* kmax, const void* kmin,
                              const int32_t* ctx_lens, float* qpn, float* scores, uint32_t* err, hipStream_t st) {
  const int V = P.dtype == 1 ? 8 : 4;
  const int nch = P.d_qk / V;
  if (P.dtype == 1) {
    if (nch <= 16) launch_score_t<BF16, 16, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else if (nch <= 32) launch_score_t<BF16, 32, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else if (nch <= 64) launch_score_t<BF16, 64, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else launch_score_t<BF16, 64, 2>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
  } else {
    if (nch <= 16) launch_score_t<F32, 16, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else if (nch <= 32) launch_score_t<F32, 32, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else if (nch <= 64) launch_score_t<F32, 64, 1>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else if (nch <= 128) launch_score_t<F32, 64, 2>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
    else launch_score_t<F32, 64, 4>(P, q, kmax, kmin, ctx_lens, qpn, scores, err, st);
  }
  return hipGetLastError();
}

hipError_t launch_block_topk(const Problem& P, const float* scores, const int32_t* ctx_lens, int K_b,
                             int32_t* block_ids, uint32_t* err, hipStream_t st) {
  (void)err;
  const size_t lds = size_t(topk_scratch_words(1024)) * sizeof(uint32_t);
  const int ept = (P.m_max + 1023) / 1024;
  auto go = [&](auto kern) {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), lds);
    if (e != hipSuccess) return e;
    kern<<<P.units, 1024, lds, st>>>(scores, ctx_lens, P.H_kv, P.T, P.B, P.m_max, K_b, block_ids);
    return hipGetLastError();
  };
  if (ept <= 1) return go(block_topk_kernel<1>);
  if (ept <= 2) return go(block_topk_kernel<2>);
  if (ept <= 4) return go(block_topk_kernel<4>);
  if (ept <= 8) return go(block_topk_kernel<8>);
  return go(block_topk_kernel<16>);
}

}  // namespace tls
