// Exact attention over the selected tokens for grouped-query layouts
// (AsyncTLS Sec. 4.1 final step; sparse attention as defined in Sec. 3):
//   o_h = softmax(sigma q_h K_S^T) V_S,   lse_h = log sum_j exp(sigma q_h . k_j)
// for the G query heads of each (sequence, KV head) unit.
//
// One work-group handles `tpw` consecutive entries of a unit's token list in
// chunks of 64 tokens.  The chunk's K and V rows are gathered straight into
// LDS with global_load_lds_dwordx4 (one 16-byte piece per lane, rows picked
// per lane), double-buffered: while a chunk is consumed the next one is in
// flight, and only LDS-side waits separate the stages.  Per chunk: scores
// (row groups of LPR lanes, reduced with a transposing butterfly), an online
// softmax update per head, then P.V into register accumulators.  The
// work-group writes its normalised partial output and log-sum-exp; the merge
// kernel combines the splits.  HBM-bound: (d_qk + d_v) * sizeof(elem) bytes
// per token.
#include "attn_gqa_mfma.hpp"

namespace tls {

constexpr int kAttnCT = 64;      // tokens per chunk
constexpr int kAttnMaxTPW = 512;  // tokens per work-group (fp32 kernel)
constexpr int kAttnMaxTPWBf16 = 1024;  // tokens per work-group (bf16 matrix-core kernel)

template <class E, int D, int G>
__global__ __launch_bounds__(256) void attn_gqa_kernel(
    const typename E::T* __restrict__ q, const typename E::T* __restrict__ Kp,
    const typename E::T* __restrict__ Vp, const int32_t* __restrict__ slot_map, int64_t n_slots,
    const TokenList tl, const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int T,
    int B, int m_max, int K_t, int tpw, float sigma, float* __restrict__ po, float* __restrict__ plse,
    uint32_t* err) {
  using S = typename E::T;
  constexpr int V = E::kVec;                // elements per 16-byte piece
  constexpr int ROWB = D * int(sizeof(S));  // bytes per K or V row
  constexpr int LPR = ROWB / 16;            // lanes per row
  constexpr int RPI = 64 / LPR;             // rows per wave-wide gather = row groups per wave
  constexpr int CT = kAttnCT;
  constexpr int RPW = CT / 4;               // rows per wave per chunk
  constexpr int NI = RPW / RPI;             // gathers per wave per chunk, for K and again for V
  constexpr int TPG = NI;                   // rows per row group per chunk
  constexpr int NZ = TPG * G;
  constexpr int NRES = NZ / LPR > 0 ? NZ / LPR : 1;
  static_assert(LPR * 16 == ROWB && RPI * LPR == 64 && NI * RPI == RPW, "row geometry");
  __shared__ __attribute__((aligned(16))) uint8_t sK0[CT * ROWB];
  __shared__ __attribute__((aligned(16))) uint8_t sV0[CT * ROWB];
  __shared__ __attribute__((aligned(16))) uint8_t sK1[CT * ROWB];
  __shared__ __attribute__((aligned(16))) uint8_t sV1[CT * ROWB];
  __shared__ float s_z[G][CT];
  __shared__ float s_m[G], s_l[G], s_sc[G];

  const int unit = blockIdx.y, split = blockIdx.x, nsplit = gridDim.x;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int li = lane % LPR, rgi = lane / LPR;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int p0 = split * tpw;
  const int cnt = max(0, min(tpw, K_t - p0));
  const int nch = (cnt + CT - 1) / CT;

  // this lane's gather rows for every chunk (row index within the unit's K/V
  // base, -1: skip); the lane's row group scores exactly these rows
  constexpr int NCH = kAttnMaxTPW / CT;
  int rreg[NCH][NI];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int idx = c * CT + wid * RPW + i * RPI + rgi;
      int row = -1;
      if (idx < cnt) {
        bool bad = false;
        const int tok = list_token(tl, unit, p0 + idx, n, &bad);
        if (bad) {
          if (li == 0) set_error(err, 4u);
        } else if (tok >= 0) {
          if (!slot_map) {
            row = tok;
          } else {
            const int slot = slot_map[size_t(unit) * m_max + tok_block(tok, B)];
            if (slot >= 0 && slot < n_slots) row = slot * B + tok_offset(tok, B);
            else if (li == 0) set_error(err, 8u);
          }
        }
      }
      rreg[c][i] = row;
    }
  if (tid < G) {
    s_m[tid] = -INFINITY;
    s_l[tid] = 0.f;
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
  const S* Kb = Kp + (slot_map ? size_t(unit) * size_t(n_slots) * B : size_t(unit) * T) * D;
  const S* Vb = Vp + (slot_map ? size_t(unit) * size_t(n_slots) * B : size_t(unit) * T) * D;
  __syncthreads();

  auto issue = [&](const int (&rows)[NI], uint8_t* bk, uint8_t* bv) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = wid * RPW + i * RPI;  // first row of this gather within the chunk
      const int row = rows[i];
      const size_t off = size_t(row < 0 ? 0 : row) * D + li * V;  // skipped rows read row 0 (masked later)
      gather16_to_lds(Kb + off, bk + r * ROWB);
      gather16_to_lds(Vb + off, bv + r * ROWB);
    }
  };

  float acc[G][V];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[h][e] = 0.f;

  // one chunk: wait for it, score, softmax update, P.V; prefetch the next
  auto step = [&](const int c, const int (&rows)[NI], const int (&next)[NI], const uint8_t* bk, const uint8_t* bv,
                  uint8_t* nk, uint8_t* nv) {
    if (c + 1 < nch) {
      issue(next, nk, nv);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NI));  // chunk c has landed
    } else {
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    }
    lds_barrier();
    uint32_t okmask = 0;
    float z[NZ];
#pragma unroll
    for (int j = 0; j < TPG; ++j) {
      const int row = wid * RPW + j * RPI + rgi;
      if (rows[j] >= 0) okmask |= 1u << j;
      float kf[V];
      unpack16<E>(*reinterpret_cast<const uint4*>(bk + row * ROWB + li * 16), kf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) dot = fmaf(qr[h][e], kf[e], dot);
        z[j * G + h] = dot;
      }
    }
    XReduceDpp<NZ, LPR>::run(z, li);
#pragma unroll
    for (int jj = 0; jj < NRES; ++jj) {
      const int idx = xreduce_index<NZ, LPR>(li, jj);
      const int j = idx / G, h = idx % G;
      s_z[h][wid * RPW + j * RPI + rgi] = ((okmask >> j) & 1u) ? z[jj] : -INFINITY;
    }
    lds_barrier();
    // online softmax update, one wave per head
    for (int h = wid; h < G; h += 4) {
      const float zz = s_z[h][lane];
      const float cmax = wave_max_f32(zz);
      const float m_old = s_m[h];
      const float m_new = fmaxf(m_old, cmax);
      const float p = zz == -INFINITY ? 0.f : expf(zz - m_new);
      const float csum = wave_sum_f32(p);
      s_z[h][lane] = p;
      if (lane == 0) {
        const float sc = m_old == -INFINITY ? 0.f : expf(m_old - m_new);
        s_sc[h] = sc;
        s_m[h] = m_new;
        s_l[h] = s_l[h] * sc + csum;
      }
    }
    lds_barrier();
    // P.V into the register accumulators
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float sc = s_sc[h];
#pragma unroll
      for (int e = 0; e < V; ++e) acc[h][e] *= sc;
    }
#pragma unroll
    for (int j = 0; j < TPG; ++j) {
      if ((okmask >> j) & 1u) {
        const int row = wid * RPW + j * RPI + rgi;
        float vf[V];
        unpack16<E>(*reinterpret_cast<const uint4*>(bv + row * ROWB + li * 16), vf);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = s_z[h][row];
#pragma unroll
          for (int e = 0; e < V; ++e) acc[h][e] = fmaf(p, vf[e], acc[h][e]);
        }
      }
    }
    lds_barrier();  // chunk buffers and scores free for reuse
  };
  if (nch > 0) issue(rreg[0], sK0, sV0);
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (c < nch) {
      const int cn = c + 1 < NCH ? c + 1 : c;
      if ((c & 1) == 0) step(c, rreg[c], rreg[cn], sK0, sV0, sK1, sV1);
      else step(c, rreg[c], rreg[cn], sK1, sV1, sK0, sV0);
    }
  }
  // combine the row groups of a wave, then the four waves through LDS
#pragma unroll
  for (int mask = LPR; mask < 64; mask <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[h][e] += __shfl_xor(acc[h][e], mask, 64);
  float* s_acc = reinterpret_cast<float*>(sK0);  // 4 * G * D floats fit in the chunk buffers
  static_assert(4 * G * D * 4 <= CT * ROWB, "accumulator staging fits in one chunk buffer");
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < V; ++e) s_acc[(wid * G + h) * D + li * V + e] = acc[h][e];
  }
  __syncthreads();
  const size_t pbase = (size_t(unit) * nsplit + split) * G;
  for (int idx = tid; idx < G * D; idx += 256) {
    const int h = idx / D;
    const float o = (s_acc[idx] + s_acc[G * D + idx]) + (s_acc[2 * G * D + idx] + s_acc[3 * G * D + idx]);
    const float L = s_l[h];
    po[pbase * D + idx] = L > 0.f ? o / L : 0.f;
    if (idx % D == 0) plse[pbase + h] = L > 0.f ? s_m[h] + logf(L) : -INFINITY;
  }
}

template <int D, int G, int NW, int TPWV, bool WHOLE>
__global__ __launch_bounds__(64 * NW) void attn_gqa_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp, const uint16_t* __restrict__ Vp,
    const int32_t* __restrict__ slot_map, int64_t n_slots, const TokenList tl,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int T, int B, int m_max, int K_t, int tpw,
    float sigma, float* __restrict__ po, float* __restrict__ plse, uint16_t* __restrict__ out,
    float* __restrict__ lse, uint32_t* err) {
  __shared__ AttnGqaLds<D, NW, TPWV> lds;
  attn_gqa_mfma_body<D, G, NW, TPWV, WHOLE>(lds, q, Kp, Vp, slot_map, n_slots, tl, ctx_lens, H_q, H_kv, T, B, m_max,
                                            K_t, tpw, sigma, po, plse, out, lse, err, blockIdx.y, blockIdx.x,
                                            gridDim.x);
}

bool gqa_whole_ok(const Problem& P, int K_t);

int gqa_tokens_per_split(const Problem& P) { return P.dtype == 1 ? kAttnMaxTPWBf16 : kAttnMaxTPW; }

// Work-groups of the bf16 kernel resident per compute unit (LDS-bound).
template <int D, int G>
static int mfma_wgs_per_cu() {
  static const int occ = [] {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &nb, attn_gqa_mfma_kernel<D, G, kAttnNW, kAttnMaxTPWBf16 / kAttnNW, false>, 64 * kAttnNW, 0) !=
            hipSuccess ||
        nb < 1)
      nb = 1;
    return nb;
  }();
  return occ;
}

template <int D>
static int mfma_wgs_per_cu_g(int G) {
  switch (G) {
    case 1: return mfma_wgs_per_cu<D, 1>();
    case 2: return mfma_wgs_per_cu<D, 2>();
    case 4: return mfma_wgs_per_cu<D, 4>();
    default: return mfma_wgs_per_cu<D, 8>();
  }
}

constexpr int kWideMinTokens = 768;  // tokens per 12-wave split work-group worth its prologue

// Split mode with 12-wave work-groups (the whole-unit kernel writing
// partials): chosen when the launch fits the compute units in one round and
// every work-group still has several tiles per wave, so each compute unit
// keeps twelve waves of gathers in flight instead of four.
static bool gqa_use_wide(const Problem& P, int K_t, int nsplit, int cus) {
  if (P.dtype != 1 || nsplit < 2 || long(P.units) * nsplit > cus) return false;
  const int tpw = (K_t + nsplit - 1) / nsplit;
  return tpw >= kWideMinTokens && tpw <= kWholeNW * kWholeTPWV - 16 * kWholeNW;
}

// Split count for the bf16 kernel: the work-groups of one launch are
// scheduled in rounds of (compute units x resident work-groups); pick the
// split count that minimises rounds x (tokens per work-group + a fixed
// per-work-group cost), fewest splits on ties.  0: not this kernel.
int gqa_auto_splits(const Problem& P, int K_t) {
  if (P.dtype != 1 || K_t < 1) return 0;
  const int cus = device_cus();
  // whole units (one 12-wave work-group each, no partials, no merge) when
  // they fill the compute units in whole rounds
  if (gqa_whole_ok(P, K_t) && P.units % cus == 0) return 1;
  // fewer units than compute units: as many 12-wave splits as fit in one
  // round, when they still occupy at least half of the compute units (with
  // fewer, many short 4-wave splits spread the gathers over more of the chip)
  if (P.units * 2 <= cus) {
    const int ns = cus / P.units;
    for (int w = ns; w >= 2; --w)
      if (gqa_use_wide(P, K_t, w, cus) && long(P.units) * w * 2 >= cus) return w;
  }
  const int occ = P.d_qk == 64 ? mfma_wgs_per_cu_g<64>(P.G) : mfma_wgs_per_cu_g<128>(P.G);
  const long slots = long(cus) * occ;
  constexpr long kFixedTokens = 64;  // prologue and merge cost of one work-group, in tokens
  const int step = 16 * kAttnNW;
  const int need = (K_t + kAttnMaxTPWBf16 - 1) / kAttnMaxTPWBf16;
  int best = need;
  long best_cost = -1;
  for (int ns = need; ns <= kMaxSplits; ++ns) {
    const int tpw = ((K_t + ns - 1) / ns + step - 1) / step * step;
    if (long(ns - 1) * tpw >= K_t) break;  // more splits would only add empty work-groups
    const long rounds = (long(P.units) * ns + slots - 1) / slots;
    const long cost = rounds * (tpw + kFixedTokens);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = ns;
    }
  }
  return best;
}

template <class E, int D, int G>
static void launch_t(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse, uint32_t* err,
                     hipStream_t st) {
  using S = typename E::T;
  dim3 grid(nsplit, P.units);
  int tpw = (K_t + nsplit - 1) / nsplit;
  if constexpr (E::kIsBf16) {
    if (gqa_use_wide(P, K_t, nsplit, device_cus())) {
      constexpr int wstep = 16 * kWholeNW;
      tpw = (tpw + wstep - 1) / wstep * wstep;
      attn_gqa_mfma_kernel<D, G, kWholeNW, kWholeTPWV, false><<<grid, 64 * kWholeNW, 0, st>>>(
          (const uint16_t*)q, (const uint16_t*)kv.k, (const uint16_t*)kv.v, kv.slot_map, kv.n_slots, tl, ctx_lens,
          P.H_q, P.H_kv, P.T, P.B, P.m_max, K_t, tpw, P.sigma, po, plse, nullptr, nullptr, err);
      return;
    }
    constexpr int step = 16 * kAttnNW;  // whole tiles for every wave
    tpw = (tpw + step - 1) / step * step;
    attn_gqa_mfma_kernel<D, G, kAttnNW, kAttnMaxTPWBf16 / kAttnNW, false><<<grid, 64 * kAttnNW, 0, st>>>(
        (const uint16_t*)q, (const uint16_t*)kv.k, (const uint16_t*)kv.v, kv.slot_map, kv.n_slots, tl,
        ctx_lens, P.H_q, P.H_kv, P.T, P.B, P.m_max, K_t, tpw, P.sigma, po, plse, nullptr, nullptr, err);
  } else {
    tpw = (tpw + kAttnCT - 1) / kAttnCT * kAttnCT;
    attn_gqa_kernel<E, D, G><<<grid, 256, 0, st>>>((const S*)q, (const S*)kv.k, (const S*)kv.v, kv.slot_map,
                                                   kv.n_slots, tl, ctx_lens, P.H_q, P.H_kv, P.T, P.B,
                                                   P.m_max, K_t, tpw, P.sigma, po, plse, err);
  }
}

template <class E, int D>
static bool launch_d(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse, uint32_t* err,
                     hipStream_t st) {
  switch (P.G) {
    case 1: launch_t<E, D, 1>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 2: launch_t<E, D, 2>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 4: launch_t<E, D, 4>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    case 8: launch_t<E, D, 8>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st); return true;
    default: return false;
  }
}

// One work-group of 12 waves per unit, output written directly: bf16 GQA
// with K_t <= 12 * 176.
bool gqa_whole_ok(const Problem& P, int K_t) {
  return P.dtype == 1 && !P.mla && (P.d_qk == 64 || P.d_qk == 128) && P.d_v == P.d_qk &&
         (P.G == 1 || P.G == 2 || P.G == 4 || P.G == 8) && K_t >= 1 && K_t <= kWholeNW * kWholeTPWV;
}

template <int D, int G>
static void launch_whole_t(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                           const int32_t* ctx_lens, int K_t, void* out, float* lse, uint32_t* err, hipStream_t st) {
  constexpr int step = 16 * kWholeNW;
  const int tpw = (K_t + step - 1) / step * step;
  attn_gqa_mfma_kernel<D, G, kWholeNW, kWholeTPWV, true><<<dim3(1, P.units), 64 * kWholeNW, 0, st>>>(
      (const uint16_t*)q, (const uint16_t*)kv.k, (const uint16_t*)kv.v, kv.slot_map, kv.n_slots, tl,
      ctx_lens, P.H_q, P.H_kv, P.T, P.B, P.m_max, K_t, tpw, P.sigma, nullptr, nullptr, (uint16_t*)out, lse, err);
}

template <int D>
static void launch_whole_d(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                           const int32_t* ctx_lens, int K_t, void* out, float* lse, uint32_t* err, hipStream_t st) {
  switch (P.G) {
    case 1: launch_whole_t<D, 1>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st); break;
    case 2: launch_whole_t<D, 2>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st); break;
    case 4: launch_whole_t<D, 4>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st); break;
    default: launch_whole_t<D, 8>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st); break;
  }
}

hipError_t launch_attention_gqa_whole(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                      const int32_t* ctx_lens, int K_t, void* out, float* lse, uint32_t* err,
                                      hipStream_t st) {
  if (!gqa_whole_ok(P, K_t)) return hipErrorInvalidValue;
  if (P.d_qk == 128) launch_whole_d<128>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st);
  else launch_whole_d<64>(P, q, kv, tl, ctx_lens, K_t, out, lse, err, st);
  return hipGetLastError();
}

hipError_t launch_attention_gqa(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                                uint32_t* err, hipStream_t st) {
  bool ok = false;
  if (P.dtype == 1) {
    if (P.d_qk == 128) ok = launch_d<BF16, 128>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
    else if (P.d_qk == 64) ok = launch_d<BF16, 64>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
  } else {
    if (P.d_qk == 128) ok = launch_d<F32, 128>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
    else if (P.d_qk == 64) ok = launch_d<F32, 64>(P, q, kv, tl, ctx_lens, K_t, nsplit, po, plse, err, st);
  }
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tls
