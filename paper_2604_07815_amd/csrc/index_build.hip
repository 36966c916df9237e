// Index construction (AsyncTLS Sec. 4.1), optionally fused with the K/V
// write-back of prefill (the prefill flow of Sec. 4.2 / Fig. 2):
//  * block index - per-channel max/min key of every block of B tokens (the
//    Quest block representation), the tail block over its valid tokens;
//  * token index - keys projected on the channel set C and quantised to
//    asymmetric uint4 per group of 32 channels (INT4 per the Sec. 5 setup),
//    with an exact float32 op sequence so the codes are reproducible bit for
//    bit.
//
// One work-group per (block, unit).  It stages the block's rows in LDS with
// coalesced 16-byte loads (taking the rows of the prefill range from the
// prefill output, and writing them to the cache on the way), then derives
// both indices from the tile, so K is read once for both.  Rows wider than
// the LDS budget are processed in passes of fewer rows; the block max/min
// then accumulate across passes in registers.
//
// Token index: one lane per (token, 32-channel group), the group uniform
// over a wave, so the channel ids are broadcast reads and every lane walks
// its own row; staged rows are padded by one word so that the 64 lanes of a
// wave reading one channel of 64 rows hit different banks.  The scale takes
// one IEEE division per (token, group); each code's quotient comes from a
// multiply by the reciprocal of the scale unless it lies within kNearHalf of
// a rounding boundary (or is not finite), where the IEEE quotient is
// computed instead, so every code equals rint of the correctly rounded
// quotient.
#include "kernels.hpp"

namespace tls {

constexpr int kIdxThreads = 256;
constexpr int kIdxTileBytes = 73984;  // LDS for staged rows: 64 padded rows of an MLA (576 x bf16) key
constexpr int kIdxMaxWords = 4;       // 4-byte words per thread in the block summary (rows <= 4 KB)
constexpr int kIdxLoadUnroll = 4;     // 16-byte loads in flight per thread
// A code from the reciprocal product is used when the product lies farther
// than this from a half-integer; its error (< 2^-17 for quotients below 16,
// with a 1-ulp reciprocal) then cannot change the rounded code.
constexpr float kNearHalf = 1.0f / 16384.0f;

enum : int { kIdxBlock = 1, kIdxToken = 2 };

struct IndexArgs {
  const uint8_t* k_src;  // prefill K rows [b][S][H_kv][d], S = tok_end - tok_begin; NULL: rows already in k
  const uint8_t* v_src;  // prefill V rows [b][S][H_kv][d_v]; NULL: no V write-back
  uint8_t* k;            // dense K cache [b][H_kv][T][d]
  uint8_t* v;            // dense V cache [b][H_kv][T][d_v]
  const int32_t* ctx_lens;
  const int32_t* channels;  // [H_kv][d_c]
  uint8_t* kmax;
  uint8_t* kmin;
  uint8_t* codes;
  float* qparams;
  int H_kv, T, d, d_v, d_c, B, m_max, tok_begin, tok_end;
  int rows_per_pass;  // rows staged in LDS at a time (B when a block fits)
  int flags;          // kIdxBlock | kIdxToken
  uint32_t* err;
};

// INT4 quantisation of one 32-channel group of a key row (the token index):
// the group's min and scale = (max - min) / 15 in IEEE float32, and the
// codes rint((x - min) / scale) clamped to [0, 15], two per byte, channel 2k
// in the low nibble of byte k (all 0 when scale == 0).  chs: the group's 32
// channel ids (already validated).  Each code's quotient comes from a
// multiply by the reciprocal of the scale unless it lies within kNearHalf of
// a rounding boundary (or is not finite), where the IEEE quotient is
// recomputed, so the codes equal rint of the correctly rounded quotient.
template <class E>
__device__ inline void quantise_group32(const typename E::T* rowp, const int* chs, float& scale_out, float& lo_out,
                                        uint4& codes_out) {
#pragma clang fp contract(off)
  float lo_v = __builtin_inff(), hi_v = -__builtin_inff();
#pragma unroll 8
  for (int j = 0; j < 32; ++j) {
    const float x = E::to_f(rowp[chs[j]]);
    lo_v = fminf(lo_v, x);
    hi_v = fmaxf(hi_v, x);
  }
  const float scale = (hi_v - lo_v) / 15.0f;  // IEEE float32 subtract and divide
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (scale != 0.0f) {
    const float rcp = __builtin_amdgcn_rcpf(scale);
    uint32_t near = 0;  // channels whose product lies near a rounding boundary
#pragma unroll 1
    for (int wi = 0; wi < 4; ++wi) {  // eight channels per 32-bit word of codes
      uint32_t acc = 0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const float q = (E::to_f(rowp[chs[wi * 8 + jj]]) - lo_v) * rcp;
        near |= uint32_t(!(fabsf(__builtin_amdgcn_fractf(q) - 0.5f) > kNearHalf && q < 16.0f)) << (wi * 8 + jj);
        // round half to even, clamp; channel 2k in the low nibble of byte k
        acc |= uint32_t(fminf(fmaxf(__builtin_rintf(q), 0.0f), 15.0f)) << (4 * jj);
      }
      w[0] = wi == 0 ? acc : w[0];
      w[1] = wi == 1 ? acc : w[1];
      w[2] = wi == 2 ? acc : w[2];
      w[3] = wi == 3 ? acc : w[3];
    }
    // rare: recompute those codes from the IEEE quotient
    for (; near != 0; near &= near - 1) {
      const int j = __builtin_ctz(near);
      const float q = fminf(fmaxf(__builtin_rintf((E::to_f(rowp[chs[j]]) - lo_v) / scale), 0.0f), 15.0f);
      const int sh = 4 * (j & 7);
      const uint32_t keep = ~(0xFu << sh), code = uint32_t(q) << sh;
      switch (j >> 3) {
        case 0: w[0] = (w[0] & keep) | code; break;
        case 1: w[1] = (w[1] & keep) | code; break;
        case 2: w[2] = (w[2] & keep) | code; break;
        default: w[3] = (w[3] & keep) | code; break;
      }
    }
  }
  scale_out = scale;
  lo_out = lo_v;
  codes_out = make_uint4(w[0], w[1], w[2], w[3]);
}

// Copies rows [r_lo, r_hi) of one unit's V from the prefill output to the cache.
__device__ inline void copy_v_rows(const IndexArgs& a, int s, int g, size_t unit, int r_lo, int r_hi, int es) {
  const int rbv = a.d_v * es;
  const size_t S = size_t(a.tok_end - a.tok_begin);
  if (rbv % 16 == 0) {
    const int cpr = rbv / 16;
    const int n = (r_hi - r_lo) * cpr;
    for (int base = 0; base < n; base += kIdxThreads * kIdxLoadUnroll) {
      uint4 x[kIdxLoadUnroll];
#pragma unroll
      for (int u = 0; u < kIdxLoadUnroll; ++u) {
        const int idx = base + u * kIdxThreads + int(threadIdx.x);
        if (idx < n) {
          const int r = r_lo + idx / cpr, c = idx % cpr;
          x[u] = ld16(a.v_src + ((size_t(s) * S + (r - a.tok_begin)) * a.H_kv + g) * rbv + c * 16);
        }
      }
#pragma unroll
      for (int u = 0; u < kIdxLoadUnroll; ++u) {
        const int idx = base + u * kIdxThreads + int(threadIdx.x);
        if (idx < n) {
          const int r = r_lo + idx / cpr, c = idx % cpr;
          *reinterpret_cast<uint4*>(a.v + (unit * a.T + r) * rbv + c * 16) = x[u];
        }
      }
    }
  } else {  // rows that are not a multiple of 16 bytes: element copies
    const int n = (r_hi - r_lo) * a.d_v;
    for (int idx = threadIdx.x; idx < n; idx += kIdxThreads) {
      const int r = r_lo + idx / a.d_v, c = idx % a.d_v;
      const uint8_t* src = a.v_src + ((size_t(s) * S + (r - a.tok_begin)) * a.H_kv + g) * rbv + c * es;
      uint8_t* dst = a.v + (unit * a.T + r) * rbv + c * es;
      if (es == 2) *reinterpret_cast<uint16_t*>(dst) = *reinterpret_cast<const uint16_t*>(src);
      else *reinterpret_cast<uint32_t*>(dst) = *reinterpret_cast<const uint32_t*>(src);
    }
  }
}

template <class E>
__global__ __launch_bounds__(kIdxThreads) void index_rows_kernel(const IndexArgs a) {
#pragma clang fp contract(off)
  constexpr int es = int(sizeof(typename E::T));
  constexpr int EPW = 4 / es;  // elements per 4-byte word
  extern __shared__ uint4 smem4[];
  const int s = blockIdx.z, g = blockIdx.y;
  const int tid = threadIdx.x;
  int n = a.ctx_lens[s];
  if (n < 0 || n > a.T) {
    if (tid == 0 && blockIdx.x == 0 && g == 0) set_error(a.err, 1u);
    n = n < 0 ? 0 : a.T;
  }
  const int hi = min(a.tok_end, n);
  const int i = a.tok_begin / a.B + int(blockIdx.x);
  const int r0 = i * a.B;
  if (r0 >= hi) return;  // block past the valid end of the range
  const int r1 = min(r0 + a.B, n);
  const size_t unit = size_t(s) * a.H_kv + g;
  const int rb = a.d * es;  // bytes per K row (multiple of 16)
  const int cpr = rb / 16;
  const int wpr = rb / 4;
  const int tsw = wpr + 1;  // words per staged row (one word of padding)
  const int R = a.rows_per_pass;
  const size_t S = size_t(a.tok_end - a.tok_begin);

  uint8_t* tile = reinterpret_cast<uint8_t*>(smem4);
  uint32_t* t32 = reinterpret_cast<uint32_t*>(smem4);
  float* part = reinterpret_cast<float*>(tile + size_t(R) * tsw * 4);  // [nph][wpr * EPW][2]
  const int nph = wpr <= kIdxThreads / 2 ? kIdxThreads / wpr : 1;
  int* s_ch = reinterpret_cast<int*>(part + (nph > 1 ? nph * wpr * EPW * 2 : 0));

  const bool do_block = a.flags & kIdxBlock, do_token = a.flags & kIdxToken;
  if (do_token) {
    for (int c = tid; c < a.d_c; c += kIdxThreads) {
      int ch = a.channels[g * a.d_c + c];
      if (ch < 0 || ch >= a.d) {  // caller-supplied channel id out of range: read channel 0
        set_error(a.err, 32u);
        ch = 0;
      }
      s_ch[c] = ch;
    }
  }
  // V write-back of the prefill rows of this block
  if (a.v_src) copy_v_rows(a, s, g, unit, max(r0, a.tok_begin), min(r1, a.tok_end), es);

  // running block max/min: thread owns word w = tid % wpr of rows ph, ph + nph, ...
  // (nph > 1), or words tid, tid + 256, ... of every row (nph == 1)
  const int ph = tid / wpr, w0 = tid % wpr;
  float mx[kIdxMaxWords][EPW], mn[kIdxMaxWords][EPW];
#pragma unroll
  for (int k = 0; k < kIdxMaxWords; ++k)
#pragma unroll
    for (int e = 0; e < EPW; ++e) {
      mx[k][e] = -__builtin_inff();
      mn[k][e] = __builtin_inff();
    }

  const int ngroups = a.d_c / 32;
  for (int pr0 = r0; pr0 < r1; pr0 += R) {
    const int nrows = min(R, r1 - pr0);
    if (pr0 != r0) __syncthreads();  // previous pass done with the tile
    // ---- stage rows [pr0, pr0 + nrows) ----
    const int nch = nrows * cpr;
    for (int base = 0; base < nch; base += kIdxThreads * kIdxLoadUnroll) {
      uint4 x[kIdxLoadUnroll];
      bool fresh[kIdxLoadUnroll];
#pragma unroll
      for (int u = 0; u < kIdxLoadUnroll; ++u) {
        const int idx = base + u * kIdxThreads + tid;
        fresh[u] = false;
        if (idx < nch) {
          const int r = pr0 + idx / cpr, cc = idx % cpr;
          fresh[u] = a.k_src && r >= a.tok_begin && r < a.tok_end;
          const uint8_t* src = fresh[u] ? a.k_src + ((size_t(s) * S + (r - a.tok_begin)) * a.H_kv + g) * rb
                                        : a.k + (unit * a.T + r) * rb;
          x[u] = ld16(src + cc * 16);
        }
      }
#pragma unroll
      for (int u = 0; u < kIdxLoadUnroll; ++u) {
        const int idx = base + u * kIdxThreads + tid;
        if (idx < nch) {
          const int rr = idx / cpr, cc = idx % cpr;
          uint32_t* dst = t32 + rr * tsw + cc * 4;
          dst[0] = x[u].x;
          dst[1] = x[u].y;
          dst[2] = x[u].z;
          dst[3] = x[u].w;
          if (fresh[u]) *reinterpret_cast<uint4*>(a.k + (unit * a.T + pr0 + rr) * rb + cc * 16) = x[u];
        }
      }
    }
    __syncthreads();

    // ---- block summary: fold the staged rows into the running max/min ----
    if (do_block) {
      if (nph > 1) {
        if (ph < nph) {
          for (int rr = ph; rr < nrows; rr += nph) {
            const uint32_t word = t32[rr * tsw + w0];
#pragma unroll
            for (int e = 0; e < EPW; ++e) {
              const float x = EPW == 2 ? (e == 0 ? bf16_lo(word) : bf16_hi(word)) : __uint_as_float(word);
              mx[0][e] = fmaxf(mx[0][e], x);
              mn[0][e] = fminf(mn[0][e], x);
            }
          }
        }
      } else {
#pragma unroll
        for (int k = 0; k < kIdxMaxWords; ++k) {
          const int w = tid + k * kIdxThreads;
          if (w < wpr) {
            for (int rr = 0; rr < nrows; ++rr) {
              const uint32_t word = t32[rr * tsw + w];
#pragma unroll
              for (int e = 0; e < EPW; ++e) {
                const float x = EPW == 2 ? (e == 0 ? bf16_lo(word) : bf16_hi(word)) : __uint_as_float(word);
                mx[k][e] = fmaxf(mx[k][e], x);
                mn[k][e] = fminf(mn[k][e], x);
              }
            }
          }
        }
      }
    }

    // ---- token index of the staged rows inside [tok_begin, hi) ----
    if (do_token) {
      const int lo = max(pr0, a.tok_begin) - pr0, up = min(pr0 + nrows, hi) - pr0;
      for (int k = tid; k < 64 * ngroups; k += kIdxThreads) {
        const int rr = k & 63, grp = k >> 6;  // lane = row of the pass, wave-uniform group
        if (rr < lo || rr >= up) continue;
        const typename E::T* rowp = reinterpret_cast<const typename E::T*>(t32 + rr * tsw);
        float scale, lo_v;
        uint4 cw;
        quantise_group32<E>(rowp, s_ch + grp * 32, scale, lo_v, cw);
        const size_t trow = unit * size_t(a.T) + (pr0 + rr);
        *reinterpret_cast<uint4*>(a.codes + trow * (a.d_c / 2) + grp * 16) = cw;
        *reinterpret_cast<float2*>(a.qparams + (trow * ngroups + grp) * 2) = make_float2(scale, lo_v + 0.0f);
      }
    }
  }

  // ---- block summary: combine the row phases and store ----
  if (do_block) {
    uint8_t* pmax = a.kmax + (unit * a.m_max + i) * rb;
    uint8_t* pmin = a.kmin + (unit * a.m_max + i) * rb;
    if (nph > 1) {
      if (ph < nph)
#pragma unroll
        for (int e = 0; e < EPW; ++e) {
          part[((ph * wpr + w0) * EPW + e) * 2 + 0] = mx[0][e];
          part[((ph * wpr + w0) * EPW + e) * 2 + 1] = mn[0][e];
        }
      __syncthreads();
      if (tid < wpr) {
        float fx[EPW], fn[EPW];
#pragma unroll
        for (int e = 0; e < EPW; ++e) {
          fx[e] = -__builtin_inff();
          fn[e] = __builtin_inff();
        }
        for (int p = 0; p < nph; ++p)
#pragma unroll
          for (int e = 0; e < EPW; ++e) {
            fx[e] = fmaxf(fx[e], part[((p * wpr + tid) * EPW + e) * 2 + 0]);
            fn[e] = fminf(fn[e], part[((p * wpr + tid) * EPW + e) * 2 + 1]);
          }
        // the values are exact copies of inputs; + 0.0f turns -0.0 into +0.0
        uint32_t wx, wn;
        if (EPW == 2) {
          wx = uint32_t(f32_to_bf16(fx[0] + 0.0f)) | (uint32_t(f32_to_bf16(fx[EPW - 1] + 0.0f)) << 16);
          wn = uint32_t(f32_to_bf16(fn[0] + 0.0f)) | (uint32_t(f32_to_bf16(fn[EPW - 1] + 0.0f)) << 16);
        } else {
          wx = __float_as_uint(fx[0] + 0.0f);
          wn = __float_as_uint(fn[0] + 0.0f);
        }
        reinterpret_cast<uint32_t*>(pmax)[tid] = wx;
        reinterpret_cast<uint32_t*>(pmin)[tid] = wn;
      }
    } else {
#pragma unroll
      for (int k = 0; k < kIdxMaxWords; ++k) {
        const int w = tid + k * kIdxThreads;
        if (w < wpr) {
          uint32_t wx, wn;
          if (EPW == 2) {
            wx = uint32_t(f32_to_bf16(mx[k][0] + 0.0f)) | (uint32_t(f32_to_bf16(mx[k][EPW - 1] + 0.0f)) << 16);
            wn = uint32_t(f32_to_bf16(mn[k][0] + 0.0f)) | (uint32_t(f32_to_bf16(mn[k][EPW - 1] + 0.0f)) << 16);
          } else {
            wx = __float_as_uint(mx[k][0] + 0.0f);
            wn = __float_as_uint(mn[k][0] + 0.0f);
          }
          reinterpret_cast<uint32_t*>(pmax)[w] = wx;
          reinterpret_cast<uint32_t*>(pmin)[w] = wn;
        }
      }
    }
  }
}

size_t index_rows_lds_bytes(int rb, int rows_per_pass, int d_c, int es) {
  const int wpr = rb / 4;
  const int nph = wpr <= kIdxThreads / 2 ? kIdxThreads / wpr : 1;
  const size_t part = nph > 1 ? size_t(nph) * wpr * (4 / es) * 2 * sizeof(float) : 0;
  return size_t(rows_per_pass) * (rb + 4) + part + size_t(d_c) * sizeof(int);
}

static hipError_t launch_index_rows(const Problem& P, const void* k_src, const void* v_src, void* K, void* V,
                                    const int32_t* ctx_lens, const int32_t* channels, int tok_begin, int tok_end,
                                    void* kmax, void* kmin, uint8_t* codes, float* qparams, int flags,
                                    uint32_t* err, hipStream_t st) {
  const int es = P.dtype == 1 ? 2 : 4;
  const int rb = P.d_qk * es;
  IndexArgs a;
  a.k_src = (const uint8_t*)k_src;
  a.v_src = (const uint8_t*)v_src;
  a.k = (uint8_t*)K;
  a.v = (uint8_t*)V;
  a.ctx_lens = ctx_lens;
  a.channels = channels;
  a.kmax = (uint8_t*)kmax;
  a.kmin = (uint8_t*)kmin;
  a.codes = codes;
  a.qparams = qparams;
  a.H_kv = P.H_kv;
  a.T = P.T;
  a.d = P.d_qk;
  a.d_v = P.d_v;
  a.d_c = P.d_c;
  a.B = P.B;
  a.m_max = P.m_max;
  a.tok_begin = tok_begin;
  a.tok_end = tok_end;
  a.rows_per_pass = kIdxTileBytes / (rb + 4) < P.B ? kIdxTileBytes / (rb + 4) : P.B;
  a.flags = flags;
  a.err = err;
  const int nblk = (tok_end + P.B - 1) / P.B - tok_begin / P.B;  // blocks overlapping the range
  dim3 grid(unsigned(nblk), unsigned(P.H_kv), unsigned(P.b));
  const size_t lds = index_rows_lds_bytes(rb, a.rows_per_pass, (flags & kIdxToken) ? P.d_c : 0, es);
  if (P.dtype == 1) index_rows_kernel<BF16><<<grid, kIdxThreads, lds, st>>>(a);
  else index_rows_kernel<F32><<<grid, kIdxThreads, lds, st>>>(a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Block summaries alone (the standalone block-index build): no staging tile.
// A work-group takes kSumBlocks consecutive blocks of one unit; thread
// (row group rg, 16-byte column c) folds the rows rg, rg + nrg, ... of a block
// in registers with four loads in flight, the nrg partials are combined
// through LDS, and the first cpr threads write the block's max and min rows
// (fmax / fmin over the block's valid rows, -0 written as +0, as the fused
// builder does).  Blocks with no valid row are left untouched.
// ---------------------------------------------------------------------------
constexpr int kSumThreads = 256;
constexpr int kSumBlocks = 4;  // blocks per work-group

template <class E>
__global__ __launch_bounds__(kSumThreads) void block_summary_kernel(
    const uint8_t* __restrict__ K, const int32_t* __restrict__ ctx_lens, int H_kv, int T, int d, int B, int m_max,
    int tok_begin, int tok_end, uint8_t* __restrict__ kmax, uint8_t* __restrict__ kmin, uint32_t* err) {
  constexpr int V = E::kVec;  // elements per 16 bytes
  __shared__ float s_mx[kSumThreads][V], s_mn[kSumThreads][V];
  const int s = blockIdx.z, g = blockIdx.y, tid = threadIdx.x;
  int n = ctx_lens[s];
  if (n < 0 || n > T) {
    if (tid == 0 && blockIdx.x == 0 && g == 0) set_error(err, 1u);
    n = n < 0 ? 0 : T;
  }
  const int hi = min(tok_end, n);
  const size_t unit = size_t(s) * H_kv + g;
  const int rb = d * int(sizeof(typename E::T));  // bytes per row (multiple of 16)
  const int cpr = rb / 16;                         // <= 256
  const int nrg = kSumThreads / cpr;
  const int c = tid % cpr, rg = tid / cpr;
  const int first = tok_begin / B + int(blockIdx.x) * kSumBlocks;
  for (int bi = 0; bi < kSumBlocks; ++bi) {
    const int i = first + bi;
    const int r0 = i * B;
    if (r0 >= hi) break;  // past the valid end of the range (uniform)
    const int nr = min(r0 + B, n) - r0;
    float mx[V], mn[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
      mx[e] = -INFINITY;
      mn[e] = INFINITY;
    }
    auto fold = [&](const uint4& x) {
      float f[V];
      unpack16<E>(x, f);
#pragma unroll
      for (int e = 0; e < V; ++e) {
        mx[e] = fmaxf(mx[e], f[e]);
        mn[e] = fminf(mn[e], f[e]);
      }
    };
    if (rg < nrg) {
      const uint8_t* base = K + (unit * T + r0) * size_t(rb) + size_t(c) * 16;
      int r = rg;
      for (; r + 3 * nrg < nr; r += 4 * nrg) {
        uint4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) x[u] = ld16_stream(base + size_t(r + u * nrg) * rb);
#pragma unroll
        for (int u = 0; u < 4; ++u) fold(x[u]);
      }
      for (; r < nr; r += nrg) fold(ld16_stream(base + size_t(r) * rb));
    }
    if (bi > 0) __syncthreads();  // the previous block's partials have been read
#pragma unroll
    for (int e = 0; e < V; ++e) {
      s_mx[tid][e] = mx[e];
      s_mn[tid][e] = mn[e];
    }
    __syncthreads();
    if (tid < cpr) {
#pragma unroll
      for (int e = 0; e < V; ++e) {
        mx[e] = s_mx[tid][e];
        mn[e] = s_mn[tid][e];
      }
      for (int q = 1; q < nrg; ++q) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          mx[e] = fmaxf(mx[e], s_mx[q * cpr + tid][e]);
          mn[e] = fminf(mn[e], s_mn[q * cpr + tid][e]);
        }
      }
      uint32_t wx[4], wn[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (E::kIsBf16) {
          wx[k] = uint32_t(f32_to_bf16(mx[2 * k] + 0.0f)) | (uint32_t(f32_to_bf16(mx[2 * k + 1] + 0.0f)) << 16);
          wn[k] = uint32_t(f32_to_bf16(mn[2 * k] + 0.0f)) | (uint32_t(f32_to_bf16(mn[2 * k + 1] + 0.0f)) << 16);
        } else {
          wx[k] = __float_as_uint(mx[k] + 0.0f);
          wn[k] = __float_as_uint(mn[k] + 0.0f);
        }
      }
      const size_t off = (unit * m_max + i) * size_t(rb) + size_t(tid) * 16;
      *reinterpret_cast<uint4*>(kmax + off) = make_uint4(wx[0], wx[1], wx[2], wx[3]);
      *reinterpret_cast<uint4*>(kmin + off) = make_uint4(wn[0], wn[1], wn[2], wn[3]);
    }
  }
}

hipError_t launch_block_index(const Problem& P, const void* K, const int32_t* ctx_lens, int tok_begin,
                              int tok_end, void* kmax, void* kmin, uint32_t* err, hipStream_t st) {
  const int rb = P.d_qk * (P.dtype == 1 ? 2 : 4);
  if (rb % 16 != 0 || rb / 16 > kSumThreads)  // not the shapes the library accepts; the general builder
    return launch_index_rows(P, nullptr, nullptr, const_cast<void*>(K), nullptr, ctx_lens, nullptr, tok_begin,
                             tok_end, kmax, kmin, nullptr, nullptr, kIdxBlock, err, st);
  const int nblk = (tok_end + P.B - 1) / P.B - tok_begin / P.B;  // blocks overlapping the range
  dim3 grid(unsigned((nblk + kSumBlocks - 1) / kSumBlocks), unsigned(P.H_kv), unsigned(P.b));
  if (P.dtype == 1)
    block_summary_kernel<BF16><<<grid, kSumThreads, 0, st>>>((const uint8_t*)K, ctx_lens, P.H_kv, P.T, P.d_qk, P.B,
                                                             P.m_max, tok_begin, tok_end, (uint8_t*)kmax,
                                                             (uint8_t*)kmin, err);
  else
    block_summary_kernel<F32><<<grid, kSumThreads, 0, st>>>((const uint8_t*)K, ctx_lens, P.H_kv, P.T, P.d_qk, P.B,
                                                            P.m_max, tok_begin, tok_end, (uint8_t*)kmax,
                                                            (uint8_t*)kmin, err);
  return hipGetLastError();
}

hipError_t launch_token_index(const Problem& P, const void* K, const int32_t* ctx_lens,
                              const int32_t* channels, int tok_begin, int tok_end, uint8_t* codes,
                              float* qparams, uint32_t* err, hipStream_t st) {
  return launch_index_rows(P, nullptr, nullptr, const_cast<void*>(K), nullptr, ctx_lens, channels, tok_begin,
                           tok_end, nullptr, nullptr, codes, qparams, kIdxToken, err, st);
}

hipError_t launch_prefill_kv(const Problem& P, const void* k_src, const void* v_src, const int32_t* ctx_lens,
                             const int32_t* channels, int tok_begin, int tok_end, void* K, void* V, void* kmax,
                             void* kmin, uint8_t* codes, float* qparams, uint32_t* err, hipStream_t st) {
  return launch_index_rows(P, k_src, v_src, K, V, ctx_lens, channels, tok_begin, tok_end, kmax, kmin, codes,
                           qparams, kIdxBlock | kIdxToken, err, st);
}

// ---------------------------------------------------------------------------
// Append during decode: the token at t = ctx_len - 1 of every sequence.  One
// work-group per unit writes the new K (and V) row to the cache (device or
// pinned host memory) and, when its block is resident in the pool, to the
// block's slot; updates the block summary incrementally (the row itself when
// t opens the block, else the elementwise max / min of the stored summary and
// the row: the exact max / min of the block's rows, as a rebuild gives); and
// quantises the row for the token index.
// ---------------------------------------------------------------------------
struct AppendArgs {
  const uint8_t* k_new;  // [b][H_kv][d]
  const uint8_t* v_new;  // [b][H_kv][d_v]; NULL when V aliases K
  uint8_t* k;            // dense K [b][H_kv][T][d]
  uint8_t* v;            // dense V, or NULL
  const int32_t* ctx_lens;
  const int32_t* channels;
  uint8_t* kmax;
  uint8_t* kmin;
  uint8_t* codes;
  float* qparams;
  uint8_t* pool_k;  // [units][n_slots][B][d], or NULL
  uint8_t* pool_v;
  const int32_t* slot_map;  // [units][m_max], or NULL
  int64_t n_slots;
  int H_kv, T, d, d_v, d_c, B, m_max;
  uint32_t* err;
};

template <class E>
__device__ inline uint32_t fold_word(uint32_t old, uint32_t x, bool take_max) {
  if constexpr (E::kIsBf16) {
    const float lo = take_max ? fmaxf(bf16_lo(old), bf16_lo(x)) : fminf(bf16_lo(old), bf16_lo(x));
    const float hi = take_max ? fmaxf(bf16_hi(old), bf16_hi(x)) : fminf(bf16_hi(old), bf16_hi(x));
    return uint32_t(f32_to_bf16(lo + 0.0f)) | (uint32_t(f32_to_bf16(hi + 0.0f)) << 16);
  } else {
    const float a = __uint_as_float(old), b = __uint_as_float(x);
    return __float_as_uint((take_max ? fmaxf(a, b) : fminf(a, b)) + 0.0f);
  }
}

template <class E>
__device__ inline uint32_t plus_zero_word(uint32_t x) {  // -0.0 -> +0.0, element by element
  if constexpr (E::kIsBf16) {
    return uint32_t(f32_to_bf16(bf16_lo(x) + 0.0f)) | (uint32_t(f32_to_bf16(bf16_hi(x) + 0.0f)) << 16);
  } else {
    return __float_as_uint(__uint_as_float(x) + 0.0f);
  }
}

template <class E>
__global__ __launch_bounds__(kIdxThreads) void append_token_kernel(const AppendArgs a) {
  constexpr int es = int(sizeof(typename E::T));
  extern __shared__ uint4 smem4[];
  uint32_t* s_row = reinterpret_cast<uint32_t*>(smem4);  // the new key row
  const int unit = blockIdx.x, tid = threadIdx.x;
  const int s = unit / a.H_kv;
  const int n = a.ctx_lens[s];
  if (n < 0 || n > a.T) {
    if (tid == 0) set_error(a.err, 1u);
    return;
  }
  if (n == 0) return;
  const int t = n - 1, blk = t / a.B, r = t % a.B;
  const int rb = a.d * es, wpr = rb / 4;
  int* s_ch = reinterpret_cast<int*>(s_row + wpr);
  int slot = -1;
  if (a.slot_map) {
    slot = a.slot_map[size_t(unit) * a.m_max + blk];
    if (slot >= a.n_slots) {
      if (tid == 0) set_error(a.err, 8u);
      slot = -1;
    }
  }
  // the row in 16-byte pieces (rows are a multiple of 16 bytes): the stores to
  // a host-memory cache then leave the chip as whole 16-byte writes
  const uint8_t* src = a.k_new + size_t(unit) * rb;
  uint8_t* dk = a.k + (size_t(unit) * a.T + t) * rb;
  uint8_t* dp = slot >= 0 ? a.pool_k + ((size_t(unit) * a.n_slots + slot) * a.B + r) * rb : nullptr;
  for (int c = tid; c < rb / 16; c += kIdxThreads) {
    const uint4 x = ld16(src + c * 16);
    reinterpret_cast<uint4*>(s_row)[c] = x;
    *reinterpret_cast<uint4*>(dk + c * 16) = x;
    if (dp) *reinterpret_cast<uint4*>(dp + c * 16) = x;
  }
  __syncthreads();
  uint32_t* smx = reinterpret_cast<uint32_t*>(a.kmax + (size_t(unit) * a.m_max + blk) * rb);
  uint32_t* smn = reinterpret_cast<uint32_t*>(a.kmin + (size_t(unit) * a.m_max + blk) * rb);
  for (int w = tid; w < wpr; w += kIdxThreads) {
    const uint32_t x = s_row[w];
    if (r == 0) {  // the row opens its block
      const uint32_t z = plus_zero_word<E>(x);
      smx[w] = z;
      smn[w] = z;
    } else {
      smx[w] = fold_word<E>(smx[w], x, true);
      smn[w] = fold_word<E>(smn[w], x, false);
    }
  }
  if (a.v_new) {
    const int rbv = a.d_v * es;
    const uint8_t* vs = a.v_new + size_t(unit) * rbv;
    uint8_t* dv = a.v + (size_t(unit) * a.T + t) * rbv;
    uint8_t* pv = slot >= 0 ? a.pool_v + ((size_t(unit) * a.n_slots + slot) * a.B + r) * rbv : nullptr;
    if (rbv % 16 == 0) {
      for (int c = tid; c < rbv / 16; c += kIdxThreads) {
        const uint4 x = ld16(vs + c * 16);
        *reinterpret_cast<uint4*>(dv + c * 16) = x;
        if (pv) *reinterpret_cast<uint4*>(pv + c * 16) = x;
      }
    } else {
      for (int e = tid; e < a.d_v; e += kIdxThreads) {  // rows that are not a multiple of 16 bytes
        if constexpr (E::kIsBf16) {
          const uint16_t x = reinterpret_cast<const uint16_t*>(vs)[e];
          reinterpret_cast<uint16_t*>(dv)[e] = x;
          if (pv) reinterpret_cast<uint16_t*>(pv)[e] = x;
        } else {
          const uint32_t x = reinterpret_cast<const uint32_t*>(vs)[e];
          reinterpret_cast<uint32_t*>(dv)[e] = x;
          if (pv) reinterpret_cast<uint32_t*>(pv)[e] = x;
        }
      }
    }
  }
  const int g = unit % a.H_kv;
  for (int c = tid; c < a.d_c; c += kIdxThreads) {
    int ch = a.channels[g * a.d_c + c];
    if (ch < 0 || ch >= a.d) {  // caller-supplied channel id out of range: read channel 0
      set_error(a.err, 32u);
      ch = 0;
    }
    s_ch[c] = ch;
  }
  __syncthreads();
  const int ngroups = a.d_c / 32;
  if (tid < ngroups) {
    float scale, lo;
    uint4 cw;
    quantise_group32<E>(reinterpret_cast<const typename E::T*>(s_row), s_ch + tid * 32, scale, lo, cw);
    const size_t trow = size_t(unit) * a.T + t;
    *reinterpret_cast<uint4*>(a.codes + trow * (a.d_c / 2) + tid * 16) = cw;
    *reinterpret_cast<float2*>(a.qparams + (trow * ngroups + tid) * 2) = make_float2(scale, lo + 0.0f);
  }
}

hipError_t launch_append_tokens(const Problem& P, const void* k_new, const void* v_new, const int32_t* ctx_lens,
                                const int32_t* channels, void* K, void* V, void* kmax, void* kmin, uint8_t* codes,
                                float* qparams, void* pool_k, void* pool_v, const int32_t* slot_map, int64_t n_slots,
                                uint32_t* err, hipStream_t st) {
  AppendArgs a;
  a.k_new = (const uint8_t*)k_new;
  a.v_new = (const uint8_t*)v_new;
  a.k = (uint8_t*)K;
  a.v = (uint8_t*)V;
  a.ctx_lens = ctx_lens;
  a.channels = channels;
  a.kmax = (uint8_t*)kmax;
  a.kmin = (uint8_t*)kmin;
  a.codes = codes;
  a.qparams = qparams;
  a.pool_k = (uint8_t*)pool_k;
  a.pool_v = (uint8_t*)pool_v;
  a.slot_map = slot_map;
  a.n_slots = n_slots;
  a.H_kv = P.H_kv;
  a.T = P.T;
  a.d = P.d_qk;
  a.d_v = P.d_v;
  a.d_c = P.d_c;
  a.B = P.B;
  a.m_max = P.m_max;
  a.err = err;
  const int es = P.dtype == 1 ? 2 : 4;
  const size_t lds = size_t(P.d_qk) * es + size_t(P.d_c) * sizeof(int);
  if (P.dtype == 1) append_token_kernel<BF16><<<P.units, kIdxThreads, lds, st>>>(a);
  else append_token_kernel<F32><<<P.units, kIdxThreads, lds, st>>>(a);
  return hipGetLastError();
}

}  // namespace tls
