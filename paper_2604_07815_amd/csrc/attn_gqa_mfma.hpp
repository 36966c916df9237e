// The matrix-core attention body for grouped-query layouts, launched by the
// attention kernels of attention_gqa.hip.
#pragma once

#include "attn_common.hpp"

namespace tls {

constexpr int kAttnNW = 4;       // waves per work-group (bf16 matrix-core kernel, split mode)
constexpr int kWholeNW = 12;     // waves per work-group when one work-group takes a whole unit
constexpr int kWholeTPWV = 176;  // tokens per wave in that mode: K_t <= 12 * 176 = 2112

// s_waitcnt immediates (gfx9 encoding): vmcnt in [3:0] and [15:14],
// expcnt in [6:4], lgkmcnt in [11:8].
__host__ __device__ constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 0xC07F;

// Work-group barrier for LDS traffic only: completes this wave's LDS
// accesses, then synchronises, leaving global loads (including the
// asynchronous LDS gathers of the next chunk) in flight.  The
// wavefront-scope fences keep the compiler from moving memory accesses
// across it.
__device__ inline void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

typedef __attribute__((address_space(3))) void lds_void;

// Asynchronous 16-byte-per-lane gather into LDS: lane i reads 16 bytes at
// `src` and the wave writes them to lds + 16*i.  Issued through inline asm so
// that the compiler does not order later LDS accesses behind it; completion
// is tracked explicitly with s_waitcnt vmcnt and a work-group barrier before
// the data is read, and the target buffer is not read or rewritten while a
// gather into it is in flight.
__device__ inline void gather16_to_lds(const void* src, const void* lds) {
  // the LDS destination is wave-uniform; readfirstlane puts it in an SGPR
  const uint32_t off = uint32_t(__builtin_amdgcn_readfirstlane(int(reinterpret_cast<uintptr_t>((lds_void*)lds))));
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" : : "s"(off), "v"(src) : "m0");
}

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// Compiler-level ordering point for LDS accesses around the inline-asm
// gathers (emits no instruction at wavefront scope).
__device__ inline void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// Max / sum over the lanes i, i^16, i^32, i^48 (one per DPP row) through the
// gfx950 row-swap permutes; every lane gets the same bits.
__device__ inline float xrows_max(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ inline float xrows_sum(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// bf16 grouped-query attention with both products on the matrix cores.
//
// Each wave owns a contiguous run of the work-group's token entries and walks
// it in tiles of 16 tokens, so the waves never wait for each other inside the
// loop.  Per tile:
//   * the tile's 16 K rows and 16 V rows are gathered into the wave's LDS
//     buffers with global_load_lds_dwordx4 (16 bytes per lane).  V is double
//     buffered and requested a full tile ahead; K has one buffer, refilled as
//     soon as the score product has read it.  Pieces are stored XOR-swizzled
//     by row so that the operand reads below spread over the LDS banks;
//   * transposed scores S^T = K Q^T by D/32 v_mfma_f32_16x16x32_bf16
//     (A = the tile's K rows, B = the G query heads padded to 16 columns).
//     Lane (g, i) then holds head i's scores of tokens 4g..4g+3, which is
//     exactly the A-operand layout of the second product;
//   * online softmax per head in base 2 (the running maximum is only raised
//     when a tile exceeds it by more than 2^8, so the accumulators are
//     rarely rescaled); the probabilities are rounded to bf16;
//   * O += P V by D/16 v_mfma_f32_16x16x16_bf16, with the V operand read
//     column-wise straight from the row-major tile by ds_read_b64_tr_b16.
// At the end the waves' (max, sum, accumulator) triples are merged in LDS.
// Split mode (WHOLE = false): the work-group writes one normalised partial
// and its log-sum-exp for the merge kernel.  Whole-unit mode (WHOLE = true,
// one work-group of 12 waves per unit, grid.x = 1): it writes the final
// output row in the input dtype and the lse directly.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;

__device__ inline short bf16_bits_rne(float f) {
  uint32_t u = __float_as_uint(f);  // finite, non-negative here
  u += 0x7fffu + ((u >> 16) & 1u);
  return short(u >> 16);
}

// LDS of the body: per wave, one K tile and two V tiles of 16 rows, the
// wave's resolved rows, and its (max, sum) pair for the final merge.
template <int D, int NW, int TPWV>
struct AttnGqaLds {
  alignas(16) uint8_t sK[NW][16 * D * 2];
  alignas(16) uint8_t sV[NW][2][16 * D * 2];
  int s_rows[NW][TPWV];
  float s_ml[NW][2][8];
};

template <int D, int G, int NW, int TPWV, bool WHOLE, int NT = 64 * NW>
__device__ inline void attn_gqa_mfma_body(
    AttnGqaLds<D, NW, TPWV>& lds, const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vp, const int32_t* __restrict__ slot_map, int64_t n_slots, const TokenList tl,
    const int32_t* __restrict__ ctx_lens, int H_q, int H_kv, int T, int B, int m_max, int K_t, int tpw,
    float sigma, float* __restrict__ po, float* __restrict__ plse, uint16_t* __restrict__ out,
    float* __restrict__ lse, uint32_t* err, const int unit, const int split, const int nsplit) {
  constexpr int ROWB = D * 2;     // bytes per K or V row
  constexpr int LPR = ROWB / 16;  // 16-byte pieces per row
  constexpr int RPI = 64 / LPR;   // rows per wave-wide gather
  constexpr int CT = 16;          // tokens per tile
  constexpr int NI = CT / RPI;    // gathers per tile, for K and again for V
  constexpr int NKK = D / 32;     // score steps per tile
  constexpr int NNT = D / 16;     // channel tiles of the output
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr float kRaise = 8.0f;  // base-2 headroom before the running maximum is raised
  static_assert(G <= 8 && (D == 64 || D == 128) && NI * RPI == CT, "tile geometry");
  static_assert(NT >= 64 * NW && NT % 64 == 0, "waves beyond NW only join the merge");
  auto& sK = lds.sK;
  auto& sV = lds.sV;
  auto& s_rows = lds.s_rows;
  auto& s_ml = lds.s_ml;

  const int s = unit / H_kv, g = unit % H_kv;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int li = lane % LPR, rgi = lane / LPR;  // gather geometry
  const int t = lane & 15, lg = lane >> 4;      // matrix-core geometry
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  f32x4_t acc[NNT];
  float m_run = -INFINITY, l_run = 0.f;  // head t, base-2 units
  if (w < NW) {
    const int p0 = split * tpw;
    const int cnt = max(0, min(tpw, K_t - p0));
    const int tpwv = tpw / NW;
    const int cw = max(0, min(tpwv, cnt - w * tpwv));
    const int nch = (cw + CT - 1) / CT;

    // resolve this wave's entries to rows of the unit's K/V base (-1: skip)
    {
      const int e0 = p0 + w * tpwv;
      for (int i = lane; i < nch * CT; i += 64) {
        int row = -1;
        if (i < cw) {
          bool bad = false;
          const int tok = list_token(tl, unit, e0 + i, n, &bad);
          if (bad) {
            set_error(err, 4u);
          } else if (tok >= 0) {
            if (!slot_map) {
              row = tok;
            } else {
              const int slot = slot_map[size_t(unit) * m_max + tok_block(tok, B)];
              if (slot >= 0 && slot < n_slots) row = slot * B + tok_offset(tok, B);
              else set_error(err, 8u);
            }
          }
        }
        s_rows[w][i] = row;
      }
    }
    // B operand of the score product: lane (lg, t) holds channels
    // kk*32 + lg*8 .. +8 of head t (zero for padding heads)
    bf16x8_t qb[NKK];
    {
      const uint16_t* qg = q + (size_t(s) * H_q + size_t(g) * G) * D;
  #pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        if (t < G) {
          qb[kk] = *reinterpret_cast<const bf16x8_t*>(qg + size_t(t) * D + kk * 32 + lg * 8);
        } else {
  #pragma unroll
          for (int e = 0; e < 8; ++e) qb[kk][e] = __bf16(0.0f);
        }
      }
    }
    const size_t ubase = slot_map ? size_t(unit) * size_t(n_slots) * B : size_t(unit) * T;
    const uint8_t* Kb = reinterpret_cast<const uint8_t*>(Kp + ubase * D);
    const uint8_t* Vb = reinterpret_cast<const uint8_t*>(Vp + ubase * D);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // prologue loads done before the gathers are counted
    wave_fence();

    // Tile c's 16-bit valid-token mask and this lane's gather rows; skipped
    // entries are replaced by a valid row of the same tile (its probability is
    // zero and its values are finite), or by row 0 when the tile has none (the
    // tile is then not consumed).
    struct Tile {
      uint32_t mask;
      int rows[NI];
    };
    auto tile_info = [&](const int c) {
      Tile tl;
      const int row_t = s_rows[w][c * CT + t];
      int rows[NI];
  #pragma unroll
      for (int j = 0; j < NI; ++j) rows[j] = s_rows[w][c * CT + j * RPI + rgi];
      tl.mask = uint32_t(__builtin_amdgcn_ballot_w64(row_t >= 0)) & 0xffffu;
      const int safe = tl.mask ? __builtin_amdgcn_readlane(row_t, __builtin_ctz(tl.mask)) : 0;
  #pragma unroll
      for (int j = 0; j < NI; ++j) tl.rows[j] = rows[j] < 0 ? safe : rows[j];
      return tl;
    };
    auto issue_v = [&](const Tile& tl, const int b) {
  #pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int r = j * RPI + rgi;
        gather16_to_lds(Vb + size_t(tl.rows[j]) * ROWB + (li ^ ((2 * r) % LPR)) * 16, &sV[w][b][j * 1024]);
      }
    };
    auto issue_k = [&](const Tile& tl) {
  #pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int r = j * RPI + rgi;
        gather16_to_lds(Kb + size_t(tl.rows[j]) * ROWB + (li ^ (r % LPR)) * 16, &sK[w][j * 1024]);
      }
    };

  #pragma unroll
    for (int nt = 0; nt < NNT; ++nt) acc[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const float sl2 = sigma * kLog2e;
    Tile cur = {};
    if (nch > 0) {
      cur = tile_info(0);
      issue_v(cur, 0);
      issue_k(cur);
    }
    for (int c = 0; c < nch; ++c) {
      const int b = c & 1;
      const bool more = c + 1 < nch;
      Tile nxt = {};
      wave_fence();
      if (more) {
        nxt = tile_info(c + 1);
        issue_v(nxt, b ^ 1);
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(NI));  // K and V of tile c have landed
      } else {
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      }
      wave_fence();
      const uint32_t mask_cur = cur.mask;
      // S^T: lane (lg, t) gets head t's scores of tokens 4lg + r
      f32x4_t st = {0.f, 0.f, 0.f, 0.f};
      if (mask_cur != 0u) {
        bf16x8_t ka[NKK];
  #pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
          ka[kk] = *reinterpret_cast<const bf16x8_t*>(&sK[w][t * ROWB + (((kk * 4 + lg) ^ (t % LPR)) * 16)]);
  #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[kk], qb[kk], st, 0, 0, 0);
      }
      // the K buffer is free once its reads have returned: refill it
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      wave_fence();
      if (more) issue_k(nxt);
      wave_fence();
      if (mask_cur != 0u) {
        float z[4];
        float cm = -INFINITY;
  #pragma unroll
        for (int r = 0; r < 4; ++r) {
          z[r] = ((mask_cur >> (lg * 4 + r)) & 1u) ? st[r] * sl2 : -INFINITY;
          cm = fmaxf(cm, z[r]);
        }
        cm = xrows_max(cm);  // > -inf: the tile has a valid token
        const float m_new = cm > m_run + kRaise ? cm : m_run;
        const float sc = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
        float ps = 0.f;
        short pb[4];
  #pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = z[r] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(z[r] - m_new);
          ps += p;
          pb[r] = bf16_bits_rne(p);
        }
        l_run = l_run * sc + xrows_sum(ps);
        // rescale the accumulators when a real head's maximum moved
        if (__builtin_amdgcn_ballot_w64(t < G && m_new != m_run) != 0) {
          float f[4];
  #pragma unroll
          for (int r = 0; r < 4; ++r) {
            f[r] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sc), r));
            if constexpr (G > 4) {
              const float f1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sc), 4 + r));
              f[r] = lg == 1 ? f1 : f[r];
            }
          }
  #pragma unroll
          for (int nt = 0; nt < NNT; ++nt)
  #pragma unroll
            for (int r = 0; r < 4; ++r) acc[nt][r] *= f[r];
        }
        m_run = m_new;
        const i16x4_t pa = {pb[0], pb[1], pb[2], pb[3]};
        // O += P V; the V operand of channel tile nt for lane (lg, t) is
        // rows 4lg + (t/4), channels 16nt + 4(t%4) .. +4, transposed on read
        const int vr = lg * 4 + (t >> 2);
  #pragma unroll
        for (int nt = 0; nt < NNT; ++nt) {
          const int piece = 2 * nt + ((t & 3) >> 1);
          const int off = vr * ROWB + ((piece ^ ((2 * vr) % LPR)) * 16) + (t & 1) * 8;
          const i16x4_t vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(&sV[w][b][off]));
          acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vb, acc[nt], 0, 0, 0);
        }
      }
      cur = nxt;
    }
  }
  // merge the waves through LDS: lane (lg, t) holds O rows (heads) 4lg + r,
  // channel 16nt + t
  __syncthreads();  // every wave is done with its tile buffers
  float* s_acc = reinterpret_cast<float*>(&sV[0][0][0]);
  static_assert(NW * G * D * 4 <= int(sizeof(lds.sV)), "accumulator staging fits in the V buffers");
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = lg * 4 + r;
    if (w < NW && h < G) {
#pragma unroll
      for (int nt = 0; nt < NNT; ++nt) s_acc[(w * G + h) * D + nt * 16 + t] = acc[nt][r];
    }
  }
  if (w < NW && lg == 0 && t < G) {
    s_ml[w][0][t] = m_run;
    s_ml[w][1][t] = l_run;
  }
  __syncthreads();
  const size_t pbase = (size_t(unit) * nsplit + split) * G;
  for (int idx = threadIdx.x; idx < G * D; idx += NT) {
    const int h = idx / D;
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < NW; ++v) M = fmaxf(M, s_ml[v][0][h]);
    float o = 0.f, L = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        const float f = __builtin_amdgcn_exp2f(s_ml[v][0][h] - M);
        L += f * s_ml[v][1][h];
        o += f * s_acc[(v * G) * D + idx];
      }
    }
    const float lv = L > 0.f ? (M + __log2f(L)) * 0.6931471805599453f : -INFINITY;
    if constexpr (WHOLE) {
      const size_t row = size_t(s) * H_q + size_t(g) * G + h;
      out[row * D + idx % D] = f32_to_bf16(L > 0.f ? o / L : 0.f);
      if (lse && idx % D == 0) lse[row] = lv;
    } else {
      po[pbase * D + idx] = L > 0.f ? o / L : 0.f;
      if (idx % D == 0) plse[pbase + h] = lv;
    }
  }
}


}  // namespace tls
