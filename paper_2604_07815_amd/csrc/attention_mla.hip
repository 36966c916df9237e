// Exact attention over the selected tokens for the absorbed MLA layout
// (AsyncTLS Sec. 4.1 final step; MLA collapsed to one shared latent head,
// Sec. 3): per unit, 32 query heads share every 576-dim row [latent; rope];
// the value is the row's first 512 dims.
//
//   scores S = Q K^T (32 x tokens x 576) and O += P V (32 x 512 x tokens) are
//   dense contractions, so both run on the matrix cores:
//   * a work-group (4 waves) walks its split in chunks of 32 tokens, double
//     buffered.  The chunk's rows are gathered into LDS with
//     global_load_lds_dwordx4 in piece-major order (16-byte piece p of row r
//     at [p][r]), so one gather instruction moves one piece of 32 rows, and
//     operand reads of 16 rows at one piece are contiguous and conflict-free;
//   * wave (token tile tt, head tile ht) computes the 16x16 tile
//     S^T = K Q^T by 18 v_mfma_f32_16x16x32_bf16 over the 576 dims, with the
//     queries staged once in LDS in the same piece-major order;
//   * the chunk's per-head max is combined through LDS, an online softmax in
//     base 2 (the running max is raised only past a 2^8 margin) turns the
//     tile into bf16 probabilities, laid out by each wave exactly as the A
//     operand of the second product;
//   * wave w owns output dims [128 w, 128 w + 128): O += P V by
//     v_mfma_f32_16x16x16_bf16 (2 token tiles x 2 head tiles x 8 dim tiles),
//     the V operand read column-wise from the piece-major chunk with
//     ds_read_b64_tr_b16.
// The work-group writes normalised partials and their log-sum-exp; the merge
// kernel combines the splits.
#include "attn_common.hpp"

namespace tls {

namespace {

constexpr int kMlaDqk = 576, kMlaDv = 512;
constexpr int kMlaPieces = kMlaDqk / 8;  // 16-byte pieces per row
constexpr int kMlaG = 32;                // query heads (two tiles of 16)
constexpr int kMlaChunk = 32;            // tokens per chunk
constexpr int kMlaMaxTPW = 1024;         // tokens per work-group
constexpr int kMlaGathers = kMlaPieces * kMlaChunk / 64 / 4;  // gathers per wave per chunk (9)

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

__host__ __device__ constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kLgkm0 = 0xC07F;

__device__ inline void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// lane i reads 16 bytes at src; the wave writes them to lds + 16*i (async)
__device__ inline void gather16(const void* src, const void* lds) {
  const uint32_t off = uint32_t(__builtin_amdgcn_readfirstlane(int(reinterpret_cast<uintptr_t>((lds_void*)lds))));
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" : : "s"(off), "v"(src) : "m0");
}

__device__ inline float xmax4(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ inline float xsum4(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ inline short bf16_rne_bits(float f) {
  uint32_t u = __float_as_uint(f);  // finite, non-negative here
  u += 0x7fffu + ((u >> 16) & 1u);
  return short(u >> 16);
}

}  // namespace

__global__ __launch_bounds__(256) void attn_mla_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp, const int32_t* __restrict__ slot_map,
    int64_t n_slots, const TokenList tl, const int32_t* __restrict__ ctx_lens, int H_q,
    int H_kv, int T, int B, int m_max, int K_t, int tpw, float sigma, float* __restrict__ po,
    float* __restrict__ plse, uint32_t* err) {
  constexpr int CT = kMlaChunk;
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr float kRaise = 8.0f;
  __shared__ __attribute__((aligned(16))) uint4 sQ[kMlaPieces][kMlaG];      // 36 KB
  __shared__ __attribute__((aligned(16))) uint4 sKV[2][kMlaPieces][CT];     // 72 KB
  __shared__ __attribute__((aligned(16))) uint2 sP[2][2][64];               // [tt][ht][lane]
  __shared__ float s_cmax[4][16], s_csum[4][16], s_sc[kMlaG], s_l[kMlaG], s_m[kMlaG];
  __shared__ int s_rows[kMlaMaxTPW];

  const int unit = blockIdx.y, split = blockIdx.x, nsplit = gridDim.x;
  const int s = unit / H_kv, g = unit % H_kv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int t16 = lane & 15, lg = lane >> 4;
  const int tt = w >> 1, ht = w & 1;  // score tile of this wave
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int p0 = split * tpw;
  const int cnt = max(0, min(tpw, K_t - p0));
  const int nch = (cnt + CT - 1) / CT;

  // resolve entries to rows of the unit's K base (-1: skip)
  {
    for (int i = tid; i < nch * CT; i += 256) {
      int row = -1;
      if (i < cnt) {
        bool bad = false;
        const int tok = list_token(tl, unit, p0 + i, n, &bad);
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
      s_rows[i] = row;
    }
  }
  const size_t ubase = slot_map ? size_t(unit) * size_t(n_slots) * B : size_t(unit) * T;
  const uint8_t* Kb = reinterpret_cast<const uint8_t*>(Kp + ubase * kMlaDqk);
  // queries, piece-major: gather i covers pieces 2i, 2i+1 of the 32 heads
  {
    const uint8_t* qb = reinterpret_cast<const uint8_t*>(q + (size_t(s) * H_q + size_t(g) * kMlaG) * kMlaDqk);
    for (int i = w; i < kMlaPieces / 2; i += 4) {
      const int piece = 2 * i + (lane >> 5), h = lane & 31;
      gather16(qb + size_t(h) * kMlaDqk * 2 + piece * 16, &sQ[2 * i][0]);
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();

  // chunk c's gathers by this wave: pieces 2(9w + j) + lane/32 of rows
  // lane%32; a skipped entry reads a valid row of the same chunk (its
  // probability is zero and its values are finite), or row 0 when the chunk
  // has none (the chunk is then not consumed)
  auto issue = [&](const int c, const int b) {
    const int r = lane & 31;
    const int row = s_rows[c * CT + r];
    const uint32_t vm = uint32_t(__builtin_amdgcn_ballot_w64(row >= 0)) & 0xffffffffu;
    const int safe = vm ? __builtin_amdgcn_readlane(row, __builtin_ctz(vm)) : 0;
    const int src = row >= 0 ? row : safe;
#pragma unroll
    for (int j = 0; j < kMlaGathers; ++j) {
      const int pp = kMlaGathers * w + j;  // piece pair
      gather16(Kb + size_t(src) * kMlaDqk * 2 + (2 * pp + (lane >> 5)) * 16, &sKV[b][2 * pp][0]);
    }
  };

  f32x4_t acc[2][8];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) acc[a][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;  // head ht*16 + t16, base 2
  const float sl2 = sigma * kLog2e;
  if (nch > 0) issue(0, 0);
  for (int c = 0; c < nch; ++c) {
    const int b = c & 1;
    wave_fence();
    if (c + 1 < nch) {
      issue(c + 1, b ^ 1);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(kMlaGathers));
    } else {
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    }
    wave_fence();
    __syncthreads();  // chunk c has landed for every wave
    {
      const uint64_t any = __builtin_amdgcn_ballot_w64(s_rows[c * CT + (lane & 31)] >= 0);
      if (any == 0) {  // uniform over the work-group: nothing to consume
        __syncthreads();
        continue;
      }
    }
    // validity of this wave's 16 tokens (lane (lg, t16): tokens 4lg + r)
    const int vrow = s_rows[c * CT + tt * 16 + t16];
    const uint32_t vmask = uint32_t(__builtin_amdgcn_ballot_w64(vrow >= 0)) & 0xffffu;
    // S^T tile: rows = tokens tt*16 + 4lg + r, col = head ht*16 + t16
    f32x4_t st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 6
    for (int kk = 0; kk < kMlaPieces / 4; ++kk) {
      const bf16x8_t ka = __builtin_bit_cast(bf16x8_t, sKV[b][kk * 4 + lg][tt * 16 + t16]);
      const bf16x8_t qb = __builtin_bit_cast(bf16x8_t, sQ[kk * 4 + lg][ht * 16 + t16]);
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb, st, 0, 0, 0);
    }
    float z[4], cm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      z[r] = ((vmask >> (lg * 4 + r)) & 1u) ? st[r] * sl2 : -INFINITY;
      cm = fmaxf(cm, z[r]);
    }
    cm = xmax4(cm);
    if (lg == 0) s_cmax[w][t16] = cm;
    __syncthreads();
    const float cmax = fmaxf(s_cmax[ht][t16], s_cmax[2 + ht][t16]);  // waves (0, ht) and (1, ht)
    const float m_new = cmax > m_run + kRaise ? cmax : m_run;
    const float sc = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
    float ps = 0.f;
    short pb[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = (z[r] == -INFINITY || m_new == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(z[r] - m_new);
      ps += p;
      pb[r] = bf16_rne_bits(p);
    }
    ps = xsum4(ps);
    sP[tt][ht][lane] = __builtin_bit_cast(uint2, i16x4_t{pb[0], pb[1], pb[2], pb[3]});
    if (lg == 0) {
      s_csum[w][t16] = ps;
      if (tt == 0) s_sc[ht * 16 + t16] = sc;
    }
    __syncthreads();
    l_run = l_run * sc + (s_csum[ht][t16] + s_csum[2 + ht][t16]);
    m_run = m_new;
    // O += P V for this wave's 128 output dims
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      float f[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) f[r] = s_sc[a * 16 + lg * 4 + r];
#pragma unroll
      for (int nt = 0; nt < 8; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[a][nt][r] *= f[r];
    }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const i16x4_t pa0 = __builtin_bit_cast(i16x4_t, sP[t2][0][lane]);
      const i16x4_t pa1 = __builtin_bit_cast(i16x4_t, sP[t2][1][lane]);
      const int vr = t2 * 16 + lg * 4 + (t16 >> 2);  // row of the V operand read
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) {
        const int dim = 128 * w + 16 * nt + 4 * (t16 & 3);
        const uint8_t* addr = reinterpret_cast<const uint8_t*>(&sKV[b][dim >> 3][vr]) + (dim & 4) * 2;
        const i16x4_t vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)addr);
        acc[0][nt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa0, vb, acc[0][nt], 0, 0, 0);
        acc[1][nt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa1, vb, acc[1][nt], 0, 0, 0);
      }
    }
    __syncthreads();  // chunk buffer, sP and the partial sums are reused next
  }
  // normalised partial output and lse; lane (lg, t16): heads a*16 + 4lg + r, dim 128w + 16nt + t16
  if (tt == 0 && lg == 0) {
    s_l[ht * 16 + t16] = l_run;
    s_m[ht * 16 + t16] = m_run;
  }
  __syncthreads();
  const size_t pbase = (size_t(unit) * nsplit + split) * kMlaG;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = a * 16 + lg * 4 + r;
      const float L = s_l[h];
      const float inv = L > 0.f ? 1.0f / L : 0.f;
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) po[(pbase + h) * kMlaDv + 128 * w + 16 * nt + t16] = acc[a][nt][r] * inv;
    }
  if (tid < kMlaG) {
    const float L = s_l[tid];
    plse[pbase + tid] = L > 0.f ? (s_m[tid] + __log2f(L)) * 0.6931471805599453f : -INFINITY;
  }
}

bool mla_mfma_ok(const Problem& P) {
  return P.mla && P.dtype == 1 && P.d_qk == kMlaDqk && P.d_v == kMlaDv && P.G == kMlaG;
}

int mla_mfma_tokens_per_split() { return kMlaMaxTPW; }

// Split count: about one work-group per compute unit, whole chunks each.
int mla_mfma_splits(const Problem& P, int K_t) {
  const int cus = device_cus();
  const int need = (K_t + kMlaMaxTPW - 1) / kMlaMaxTPW;
  int ns = (cus + P.units - 1) / P.units;
  const int max_ns = (K_t + kMlaChunk - 1) / kMlaChunk;
  if (ns > max_ns) ns = max_ns;
  if (ns > kMaxSplits) ns = kMaxSplits;
  return ns < need ? need : ns;
}

hipError_t launch_attention_mla_mfma(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                     const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                                     uint32_t* err, hipStream_t st) {
  int tpw = (K_t + nsplit - 1) / nsplit;
  tpw = (tpw + kMlaChunk - 1) / kMlaChunk * kMlaChunk;
  if (tpw > kMlaMaxTPW) return hipErrorInvalidValue;
  attn_mla_mfma_kernel<<<dim3(nsplit, P.units), 256, 0, st>>>(
      (const uint16_t*)q, (const uint16_t*)kv.k, kv.slot_map, kv.n_slots, tl, ctx_lens, P.H_q, P.H_kv, P.T,
      P.B, P.m_max, K_t, tpw, P.sigma, po, plse, err);
  return hipGetLastError();
}

}  // namespace tls
