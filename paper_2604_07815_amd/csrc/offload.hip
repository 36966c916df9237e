// Hierarchical KV cache: incremental block transmission (AsyncTLS Sec. 4.2).
//
// Per unit, the HBM pool holds n_slots blocks of K (and V) rows.  slot_map
// maps a block id to its slot (-1: not resident) and slot_owner maps a slot
// back to its block (-1: free).  One prefetch call for a new selection M_t:
//   1. release every slot whose block is in neither M_t nor the live set
//      (the blocks the in-flight attention step may still read);
//   2. T_t = blocks of M_t without a slot (= M_t minus the resident set C_t);
//   3. give the k-th block of T_t (ascending id) the k-th free slot
//      (ascending), updating slot_map and slot_owner;
//   4. copy those blocks' rows from pinned host memory into the pool with
//      device-side loads over PCIe (no host round trip for T_t), on a few
//      work-groups that leave the chip to the overlapping decode step.
// The copy reads rows [iB, min((i+1)B, ctx_len)) of block i.
//
// The prefill side of the tier (Sec. 4.2, Fig. 2) has two more pieces:
// offload_rows_kernel copies the K/V rows written at prefill from HBM to the
// pinned host arrays the prefetch later reads, and the initial residency
// (the blocks chosen by the final prefill query) is the same plan run on an
// emptied pool, then a copy with one work-group per transfer entry.
#include "kernels.hpp"

namespace tls {

__global__ __launch_bounds__(256) void prefetch_plan_kernel(
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ newb, const int32_t* __restrict__ live,
    int K_b, int H_kv, int T, int B, int m_max, int64_t n_slots, int32_t* __restrict__ slot_map,
    int32_t* __restrict__ slot_owner, int32_t* __restrict__ transfer_count, int32_t* __restrict__ xfer,
    uint32_t* err) {
  extern __shared__ uint32_t smem[];
  uint32_t* keep = smem;                      // bitmap over the unit's blocks
  uint32_t* wsum = smem + (m_max + 31) / 32;  // 2 x 4 wave partials
  const int unit = blockIdx.x;
  const int s = unit / H_kv;
  int n = ctx_lens[s];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int m = (n + B - 1) / B;
  const int words = (m_max + 31) / 32;
  int32_t* smap = slot_map + size_t(unit) * m_max;
  int32_t* sown = slot_owner + size_t(unit) * n_slots;
  const int32_t* nb = newb + size_t(unit) * K_b;
  for (int i = threadIdx.x; i < words; i += 256) keep[i] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < K_b; i += 256) {
    const int b = nb[i];
    if (b >= 0 && b < m) atomicOr(&keep[b >> 5], 1u << (b & 31));
    else if (b >= m) set_error(err, 2u);
    if (live) {
      const int lb = live[size_t(unit) * K_b + i];
      if (lb >= 0 && lb < m) atomicOr(&keep[lb >> 5], 1u << (lb & 31));
    }
  }
  __syncthreads();
  // 1. release
  for (int64_t sl = threadIdx.x; sl < n_slots; sl += 256) {
    const int ow = sown[sl];
    if (ow >= 0 && (ow >= m || !((keep[ow >> 5] >> (ow & 31)) & 1u))) {
      if (ow < m_max && smap[ow] == int32_t(sl)) smap[ow] = -1;
      sown[sl] = -1;
    }
  }
  __syncthreads();
  // 2 + 3. ordered compaction of the new blocks and the free slots
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int32_t* list = xfer + size_t(unit) * (2 * K_b + 1);
  int ntr = 0;
  for (int base = 0; base < K_b; base += 256) {
    const int i = base + threadIdx.x;
    const int b = i < K_b ? nb[i] : -1;
    const bool need = b >= 0 && b < m && smap[b] < 0;
    const uint64_t bal = __ballot(need);
    if (lane == 0) wsum[wid] = __popcll(bal);
    __syncthreads();
    int before = ntr, tot = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wid) before += wsum[w];
      tot += wsum[w];
    }
    if (need) list[1 + 2 * (before + lanes_below(bal))] = b;
    ntr += tot;
    __syncthreads();
  }
  int nfree = 0;
  for (int64_t base = 0; base < n_slots && nfree < ntr; base += 256) {
    const int64_t sl = base + threadIdx.x;
    const bool fr = sl < n_slots && sown[sl] < 0;
    const uint64_t bal = __ballot(fr);
    if (lane == 0) wsum[wid] = __popcll(bal);
    __syncthreads();
    int before = nfree, tot = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wid) before += wsum[w];
      tot += wsum[w];
    }
    const int k = before + lanes_below(bal);
    if (fr && k < ntr) list[2 + 2 * k] = int32_t(sl);
    nfree += tot;
    __syncthreads();
  }
  const int done = min(ntr, nfree);
  if (ntr > nfree && threadIdx.x == 0) set_error(err, 16u);
  for (int k = threadIdx.x; k < done; k += 256) {
    const int b = list[1 + 2 * k], sl = list[2 + 2 * k];
    smap[b] = sl;
    sown[sl] = b;
  }
  if (threadIdx.x == 0) {
    list[0] = done;
    if (transfer_count) transfer_count[unit] = ntr;
  }
}

// The copy runs on a small, fixed number of work-groups so that it never
// holds more than a few compute units while it waits on PCIe: the decode step
// it overlaps with keeps the rest of the chip.  Work-group w walks units w,
// w + gridDim.x, ...; for each entry of a unit's transfer list it copies the
// block's K and V rows.  Every thread first requests all of its pieces of the
// block (kCopyPieces 16-byte loads per row array, enough for B rows of up to
// kCopyPieces * 4 KB / B bytes), then stores them, so each work-group keeps a
// whole block in flight over the link.
constexpr int kCopyWGs = 64;
constexpr int kCopyThreads = 256;
constexpr int kCopyPieces = 4;  // 16-byte pieces per thread and row array: 256 * 16 * 4 = 16 KB per block

__device__ inline void copy_block_rows(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, size_t bytes) {
  uint4 v[kCopyPieces];
#pragma unroll
  for (int i = 0; i < kCopyPieces; ++i) {
    const size_t o = (size_t(i) * kCopyThreads + threadIdx.x) * 16;
    if (o < bytes) v[i] = ld16(src + o);
  }
#pragma unroll
  for (int i = 0; i < kCopyPieces; ++i) {
    const size_t o = (size_t(i) * kCopyThreads + threadIdx.x) * 16;
    if (o < bytes) *reinterpret_cast<uint4*>(dst + o) = v[i];
  }
  // rows larger than the unrolled span (not used by the supported shapes)
  for (size_t o = (size_t(kCopyPieces) * kCopyThreads + threadIdx.x) * 16; o < bytes; o += kCopyThreads * 16)
    *reinterpret_cast<uint4*>(dst + o) = ld16(src + o);
}

__global__ __launch_bounds__(kCopyThreads) void prefetch_copy_kernel(
    const uint8_t* __restrict__ host_k, const uint8_t* __restrict__ host_v, const int32_t* __restrict__ ctx_lens,
    const int32_t* __restrict__ xfer, int units, int K_b, int H_kv, int T, int B, int row_k, int row_v,
    int64_t n_slots, uint8_t* __restrict__ pool_k, uint8_t* __restrict__ pool_v) {
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const int32_t* list = xfer + size_t(unit) * (2 * K_b + 1);
    const int cnt = list[0];
    const int s = unit / H_kv;
    int n = ctx_lens[s];
    n = n < 0 ? 0 : (n > T ? T : n);
    for (int k = 0; k < cnt; ++k) {
      const int b = list[1 + 2 * k], sl = list[2 + 2 * k];
      const int r0 = b * B, r1 = min(r0 + B, n);
      if (r1 <= r0) continue;
      const size_t rows = size_t(r1 - r0);
      copy_block_rows(host_k + (size_t(unit) * T + r0) * row_k,
                      pool_k + (size_t(unit) * n_slots + sl) * size_t(B) * row_k, rows * row_k);
      if (host_v)
        copy_block_rows(host_v + (size_t(unit) * T + r0) * row_v,
                        pool_v + (size_t(unit) * n_slots + sl) * size_t(B) * row_v, rows * row_v);
    }
  }
}

static hipError_t launch_plan_and_copy(const Problem& P, const void* src_k, const void* src_v,
                                       const int32_t* ctx_lens, const int32_t* block_ids_new,
                                       const int32_t* block_ids_live, int K_b, void* pool_k, void* pool_v,
                                       int64_t n_slots, int32_t* slot_map, int32_t* slot_owner,
                                       int32_t* transfer_count, int32_t* transfer_list, uint32_t* err, int copy_wgs,
                                       hipStream_t st) {
  const size_t lds = ((P.m_max + 31) / 32 + 8) * sizeof(uint32_t);
  prefetch_plan_kernel<<<P.units, 256, lds, st>>>(ctx_lens, block_ids_new, block_ids_live, K_b, P.H_kv, P.T, P.B,
                                                  P.m_max, n_slots, slot_map, slot_owner, transfer_count,
                                                  transfer_list, err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int es = P.dtype == 1 ? 2 : 4;
  const int wgs = P.units < copy_wgs ? P.units : copy_wgs;
  prefetch_copy_kernel<<<wgs, kCopyThreads, 0, st>>>((const uint8_t*)src_k, (const uint8_t*)src_v, ctx_lens,
                                                     transfer_list, P.units, K_b, P.H_kv, P.T, P.B, P.d_qk * es,
                                                     P.d_v * es, n_slots, (uint8_t*)pool_k, (uint8_t*)pool_v);
  return hipGetLastError();
}

hipError_t launch_prefetch(const Problem& P, const void* host_k, const void* host_v, const int32_t* ctx_lens,
                           const int32_t* block_ids_new, const int32_t* block_ids_live, int K_b, void* pool_k,
                           void* pool_v, int64_t n_slots, int32_t* slot_map, int32_t* slot_owner,
                           int32_t* transfer_count, int32_t* transfer_list, uint32_t* err, hipStream_t st) {
  return launch_plan_and_copy(P, host_k, host_v, ctx_lens, block_ids_new, block_ids_live, K_b, pool_k, pool_v,
                              n_slots, slot_map, slot_owner, transfer_count, transfer_list, err, kCopyWGs, st);
}

// Initial residency copy: nothing runs beside it, so every transfer entry
// gets its own work-group (grid K_b x units; entries past the unit's count
// exit at once).
__global__ __launch_bounds__(kCopyThreads) void residency_copy_kernel(
    const uint8_t* __restrict__ src_k, const uint8_t* __restrict__ src_v, const int32_t* __restrict__ ctx_lens,
    const int32_t* __restrict__ xfer, int K_b, int H_kv, int T, int B, int row_k, int row_v, int64_t n_slots,
    uint8_t* __restrict__ pool_k, uint8_t* __restrict__ pool_v) {
  const int unit = blockIdx.y, k = blockIdx.x;
  const int32_t* list = xfer + size_t(unit) * (2 * K_b + 1);
  if (k >= list[0]) return;
  int n = ctx_lens[unit / H_kv];
  n = n < 0 ? 0 : (n > T ? T : n);
  const int b = list[1 + 2 * k], sl = list[2 + 2 * k];
  const int r0 = b * B, r1 = min(r0 + B, n);
  if (r1 <= r0) return;
  const size_t rows = size_t(r1 - r0);
  copy_block_rows(src_k + (size_t(unit) * T + r0) * row_k, pool_k + (size_t(unit) * n_slots + sl) * size_t(B) * row_k,
                  rows * row_k);
  if (src_v)
    copy_block_rows(src_v + (size_t(unit) * T + r0) * row_v,
                    pool_v + (size_t(unit) * n_slots + sl) * size_t(B) * row_v, rows * row_v);
}

hipError_t launch_init_residency(const Problem& P, const void* src_k, const void* src_v, const int32_t* ctx_lens,
                                 const int32_t* block_ids, int K_b, void* pool_k, void* pool_v, int64_t n_slots,
                                 int32_t* slot_map, int32_t* slot_owner, int32_t* transfer_list, uint32_t* err,
                                 hipStream_t st) {
  // empty pool: every block unmapped, every slot free
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(slot_map), 0xffffffffu, size_t(P.units) * P.m_max, st);
  if (e == hipSuccess)
    e = launch_fill_u32(reinterpret_cast<uint32_t*>(slot_owner), 0xffffffffu, size_t(P.units) * n_slots, st);
  if (e != hipSuccess) return e;
  const size_t lds = ((P.m_max + 31) / 32 + 8) * sizeof(uint32_t);
  prefetch_plan_kernel<<<P.units, 256, lds, st>>>(ctx_lens, block_ids, nullptr, K_b, P.H_kv, P.T, P.B, P.m_max,
                                                  n_slots, slot_map, slot_owner, nullptr, transfer_list, err);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int es = P.dtype == 1 ? 2 : 4;
  residency_copy_kernel<<<dim3(unsigned(K_b), unsigned(P.units)), kCopyThreads, 0, st>>>(
      (const uint8_t*)src_k, (const uint8_t*)src_v, ctx_lens, transfer_list, K_b, P.H_kv, P.T, P.B, P.d_qk * es,
      P.d_v * es, n_slots, (uint8_t*)pool_k, (uint8_t*)pool_v);
  return hipGetLastError();
}

// Device -> pinned host copy of the rows [tok_begin, min(tok_end, ctx_len))
// of every unit (K, and V unless it aliases K).  In the dense layouts those
// rows are one contiguous byte range per unit on both sides.  Work-group w
// copies units w, w + gridDim.x, ...; a few work-groups keep enough stores in
// flight for the link and leave the rest of the chip to other work.
constexpr int kOffloadWGs = 64;

__device__ inline void copy_span(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, size_t bytes) {
  constexpr size_t step = size_t(kCopyPieces) * kCopyThreads * 16;
  for (size_t base = 0; base < bytes; base += step) {
    uint4 v[kCopyPieces];
#pragma unroll
    for (int i = 0; i < kCopyPieces; ++i) {
      const size_t o = base + (size_t(i) * kCopyThreads + threadIdx.x) * 16;
      if (o < bytes) v[i] = ld16_stream(src + o);
    }
#pragma unroll
    for (int i = 0; i < kCopyPieces; ++i) {
      const size_t o = base + (size_t(i) * kCopyThreads + threadIdx.x) * 16;
      if (o < bytes) *reinterpret_cast<uint4*>(dst + o) = v[i];
    }
  }
}

__global__ __launch_bounds__(kCopyThreads) void offload_rows_kernel(
    const uint8_t* __restrict__ k, const uint8_t* __restrict__ v, const int32_t* __restrict__ ctx_lens, int units,
    int H_kv, int T, int tok_begin, int tok_end, int row_k, int row_v, uint8_t* __restrict__ host_k,
    uint8_t* __restrict__ host_v, uint32_t* err) {
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    int n = ctx_lens[unit / H_kv];
    if (n < 0 || n > T) {
      if (threadIdx.x == 0 && unit % H_kv == 0) set_error(err, 1u);
      n = n < 0 ? 0 : T;
    }
    const int hi = min(tok_end, n);
    if (hi <= tok_begin) continue;
    const size_t rows = size_t(hi - tok_begin);
    const size_t first = size_t(unit) * T + tok_begin;
    copy_span(k + first * row_k, host_k + first * row_k, rows * row_k);
    if (v) copy_span(v + first * row_v, host_v + first * row_v, rows * row_v);
  }
}

hipError_t launch_offload_rows(const Problem& P, const void* K, const void* V, const int32_t* ctx_lens,
                               int tok_begin, int tok_end, void* host_k, void* host_v, uint32_t* err,
                               hipStream_t st) {
  const int es = P.dtype == 1 ? 2 : 4;
  const int wgs = P.units < kOffloadWGs ? P.units : kOffloadWGs;
  offload_rows_kernel<<<wgs, kCopyThreads, 0, st>>>((const uint8_t*)K, (const uint8_t*)V, ctx_lens, P.units,
                                                    P.H_kv, P.T, tok_begin, tok_end, P.d_qk * es, P.d_v * es,
                                                    (uint8_t*)host_k, (uint8_t*)host_v, err);
  return hipGetLastError();
}

}  // namespace tls
