// C ABI of libtls.so: host-side validation (nothing is enqueued on error),
// workspace carving and stage dispatch.  See include/tls.h for the contract.
#include <math.h>
#include <string.h>

#include <mutex>

#include "tls.h"
#include "kernels.hpp"

using tls::Problem;

// Scratch of tls_sparse_decode_noalloc, 64 MiB per device (see
// scratch_of_current_device for how host code reaches it).
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kHeaderBytes = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

tls_status make_problem(const tls_layout* L, Problem* P) {
  if (!L) return TLS_ERR_INVALID_ARGUMENT;
  if (L->batch < 1 || L->num_q_heads < 1 || L->num_kv_heads < 1) return TLS_ERR_INVALID_ARGUMENT;
  if (L->num_q_heads % L->num_kv_heads != 0) return TLS_ERR_INVALID_ARGUMENT;
  if (L->head_dim_qk < 1 || L->head_dim_v < 1 || L->block_size < 1 || L->max_ctx < 1) return TLS_ERR_INVALID_ARGUMENT;
  if (L->index_channels < 32 || L->index_channels % 32 != 0 || L->index_channels > L->head_dim_qk)
    return TLS_ERR_INVALID_ARGUMENT;
  if (L->dtype != TLS_DTYPE_F32 && L->dtype != TLS_DTYPE_BF16) return TLS_ERR_INVALID_ARGUMENT;
  if (L->mla_shared_kv != 0 && L->mla_shared_kv != 1) return TLS_ERR_INVALID_ARGUMENT;
  if (L->mla_shared_kv && L->head_dim_v > L->head_dim_qk) return TLS_ERR_INVALID_ARGUMENT;
  if (!(L->softmax_scale == L->softmax_scale) || isinf(L->softmax_scale)) return TLS_ERR_INVALID_ARGUMENT;
  // supported subset of the library
  if (L->block_size != 64) return TLS_ERR_UNSUPPORTED;
  if (L->head_dim_qk % 8 != 0 || L->head_dim_qk > 1024) return TLS_ERR_UNSUPPORTED;
  if (L->index_channels > 256) return TLS_ERR_UNSUPPORTED;
  const int G = L->num_q_heads / L->num_kv_heads;
  if (G > 32) return TLS_ERR_UNSUPPORTED;
  const long m_max = (long(L->max_ctx) + L->block_size - 1) / L->block_size;
  if (m_max > tls::kMaxKeys) return TLS_ERR_UNSUPPORTED;
  const long units = long(L->batch) * L->num_kv_heads;
  if (units > 65535) return TLS_ERR_UNSUPPORTED;
  P->b = L->batch;
  P->H_q = L->num_q_heads;
  P->H_kv = L->num_kv_heads;
  P->G = G;
  P->d_qk = L->head_dim_qk;
  P->d_v = L->head_dim_v;
  P->B = L->block_size;
  P->d_c = L->index_channels;
  P->T = L->max_ctx;
  P->m_max = int(m_max);
  P->dtype = L->dtype;
  P->mla = L->mla_shared_kv;
  P->sigma = L->softmax_scale > 0.f ? L->softmax_scale : float(1.0 / sqrt(double(L->head_dim_qk)));
  P->units = int(units);
  return TLS_OK;
}

// Device address of caller-owned pinned host memory (hipHostMalloc or
// registered); false for pageable host memory or device memory.
bool pinned_device_ptr(const void* p, const void** out) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess || a.type != hipMemoryTypeHost || !a.devicePointer) {
    (void)hipGetLastError();
    return false;
  }
  *out = static_cast<const char*>(a.devicePointer) + (static_cast<const char*>(p) - static_cast<const char*>(a.hostPointer));
  return true;
}

// Device address of either device memory or pinned host memory.
bool readable_ptr(const void* p, const void** out) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (a.type == hipMemoryTypeDevice) {
    *out = p;
    return true;
  }
  return pinned_device_ptr(p, out);
}

tls_status check_budgets(const Problem& P, int K_b, int K_t) {
  if (K_b < 1 || K_t < 1) return TLS_ERR_INVALID_ARGUMENT;
  if (long(K_b) * P.B > tls::kMaxKeys) return TLS_ERR_UNSUPPORTED;
  return TLS_OK;
}

tls_status check_attention(const Problem& P, int K_t) {
  if (P.mla) {
    if (P.dtype != TLS_DTYPE_BF16 || P.d_qk > 576 || P.d_v > 512 || P.d_v % 2 != 0) return TLS_ERR_UNSUPPORTED;
  } else {
    if (P.d_qk != P.d_v || (P.d_qk != 128 && P.d_qk != 64)) return TLS_ERR_UNSUPPORTED;
    if (P.G != 1 && P.G != 2 && P.G != 4 && P.G != 8) return TLS_ERR_UNSUPPORTED;
  }
  if (long(K_t) > long(tls::kMaxSplits) * tls::attn_tokens_per_split(P)) return TLS_ERR_UNSUPPORTED;
  return TLS_OK;
}

tls_status hip_status(hipError_t e) { return e == hipSuccess ? TLS_OK : TLS_ERR_HIP; }

template <class T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

uint32_t* err_word(void* ws) { return static_cast<uint32_t*>(ws); }

hipError_t run_token_select(const Problem& P, const tls::Workspace& W, const void* q, const uint8_t* codes,
                            const float* qparams, const int32_t* channels, const int32_t* block_ids, int K_b,
                            const int32_t* ctx_lens, int K_t, int32_t* token_ids, float* token_scores, void* ws,
                            uint32_t* err, hipStream_t stream, hipEvent_t* ev) {
  hipError_t e = tls::launch_token_score(P, q, codes, qparams, channels, block_ids, K_b, ctx_lens,
                                         at<float>(ws, W.logits), at<float>(ws, W.stats), W.n_tchunks, err, stream);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[0], stream);
  e = tls::launch_token_alpha(P, at<float>(ws, W.logits), at<float>(ws, W.stats), W.n_tchunks, block_ids, K_b,
                              ctx_lens, at<uint32_t>(ws, W.keys), at<uint32_t>(ws, W.kinfo), stream);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[1], stream);
  return tls::launch_token_topk(P, at<uint32_t>(ws, W.keys), at<uint32_t>(ws, W.kinfo), block_ids, K_b, K_t,
                                token_ids, token_scores, stream);
}

}  // namespace

namespace tls {

Workspace plan_workspace(const Problem& P, int K_b, int K_t, unsigned regions, int nsplit) {
  Workspace w{};
  const size_t U = size_t(P.units);
  const size_t S = size_t(K_b) * P.B;
  const size_t ns = size_t(nsplit);
  w.n_tchunks = int((S + kTokenSlotsPerWG - 1) / kTokenSlotsPerWG);
  size_t off = 0;
  // a region outside `regions` takes no bytes (its offset is never used)
  auto take = [&](size_t* at, unsigned region, size_t bytes) {
    *at = off;
    if (regions & region) off = align_up(off + bytes);
  };
  w.err = off;      off += kHeaderBytes;
  take(&w.xfer, kWsXfer, U * (2 * size_t(K_b) + 1) * sizeof(int32_t));  // prefetch lists
  take(&w.qpn, kWsBlockSel, U * 2 * size_t(P.d_qk) * sizeof(float));
  take(&w.bscores, kWsBlockSel, U * P.m_max * sizeof(float));
  take(&w.bids, kWsBids, U * K_b * sizeof(int32_t));
  take(&w.logits, kWsTokenSel, U * P.G * S * sizeof(float));
  take(&w.stats, kWsTokenSel, U * w.n_tchunks * P.G * 2 * sizeof(float));
  take(&w.keys, kWsTokenSel, U * S * sizeof(uint32_t));
  take(&w.kinfo, kWsTokenSel, U * 2 * sizeof(uint32_t));  // per unit: valid candidates, key bound
  take(&w.tids, kWsTids, U * size_t(K_t) * sizeof(int32_t));
  take(&w.po, kWsSplit, U * ns * P.G * size_t(P.d_v) * sizeof(float));
  take(&w.plse, kWsSplit, U * ns * P.G * sizeof(float));
  take(&w.dkeys, kWsDense, U * size_t(P.T) * sizeof(uint32_t));  // token-only operator
  take(&w.dstats, kWsDense, ds_stats_floats(P) * sizeof(float));
  w.total = off;
  return w;
}

}  // namespace tls

extern "C" {

const char* tls_version(void) { return "0.1.0 gfx950"; }

const char* tls_status_string(tls_status s) {
  switch (s) {
    case TLS_OK: return "TLS_OK";
    case TLS_ERR_INVALID_ARGUMENT: return "TLS_ERR_INVALID_ARGUMENT";
    case TLS_ERR_UNSUPPORTED: return "TLS_ERR_UNSUPPORTED";
    case TLS_ERR_WORKSPACE_TOO_SMALL: return "TLS_ERR_WORKSPACE_TOO_SMALL";
    case TLS_ERR_HIP: return "TLS_ERR_HIP";
    default: return "TLS_ERR_UNKNOWN";
  }
}

tls_status tls_workspace_size(const tls_layout* layout, int32_t K_b, int32_t K_t, size_t* bytes) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!bytes) return TLS_ERR_INVALID_ARGUMENT;
  st = check_budgets(P, K_b, K_t);
  if (st != TLS_OK) return st;
  *bytes = tls::plan_workspace(P, K_b, K_t).total;
  return TLS_OK;
}

tls_status tls_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!ws || ws_bytes < kHeaderBytes) return TLS_ERR_INVALID_ARGUMENT;
  return hip_status(tls::launch_fill_u32(static_cast<uint32_t*>(ws), 0u, kHeaderBytes / 4, stream));
}

tls_status tls_build_block_index(const tls_layout* layout, const void* K, const int32_t* ctx_lens, int32_t tok_begin,
                                 int32_t tok_end, void* kmax, void* kmin, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!K || !ctx_lens || !kmax || !kmin) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_begin < 0 || tok_end < tok_begin || tok_end > P.T) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_end == tok_begin) return TLS_OK;
  return hip_status(tls::launch_block_index(P, K, ctx_lens, tok_begin, tok_end, kmax, kmin, nullptr, stream));
}

tls_status tls_build_token_index(const tls_layout* layout, const void* K, const int32_t* ctx_lens,
                                 const int32_t* channels, int32_t tok_begin, int32_t tok_end, uint8_t* codes,
                                 float* qparams, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!K || !ctx_lens || !channels || !codes || !qparams) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_begin < 0 || tok_end < tok_begin || tok_end > P.T) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_end == tok_begin) return TLS_OK;
  return hip_status(
      tls::launch_token_index(P, K, ctx_lens, channels, tok_begin, tok_end, codes, qparams, nullptr, stream));
}

tls_status tls_prefill_kv(const tls_layout* layout, const void* k_src, const void* v_src, const int32_t* ctx_lens,
                          const int32_t* channels, int32_t tok_begin, int32_t tok_end, void* K, void* V, void* kmax,
                          void* kmin, uint8_t* codes, float* qparams, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!k_src || !ctx_lens || !channels || !K || !kmax || !kmin || !codes || !qparams) return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla ? (v_src != nullptr || V != nullptr) : (!v_src || !V)) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_begin < 0 || tok_end < tok_begin || tok_end > P.T) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_end == tok_begin) return TLS_OK;
  return hip_status(tls::launch_prefill_kv(P, k_src, v_src, ctx_lens, channels, tok_begin, tok_end, K, V, kmax, kmin,
                                           codes, qparams, nullptr, stream));
}

tls_status tls_append_tokens(const tls_layout* layout, const void* k_new, const void* v_new, const int32_t* ctx_lens,
                             const int32_t* channels, void* K, void* V, void* kmax, void* kmin, uint8_t* codes,
                             float* qparams, const tls_kv_view* pool, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!k_new || !ctx_lens || !channels || !K || !kmax || !kmin || !codes || !qparams) return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla ? (v_new != nullptr || V != nullptr) : (!v_new || !V)) return TLS_ERR_INVALID_ARGUMENT;
  void* pk = nullptr;
  void* pv = nullptr;
  const int32_t* smap = nullptr;
  int64_t n_slots = 0;
  if (pool) {
    if (!pool->k || !pool->slot_map || pool->n_slots < 1 || pool->n_slots > (int64_t(1) << 30))
      return TLS_ERR_INVALID_ARGUMENT;
    if (P.mla ? pool->v != nullptr : !pool->v) return TLS_ERR_INVALID_ARGUMENT;
    pk = const_cast<void*>(pool->k);
    pv = const_cast<void*>(pool->v);
    smap = pool->slot_map;
    n_slots = pool->n_slots;
  }
  // the cache may be device memory or pinned host memory (the offloaded tier's host copy)
  const void* dk = nullptr;
  const void* dv = nullptr;
  if (!readable_ptr(K, &dk) || (V && !readable_ptr(V, &dv))) return TLS_ERR_INVALID_ARGUMENT;
  return hip_status(tls::launch_append_tokens(P, k_new, v_new, ctx_lens, channels, const_cast<void*>(dk),
                                              const_cast<void*>(dv), kmax, kmin, codes, qparams, pk, pv, smap,
                                              n_slots, nullptr, stream));
}

tls_status tls_offload_kv(const tls_layout* layout, const void* K, const void* V, const int32_t* ctx_lens,
                          int32_t tok_begin, int32_t tok_end, void* host_k, void* host_v, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!K || !ctx_lens || !host_k) return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla ? (V != nullptr || host_v != nullptr) : (!V || !host_v)) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_begin < 0 || tok_end < tok_begin || tok_end > P.T) return TLS_ERR_INVALID_ARGUMENT;
  const void* dk = nullptr;
  const void* dv = nullptr;
  if (!pinned_device_ptr(host_k, &dk) || (host_v && !pinned_device_ptr(host_v, &dv))) return TLS_ERR_INVALID_ARGUMENT;
  if (tok_end == tok_begin) return TLS_OK;
  return hip_status(tls::launch_offload_rows(P, K, V, ctx_lens, tok_begin, tok_end, const_cast<void*>(dk),
                                             const_cast<void*>(dv), nullptr, stream));
}

tls_status tls_init_residency(const tls_layout* layout, const void* src_k, const void* src_v, const int32_t* ctx_lens,
                              const int32_t* block_ids, int32_t K_b, void* pool_k, void* pool_v, int64_t n_slots,
                              int32_t* slot_map, int32_t* slot_owner, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!src_k || !ctx_lens || !block_ids || !pool_k || !slot_map || !slot_owner || !ws) return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla ? (src_v != nullptr || pool_v != nullptr) : (!src_v || !pool_v)) return TLS_ERR_INVALID_ARGUMENT;
  st = check_budgets(P, K_b, 1);
  if (st != TLS_OK) return st;
  if (n_slots < int64_t(K_b) || n_slots > (int64_t(1) << 30)) return TLS_ERR_INVALID_ARGUMENT;
  const void* dk = nullptr;
  const void* dv = nullptr;
  if (!readable_ptr(src_k, &dk) || (src_v && !readable_ptr(src_v, &dv))) return TLS_ERR_INVALID_ARGUMENT;
  const tls::Workspace W = tls::plan_workspace(P, K_b, 1);
  if (ws_bytes < W.total) return TLS_ERR_WORKSPACE_TOO_SMALL;
  return hip_status(tls::launch_init_residency(P, dk, dv, ctx_lens, block_ids, K_b, pool_k, pool_v, n_slots, slot_map,
                                               slot_owner, at<int32_t>(ws, W.xfer), err_word(ws), stream));
}

tls_status tls_calibrate_absmax(const tls_layout* layout, const void* q_cal, const void* k_cal, int32_t n_cal,
                                float* q_absmax, float* k_absmax, int32_t accumulate, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (n_cal < 0 || (accumulate != 0 && accumulate != 1) || !q_absmax || !k_absmax) return TLS_ERR_INVALID_ARGUMENT;
  if (n_cal > 0 && (!q_cal || !k_cal)) return TLS_ERR_INVALID_ARGUMENT;
  hipError_t e = hipSuccess;
  if (!accumulate) {
    e = tls::launch_fill_u32(reinterpret_cast<uint32_t*>(q_absmax), 0u, size_t(P.H_q) * P.d_qk, stream);
    if (e == hipSuccess)
      e = tls::launch_fill_u32(reinterpret_cast<uint32_t*>(k_absmax), 0u, size_t(P.H_kv) * P.d_qk, stream);
  }
  if (e == hipSuccess) e = tls::launch_calib_absmax(P, q_cal, n_cal, P.H_q, q_absmax, stream);
  if (e == hipSuccess) e = tls::launch_calib_absmax(P, k_cal, n_cal, P.H_kv, k_absmax, stream);
  return hip_status(e);
}

tls_status tls_calibrate_channels(const tls_layout* layout, const float* q_absmax, const float* k_absmax,
                                  int32_t* channels, float* scores, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!q_absmax || !k_absmax || !channels) return TLS_ERR_INVALID_ARGUMENT;
  return hip_status(tls::launch_calib_select(P, q_absmax, k_absmax, channels, scores, stream));
}

tls_status tls_select_blocks(const tls_layout* layout, const void* q, const void* kmax, const void* kmin,
                             const int32_t* ctx_lens, int32_t K_b, int32_t* block_ids, float* block_scores, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!q || !kmax || !kmin || !ctx_lens || !block_ids || !ws) return TLS_ERR_INVALID_ARGUMENT;
  st = check_budgets(P, K_b, 1);
  if (st != TLS_OK) return st;
  const tls::Workspace W = tls::plan_workspace(P, K_b, 1);
  if (ws_bytes < W.total) return TLS_ERR_WORKSPACE_TOO_SMALL;
  float* scores = block_scores ? block_scores : at<float>(ws, W.bscores);
  hipError_t e = tls::launch_block_score(P, q, kmax, kmin, ctx_lens, at<float>(ws, W.qpn), scores, err_word(ws), stream);
  if (e == hipSuccess) e = tls::launch_block_topk(P, scores, ctx_lens, K_b, block_ids, err_word(ws), stream);
  return hip_status(e);
}

tls_status tls_select_tokens(const tls_layout* layout, const void* q, const uint8_t* codes, const float* qparams,
                             const int32_t* channels, const int32_t* block_ids, int32_t K_b, const int32_t* ctx_lens,
                             int32_t K_t, int32_t* token_ids, float* token_scores, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!q || !codes || !qparams || !channels || !block_ids || !ctx_lens || !token_ids || !ws)
    return TLS_ERR_INVALID_ARGUMENT;
  st = check_budgets(P, K_b, K_t);
  if (st != TLS_OK) return st;
  const tls::Workspace W = tls::plan_workspace(P, K_b, K_t);
  if (ws_bytes < W.total) return TLS_ERR_WORKSPACE_TOO_SMALL;
  if (tls::fused_token_select_ok(P, K_b, K_t))
    return hip_status(tls::launch_token_select_fused(P, q, codes, qparams, channels, nullptr, block_ids, nullptr,
                                                     ctx_lens, K_b, K_t, token_ids, token_scores, err_word(ws),
                                                     stream));
  return hip_status(run_token_select(P, W, q, codes, qparams, channels, block_ids, K_b, ctx_lens, K_t, token_ids,
                                     token_scores, ws, err_word(ws), stream, nullptr));
}

}  // extern "C"

namespace {

// Where a decode call's scratch lives: a caller workspace (the public plan,
// every region, sized by tls_workspace_size), or the library's own static
// scratch (compact plan: only the regions the call's route uses).  `err` is
// the device error word the kernels set bits in.
// The library's own scratch for tls_sparse_decode_noalloc: one array per
// device, resident from the library's load until the process ends.  Host
// code never uses the array's name as an address: the device address comes
// from hipGetSymbolAddress, once per device, with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];  // guarded by g_scratch_mutex

tls_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TLS_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return TLS_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TLS_OK;
}

// Where a decode call's scratch lives: the caller's workspace (base, bytes,
// its error word), or the library's own scratch (base == nullptr, compact
// plan; the error word is the caller's device_error, else the scratch's
// first word, which nothing reads).
struct WsTarget {
  void* base;
  size_t bytes;
  uint32_t* err;
  bool compact;
  // Plans the workspace for a route using `regions` (split partials for
  // `nsplit` splits) and binds its memory: TLS_ERR_WORKSPACE_TOO_SMALL when
  // the plan does not fit.  The library scratch is looked up only here, after
  // every argument check, so a rejected call touches no device.
  tls_status bind(const Problem& P, int K_b, int K_t, unsigned regions, int nsplit, tls::Workspace* W, void** ws,
                  uint32_t** err_word_out) const {
    *W = compact ? tls::plan_workspace(P, K_b, K_t, regions, nsplit) : tls::plan_workspace(P, K_b, K_t);
    if (bytes < W->total) return TLS_ERR_WORKSPACE_TOO_SMALL;
    if (base) {
      *ws = base;
      *err_word_out = err;
      return TLS_OK;
    }
    const tls_status st = scratch_of_current_device(ws);
    if (st != TLS_OK) return st;
    *err_word_out = err ? err : static_cast<uint32_t*>(*ws);
    return TLS_OK;
  }
};

// Split count of the attention stage over n_list entries per unit, and
// whether it writes partials (everything but the whole-unit kernel does).
int attention_route(const Problem& P, int n_list, int requested, unsigned* regions) {
  const int nsplit = tls::attn_splits_for(P, n_list, requested);
  if (!(nsplit == 1 && tls::gqa_whole_ok(P, n_list))) *regions |= tls::kWsSplit;
  return nsplit;
}

// Attention over a work list (stages 6 and 7): n_list entries per unit.
tls_status finish_decode(const Problem& P, const tls::Workspace& W, const void* q, const tls_kv_view* kv,
                         const int32_t* ctx_lens, int n_list, int nsplit, const tls::TokenList& tl, void* out,
                         float* lse, void* ws, uint32_t* err, hipEvent_t* ev, hipStream_t stream) {
  tls::KvView view{kv->k, kv->v, kv->slot_map, kv->n_slots};
  if (nsplit == 1 && tls::gqa_whole_ok(P, n_list)) {
    const hipError_t e = tls::launch_attention_gqa_whole(P, q, view, tl, ctx_lens, n_list, out, lse, err, stream);
    if (ev) (void)hipEventRecord(ev[6], stream);
    if (ev) (void)hipEventRecord(ev[7], stream);
    return hip_status(e);
  }
  hipError_t e = tls::launch_attention(P, q, view, tl, ctx_lens, n_list, nsplit, at<float>(ws, W.po),
                                       at<float>(ws, W.plse), err, stream);
  if (ev) (void)hipEventRecord(ev[6], stream);
  if (e == hipSuccess) e = tls::launch_merge(P, at<float>(ws, W.po), at<float>(ws, W.plse), nsplit, out, lse, stream);
  if (ev) (void)hipEventRecord(ev[7], stream);
  return hip_status(e);
}

// Token-level selection alone (TLS_MODE_TOKEN_SPARSE): alpha over every valid
// token of each unit, its top-K_t, then attention over those tokens.
tls_status token_level_decode(const Problem& P, const void* q, const tls_kv_view* kv, const int32_t* ctx_lens,
                              const uint8_t* codes, const float* qparams, const int32_t* channels, int K_b, int K_t,
                              const int32_t* block_ids_in, const int32_t* token_ids_in, void* out, float* lse,
                              int32_t* block_ids_out, int32_t* token_ids_out, const WsTarget& tgt, int requested,
                              hipEvent_t* ev, hipStream_t stream) {
  if (block_ids_in || token_ids_in || block_ids_out) return TLS_ERR_INVALID_ARGUMENT;
  if (!codes || !qparams || !channels) return TLS_ERR_INVALID_ARGUMENT;
  if (K_t < 1) return TLS_ERR_INVALID_ARGUMENT;
  if (!tls::ds_supported(P)) return TLS_ERR_UNSUPPORTED;
  tls_status st = check_attention(P, K_t);
  if (st != TLS_OK) return st;
  unsigned regions = tls::kWsDense | (token_ids_out ? 0u : tls::kWsTids);
  const int nsplit = attention_route(P, K_t, requested, &regions);
  tls::Workspace W;
  void* ws = nullptr;
  uint32_t* err = nullptr;
  st = tgt.bind(P, K_b > 0 ? K_b : 1, K_t, regions, nsplit, &W, &ws, &err);
  if (st != TLS_OK) return st;
  auto mark = [&](int i) {
    if (ev) (void)hipEventRecord(ev[i], stream);
  };
  mark(0);
  mark(1);
  mark(2);
  int32_t* to = token_ids_out ? token_ids_out : at<int32_t>(ws, W.tids);
  const hipError_t e = tls::launch_token_select_dense(P, q, codes, qparams, channels, ctx_lens, K_t,
                                                      at<float>(ws, W.dstats), at<uint32_t>(ws, W.dkeys), to, err,
                                                      stream);
  mark(3);
  mark(4);
  mark(5);
  if (e != hipSuccess) return TLS_ERR_HIP;
  return finish_decode(P, W, q, kv, ctx_lens, K_t, nsplit, tls::TokenList{to, K_t, tls::kListIds, P.B}, out, lse,
                       ws, err, ev, stream);
}

// The single-level baselines (TLS_MODE_BLOCK_SPARSE, TLS_MODE_DENSE): block
// selection (unless given) and attention over every valid token of the
// selected blocks, or attention over the whole context.
tls_status single_level_decode(const Problem& P, int mode, const void* q, const tls_kv_view* kv,
                               const int32_t* ctx_lens, const void* kmax, const void* kmin, const uint8_t* codes,
                               const float* qparams, const int32_t* channels, int K_b, int K_t,
                               const int32_t* block_ids_in, const int32_t* token_ids_in, void* out, float* lse,
                               int32_t* block_ids_out, int32_t* token_ids_out, const WsTarget& tgt, int requested,
                               hipEvent_t* ev, hipStream_t stream) {
  if (mode == TLS_MODE_TOKEN_SPARSE)
    return token_level_decode(P, q, kv, ctx_lens, codes, qparams, channels, K_b, K_t, block_ids_in, token_ids_in,
                              out, lse, block_ids_out, token_ids_out, tgt, requested, ev, stream);
  if (token_ids_in || token_ids_out) return TLS_ERR_INVALID_ARGUMENT;
  const bool dense = mode == TLS_MODE_DENSE;
  if (dense && (block_ids_in || block_ids_out)) return TLS_ERR_INVALID_ARGUMENT;
  if (!dense && !block_ids_in && (!kmax || !kmin)) return TLS_ERR_INVALID_ARGUMENT;
  tls_status st = check_budgets(P, dense ? 1 : K_b, 1);
  if (st != TLS_OK) return st;
  const int n_list = dense ? P.T : K_b * P.B;  // work-list entries per unit
  st = check_attention(P, n_list);
  if (st != TLS_OK) return st;
  const bool sel = !dense && !block_ids_in;
  unsigned regions = sel ? (tls::kWsBlockSel | (block_ids_out ? 0u : tls::kWsBids)) : 0u;
  const int nsplit = attention_route(P, n_list, requested, &regions);
  tls::Workspace W;
  void* ws = nullptr;
  uint32_t* err = nullptr;
  st = tgt.bind(P, dense ? 1 : K_b, K_t > 0 ? K_t : 1, regions, nsplit, &W, &ws, &err);
  if (st != TLS_OK) return st;
  auto mark = [&](int i) {
    if (ev) (void)hipEventRecord(ev[i], stream);
  };
  mark(0);
  hipError_t e = hipSuccess;
  const int32_t* bids = block_ids_in;
  if (sel) {
    int32_t* bo = block_ids_out ? block_ids_out : at<int32_t>(ws, W.bids);
    e = tls::launch_block_score(P, q, kmax, kmin, ctx_lens, at<float>(ws, W.qpn), at<float>(ws, W.bscores), err,
                                stream);
    mark(1);
    if (e == hipSuccess) e = tls::launch_block_topk(P, at<float>(ws, W.bscores), ctx_lens, K_b, bo, err, stream);
    bids = bo;
  } else {
    mark(1);
  }
  for (int i = 2; i < 6; ++i) mark(i);
  if (e != hipSuccess) return TLS_ERR_HIP;
  const tls::TokenList tl = dense ? tls::TokenList{nullptr, 0, tls::kListAll, P.B}
                                  : tls::TokenList{bids, K_b, tls::kListBlocks, P.B};
  return finish_decode(P, W, q, kv, ctx_lens, n_list, nsplit, tl, out, lse, ws, err, ev, stream);
}

// tls_sparse_decode after the layout is validated, on a workspace target.
tls_status sparse_decode_on(const Problem& P, const void* q, const tls_kv_view* kv, const int32_t* ctx_lens,
                            const void* kmax, const void* kmin, const uint8_t* codes, const float* qparams,
                            const int32_t* channels, int32_t K_b, int32_t K_t, const int32_t* block_ids_in,
                            const int32_t* token_ids_in, void* out, float* lse, int32_t* block_ids_out,
                            int32_t* token_ids_out, const tls_decode_opts* opts, const WsTarget& tgt,
                            hipStream_t stream) {
  if (!q || !kv || !kv->k || !ctx_lens || !out) return TLS_ERR_INVALID_ARGUMENT;
  if (!P.mla && !kv->v) return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla && kv->v) return TLS_ERR_INVALID_ARGUMENT;
  if (kv->slot_map && kv->n_slots < 1) return TLS_ERR_INVALID_ARGUMENT;
  int requested = 0, mode = TLS_MODE_TWO_LEVEL;
  hipEvent_t* ev = nullptr;
  if (opts) {
    for (int i = 0; i < 6; ++i)
      if (opts->reserved[i] != 0) return TLS_ERR_INVALID_ARGUMENT;
    if (opts->attn_splits < 0 || opts->attn_splits > tls::kMaxSplits) return TLS_ERR_INVALID_ARGUMENT;
    if (opts->mode < TLS_MODE_TWO_LEVEL || opts->mode > TLS_MODE_LAGGED) return TLS_ERR_INVALID_ARGUMENT;
    requested = opts->attn_splits;
    mode = opts->mode;
    ev = opts->stage_events;
    if (ev)
      for (int i = 0; i < TLS_NUM_STAGE_EVENTS; ++i)
        if (!ev[i]) return TLS_ERR_INVALID_ARGUMENT;
  }
  const bool lagged = mode == TLS_MODE_LAGGED;
  if (mode != TLS_MODE_TWO_LEVEL && !lagged)
    return single_level_decode(P, mode, q, kv, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t,
                               block_ids_in, token_ids_in, out, lse, block_ids_out, token_ids_out, tgt, requested,
                               ev, stream);
  if (lagged) {
    // tokens from the given (previous step's) blocks, this step's block
    // selection to block_ids_out; the two lists must not overlap
    if (!block_ids_in || !block_ids_out || token_ids_in) return TLS_ERR_INVALID_ARGUMENT;
    const uintptr_t bytes = uintptr_t(P.units) * uintptr_t(K_b > 0 ? K_b : 0) * sizeof(int32_t);
    const uintptr_t a = reinterpret_cast<uintptr_t>(block_ids_in), b = reinterpret_cast<uintptr_t>(block_ids_out);
    if (a < b + bytes && b < a + bytes) return TLS_ERR_INVALID_ARGUMENT;
  }
  const bool sel_tokens = token_ids_in == nullptr;
  const bool sel_blocks = lagged || (sel_tokens && block_ids_in == nullptr);
  if (sel_blocks && (!kmax || !kmin)) return TLS_ERR_INVALID_ARGUMENT;
  if (sel_tokens && (!codes || !qparams || !channels)) return TLS_ERR_INVALID_ARGUMENT;
  tls_status st = check_budgets(P, K_b, K_t);
  if (st != TLS_OK) return st;
  st = check_attention(P, K_t);
  if (st != TLS_OK) return st;
  // the route: fused selection (block scores, then one kernel for block
  // top-k and token selection), or the general stages
  const bool fused = sel_tokens && tls::fused_token_select_ok(P, K_b, K_t);
  unsigned regions = 0u;
  if (sel_blocks) regions |= tls::kWsBlockSel | (fused || block_ids_out ? 0u : tls::kWsBids);
  if (sel_tokens) regions |= (fused ? 0u : tls::kWsTokenSel) | (token_ids_out ? 0u : tls::kWsTids);
  const int nsplit = attention_route(P, K_t, requested, &regions);
  tls::Workspace W;
  void* ws = nullptr;
  uint32_t* err = nullptr;
  st = tgt.bind(P, K_b, K_t, regions, nsplit, &W, &ws, &err);
  if (st != TLS_OK) return st;

  hipError_t e = hipSuccess;
  auto mark = [&](int i) {
    if (ev) (void)hipEventRecord(ev[i], stream);
  };
  mark(0);
  const int32_t* bids = block_ids_in;
  if (fused) {
    // the token-score stage events bracket the fused kernel
    int32_t* to = token_ids_out ? token_ids_out : at<int32_t>(ws, W.tids);
    const float* bsc = nullptr;
    if (sel_blocks) {
      e = tls::launch_block_score(P, q, kmax, kmin, ctx_lens, at<float>(ws, W.qpn), at<float>(ws, W.bscores), err,
                                  stream);
      bsc = at<float>(ws, W.bscores);
    }
    mark(1);
    mark(2);
    if (e == hipSuccess)
      e = tls::launch_token_select_fused(P, q, codes, qparams, channels, bsc, block_ids_in,
                                         sel_blocks ? block_ids_out : nullptr, ctx_lens, K_b, K_t, to, nullptr, err,
                                         stream);  // scores and a given list: the lagged operator
    mark(3);
    mark(4);
    mark(5);
    if (e != hipSuccess) return TLS_ERR_HIP;
    return finish_decode(P, W, q, kv, ctx_lens, K_t, nsplit, tls::TokenList{to, K_t, tls::kListIds, P.B}, out, lse,
                         ws, err, ev, stream);
  }
  if (sel_blocks) {
    int32_t* bo = block_ids_out ? block_ids_out : at<int32_t>(ws, W.bids);
    e = tls::launch_block_score(P, q, kmax, kmin, ctx_lens, at<float>(ws, W.qpn), at<float>(ws, W.bscores), err,
                                stream);
    mark(1);
    if (e == hipSuccess) e = tls::launch_block_topk(P, at<float>(ws, W.bscores), ctx_lens, K_b, bo, err, stream);
    if (!lagged) bids = bo;  // the lagged operator selects tokens from the given blocks
  } else {
    mark(1);
  }
  mark(2);
  if (e != hipSuccess) return TLS_ERR_HIP;
  const int32_t* tids = token_ids_in;
  if (sel_tokens) {
    int32_t* to = token_ids_out ? token_ids_out : at<int32_t>(ws, W.tids);
    e = run_token_select(P, W, q, codes, qparams, channels, bids, K_b, ctx_lens, K_t, to, nullptr, ws, err, stream,
                         ev ? ev + 3 : nullptr);
    tids = to;
  } else {
    mark(3);
    mark(4);
  }
  mark(5);
  if (e != hipSuccess) return TLS_ERR_HIP;
  return finish_decode(P, W, q, kv, ctx_lens, K_t, nsplit, tls::TokenList{tids, K_t, tls::kListIds, P.B}, out, lse,
                       ws, err, ev, stream);
}

}  // namespace

extern "C" {

tls_status tls_sparse_decode(const tls_layout* layout, const void* q, const tls_kv_view* kv, const int32_t* ctx_lens,
                             const void* kmax, const void* kmin, const uint8_t* codes, const float* qparams,
                             const int32_t* channels, int32_t K_b, int32_t K_t, const int32_t* block_ids_in,
                             const int32_t* token_ids_in, void* out, float* lse, int32_t* block_ids_out,
                             int32_t* token_ids_out, void* ws, size_t ws_bytes, const tls_decode_opts* opts,
                             hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!ws) return TLS_ERR_INVALID_ARGUMENT;
  const WsTarget tgt{ws, ws_bytes, err_word(ws), false};
  return sparse_decode_on(P, q, kv, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t, block_ids_in,
                          token_ids_in, out, lse, block_ids_out, token_ids_out, opts, tgt, stream);
}

tls_status tls_sparse_decode_noalloc(const tls_layout* layout, const void* q, const tls_kv_view* kv,
                                     const int32_t* ctx_lens, const void* kmax, const void* kmin,
                                     const uint8_t* codes, const float* qparams, const int32_t* channels, int32_t K_b,
                                     int32_t K_t, const int32_t* block_ids_in, const int32_t* token_ids_in, void* out,
                                     float* lse, int32_t* block_ids_out, int32_t* token_ids_out,
                                     uint32_t* device_error, const tls_decode_opts* opts, hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  // the scratch address is resolved once the arguments have passed (bind)
  const WsTarget tgt{nullptr, kScratchBytes, device_error, true};
  return sparse_decode_on(P, q, kv, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t, block_ids_in,
                          token_ids_in, out, lse, block_ids_out, token_ids_out, opts, tgt, stream);
}

tls_status tls_prefetch_blocks(const tls_layout* layout, const void* host_k, const void* host_v,
                               const int32_t* ctx_lens, const int32_t* block_ids_new, const int32_t* block_ids_live,
                               int32_t K_b, void* pool_k, void* pool_v, int64_t n_slots, int32_t* slot_map,
                               int32_t* slot_owner, int32_t* transfer_count, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  Problem P;
  tls_status st = make_problem(layout, &P);
  if (st != TLS_OK) return st;
  if (!host_k || !ctx_lens || !block_ids_new || !pool_k || !slot_map || !slot_owner || !ws)
    return TLS_ERR_INVALID_ARGUMENT;
  if (P.mla ? (host_v != nullptr || pool_v != nullptr) : (!host_v || !pool_v)) return TLS_ERR_INVALID_ARGUMENT;
  st = check_budgets(P, K_b, 1);
  if (st != TLS_OK) return st;
  if (n_slots < (block_ids_live ? 2 * int64_t(K_b) : int64_t(K_b)) || n_slots > (int64_t(1) << 30))
    return TLS_ERR_INVALID_ARGUMENT;
  // host K/V must be pinned (device-accessible) host memory
  const void* dk = nullptr;
  const void* dv = nullptr;
  if (!pinned_device_ptr(host_k, &dk) || (host_v && !pinned_device_ptr(host_v, &dv))) return TLS_ERR_INVALID_ARGUMENT;
  const tls::Workspace W = tls::plan_workspace(P, K_b, 1);
  if (ws_bytes < W.total) return TLS_ERR_WORKSPACE_TOO_SMALL;
  int32_t* xfer = at<int32_t>(ws, W.xfer);
  return hip_status(tls::launch_prefetch(P, dk, dv, ctx_lens, block_ids_new, block_ids_live, K_b, pool_k, pool_v,
                                         n_slots, slot_map, slot_owner, transfer_count, xfer, err_word(ws), stream));
}

tls_status tls_check_device_error(const void* ws, size_t ws_bytes, int32_t clear, int32_t* flags, hipStream_t stream) {
  if (!ws || ws_bytes < kHeaderBytes || !flags) return TLS_ERR_INVALID_ARGUMENT;
  uint32_t h = 0;
  if (hipMemcpyAsync(&h, ws, sizeof(h), hipMemcpyDeviceToHost, stream) != hipSuccess) return TLS_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return TLS_ERR_HIP;
  *flags = int32_t(h);
  if (clear) {
    if (tls::launch_fill_u32(static_cast<uint32_t*>(const_cast<void*>(ws)), 0u, 1, stream) != hipSuccess)
      return TLS_ERR_HIP;
  }
  return TLS_OK;
}

}  // extern "C"
