// Internal launch interface between the C ABI (tls_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "host_cache.hpp"

namespace tls {

// Validated shape of one call (see tls_layout in include/tls.h).
struct Problem {
  int b, H_q, H_kv, G;
  int d_qk, d_v, B, d_c, T, m_max;
  int dtype;  // 0 f32, 1 bf16
  int mla;    // V aliases K[..., :d_v]
  float sigma;
  int units;  // b * H_kv
};

// Capacity limits of the library (host validation rejects larger requests).
constexpr int kMaxKeys = 12288;     // blocks per sequence, and K_b * B candidate slots
constexpr int kMaxSplits = 128;     // attention splits per unit
constexpr int kMaxGroupGqa = 8;     // G for the VALU attention path
constexpr int kTokenSlotsPerWG = 256;

// Workspace carving (byte offsets from the workspace base, 256-aligned).
struct Workspace {
  size_t err, xfer, qpn, bscores, bids, logits, stats, keys, kinfo, tids, po, plse, dkeys, dstats, total;
  int n_tchunks;  // token-score work-groups per unit
};
// Regions of the workspace, as a mask: a route of a call names the regions
// it uses; the public size holds all of them (partials for kMaxSplits).
enum : unsigned {
  kWsXfer = 1u,       // prefetch transfer lists
  kWsBlockSel = 2u,   // pre-reduced queries and block scores
  kWsBids = 4u,       // block ids when the caller takes none
  kWsTokenSel = 8u,   // logits, per-chunk statistics and keys of the general token stage
  kWsTids = 16u,      // token ids when the caller takes none
  kWsSplit = 32u,     // split-attention partials and their lse
  kWsDense = 64u,     // keys and statistics of the token-level operator
  kWsAll = 127u,
};
Workspace plan_workspace(const Problem& P, int K_b, int K_t, unsigned regions = kWsAll, int nsplit = kMaxSplits);

hipError_t launch_block_index(const Problem& P, const void* K, const int32_t* ctx_lens, int tok_begin,
                              int tok_end, void* kmax, void* kmin, uint32_t* err, hipStream_t st);
hipError_t launch_token_index(const Problem& P, const void* K, const int32_t* ctx_lens,
                              const int32_t* channels, int tok_begin, int tok_end, uint8_t* codes,
                              float* qparams, uint32_t* err, hipStream_t st);
// Prefill write-back of the K/V rows [tok_begin, tok_end) fused with both
// index builds over the same range (one read of every touched block).
hipError_t launch_prefill_kv(const Problem& P, const void* k_src, const void* v_src, const int32_t* ctx_lens,
                             const int32_t* channels, int tok_begin, int tok_end, void* K, void* V, void* kmax,
                             void* kmin, uint8_t* codes, float* qparams, uint32_t* err, hipStream_t st);
// Decode-time append of the token at ctx_len - 1 of every sequence: cache row,
// pool row when its block is resident (slot_map non-null), incremental block
// summary, token-index row.
hipError_t launch_append_tokens(const Problem& P, const void* k_new, const void* v_new, const int32_t* ctx_lens,
                                const int32_t* channels, void* K, void* V, void* kmax, void* kmin, uint8_t* codes,
                                float* qparams, void* pool_k, void* pool_v, const int32_t* slot_map, int64_t n_slots,
                                uint32_t* err, hipStream_t st);

hipError_t launch_block_score(const Problem& P, const void* q, const void* kmax, const void* kmin,
                              const int32_t* ctx_lens, float* qpn, float* scores, uint32_t* err, hipStream_t st);
hipError_t launch_block_topk(const Problem& P, const float* scores, const int32_t* ctx_lens, int K_b,
                             int32_t* block_ids, uint32_t* err, hipStream_t st);

hipError_t launch_token_score(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                              const int32_t* channels, const int32_t* block_ids, int K_b,
                              const int32_t* ctx_lens, float* logits, float* stats, int n_tchunks,
                              uint32_t* err, hipStream_t st);
hipError_t launch_token_alpha(const Problem& P, const float* logits, const float* stats, int n_tchunks,
                              const int32_t* block_ids, int K_b, const int32_t* ctx_lens, uint32_t* keys, uint32_t* kinfo,
                              hipStream_t st);
hipError_t launch_token_topk(const Problem& P, const uint32_t* keys, const uint32_t* kinfo, const int32_t* block_ids, int K_b,
                             int K_t, int32_t* token_ids, float* token_scores, hipStream_t st);

// One work-group per unit: (optional) block top-k from block_scores, then the
// whole token selection on chip, over the selected blocks or, when
// block_ids_in is given, over those (with block_scores as well, the new
// selection is written to block_ids_out: the lagged operator).  Valid when
// fused_token_select_ok().
bool fused_token_select_ok(const Problem& P, int K_b, int K_t);
hipError_t launch_token_select_fused(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                                     const int32_t* channels, const float* block_scores,
                                     const int32_t* block_ids_in, int32_t* block_ids_out, const int32_t* ctx_lens,
                                     int K_b, int K_t, int32_t* token_ids, float* token_scores, uint32_t* err,
                                     hipStream_t st);

// Token-level selection over every valid token of each unit (the token-only
// operator): alpha keys [units][T] and per-chunk statistics in the workspace.
bool ds_supported(const Problem& P);
size_t ds_stats_floats(const Problem& P);
hipError_t launch_token_select_dense(const Problem& P, const void* q, const uint8_t* codes, const float* qparams,
                                     const int32_t* channels, const int32_t* ctx_lens, int K_t, float* stats,
                                     uint32_t* keys, int32_t* token_ids, uint32_t* err, hipStream_t st);

struct KvView {
  const void* k;
  const void* v;
  const int32_t* slot_map;
  int64_t n_slots;
};

// The work list of the attention stage: which tokens each unit attends.
//   kListIds:    ids = [units][stride] token positions (the two-level
//                selection, or ids given by the caller), -1 = empty;
//   kListBlocks: ids = [units][stride] block ids, entry p is token
//                ids[p / B] * B + p % B (block-sparse attention over every
//                token of the selected blocks), -1 blocks are empty;
//   kListAll:    entry p is token p (dense attention), ids unused.
// Derived positions at or past ctx_len are empty entries, not errors.
enum : int { kListIds = 0, kListBlocks = 1, kListAll = 2 };
struct TokenList {
  const int32_t* ids;
  int stride;
  int kind;
  int B;
};
int attn_tokens_per_split(const Problem& P);  // token capacity of one attention work-group
int attn_splits_for(const Problem& P, int K_t, int requested);
// Whole-unit attention (one work-group per unit writes the output directly;
// no partials, no merge).  Valid when gqa_whole_ok().
bool gqa_whole_ok(const Problem& P, int K_t);
hipError_t launch_attention_gqa_whole(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                                      const int32_t* ctx_lens, int K_t, void* out, float* lse, uint32_t* err,
                                      hipStream_t st);
// K_t here is the number of list entries per unit (the budget for kListIds,
// stride * B for kListBlocks, max_ctx for kListAll).
hipError_t launch_attention(const Problem& P, const void* q, const KvView& kv, const TokenList& tl,
                            const int32_t* ctx_lens, int K_t, int nsplit, float* po, float* plse,
                            uint32_t* err, hipStream_t st);
hipError_t launch_merge(const Problem& P, const float* po, const float* plse, int nsplit, void* out,
                        float* lse, hipStream_t st);

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, size_t n, hipStream_t st);

// Channel calibration (token-index channel set): running max |x| per (head,
// channel) over n token-major rows [n][H][d_qk], merged into `out` (>= 0);
// then scores and the top-d_c channels per KV head.
hipError_t launch_calib_absmax(const Problem& P, const void* x, int n, int H, float* out, hipStream_t st);
hipError_t launch_calib_select(const Problem& P, const float* q_absmax, const float* k_absmax, int32_t* channels,
                               float* scores, hipStream_t st);

hipError_t launch_prefetch(const Problem& P, const void* host_k, const void* host_v, const int32_t* ctx_lens,
                           const int32_t* block_ids_new, const int32_t* block_ids_live, int K_b,
                           void* pool_k, void* pool_v, int64_t n_slots, int32_t* slot_map,
                           int32_t* slot_owner, int32_t* transfer_count, int32_t* transfer_list,
                           uint32_t* err, hipStream_t st);
hipError_t launch_init_residency(const Problem& P, const void* src_k, const void* src_v, const int32_t* ctx_lens,
                                 const int32_t* block_ids, int K_b, void* pool_k, void* pool_v, int64_t n_slots,
                                 int32_t* slot_map, int32_t* slot_owner, int32_t* transfer_list, uint32_t* err,
                                 hipStream_t st);
hipError_t launch_offload_rows(const Problem& P, const void* K, const void* V, const int32_t* ctx_lens,
                               int tok_begin, int tok_end, void* host_k, void* host_v, uint32_t* err,
                               hipStream_t st);

}  // namespace tls
