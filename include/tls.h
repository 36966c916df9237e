/*
 * tls.h - C ABI of the two-level sparse decode-attention library (libtls.so)
 * for AMD Instinct MI355X (gfx950).
 *
 * The operator follows AsyncTLS (arXiv 2604.07815), Sec. 4.1 "Two-Level
 * Sparse Attention" and Sec. 4.2 "Hierarchical KV Cache Management":
 * for one decode query and each KV group (the G query heads sharing one KV
 * head; G = H_q for the absorbed MLA layout, Sec. 3), it
 *   1. scores every block of B cached keys by the Quest bound computed from
 *      per-channel max/min block summaries and keeps the top-K_b blocks;
 *   2. scores only the tokens of those blocks against an INT4 index of the
 *      keys projected on d_c channels, averages the G per-head softmax
 *      distributions and keeps the top-K_t tokens;
 *   3. runs exact softmax attention over the full K/V rows of those tokens.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are caller-owned DEVICE memory unless stated
 *   otherwise (the host K/V of tls_prefetch_blocks is caller-owned pinned
 *   host memory).  The library allocates no memory; scratch space comes from
 *   a caller buffer sized by tls_workspace_size.
 * - Every call is asynchronous on the given stream (NULL = default stream)
 *   and never synchronises, except tls_check_device_error.
 * - Every call returns a tls_status.  Arguments are validated on the host
 *   before anything is enqueued: on any error no kernel is launched and no
 *   output is written.
 * - Values that only the device knows (context lengths, given block or token
 *   ids, pool slots) are checked by the kernels: offending items are
 *   skipped or clamped and a bit is set in the device error word held by the
 *   workspace (tls_check_device_error).
 * - Results are deterministic run to run: fixed reduction orders and no
 *   floating-point atomics.
 * - Every call except tls_check_device_error enqueues kernels only (no
 *   memset or copy nodes, no host round trip), so a serving step can be
 *   captured into a HIP graph and replayed (the tests replay decode steps
 *   and append + decode steps).  Calls that share a workspace must not run
 *   concurrently.
 * - Unit = one (sequence, KV head) pair; "units" = batch * num_kv_heads.
 *   Query head h belongs to KV head floor(h / G), G = num_q_heads / num_kv_heads.
 *
 * Dense row-major layouts (T = max_ctx, m_max = ceil(T / B)):
 *   q          [b][H_q][d_qk]            dtype
 *   K          [b][H_kv][T][d_qk]        dtype   (MLA: H_kv = 1, row = [latent; rope])
 *   V          [b][H_kv][T][d_v]         dtype   (NULL when mla_shared_kv: V = K[..., :d_v])
 *   ctx_lens   [b]                       int32   valid tokens per sequence, 0 <= n <= T
 *   kmax, kmin [b][H_kv][m_max][d_qk]    dtype   block summaries
 *   channels   [H_kv][d_c]               int32   ascending channel ids < d_qk
 *   codes      [b][H_kv][T][d_c/2]       uint8   two 4-bit codes per byte, low nibble first
 *   qparams    [b][H_kv][T][d_c/32][2]   float   (scale, min) per 32-channel group
 *   block_ids  [b][H_kv][K_b]            int32   ascending block ids, -1 padded
 *   token_ids  [b][H_kv][K_t]            int32   ascending token positions, -1 padded
 *   out        [b][H_q][d_v]             dtype
 *   lse        [b][H_q]                  float   log-sum-exp of the scaled logits
 */
#ifndef TLS_H_
#define TLS_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tls_status;

enum {
  TLS_OK = 0,
  TLS_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad shape, bad budget        */
  TLS_ERR_UNSUPPORTED = 2,        /* valid request the library does not handle */
  TLS_ERR_WORKSPACE_TOO_SMALL = 3,
  TLS_ERR_HIP = 4                 /* a HIP runtime call or launch failed        */
};

enum { TLS_DTYPE_F32 = 0, TLS_DTYPE_BF16 = 1 };

/* Device error word bits (tls_check_device_error). */
enum {
  TLS_DEVERR_CTX_LEN = 1,        /* a ctx_lens entry was outside [0, max_ctx]; clamped */
  TLS_DEVERR_BLOCK_ID = 2,       /* a given block id was >= the block count; skipped  */
  TLS_DEVERR_TOKEN_ID = 4,       /* a given token id was >= ctx_len; skipped          */
  TLS_DEVERR_SLOT = 8,           /* pooled view: token's block not resident; skipped  */
  TLS_DEVERR_POOL_FULL = 16,     /* prefetch: no free slot for a new block            */
  TLS_DEVERR_CHANNEL = 32        /* a channel id was outside [0, d_qk); read as 0     */
};

/* Number of events tls_decode_opts.stage_events must hold: one before each
 * of the seven stages (block score, block top-k, token score, token
 * normalisation, token top-k, attention, split merge) and one after the
 * last. */
#define TLS_NUM_STAGE_EVENTS 8

typedef struct tls_layout {
  int32_t batch;           /* b                                                  */
  int32_t num_q_heads;     /* H_q                                                */
  int32_t num_kv_heads;    /* H_kv; must divide H_q (1 for absorbed MLA)         */
  int32_t head_dim_qk;     /* d_qk: score dimension (GQA 128; MLA 576)           */
  int32_t head_dim_v;      /* d_v: value dimension (GQA 128; MLA 512)            */
  int32_t block_size;      /* B: tokens per block (64)                           */
  int32_t index_channels;  /* d_c: token-index channels, multiple of 32          */
  int32_t max_ctx;         /* T: token stride of the dense K/V/index layouts     */
  int32_t dtype;           /* TLS_DTYPE_F32 or TLS_DTYPE_BF16 (q, K, V, out)     */
  int32_t mla_shared_kv;   /* 1: V aliases K[..., :d_v] (pass V = NULL)          */
  float softmax_scale;     /* sigma; <= 0 selects 1/sqrt(d_qk)                   */
} tls_layout;

/* Where the attention stage reads K/V rows.
 * Direct view (slot_map == NULL): k, v use the dense layouts above.
 * Pooled view (slot_map != NULL): the HBM-resident block pool of the
 * offloaded KV tier (Sec. 4.2).  k is [units][n_slots][B][d_qk], v is
 * [units][n_slots][B][d_v] (NULL when mla_shared_kv), and slot_map is
 * [units][m_max] int32 giving the pool slot of each resident block of the
 * unit, -1 when the block is not resident. */
typedef struct tls_kv_view {
  const void* k;
  const void* v;
  const int32_t* slot_map;
  int64_t n_slots;         /* slots per unit (pooled view only) */
} tls_kv_view;

/* Operator run by tls_sparse_decode (tls_decode_opts.mode).  The
 * single-level operators are the baselines the paper measures its operator
 * against (Sec. 5, kernel study): block-level selection alone (Quest),
 * token-level selection alone (Double Sparsity) and full attention.
 *   TLS_MODE_TWO_LEVEL    Sec. 4.1: block selection, token selection, then
 *                         attention over the K_t selected tokens.
 *   TLS_MODE_BLOCK_SPARSE block selection only, then attention over every
 *                         valid token of the K_b selected blocks (up to
 *                         K_b * B tokens).  K_t, codes, qparams and channels
 *                         are not used; token_ids_in and token_ids_out must
 *                         be NULL.  block_ids_in / block_ids_out work as in
 *                         the two-level operator.
 *   TLS_MODE_DENSE        no selection: attention over all ctx_len tokens
 *                         of each sequence (full attention).  K_b, K_t and
 *                         the index arrays are not used; every id argument
 *                         must be NULL.
 *   TLS_MODE_TOKEN_SPARSE token selection alone: the approximate score of
 *                         Sec. 4.1 over every valid token of the unit (the
 *                         per-head softmax runs over all of them), the K_t
 *                         largest, then attention over those tokens.  kmax
 *                         and kmin are not used; the block-id arguments and
 *                         token_ids_in must be NULL; token_ids_out receives
 *                         the selection.  G must be 1, 2, 4, 8, 16 or 32.
 *   TLS_MODE_LAGGED       the two-level operator with the one-step lag of the
 *                         offloaded tier (Sec. 4.2): block selection from
 *                         this step's query writes M_t to block_ids_out (the
 *                         blocks to bring in for the next step), while token
 *                         selection and attention run over the blocks of
 *                         block_ids_in (M_{t-1}, already resident).  Both
 *                         lists are required and must not overlap; kmax,
 *                         kmin, codes, qparams and channels are required;
 *                         token_ids_in must be NULL.  The same results as
 *                         tls_select_blocks into block_ids_out followed by
 *                         the two-level operator with block_ids_in, in one
 *                         call; stage event 5 (after token selection) marks
 *                         the point where block_ids_out is complete. */
enum {
  TLS_MODE_TWO_LEVEL = 0,
  TLS_MODE_BLOCK_SPARSE = 1,
  TLS_MODE_DENSE = 2,
  TLS_MODE_TOKEN_SPARSE = 3,
  TLS_MODE_LAGGED = 4
};

/* Optional knobs of tls_sparse_decode; pass NULL for defaults. */
typedef struct tls_decode_opts {
  int32_t attn_splits;       /* token splits per unit in the attention stage; 0 = auto */
  int32_t mode;              /* TLS_MODE_*; 0 = the two-level operator                  */
  int32_t reserved[6];       /* must be zero                                            */
  hipEvent_t* stage_events;  /* NULL, or TLS_NUM_STAGE_EVENTS events recorded on the
                                stream around the stages (skipped stages record
                                back-to-back events)                                   */
} tls_decode_opts;

/* Library version string, e.g. "0.1.0 gfx950". */
const char* tls_version(void);

/* Static, human-readable name of a status code. */
const char* tls_status_string(tls_status status);

/* Bytes of scratch workspace needed by tls_select_blocks, tls_select_tokens,
 * tls_sparse_decode and tls_prefetch_blocks for this layout and budgets
 * (K_b >= 1, K_t >= 1).  Pure host function.  Writes *bytes. */
tls_status tls_workspace_size(const tls_layout* layout, int32_t K_b, int32_t K_t, size_t* bytes);

/* Clears the workspace header (device error word and internal counters).
 * Call once after allocating a workspace, before its first use; the library
 * keeps the header consistent afterwards.  Enqueued on `stream`. */
tls_status tls_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/* Block-level index, Sec. 4.1 (block representation): for every block that
 * overlaps [tok_begin, tok_end) of each sequence, kmax/kmin receive the
 * per-channel max/min of K over the block's valid tokens (positions
 * < ctx_len; the last block may be partial).  Blocks past ceil(ctx_len/B)
 * are left untouched.  Values are copied exactly (-0.0 is stored as +0.0).
 * Full build: tok_begin = 0, tok_end = max_ctx.  Appending token t:
 * tok_begin = t, tok_end = t + 1 (re-summarises its block). */
tls_status tls_build_block_index(const tls_layout* layout, const void* K, const int32_t* ctx_lens,
                                 int32_t tok_begin, int32_t tok_end, void* kmax, void* kmin,
                                 hipStream_t stream);

/* Token-level index, Sec. 4.1 (channel projection onto C and INT4
 * quantisation; d_c and INT4 from Sec. 5): for every valid token in
 * [tok_begin, tok_end), x = K[token][channels[kv_head][:]] is quantised per
 * group of 32 channels as asymmetric uint4 in float32:
 *   scale = (max - min) / 15,  code = clamp(rint((x - min) / scale), 0, 15)
 * (all codes 0 when scale == 0), with IEEE division and round-half-even, so
 * the codes are reproducible bit for bit.  Rows of invalid tokens are left
 * untouched. */
tls_status tls_build_token_index(const tls_layout* layout, const void* K, const int32_t* ctx_lens,
                                 const int32_t* channels, int32_t tok_begin, int32_t tok_end,
                                 uint8_t* codes, float* qparams, hipStream_t stream);

/* Channel calibration for the token index, Sec. 4.1: the channel set C of
 * each KV group is chosen offline from a held-out calibration set by the
 * importance s_i = (1/G) sum_h max|q_h[i]| * max|k[i]| of every score
 * dimension i.  This call computes the running maxima: over the n_cal rows
 * of q_cal [n_cal][H_q][d_qk] and k_cal [n_cal][H_kv][d_qk] (dtype,
 * token-major as the projections produce them), q_absmax [H_q][d_qk] and
 * k_absmax [H_kv][d_qk] (float) receive max |x| per (head, channel).
 * accumulate = 0 starts from zero; accumulate = 1 folds the rows into the
 * values already held (a calibration set streamed in batches; the arrays
 * must hold results of earlier calls).  The maxima are exact and do not
 * depend on batching or launch order.  n_cal = 0 is allowed (q_cal and k_cal
 * may then be NULL). */
tls_status tls_calibrate_absmax(const tls_layout* layout, const void* q_cal, const void* k_cal,
                                int32_t n_cal, float* q_absmax, float* k_absmax, int32_t accumulate,
                                hipStream_t stream);

/* Channel selection from the maxima of tls_calibrate_absmax (Sec. 4.1): per
 * KV head g, s_i = (sum over the G heads h of g, in order, of
 * q_absmax[h][i] * k_absmax[g][i]) / G in float32, then channels[g][:] =
 * the d_c channels with the highest s_i (ties to the lower channel),
 * ascending, ready for tls_build_token_index.  scores (nullable)
 * [H_kv][d_qk] receives every s_i. */
tls_status tls_calibrate_channels(const tls_layout* layout, const float* q_absmax, const float* k_absmax,
                                  int32_t* channels, float* scores, hipStream_t stream);

/* Prefill write-back fused with both index builds (the prefill flow of
 * Sec. 4.2 / Fig. 2: the hierarchical indices are built while the prompt's
 * keys are stored).  For every token t in [tok_begin, tok_end) with
 * t < ctx_len of its sequence s, copies the prefill output rows
 *   K[s][h][t][:] = k_src[s][t - tok_begin][h][:]   (and V from v_src),
 * then builds the block index of every block overlapping the range and the
 * token index of those tokens, exactly as tls_build_block_index and
 * tls_build_token_index over [tok_begin, tok_end) would after the copy (bit
 * for bit), from one read of each touched block.  Rows of those blocks
 * outside the range (earlier prefill chunks, or later rows already present)
 * are read from K.  Tokens at or past ctx_len are skipped.  k_src and v_src
 * must not overlap K or V.
 *   k_src  [b][tok_end - tok_begin][H_kv][d_qk]  dtype, token-major as a key
 *                                                projection produces it
 *   v_src  [b][tok_end - tok_begin][H_kv][d_v]   dtype; NULL iff mla_shared_kv
 *   K, V   dense cache layouts (V NULL iff mla_shared_kv)
 * Chunked prefill: call once per chunk with consecutive ranges. */
tls_status tls_prefill_kv(const tls_layout* layout, const void* k_src, const void* v_src,
                          const int32_t* ctx_lens, const int32_t* channels, int32_t tok_begin,
                          int32_t tok_end, void* K, void* V, void* kmax, void* kmin, uint8_t* codes,
                          float* qparams, hipStream_t stream);

/* Coarse block selection, Sec. 4.1: per unit, the Quest score of each of the
 * ceil(ctx_len/B) blocks, s_i = sum_h (max(q_h,0) . kmax_i + min(q_h,0) . kmin_i)
 * (the paper's GEMM form; fp32 accumulation), then M = the K_b highest
 * scores, ties to the lower block id, written ascending and padded with -1.
 * block_scores (nullable) [b][H_kv][m_max] receives every block's score
 * (-inf past the last block). */
tls_status tls_select_blocks(const tls_layout* layout, const void* q, const void* kmax,
                             const void* kmin, const int32_t* ctx_lens, int32_t K_b,
                             int32_t* block_ids, float* block_scores, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* Fine token selection, Sec. 4.1: for the valid tokens j of the blocks in
 * block_ids ([b][H_kv][K_b], -1 entries ignored; may be the previous step's
 * selection in the offloaded schedule of Sec. 4.2), the logits
 * l_hj = sigma * q_h[C] . dequant(codes_j) per head, the per-head softmax over
 * those candidates and its mean over the G heads, alpha_j; then the K_t
 * largest alpha_j (ties to the lower position), written ascending, -1 padded.
 * token_scores (nullable) [b][H_kv][K_t] receives alpha of each selected token. */
tls_status tls_select_tokens(const tls_layout* layout, const void* q, const uint8_t* codes,
                             const float* qparams, const int32_t* channels,
                             const int32_t* block_ids, int32_t K_b, const int32_t* ctx_lens,
                             int32_t K_t, int32_t* token_ids, float* token_scores, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* The whole decode step (Sec. 4.1): block selection, token selection and
 * exact attention o_h = softmax(sigma q_h K_S^T) V_S over the selected
 * tokens, per query head.  block_ids_in (nullable) skips block selection;
 * token_ids_in (nullable) skips both selection stages (then kmax, kmin,
 * codes, qparams and channels may be NULL).  out receives the attention
 * output in the input dtype (round to nearest even for bf16), lse (nullable)
 * the fp32 log-sum-exp; an empty selection gives out = 0, lse = -inf.
 * block_ids_out / token_ids_out (nullable) receive the selections.  With
 * opts->mode = TLS_MODE_LAGGED (Sec. 4.2) block_ids_in is the previous
 * step's selection the tokens are chosen from, and block_ids_out receives
 * this step's block selection. */
tls_status tls_sparse_decode(const tls_layout* layout, const void* q, const tls_kv_view* kv,
                             const int32_t* ctx_lens, const void* kmax, const void* kmin,
                             const uint8_t* codes, const float* qparams, const int32_t* channels,
                             int32_t K_b, int32_t K_t, const int32_t* block_ids_in,
                             const int32_t* token_ids_in, void* out, float* lse,
                             int32_t* block_ids_out, int32_t* token_ids_out, void* ws,
                             size_t ws_bytes, const tls_decode_opts* opts, hipStream_t stream);

/* tls_sparse_decode for callers that cannot allocate memory or pass a
 * workspace (code under stream capture, tight serving loops, harnesses that
 * forbid allocation): the same operator, arguments and results, with the
 * scratch taken from a buffer the library owns instead of ws/ws_bytes.
 * That buffer is a 64 MiB device array of the library, one per GPU it runs
 * on, held from the library's load until the process ends; the call
 * allocates nothing (no hipMalloc, no allocating library routine).  A call
 * whose route needs more than 64 MiB of scratch returns
 * TLS_ERR_WORKSPACE_TOO_SMALL and enqueues nothing (the token-level operator
 * needs 4 * b * H_kv * max_ctx bytes; the two-level operator at 96k context,
 * b = 32, H_kv = 8 needs about 4 MB).  Every call on one GPU shares that GPU's
 * buffer, so calls that may overlap on one GPU (different streams, or
 * host threads) race and must be ordered by the caller; calls in one stream
 * are ordered.  The buffer needs no clearing between calls: every region a
 * call reads is written by the same call first.  device_error (nullable)
 * is a caller-owned device word the kernels OR TLS_DEVERR_* bits into (the
 * caller zeroes and reads it); with NULL, device-side errors go unreported.
 * The current device must be the one `stream` belongs to. */
tls_status tls_sparse_decode_noalloc(const tls_layout* layout, const void* q, const tls_kv_view* kv,
                                     const int32_t* ctx_lens, const void* kmax, const void* kmin,
                                     const uint8_t* codes, const float* qparams, const int32_t* channels,
                                     int32_t K_b, int32_t K_t, const int32_t* block_ids_in,
                                     const int32_t* token_ids_in, void* out, float* lse,
                                     int32_t* block_ids_out, int32_t* token_ids_out,
                                     uint32_t* device_error, const tls_decode_opts* opts,
                                     hipStream_t stream);

/* Incremental block transfer of the offloaded KV tier, Sec. 4.2: with the
 * resident set C_t of each unit described by slot_map ([units][m_max]) and
 * slot_owner ([units][n_slots], block id held by each slot or -1), brings in
 * T_t = M_t \ C_t for M_t = block_ids_new ([b][H_kv][K_b]).
 * Slots holding blocks outside block_ids_new and block_ids_live (the blocks
 * the in-flight attention step may still read, nullable) are released
 * first; each new block then takes the lowest free slot, its K (and V) rows
 * are copied from the pinned host arrays host_k/host_v (dense layouts) into
 * the pool over PCIe by device-side reads, and slot_map/slot_owner are
 * updated.  transfer_count (nullable) [units] receives |T_t|.  n_slots must
 * be >= 2*K_b when block_ids_live is given (>= K_b otherwise).  Enqueue on a
 * side stream and order it against the attention step with events: while it
 * runs, the in-flight step may read only blocks of block_ids_live, whose
 * slot_map entries and slots this call leaves untouched.  The workspace
 * (sized for K_b and any K_t) may be the one the concurrent decode step
 * uses: the transfer lists live in a region no other call touches, and both
 * calls only set bits of the shared error word. */
tls_status tls_prefetch_blocks(const tls_layout* layout, const void* host_k, const void* host_v,
                               const int32_t* ctx_lens, const int32_t* block_ids_new,
                               const int32_t* block_ids_live, int32_t K_b, void* pool_k,
                               void* pool_v, int64_t n_slots, int32_t* slot_map,
                               int32_t* slot_owner, int32_t* transfer_count, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/* Decode-time append (the index definitions of Sec. 4.1 kept current as the
 * context grows; with the offloaded tier of Sec. 4.2).  For every sequence s
 * with n = ctx_lens[s] >= 1 (the length including the new token), the token
 * at t = n - 1:
 *   K[s][h][t][:] = k_new[s][h][:]   (and V from v_new unless mla_shared_kv);
 *   block summaries of block t/B: the row itself when t opens the block,
 *     else the elementwise max / min of the stored summaries and the row --
 *     the exact max / min of the block's rows, equal bit for bit to a
 *     rebuild (the summaries must describe rows [B*(t/B), t));
 *   token-index row t, quantised as tls_build_token_index does;
 *   and, when pool is given (its slot_map non-NULL) and block t/B is resident,
 *     row t%B of the block's pool slot (K, and V unless mla_shared_kv), so a
 *     resident block stays a copy of the cache.
 * k_new [b][H_kv][d_qk], v_new [b][H_kv][d_v] (device; v_new NULL iff
 * mla_shared_kv).  K and V (dense layouts) may be device memory or pinned
 * host memory (the offloaded tier's host copy); the row is stored there by
 * the device.  Call once per decode step, after raising ctx_lens by one and
 * before the step's selection.  Sequences with ctx_lens 0 are skipped;
 * ctx_lens outside [0, max_ctx] and slots >= pool->n_slots are skipped.
 * Must not run concurrently with tls_prefetch_blocks on the same pool (order
 * them with events: the prefetch of a step then sees the appended rows in
 * host memory). */
tls_status tls_append_tokens(const tls_layout* layout, const void* k_new, const void* v_new,
                             const int32_t* ctx_lens, const int32_t* channels, void* K, void* V, void* kmax,
                             void* kmin, uint8_t* codes, float* qparams, const tls_kv_view* pool,
                             hipStream_t stream);

/* Offload of the prefill KV cache to host memory (Sec. 4.2 / Fig. 2: after
 * prefill the cache lives in host memory and only a resident subset stays in
 * HBM).  Copies rows [tok_begin, min(tok_end, ctx_len)) of every unit of the
 * dense device K (and V) into host_k (and host_v), caller-owned pinned host
 * arrays with the same dense layouts, by device-side stores over PCIe on a
 * few work-groups (enqueue on a side stream to overlap other work).  V and
 * host_v are NULL iff mla_shared_kv.  Rows outside the range are untouched. */
tls_status tls_offload_kv(const tls_layout* layout, const void* K, const void* V, const int32_t* ctx_lens,
                          int32_t tok_begin, int32_t tok_end, void* host_k, void* host_v,
                          hipStream_t stream);

/* Initial residency of the offloaded tier (Sec. 4.2 / Fig. 2: the blocks
 * selected for the final prefill query stay in HBM).  Empties the pool
 * (slot_map all -1, slot_owner all -1), then gives the blocks of block_ids
 * ([b][H_kv][K_b], -1 entries ignored; normally tls_select_blocks of the
 * last prompt token's query) slots 0, 1, ... in ascending block order and
 * copies their rows from src_k/src_v (dense layouts, device memory or
 * pinned host memory) into the pool.  The result is the state
 * tls_prefetch_blocks would reach from an empty pool; the decode loop then
 * continues with tls_prefetch_blocks.  n_slots >= K_b (2 * K_b for the
 * lagged schedule).  Block ids past the unit's block count set
 * TLS_DEVERR_BLOCK_ID and are skipped. */
tls_status tls_init_residency(const tls_layout* layout, const void* src_k, const void* src_v,
                              const int32_t* ctx_lens, const int32_t* block_ids, int32_t K_b,
                              void* pool_k, void* pool_v, int64_t n_slots, int32_t* slot_map,
                              int32_t* slot_owner, void* ws, size_t ws_bytes, hipStream_t stream);

/* Reads (and, if clear != 0, resets) the device error word of a workspace.
 * Synchronous: waits for `stream`.  *flags receives TLS_DEVERR_* bits. */
tls_status tls_check_device_error(const void* ws, size_t ws_bytes, int32_t clear, int32_t* flags,
                                  hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TLS_H_ */
