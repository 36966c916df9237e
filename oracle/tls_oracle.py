"""CPU oracle of two-level sparse decode attention (AsyncTLS, arXiv 2604.07815).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
calls it.  It shares no code with the GPU implementation: both sides only
consume the same seeded input arrays.

Everything here is a plain, slow, step-by-step restatement of the method in
float64 (NumPy), except the INT4 token-index quantisation, which is carried
out in float32 because its codes must be reproduced bit for bit.  Library
primitives (a matrix product, a sort, ``exp``) serve as single steps; there
is no blocking, fusion or reordering beyond what the paper writes down.

Notation follows the paper: per KV group ("unit") there are G query heads
q_h in R^d, cached keys K and values V (n rows), blocks of B tokens,
block summaries k^max / k^min, the block budget k_b, the channel set C with
|C| = d_c, the token budget k_t and the softmax scale sigma (1/sqrt(d)).

Readings taken where the paper is silent or ambiguous:

* tail block: the cache is cut into ceil(n/B) blocks and the last one
  summarises only its valid tokens (the paper writes floor(n/B), which would
  make the newest tokens unselectable);
* top-k: ties go to the lowest index, -0.0 equals +0.0, the budget is clamped
  to the number of valid items, selections are returned in ascending order;
* quantisation ("INT4", Sec. 4.1 / Sec. 5 setup): per token and per group of
  32 consecutive entries of C, asymmetric uint4 with float32 parameters
  scale = (max - min)/15 and min, code = rint_half_even((x - min)/scale)
  clamped to [0, 15] (all codes 0 when scale == 0); dequantised value
  min + code*scale; two codes per byte, low nibble first;
* the query side of the token index is not quantised;
* the softmax inside the approximate score runs per head over the candidate
  tokens of the selected blocks, then the G head distributions are averaged;
* sigma = 1/sqrt(d_qk) in both the approximate score and the attention;
* an empty selection gives a zero output row and lse = -inf.
"""
from __future__ import annotations

import numpy as np

QUANT_GROUP = 32
QUANT_LEVELS = 15


# ----------------------------------------------------------------------------
# Block level (Sec. 4.1, "Coarse-grained Block Selection")
# ----------------------------------------------------------------------------

def num_blocks(n: int, B: int) -> int:
    """Block count for n valid tokens: ceil(n/B) (tail-block reading)."""
    return -(-int(n) // int(B))


def block_summaries(K: np.ndarray, n: int, B: int):
    """Per-channel max and min key over the tokens of each block
    (Sec. 4.1, block representation k^max_i, k^min_i).

    K: [>= n][d] float64.  Returns (kmax, kmin), each [ceil(n/B)][d]."""
    m = num_blocks(n, B)
    d = K.shape[1]
    kmax = np.empty((m, d), dtype=np.float64)
    kmin = np.empty((m, d), dtype=np.float64)
    for i in range(m):
        rows = K[i * B:min((i + 1) * B, n)]
        kmax[i] = rows.max(axis=0)
        kmin[i] = rows.min(axis=0)
    return kmax, kmin


def quest_scores(q_group: np.ndarray, kmax: np.ndarray, kmin: np.ndarray) -> np.ndarray:
    """Block importance, literal Quest form (Sec. 4.1):
    s_i = sum_h sum_k max(q_{h,k} kmax_{i,k}, q_{h,k} kmin_{i,k}).

    q_group: [G][d]; kmax/kmin: [m][d].  Returns [m]."""
    s = np.zeros(kmax.shape[0], dtype=np.float64)
    for h in range(q_group.shape[0]):
        a = q_group[h][None, :] * kmax
        b = q_group[h][None, :] * kmin
        s += np.maximum(a, b).sum(axis=1)
    return s


def quest_scores_gemm(q_group: np.ndarray, kmax: np.ndarray, kmin: np.ndarray) -> np.ndarray:
    """The same scores via the paper's GEMM reformulation (Sec. 4.1):
    q^max = max(q, 0), q^min = min(q, 0),
    s_i = sum_h (q^max_h . kmax_i + q^min_h . kmin_i)."""
    qmax = np.maximum(q_group, 0.0)
    qmin = np.minimum(q_group, 0.0)
    return (qmax @ kmax.T + qmin @ kmin.T).sum(axis=0)


def topk_ascending(scores: np.ndarray, k: int, valid: np.ndarray | None = None) -> np.ndarray:
    """Indices of the k largest scores (ties -> lower index), ascending.

    `valid` (bool mask) restricts the candidates; k is clamped to their count."""
    idx = np.arange(len(scores))
    if valid is not None:
        idx = idx[valid]
    s = np.asarray(scores, dtype=np.float64)[idx] + 0.0  # -0.0 -> +0.0
    k = min(int(k), len(idx))
    # primary key: score descending; secondary: index ascending
    order = np.lexsort((idx, -s))
    return np.sort(idx[order[:k]]).astype(np.int64)


def select_blocks(q_group: np.ndarray, kmax: np.ndarray, kmin: np.ndarray, k_b: int):
    """M_t: the top-k_b blocks of the unit (Sec. 4.1).  Returns (ids, scores)."""
    s = quest_scores(q_group, kmax, kmin)
    return topk_ascending(s, k_b), s


# ----------------------------------------------------------------------------
# Token index (Sec. 4.1, "Fine-grained Token Selection": channel projection
# onto C followed by INT4 quantisation; d_c and INT4 from Sec. 5 setup)
# ----------------------------------------------------------------------------

def quantize_group(x: np.ndarray):
    """Asymmetric uint4 quantisation of rows of QUANT_GROUP values, float32.

    x: [rows][32] float32 (exact copies of the key entries).
    Returns (codes uint8 [rows][32], scale f32 [rows], mn f32 [rows])."""
    x = np.asarray(x, dtype=np.float32)
    mn = x.min(axis=1)
    mx = x.max(axis=1)
    scale = (mx - mn) / np.float32(QUANT_LEVELS)          # float32 ops
    codes = np.zeros(x.shape, dtype=np.uint8)
    nz = scale != np.float32(0.0)
    if nz.any():
        v = (x[nz] - mn[nz][:, None]) / scale[nz][:, None]  # float32 ops
        codes[nz] = np.clip(np.rint(v), 0, QUANT_LEVELS).astype(np.uint8)
    return codes, scale.astype(np.float32), mn.astype(np.float32)


def token_index(K: np.ndarray, n: int, channels: np.ndarray):
    """Token-level index rows for tokens [0, n): k~_j = Quantize(k_j[C]).

    K: [>= n][d] (float32 or float64 holding values exact in float32).
    Returns (codes_packed uint8 [n][d_c/2], qparams float32 [n][d_c/32][2])
    with qparams[..., 0] = scale and qparams[..., 1] = min."""
    channels = np.asarray(channels)
    d_c = len(channels)
    assert d_c % QUANT_GROUP == 0
    x = np.asarray(K[:n][:, channels], dtype=np.float32)
    ng = d_c // QUANT_GROUP
    codes = np.zeros((n, d_c), dtype=np.uint8)
    qp = np.zeros((n, ng, 2), dtype=np.float32)
    for g in range(ng):
        c, sc, mn = quantize_group(x[:, g * QUANT_GROUP:(g + 1) * QUANT_GROUP])
        codes[:, g * QUANT_GROUP:(g + 1) * QUANT_GROUP] = c
        qp[:, g, 0] = sc
        qp[:, g, 1] = mn
    return pack_codes(codes), qp


def pack_codes(codes: np.ndarray) -> np.ndarray:
    """Two 4-bit codes per byte: byte i = code[2i] | code[2i+1] << 4."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


def unpack_codes(packed: np.ndarray) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty((packed.shape[0], packed.shape[1] * 2), dtype=np.uint8)
    out[:, 0::2] = packed & 0xF
    out[:, 1::2] = packed >> 4
    return out


def dequantize(packed: np.ndarray, qparams: np.ndarray) -> np.ndarray:
    """x^ = min + code*scale, per 32-channel group, in float64.  Returns [n][d_c]."""
    codes = unpack_codes(packed).astype(np.float64)
    n, d_c = codes.shape
    scale = np.repeat(qparams[:, :, 0].astype(np.float64), QUANT_GROUP, axis=1)
    mn = np.repeat(qparams[:, :, 1].astype(np.float64), QUANT_GROUP, axis=1)
    return mn + codes * scale


# ----------------------------------------------------------------------------
# Channel set C (Sec. 4.1, "Fine-grained Token Selection": the importance of
# each channel over a held-out calibration set, then the top-d_c channels)
# ----------------------------------------------------------------------------

def channel_absmax(x: np.ndarray) -> np.ndarray:
    """max over the calibration rows of |x|, per (head, channel).

    x: [N][H][d] (token-major activations).  An empty set gives zeros (the
    identity of a maximum of absolute values)."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    if x.shape[0] == 0:
        return np.zeros(x.shape[1:], dtype=np.float64)
    return x.max(axis=0)


def channel_importance(q_absmax_group: np.ndarray, k_absmax: np.ndarray) -> np.ndarray:
    """s_i = (1/G) sum_h max|q_h[i]| * max|k[i]| over the G query heads that
    share the key (q_absmax_group [G][d], k_absmax [d])."""
    G = q_absmax_group.shape[0]
    return (q_absmax_group * k_absmax[None, :]).sum(axis=0) / G


def calibrate_channels(q_cal: np.ndarray, k_cal: np.ndarray, G: int, d_c: int):
    """C per KV head: the d_c channels of highest importance (ties -> lower
    channel), ascending.  q_cal [N][H_q][d], k_cal [N][H_kv][d].

    Returns (channels [H_kv][d_c], scores [H_kv][d], q_absmax, k_absmax)."""
    qa, ka = channel_absmax(q_cal), channel_absmax(k_cal)
    H_kv = ka.shape[0]
    scores = np.stack([channel_importance(qa[g * G:(g + 1) * G], ka[g]) for g in range(H_kv)])
    chans = np.stack([topk_ascending(scores[g], d_c) for g in range(H_kv)])
    return chans, scores, qa, ka


# ----------------------------------------------------------------------------
# Token selection inside the selected blocks (Sec. 4.1)
# ----------------------------------------------------------------------------

def candidates(block_ids: np.ndarray, n: int, B: int) -> np.ndarray:
    """Token positions of the selected blocks, ascending (valid tokens only)."""
    out = []
    for i in sorted(int(b) for b in block_ids if b >= 0):
        out.extend(range(i * B, min((i + 1) * B, n)))
    return np.asarray(out, dtype=np.int64)


def token_logits(q_group: np.ndarray, channels: np.ndarray, xhat: np.ndarray, sigma: float) -> np.ndarray:
    """sigma * q~^(h) . k~_j for every head h and candidate row j: [G][rows]."""
    qt = q_group[:, np.asarray(channels)]
    return sigma * (qt @ xhat.T)


def approx_scores(logits: np.ndarray) -> np.ndarray:
    """alpha~_j = (1/G) sum_h softmax_j(logits_h) - each head normalised over
    the candidate set, then the G distributions averaged (Sec. 4.1)."""
    G = logits.shape[0]
    if logits.shape[1] == 0:
        return np.zeros(0)
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    p = e / e.sum(axis=1, keepdims=True)
    return p.sum(axis=0) / G


def select_tokens(q_group, channels, codes_packed, qparams, block_ids, n, B, k_t, sigma,
                  xhat_all=None):
    """S_t = TopK_{k_t}(alpha~_j, j in the tokens of M_t) (Sec. 4.1).

    codes_packed/qparams cover tokens [0, n).  `xhat_all` ([n][d_c], float64)
    replaces the dequantised index when given (quantisation switched off).
    Returns (token_ids ascending, alpha~ of the candidates, candidate ids)."""
    cand = candidates(block_ids, n, B)
    if xhat_all is None:
        xhat = dequantize(codes_packed[cand], qparams[cand]) if len(cand) else np.zeros((0, len(channels)))
    else:
        xhat = xhat_all[cand]
    alpha = approx_scores(token_logits(q_group, channels, xhat, sigma))
    pick = topk_ascending(alpha, k_t)
    return cand[pick], alpha, cand


# ----------------------------------------------------------------------------
# Sparse attention over the selected tokens (Sec. 3 sparse attention;
# Sec. 4.1 final attention with full-dimensional K/V)
# ----------------------------------------------------------------------------

def sparse_attention(q_group: np.ndarray, K: np.ndarray, V: np.ndarray, ids: np.ndarray, sigma: float):
    """o_h = softmax(sigma q_h K_S^T) V_S and lse_h = log sum_j exp(sigma q_h.k_j)."""
    G = q_group.shape[0]
    ids = np.asarray(ids, dtype=np.int64)
    if len(ids) == 0:
        return np.zeros((G, V.shape[1])), np.full(G, -np.inf)
    z = sigma * (q_group @ K[ids].T)
    mz = z.max(axis=1, keepdims=True)
    e = np.exp(z - mz)
    Z = e.sum(axis=1, keepdims=True)
    o = (e / Z) @ V[ids]
    lse = (mz + np.log(Z))[:, 0]
    return o, lse


# ----------------------------------------------------------------------------
# One unit, one batch, and the offloaded (lagged) schedule
# ----------------------------------------------------------------------------

def decode_unit(q_group, K, V, n, channels, k_b, k_t, B, sigma, index=None, block_ids=None,
                token_ids=None, summaries=None):
    """Whole decode step for one (sequence, KV group).

    index: optional prebuilt (codes_packed, qparams) for tokens [0, n).
    summaries: optional prebuilt (kmax, kmin) block summaries.
    block_ids / token_ids: optional given selections (skip those stages)."""
    res = {}
    if token_ids is None:
        if block_ids is None:
            kmax, kmin = block_summaries(K, n, B) if summaries is None else summaries
            block_ids, bscores = select_blocks(q_group, kmax, kmin, k_b)
            res["block_scores"] = bscores
        if index is None:
            index = token_index(K, n, channels)
        token_ids, alpha, cand = select_tokens(q_group, channels, index[0], index[1],
                                               block_ids, n, B, k_t, sigma)
        res["alpha"] = alpha
        res["cand"] = cand
    o, lse = sparse_attention(q_group, K, V, token_ids, sigma)
    res.update(block_ids=np.asarray(block_ids) if block_ids is not None else None,
               token_ids=np.asarray(token_ids), out=o, lse=lse)
    return res


# ----------------------------------------------------------------------------
# The single-level operators the paper measures against (Sec. 5, kernel
# study): block-level selection alone (Quest) and full attention
# ----------------------------------------------------------------------------

def block_sparse_unit(q_group, K, V, n, k_b, B, sigma, summaries=None, block_ids=None):
    """Block-level selection alone: M = the top-k_b blocks (Sec. 4.1 coarse
    stage), then attention over every valid token of M."""
    res = {}
    if block_ids is None:
        kmax, kmin = block_summaries(K, n, B) if summaries is None else summaries
        block_ids, bscores = select_blocks(q_group, kmax, kmin, k_b)
        res["block_scores"] = bscores
    ids = candidates(block_ids, n, B)
    o, lse = sparse_attention(q_group, K, V, ids, sigma)
    res.update(block_ids=np.asarray(block_ids), token_ids=ids, out=o, lse=lse)
    return res


def token_sparse_unit(q_group, K, V, n, channels, k_t, B, sigma, index=None):
    """Token-level selection alone (the Double Sparsity baseline): the
    approximate score of Sec. 4.1 over every valid token (the candidate set is
    every block), the top-k_t, then attention over them."""
    if index is None:
        index = token_index(K, n, channels)
    every_block = np.arange(num_blocks(n, B))
    ids, alpha, cand = select_tokens(q_group, channels, index[0], index[1], every_block, n, B, k_t, sigma)
    o, lse = sparse_attention(q_group, K, V, ids, sigma)
    return dict(token_ids=np.asarray(ids), alpha=alpha, cand=cand, out=o, lse=lse)


def dense_unit(q_group, K, V, n, sigma):
    """Full attention over the n cached tokens."""
    o, lse = sparse_attention(q_group, K, V, np.arange(int(n)), sigma)
    return dict(out=o, lse=lse)


def unit_views(q, K, V, s, g, group, mla, d_v):
    """(q_group, K_unit, V_unit) for sequence s and KV head g (float64 arrays)."""
    qg = q[s, g * group:(g + 1) * group]
    Ku = K[s, g]
    Vu = Ku[:, :d_v] if mla else V[s, g]
    return qg, Ku, Vu


def decode_batch(q, K, V, ctx_lens, channels, k_b, k_t, B, sigma, mla=False, units=None,
                 d_v=None):
    """Run decode_unit over the requested (s, g) units (default: all).

    q: [b][H_q][d_qk]; K: [b][H_kv][T][d_qk]; V: [b][H_kv][T][d_v] or None (MLA).
    Returns {(s, g): result dict}."""
    b, H_q, _ = q.shape
    H_kv = K.shape[1]
    G = H_q // H_kv
    d_v = d_v if d_v is not None else (V.shape[-1] if V is not None else K.shape[-1])
    if units is None:
        units = [(s, g) for s in range(b) for g in range(H_kv)]
    out = {}
    for (s, g) in units:
        qg, Ku, Vu = unit_views(q, K, V, s, g, G, mla, d_v)
        out[(s, g)] = decode_unit(qg, Ku, Vu, int(ctx_lens[s]), channels[g], k_b, k_t, B, sigma)
    return out


def lagged_decode(q_steps, K, V, n, channels, k_b, k_t, B, sigma, d_v, mla=False, s=0, g=0):
    """Offloaded schedule for one unit (Sec. 4.2): with a one-step lag,
    M_t = BlockSelect(q_t) and S_t = TokenSelect(q_t, M_{t-1}); the resident
    set evolves as T_t = M_t minus C_t, C_{t+1} = M_t, with C_1 = M_0.

    q_steps: [T+1][b][H_q][d] float64.  n: the context length, or a sequence
    of T+1 lengths when the context grows during decoding (n[0] at the
    prefill's selection of M_0; at step t the tokens below n[t] exist, the
    block and token indices are those of that length, and the candidates of
    M_{t-1} are its blocks' tokens below n[t]).  Attention always reads the
    full K/V, so offloading must not change any result.  Returns a list over
    t = 1..T."""
    H_kv = K.shape[1]
    G = q_steps.shape[2] // H_kv
    n_at = [int(n)] * q_steps.shape[0] if np.ndim(n) == 0 else [int(x) for x in n]
    qg0, Ku, Vu = unit_views(q_steps[0], K, V, s, g, G, mla, d_v)
    kmax, kmin = block_summaries(Ku, n_at[0], B)
    M_prev, _ = select_blocks(qg0, kmax, kmin, k_b)
    resident = set(int(x) for x in M_prev)
    steps = []
    index, index_n = None, -1
    for t in range(1, q_steps.shape[0]):
        nt = n_at[t]
        if index_n != nt:  # the indices of the context as it stands at step t
            kmax, kmin = block_summaries(Ku, nt, B)
            index, index_n = token_index(Ku, nt, channels), nt
        qg = q_steps[t, s, g * G:(g + 1) * G]
        M_t, bscores = select_blocks(qg, kmax, kmin, k_b)
        S_t, alpha, cand = select_tokens(qg, channels, index[0], index[1], M_prev, nt, B, k_t, sigma)
        o, lse = sparse_attention(qg, Ku, Vu, S_t, sigma)
        Mset = set(int(x) for x in M_t)
        transfer = sorted(Mset - resident)
        repeat = len(Mset & set(int(x) for x in M_prev)) / max(1, len(Mset))
        steps.append(dict(block_ids=M_t, block_scores=bscores, lag_block_ids=M_prev, token_ids=S_t, alpha=alpha,
                          cand=cand, out=o, lse=lse, transfer=np.asarray(transfer, dtype=np.int64),
                          repeat=repeat, index=index))
        resident = Mset
        M_prev = M_t
    return steps
