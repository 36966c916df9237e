"""Plant plausible mistakes in the oracle (on the CPU) and check that at
least one pin fails for each: the pins constrain every step."""
import numpy as np
import pytest

import oracle_pins as P
from oracle import tls_oracle as O


def _swap_max_min(q, kmax, kmin):            # lower bound instead of upper bound
    s = np.zeros(kmax.shape[0])
    for h in range(q.shape[0]):
        s += np.minimum(q[h] * kmax, q[h] * kmin).sum(axis=1)
    return s


def _floor_blocks(K, n, B):                  # drops the tail block
    m = n // B
    return (np.array([K[i * B:(i + 1) * B].max(axis=0) for i in range(m)]).reshape(m, K.shape[1]),
            np.array([K[i * B:(i + 1) * B].min(axis=0) for i in range(m)]).reshape(m, K.shape[1]))


def _single_softmax(logits):                 # softmax of summed logits
    s = logits.sum(axis=0)
    e = np.exp(s - s.max())
    return e / e.sum()


def _no_mean(logits):                        # drops the 1/G
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    return (e / e.sum(axis=1, keepdims=True)).sum(axis=0)


def _floor_quant(x):                         # floor instead of round-half-even
    x = np.asarray(x, dtype=np.float32)
    mn, mx = x.min(axis=1), x.max(axis=1)
    sc = (mx - mn) / np.float32(15)
    c = np.zeros(x.shape, np.uint8)
    nz = sc != 0
    c[nz] = np.clip(np.floor((x[nz] - mn[nz][:, None]) / sc[nz][:, None]), 0, 15).astype(np.uint8)
    return c, sc, mn


def _high_nibble_first(codes):
    codes = np.asarray(codes, dtype=np.uint8)
    return ((codes[:, 0::2] << 4) | codes[:, 1::2]).astype(np.uint8)


def _ties_high(scores, k, valid=None):      # ties go to the higher index
    idx = np.arange(len(scores))
    k = min(int(k), len(idx))
    order = np.lexsort((-idx, -np.asarray(scores, dtype=np.float64)))
    return np.sort(idx[order[:k]])


def _attn_no_scale(q, K, V, ids, sigma):    # forgets the softmax scale
    return _REAL_ATTN(q, K, V, ids, 1.0)


def _attn_transposed_values(q, K, V, ids, sigma):   # wrong gather for V
    rev = np.asarray(ids)[::-1].copy()
    o, lse = _REAL_ATTN(q, K, V, ids, sigma)
    o2, _ = _REAL_ATTN(q, K, V[::-1].copy(), len(V) - 1 - np.asarray(ids), sigma) if len(ids) else (o, lse)
    return o2, lse


def _wrong_candidates(block_ids, n, B):      # ignores the ragged tail
    out = []
    for i in sorted(int(b) for b in block_ids if b >= 0):
        out.extend(range(i * B, (i + 1) * B))
    return np.asarray(out, dtype=np.int64)


_REAL_ATTN = O.sparse_attention
_REAL_INDEX = O.token_index


def _logits_prefix_channels(q, channels, xhat, sigma):   # q~ = q[:, :d_c] instead of q[:, C]
    return sigma * (q[:, :len(channels)] @ xhat.T)


def _logits_no_sigma(q, channels, xhat, sigma):          # forgets the scale in the approximate score
    return q[:, np.asarray(channels)] @ xhat.T

def _summaries_past_n(K, n, B):              # reads whole blocks, past the valid tokens
    m = -(-n // B)
    return (np.array([K[i * B:(i + 1) * B].max(axis=0) for i in range(m)]),
            np.array([K[i * B:(i + 1) * B].min(axis=0) for i in range(m)]))


def _index_prefix_channels(K, n, channels):   # k~ = Quantize(k[:d_c]) instead of k[C]
    return _REAL_INDEX(K, n, np.arange(len(channels)))


def _absmax_signed(x):                       # max of x instead of max of |x|
    x = np.asarray(x, dtype=np.float64)
    return np.zeros(x.shape[1:]) if x.shape[0] == 0 else x.max(axis=0)


def _importance_sum(qa, ka):                 # drops the 1/G
    return (qa * ka[None, :]).sum(axis=0)


def _importance_max_heads(qa, ka):           # max over the heads instead of their mean
    return (qa * ka[None, :]).max(axis=0)


MUTATIONS = [
    ("quest_scores", _swap_max_min),
    ("block_summaries", _floor_blocks),
    ("block_summaries", _summaries_past_n),
    ("token_index", _index_prefix_channels),
    ("approx_scores", _single_softmax),
    ("approx_scores", _no_mean),
    ("token_logits", _logits_prefix_channels),
    ("token_logits", _logits_no_sigma),
    ("quantize_group", _floor_quant),
    ("pack_codes", _high_nibble_first),
    ("topk_ascending", _ties_high),
    ("sparse_attention", _attn_no_scale),
    ("sparse_attention", _attn_transposed_values),
    ("candidates", _wrong_candidates),
    ("channel_absmax", _absmax_signed),
    ("channel_importance", _importance_sum),
    ("channel_importance", _importance_max_heads),
]


@pytest.mark.parametrize("name,bad", MUTATIONS, ids=[f"{n}:{b.__name__}" for n, b in MUTATIONS])
def test_mutation_is_caught(monkeypatch, name, bad):
    monkeypatch.setattr(O, name, bad)
    failures = 0
    for pin in P.ALL_PINS:
        try:
            pin()
        except Exception:
            failures += 1
    assert failures > 0, f"no pin caught the mutation of {name}"
