"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin reads the oracle's functions through the module object at call
time, so the mutation tests can replace one function with a plausible
mistake and check that some pin fails.  Nothing here retypes the oracle's
formulas: the expected values are hand-derived fixtures (tests/golden),
closed forms, invariants, brute force, or independent library routines.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
import scipy.special
import torch

from oracle import tls_oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --- block level -------------------------------------------------------------

def pin_quest_golden():
    """Hand-derived block summaries, Quest scores and selections (Sec. 4.1)."""
    g = _golden("quest_tiny.json")
    K = np.array(g["keys"], dtype=np.float64)
    q = np.array(g["queries"], dtype=np.float64)
    kmax, kmin = O.block_summaries(K, g["n"], g["B"])
    assert kmax.shape == (3, 2), kmax.shape
    np.testing.assert_array_equal(kmax, np.array(g["kmax"], dtype=np.float64))
    np.testing.assert_array_equal(kmin, np.array(g["kmin"], dtype=np.float64))
    s = O.quest_scores(q, kmax, kmin)
    np.testing.assert_array_equal(s, np.array(g["scores"], dtype=np.float64))
    for k, ids in g["topk"].items():
        got, _ = O.select_blocks(q, kmax, kmin, int(k))
        assert list(got) == ids, (k, got, ids)


def pin_quest_forms_agree(seed=11):
    """The literal Quest score equals the GEMM reformulation (Sec. 4.1)."""
    r = np.random.default_rng(seed)
    for G, d, m in [(1, 8, 5), (4, 128, 37), (32, 576, 9)]:
        q = r.standard_normal((G, d))
        a, b = r.standard_normal((m, d)), r.standard_normal((m, d))
        kmax, kmin = np.maximum(a, b), np.minimum(a, b)
        lit = O.quest_scores(q, kmax, kmin)
        gem = O.quest_scores_gemm(q, kmax, kmin)
        np.testing.assert_allclose(lit, gem, rtol=1e-12, atol=1e-12)


def pin_quest_upper_bound(seed=12):
    """Every token of a block scores at most the block's Quest score:
    sum_h q_h.k_j <= s_i for j in block i; equality for one-token blocks."""
    r = np.random.default_rng(seed)
    G, d, B, n = 4, 32, 16, 16 * 7 + 5
    q = r.standard_normal((G, d))
    K = r.standard_normal((n, d))
    kmax, kmin = O.block_summaries(K, n, B)
    assert kmax.shape[0] == 8
    s = O.quest_scores(q, kmax, kmin)
    true = (q @ K.T).sum(axis=0)
    for i in range(kmax.shape[0]):
        blk = true[i * B:min((i + 1) * B, n)]
        assert blk.max() <= s[i] + 1e-9, (i, blk.max(), s[i])
    # B = 1: the bound is tight
    kmax1, kmin1 = O.block_summaries(K, n, 1)
    np.testing.assert_allclose(O.quest_scores(q, kmax1, kmin1), true, rtol=1e-12, atol=1e-12)


# --- selection ---------------------------------------------------------------

def _brute_topk(scores, k):
    """Unique k-subset S with s_i > s_j or (s_i == s_j and i < j) for i in S, j not in S."""
    n = len(scores)
    k = min(k, n)
    found = []
    for S in itertools.combinations(range(n), k):
        Sset = set(S)
        ok = all((scores[i] > scores[j]) or (scores[i] == scores[j] and i < j)
                 for i in S for j in range(n) if j not in Sset)
        if ok:
            found.append(list(S))
    assert len(found) == 1, found
    return found[0]


def pin_topk_bruteforce(seed=13):
    """Top-k with lowest-index tie-break equals exhaustive search on tiny inputs."""
    r = np.random.default_rng(seed)
    for trial in range(40):
        n = int(r.integers(1, 9))
        s = r.integers(-3, 4, size=n).astype(np.float64)   # many ties
        if trial % 5 == 0:
            s[s == 0] = -0.0                               # -0.0 ties with +0.0
            s[: n // 2][s[: n // 2] == -0.0] = 0.0
        k = int(r.integers(0, n + 2))
        got = list(O.topk_ascending(s, k))
        assert got == _brute_topk(list(s), k), (s, k, got)


def pin_candidates():
    """Candidates are the valid tokens of the selected blocks, ascending."""
    got = list(O.candidates(np.array([2, 0, -1]), 10, 4))
    assert got == [0, 1, 2, 3, 8, 9], got


# --- token index ---------------------------------------------------------------

def pin_quant_golden():
    """Hand-derived INT4 codes, packing and dequantised values."""
    g = _golden("quant_tiny.json")
    for case in g["cases"]:
        x = np.array([case["x"]], dtype=np.float32)
        codes, scale, mn = O.quantize_group(x)
        assert list(codes[0]) == case["codes"], (list(codes[0]), case["codes"])
        assert float(scale[0]) == case["scale"] and float(mn[0]) == case["min"]
        packed, qp = O.token_index(x, 1, np.arange(32))
        assert list(packed[0]) == case["packed"], (list(packed[0]), case["packed"])
        deq = O.dequantize(packed, qp)[0]
        assert list(deq) == case["dequant"], (list(deq), case["dequant"])


def pin_quant_bound(seed=14):
    """codes in [0,15]; |x - x^| <= scale/2 (+ float32 rounding); the group's
    min and max are reproduced exactly (codes 0 and 15)."""
    r = np.random.default_rng(seed)
    x = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(r.standard_normal((500, 64)).astype(np.float32)))
    ch = np.arange(64)
    packed, qp = O.token_index(x, 500, ch)
    codes = O.unpack_codes(packed)
    assert codes.max() <= 15
    deq = O.dequantize(packed, qp)
    for g in range(2):
        sl = slice(32 * g, 32 * g + 32)
        xs = x[:, sl].astype(np.float64)
        sc = qp[:, g, 0].astype(np.float64)
        err = np.abs(xs - deq[:, sl])
        assert np.all(err <= sc[:, None] * (0.5 + 1e-5)), err.max()
        rows = np.arange(500)
        assert np.all(deq[rows, 32 * g + xs.argmin(axis=1)] == xs.min(axis=1))
        assert np.all(codes[rows, 32 * g + xs.argmax(axis=1)] == 15)
        np.testing.assert_allclose(deq[rows, 32 * g + xs.argmax(axis=1)], xs.max(axis=1),
                                   rtol=1e-6)


# --- approximate score -----------------------------------------------------------

def pin_alpha_golden():
    """Per-head softmax average, hand-derived; it is not monotone in the
    summed logits, so the ranking differs from a single softmax."""
    g = _golden("alpha_tiny.json")
    a = O.approx_scores(np.array(g["logits"], dtype=np.float64))
    np.testing.assert_allclose(a, g["alpha"], atol=g["abs_tol"], rtol=0)
    for k, ids in g["topk"].items():
        assert list(O.topk_ascending(a, int(k))) == ids


def pin_alpha_distribution(seed=15):
    """alpha~ is a probability distribution over the candidates, and with
    G = 1, C = all channels and quantisation off it is the exact attention
    distribution (a textbook softmax), whose top-k it then selects."""
    r = np.random.default_rng(seed)
    d, n, B = 32, 200, 16
    K = r.standard_normal((n, d))
    for G in (1, 3):
        q = r.standard_normal((G, d))
        lg = O.token_logits(q, np.arange(d), K, 0.3)
        a = O.approx_scores(lg)
        assert abs(a.sum() - 1.0) < 1e-12
    q = r.standard_normal((1, d))
    sigma = 1.0 / math.sqrt(d)
    blocks = np.array([1, 4, 7, 12])
    ids, alpha, cand = O.select_tokens(q, np.arange(d), None, None, blocks, n, B, 10, sigma,
                                       xhat_all=K)
    w = scipy.special.softmax(sigma * (K[cand] @ q[0]))
    np.testing.assert_allclose(alpha, w, rtol=1e-12, atol=1e-15)
    ref = np.sort(cand[np.argsort(-w, kind="stable")[:10]])
    assert list(ids) == list(ref)


def pin_channel_projection_golden():
    """Hand-derived logits and alpha~ with a channel set that is not a prefix
    of the channels: the query side is gathered at C (q~ = q[C])."""
    g = _golden("channel_projection_tiny.json")
    q = np.array(g["queries"], dtype=np.float64)
    xhat = np.array(g["xhat"], dtype=np.float64)
    lg = O.token_logits(q, np.array(g["channels"]), xhat, g["sigma"])
    np.testing.assert_array_equal(lg, np.array(g["logits"], dtype=np.float64))
    a = O.approx_scores(lg)
    np.testing.assert_allclose(a, g["alpha"], atol=g["abs_tol"], rtol=0)
    assert list(O.topk_ascending(a, 1)) == g["top1"]


def pin_channel_projection_property(seed=19):
    """The token selection reads the query only at the channels of C: noise
    added to the other channels changes neither alpha~ nor S_t, while a query
    that is zero on C (and arbitrary elsewhere) gives the uniform alpha~ of a
    zero query, whose top-k is the lowest candidate positions.  C is a random,
    non-contiguous subset, quantisation on."""
    r = np.random.default_rng(seed)
    d, n, B, G, k_t = 96, 300, 16, 3, 20
    K = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(r.standard_normal((n, d)).astype(np.float32)))
    C = np.sort(r.choice(np.arange(1, d), size=32, replace=False))
    assert not np.array_equal(C, np.arange(32))
    codes, qp = O.token_index(K, n, C)
    blocks = np.array([0, 3, 7, 11, 18])
    sigma = 1.0 / math.sqrt(d)
    q = r.standard_normal((G, d))
    off = np.setdiff1d(np.arange(d), C)
    q_noise = q.copy()
    q_noise[:, off] += 5.0 * r.standard_normal((G, len(off)))
    ids, alpha, cand = O.select_tokens(q, C, codes, qp, blocks, n, B, k_t, sigma)
    ids2, alpha2, _ = O.select_tokens(q_noise, C, codes, qp, blocks, n, B, k_t, sigma)
    np.testing.assert_array_equal(alpha2, alpha)
    np.testing.assert_array_equal(ids2, ids)
    q_off = np.zeros_like(q)
    q_off[:, off] = r.standard_normal((G, len(off)))
    ids3, alpha3, cand3 = O.select_tokens(q_off, C, codes, qp, blocks, n, B, k_t, sigma)
    np.testing.assert_array_equal(alpha3, np.full(len(cand3), 1.0 / len(cand3)))
    np.testing.assert_array_equal(ids3, cand3[:k_t])


def pin_token_index_projection(seed=21):
    """The token index reads the key only at the channels of C (Sec. 4.1,
    k~ = Quantize(k[C])): it equals the index of the projected key matrix
    K[:, C] built on its own channels 0..d_c-1, and noise on the channels
    outside C changes no code and no (scale, min).  C is a random,
    non-contiguous subset."""
    r = np.random.default_rng(seed)
    d, n = 80, 45
    K = r.standard_normal((n, d)).astype(np.float32).astype(np.float64)
    C = np.sort(r.choice(np.arange(1, d), size=32, replace=False))
    assert not np.array_equal(C, np.arange(32))
    codes, qp = O.token_index(K, n, C)
    codes_p, qp_p = O.token_index(np.ascontiguousarray(K[:, C]), n, np.arange(32))
    np.testing.assert_array_equal(codes, codes_p)
    np.testing.assert_array_equal(qp, qp_p)
    off = np.setdiff1d(np.arange(d), C)
    K2 = K.copy()
    K2[:, off] = (K2[:, off] + 7.0 * r.standard_normal((n, len(off)))).astype(np.float32)
    codes2, qp2 = O.token_index(K2, n, C)
    np.testing.assert_array_equal(codes2, codes)
    np.testing.assert_array_equal(qp2, qp)


def pin_block_summaries_tail(seed=20):
    """The block summaries cover only the n valid tokens (R1): rows at or past
    n — here huge values of both signs, and NaN — change nothing, the tail
    block is summarised over its valid rows alone, and every summary is
    finite; each summary is the brute-force max / min of its block's rows."""
    r = np.random.default_rng(seed)
    B, d, n = 16, 8, 53  # 4 blocks, the last with 5 valid rows
    K = r.standard_normal((n, d))
    pad = np.full((3 * B, d), 1e30)
    pad[1::2] = -1e30
    pad[5] = np.nan
    kmax, kmin = O.block_summaries(np.vstack([K, pad]), n, B)
    kmax0, kmin0 = O.block_summaries(K, n, B)
    assert kmax.shape == (4, d) and np.all(np.isfinite(kmax)) and np.all(np.isfinite(kmin))
    np.testing.assert_array_equal(kmax, kmax0)
    np.testing.assert_array_equal(kmin, kmin0)
    for i in range(4):
        for c in range(d):
            vals = [K[j, c] for j in range(i * B, min((i + 1) * B, n))]
            assert kmax[i, c] == max(vals) and kmin[i, c] == min(vals)


# --- attention -------------------------------------------------------------------

def pin_attention_library(seed=16):
    """Sparse attention equals torch's float64 scaled-dot-product attention on
    the gathered rows; lse equals scipy's logsumexp."""
    r = np.random.default_rng(seed)
    G, d, dv, n = 4, 64, 48, 300
    q = r.standard_normal((G, d))
    K = r.standard_normal((n, d))
    V = r.standard_normal((n, dv))
    ids = np.sort(r.choice(n, 77, replace=False))
    sigma = 0.21
    o, lse = O.sparse_attention(q, K, V, ids, sigma)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :], torch.from_numpy(K[ids])[None, None].expand(1, G, -1, -1),
        torch.from_numpy(V[ids])[None, None].expand(1, G, -1, -1), scale=sigma)[0, :, 0].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(sigma * q @ K[ids].T, axis=1),
                               rtol=1e-12)


def pin_attention_closed_form():
    """All selected keys equal -> uniform weights: o = mean of the selected V
    rows and lse = log|S| + sigma q.k; an empty selection gives o = 0,
    lse = -inf."""
    G, d, dv, n = 2, 8, 4, 12
    q = np.arange(G * d, dtype=np.float64).reshape(G, d) / 10
    K = np.tile(np.linspace(-1, 1, d), (n, 1))
    V = np.arange(n * dv, dtype=np.float64).reshape(n, dv)
    ids = np.array([1, 5, 6, 11])
    o, lse = O.sparse_attention(q, K, V, ids, 0.5)
    np.testing.assert_allclose(o, np.tile(V[ids].mean(axis=0), (G, 1)), rtol=1e-13)
    np.testing.assert_allclose(lse, math.log(4) + 0.5 * q @ K[0], rtol=1e-13)
    o0, l0 = O.sparse_attention(q, K, V, np.array([], dtype=np.int64), 0.5)
    assert np.all(o0 == 0) and np.all(np.isneginf(l0))


# --- whole pipeline on the toy workload ---------------------------------------------

def _toy_f64(n_override=None):
    cfg = synth.config("toy")
    if n_override is not None:
        cfg = cfg.replace(ctx_lo=n_override, ctx_hi=n_override)
    d = synth.make_host(cfg, pad="nan")
    q = synth.to_f64(d["q"], cfg.dtype)
    K = synth.to_f64(d["k"], cfg.dtype)
    V = synth.to_f64(d["v"], cfg.dtype)
    return cfg, d, q, K, V


def pin_dense_equivalence(n_override=None):
    """With k_b = all blocks and k_t = all tokens the operator is dense
    attention (Sec. 3), checked against torch's float64 SDPA."""
    cfg, d, q, K, V = _toy_f64(n_override)
    n = int(d["ctx_lens"][0])
    m = O.num_blocks(n, cfg.block)
    res = O.decode_batch(q, K, V, d["ctx_lens"], d["channels"], m, n, cfg.block, cfg.sigma)
    for (s, g), r in res.items():
        assert len(r["block_ids"]) == m and len(r["token_ids"]) == n
        qg = torch.from_numpy(q[s, g * cfg.group:(g + 1) * cfg.group])
        kk = torch.from_numpy(K[s, g, :n])[None, None].expand(1, cfg.group, -1, -1)
        vv = torch.from_numpy(V[s, g, :n])[None, None].expand(1, cfg.group, -1, -1)
        ref = torch.nn.functional.scaled_dot_product_attention(qg[None, :, None, :], kk, vv,
                                                               scale=cfg.sigma)[0, :, 0].numpy()
        np.testing.assert_allclose(r["out"], ref, rtol=1e-10, atol=1e-12)
        lse_ref = scipy.special.logsumexp(cfg.sigma * qg.numpy() @ K[s, g, :n].T, axis=1)
        np.testing.assert_allclose(r["lse"], lse_ref, rtol=1e-12)


def pin_invariants_and_planted(n_override=None):
    """|M| = min(k_b, m), |S| = min(k_t, |cand|), ids unique and ascending,
    S inside the selected blocks; planted high-affinity tokens are recovered."""
    cfg, d, q, K, V = _toy_f64(n_override)
    n = int(d["ctx_lens"][0])
    res = O.decode_batch(q, K, V, d["ctx_lens"], d["channels"], cfg.k_b, cfg.k_t, cfg.block,
                         cfg.sigma)
    for (s, g), r in res.items():
        M, S = r["block_ids"], r["token_ids"]
        assert len(M) == min(cfg.k_b, O.num_blocks(n, cfg.block))
        assert np.all(np.diff(M) > 0) and np.all(np.diff(S) > 0)
        cand = O.candidates(M, n, cfg.block)
        assert len(S) == min(cfg.k_t, len(cand))
        assert set(S.tolist()) <= set(cand.tolist())
        assert S.max() < n
        planted = [st + i for st in d["plant_starts"][s, g] for i in range(cfg.cluster_len)]
        assert set(p // cfg.block for p in planted) <= set(M.tolist())
        assert set(planted) <= set(S.tolist())
        assert np.all(np.isfinite(r["out"]))


def pin_single_level_operators(n_override=None):
    """The baselines: full attention equals torch's float64 SDPA over the n
    tokens; block-sparse attention attends exactly the valid tokens of the
    top-k_b blocks, equals the two-level operator with k_t >= those tokens,
    equals full attention when k_b covers every block, and keeps the planted
    blocks; token-level selection alone scores every token, equals the
    two-level operator with k_b = every block and keeps the planted tokens."""
    cfg, d, q, K, V = _toy_f64(n_override)
    n = int(d["ctx_lens"][0])
    m = O.num_blocks(n, cfg.block)
    G = cfg.group
    for g in range(cfg.h_kv):
        qg = q[0, g * G:(g + 1) * G]
        dn = O.dense_unit(qg, K[0, g], V[0, g], n, cfg.sigma)
        kk = torch.from_numpy(K[0, g, :n])[None, None].expand(1, G, -1, -1)
        vv = torch.from_numpy(V[0, g, :n])[None, None].expand(1, G, -1, -1)
        ref = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(qg)[None, :, None, :], kk, vv,
                                                               scale=cfg.sigma)[0, :, 0].numpy()
        np.testing.assert_allclose(dn["out"], ref, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(dn["lse"], scipy.special.logsumexp(cfg.sigma * qg @ K[0, g, :n].T, axis=1),
                                   rtol=1e-12)
        bs = O.block_sparse_unit(qg, K[0, g], V[0, g], n, cfg.k_b, cfg.block, cfg.sigma)
        M = bs["block_ids"]
        want = [j for j in range(n) if j // cfg.block in set(M.tolist())]
        assert bs["token_ids"].tolist() == want
        two = O.decode_unit(qg, K[0, g], V[0, g], n, d["channels"][g], cfg.k_b, cfg.k_b * cfg.block, cfg.block,
                            cfg.sigma)
        assert np.array_equal(two["block_ids"], M) and np.array_equal(two["token_ids"], bs["token_ids"])
        np.testing.assert_array_equal(two["out"], bs["out"])
        planted = [st + i for st in d["plant_starts"][0, g] for i in range(cfg.cluster_len)]
        assert set(p // cfg.block for p in planted) <= set(M.tolist())
        full = O.block_sparse_unit(qg, K[0, g], V[0, g], n, m, cfg.block, cfg.sigma)
        np.testing.assert_allclose(full["out"], dn["out"], rtol=1e-12, atol=1e-14)
        # token-level selection alone: its candidates are every valid token,
        # it equals the two-level operator with k_b = every block, keeps the
        # planted tokens, and with k_t = n it is full attention
        ts = O.token_sparse_unit(qg, K[0, g], V[0, g], n, d["channels"][g], cfg.k_t, cfg.block, cfg.sigma)
        assert ts["cand"].tolist() == list(range(n)) and len(ts["token_ids"]) == min(cfg.k_t, n)
        two_all = O.decode_unit(qg, K[0, g], V[0, g], n, d["channels"][g], m, cfg.k_t, cfg.block, cfg.sigma)
        assert np.array_equal(two_all["token_ids"], ts["token_ids"])
        assert set(planted) <= set(ts["token_ids"].tolist())
        ts_all = O.token_sparse_unit(qg, K[0, g], V[0, g], n, d["channels"][g], n, cfg.block, cfg.sigma)
        np.testing.assert_allclose(ts_all["out"], dn["out"], rtol=1e-12, atol=1e-14)


def pin_lagged_schedule():
    """Offloaded schedule (Sec. 4.2): T_t = M_t minus C_t, C_{t+1} = M_t; with a
    frozen query (rho = 1) nothing is transferred after the first step and the
    lagged result equals the same-step result."""
    cfg = synth.config("toy").replace(ctx_lo=1024, ctx_hi=1024, k_b=4, k_t=64, steps=3)
    d = synth.make_host(cfg)
    K = synth.to_f64(d["k"], cfg.dtype)
    V = synth.to_f64(d["v"], cfg.dtype)
    for rho in (1.0, 0.5):
        walk = synth.draw_query_walk(cfg.replace(rho=rho))
        qs = synth.to_f64(walk, cfg.dtype)
        steps = O.lagged_decode(qs, K, V, 1024, d["channels"][0], cfg.k_b, cfg.k_t, cfg.block,
                                cfg.sigma, cfg.d_v)
        prev = None
        for t, st in enumerate(steps, start=1):
            M, T = set(st["block_ids"].tolist()), set(st["transfer"].tolist())
            C = set(st["lag_block_ids"].tolist())     # C_t = M_{t-1}
            assert T == M - C and not (T & C)
            assert len(T) == len(M) - len(M & C)
            assert set(st["token_ids"].tolist()) <= set(O.candidates(st["lag_block_ids"], 1024, 64).tolist())
            if rho == 1.0:
                assert len(T) == 0 and st["repeat"] == 1.0
                same = O.decode_batch(qs[t], K, V, d["ctx_lens"], d["channels"], cfg.k_b,
                                      cfg.k_t, cfg.block, cfg.sigma, units=[(0, 0)])[(0, 0)]
                assert np.array_equal(same["token_ids"], st["token_ids"])
                np.testing.assert_array_equal(same["out"], st["out"])
            prev = st
        assert prev is not None


def pin_lagged_schedule_growth(seed=18):
    """Offloaded schedule with the context growing by one token per step: a
    constant length reproduces the fixed-length schedule exactly; every step's
    tokens lie in the candidates of M_{t-1} at that step's length; a token
    appended with a key along the step's queries, inside a block of M_{t-1},
    is selected at once."""
    cfg = synth.config("toy").replace(ctx_lo=1024, ctx_hi=1024, k_b=4, k_t=64, steps=6)
    d = synth.make_host(cfg)
    K = synth.to_f64(d["k"], cfg.dtype)
    V = synth.to_f64(d["v"], cfg.dtype)
    qs = synth.to_f64(synth.draw_query_walk(cfg.replace(rho=0.8)), cfg.dtype)
    args = (d["channels"][0], cfg.k_b, cfg.k_t, cfg.block, cfg.sigma, cfg.d_v)
    fixed = O.lagged_decode(qs, K, V, 1000, *args)
    same = O.lagged_decode(qs, K, V, [1000] * qs.shape[0], *args)
    for a, b in zip(fixed, same):
        assert np.array_equal(a["token_ids"], b["token_ids"]) and np.array_equal(a["out"], b["out"])
    n_steps = [1000 + t for t in range(qs.shape[0])]
    steps = O.lagged_decode(qs, K, V, n_steps, *args)
    for t, st in enumerate(steps, start=1):
        cand = set(O.candidates(st["lag_block_ids"], n_steps[t], cfg.block).tolist())
        assert set(st["token_ids"].tolist()) <= cand
        assert max(st["token_ids"]) < n_steps[t]
    # plant: the token appended at step t (position n_t - 1) gets a key along
    # the group's (frozen) query; an earlier planted key in the same block
    # keeps that block in every M, so the new token is a candidate at once
    # and must be selected
    Kp = K.copy()
    qf = np.repeat(qs[:1], qs.shape[0], axis=0)
    u = qf[0, 0, 0:cfg.group].mean(axis=0)
    u /= np.linalg.norm(u)
    t_plant = 3
    pos = n_steps[t_plant] - 1
    Kp[0, 0, pos] = 4.0 * math.sqrt(cfg.d_qk) * u
    Kp[0, 0, (pos // cfg.block) * cfg.block + 5] = 4.0 * math.sqrt(cfg.d_qk) * u
    blocks0 = O.select_blocks(qf[0, 0, 0:cfg.group], *O.block_summaries(Kp[0, 0], n_steps[0], cfg.block), cfg.k_b)[0]
    assert pos // cfg.block in set(blocks0.tolist())
    st = O.lagged_decode(qf, Kp, V, n_steps, *args)[t_plant - 1]
    assert pos in set(st["token_ids"].tolist())
    before = O.lagged_decode(qf, Kp, V, n_steps, *args)[t_plant - 2]   # one step earlier it does not exist yet
    assert pos not in set(before["token_ids"].tolist())


# --- channel calibration (Sec. 4.1) -------------------------------------------

def pin_calibration_golden():
    """Hand-derived worked example, including a tie at the cut."""
    g = _golden("calibration_worked.json")
    q, k = np.asarray(g["q_cal"], float), np.asarray(g["k_cal"], float)
    for d_c, want in g["channels"].items():
        ch, sc, qa, ka = O.calibrate_channels(q, k, g["G"], int(d_c))
        np.testing.assert_array_equal(qa, g["q_absmax"])
        np.testing.assert_array_equal(ka, g["k_absmax"])
        np.testing.assert_array_equal(sc, g["scores"])
        np.testing.assert_array_equal(ch, want)


def pin_calibration_properties(seed=17):
    """Planted outlier channels are found; the result does not depend on the
    order or signs of the calibration rows and scales with the activations;
    every score bounds the per-channel logit magnitude of every calibration
    row; a channel no key uses is never chosen; an empty set gives zeros."""
    r = np.random.default_rng(seed)
    N, H_kv, G, d, d_c = 300, 2, 4, 64, 16
    q = r.standard_normal((N, H_kv * G, d))
    k = r.standard_normal((N, H_kv, d))
    planted = [np.sort(r.choice(d, size=8, replace=False)) for _ in range(H_kv)]
    for g in range(H_kv):
        q[:, g * G:(g + 1) * G, planted[g]] *= 10.0
        k[:, g, planted[g]] *= 10.0
    ch, sc, qa, ka = O.calibrate_channels(q, k, G, d_c)
    for g in range(H_kv):
        assert set(planted[g].tolist()) <= set(ch[g].tolist())
        assert np.all(np.diff(ch[g]) > 0) and len(ch[g]) == d_c
    # order and signs of the rows do not matter
    perm = r.permutation(N)
    flip_q = np.where(r.random(q.shape) < 0.5, -1.0, 1.0)
    flip_k = np.where(r.random(k.shape) < 0.5, -1.0, 1.0)
    ch2, sc2, _, _ = O.calibrate_channels((q * flip_q)[perm], (k * flip_k)[perm], G, d_c)
    np.testing.assert_array_equal(ch2, ch)
    np.testing.assert_array_equal(sc2, sc)
    # scaling q by 4 and k by 0.5 (exact in binary) scales the scores by 2
    ch3, sc3, _, _ = O.calibrate_channels(4.0 * q, 0.5 * k, G, d_c)
    np.testing.assert_array_equal(ch3, ch)
    np.testing.assert_array_equal(sc3, 2.0 * sc)
    # the score bounds every row's per-channel logit mass: G s_i >= sum_h |q_h[i] k[i]|
    for g in range(H_kv):
        mass = np.abs(q[:, g * G:(g + 1) * G, :] * k[:, g:g + 1, :]).sum(axis=1)  # [N][d]
        assert np.all(mass <= G * sc[g][None, :] * (1 + 1e-12))
    # equality when one row holds every maximum: append that row
    row_q = np.abs(q).max(axis=0, keepdims=True)
    row_k = np.abs(k).max(axis=0, keepdims=True)
    _, sc4, _, _ = O.calibrate_channels(np.concatenate([q, row_q]), np.concatenate([k, row_k]), G, d_c)
    for g in range(H_kv):
        mass = (row_q[0, g * G:(g + 1) * G, :] * row_k[0, g][None, :]).sum(axis=0)
        np.testing.assert_allclose(G * sc4[g], mass, rtol=1e-15)
    # heads with identical activations: the score is the plain product of the maxima
    q_same = np.repeat(q[:, ::G, :], G, axis=1)
    _, sc5, qa5, ka5 = O.calibrate_channels(q_same, k, G, d_c)
    for g in range(H_kv):
        np.testing.assert_allclose(sc5[g], np.abs(q[:, g * G, :]).max(axis=0) * np.abs(k[:, g, :]).max(axis=0),
                                   rtol=1e-15)
    # a channel that no key uses scores 0 and is never chosen
    k0 = k.copy()
    k0[:, :, 5] = 0.0
    ch6, sc6, _, _ = O.calibrate_channels(q, k0, G, d_c)
    assert np.all(sc6[:, 5] == 0.0) and not np.any(ch6 == 5)
    # empty calibration set: zero scores, ties to the lowest channels
    ch7, sc7, _, _ = O.calibrate_channels(q[:0], k[:0], G, d_c)
    assert np.all(sc7 == 0.0)
    np.testing.assert_array_equal(ch7, np.tile(np.arange(d_c), (H_kv, 1)))


ALL_PINS = [
    pin_quest_golden, pin_quest_forms_agree, pin_quest_upper_bound, pin_topk_bruteforce,
    pin_candidates, pin_quant_golden, pin_quant_bound, pin_alpha_golden, pin_alpha_distribution,
    pin_channel_projection_golden, pin_channel_projection_property, pin_token_index_projection,
    pin_block_summaries_tail, pin_attention_library, pin_attention_closed_form, pin_dense_equivalence,
    pin_invariants_and_planted, pin_single_level_operators, pin_lagged_schedule, pin_lagged_schedule_growth,
    pin_calibration_golden,
    pin_calibration_properties,
]
