"""Inputs whose selections have exact ties at the top-k cuts, and their
oracle references (shared by the CPU precondition checks and the GPU tests).

Sec. 4.1 selects the top-K_b blocks and the top-K_t tokens; ties go to the
lowest block id / token position.  Each case plants byte-identical blocks
(equal summaries, hence exactly equal block scores) or byte-identical token
rows (equal index rows, hence exactly equal approximate scores) so that the
cut falls inside a group of equal scores, and everything else is far from
the cut.  The GPU must then pick exactly the oracle's ids: no near-tie
allowance applies.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

import synth
from oracle import tls_oracle as O


@dataclass(frozen=True)
class TieCase:
    base: str
    over: dict
    n_hi: int    # blocks clearly above the block cut
    n_dup: int   # identical blocks straddling it (K_b - n_hi of them selected)
    n_a: int     # tokens clearly above the token cut
    n_b: int     # identical tokens straddling it (K_t - n_a of them selected)
    logit_a: float = 12.0  # approximate logits of the two planted kinds
    logit_b: float = 9.0   # (sigma * mean query . key)

    def cfg(self):
        return synth.config(self.base).replace(**self.over)


CASES = {
    # bf16 GQA, G = 4: the fused selection kernel (block top-k + token scoring + token top-k)
    "gqa_bf16_fused": TieCase("qwen3_gqa_48k", dict(batch=2, h_q=8, h_kv=2, ctx_lo=3000, ctx_hi=4096, k_b=8,
                                                    k_t=128, clusters=0, seed=7100), 5, 10, 100, 60),
    # the same kernel at the 96k budget: 1536 blocks (two block keys per thread),
    # 8192 candidates (eight slots per thread)
    "gqa_bf16_fused_96k": TieCase("qwen3_gqa_48k", dict(batch=1, h_q=8, h_kv=2, ctx_lo=98304, ctx_hi=98304,
                                                        k_b=128, k_t=2048, clusters=0, seed=7200),
                                  100, 60, 1500, 1200),
    # bf16 GQA, G = 8: block_topk_kernel + vector-unit token scoring + token_topk_kernel
    "gqa_bf16_g8": TieCase("qwen3_gqa_48k", dict(batch=1, h_q=16, h_kv=2, ctx_lo=4000, ctx_hi=4000, k_b=8,
                                                 k_t=128, clusters=0, seed=7300), 5, 10, 100, 60),
    # fp32 GQA
    "gqa_f32": TieCase("toy", dict(batch=2, ctx_lo=3000, ctx_hi=4096, clusters=0, seed=7400), 5, 10, 100, 60),
    # bf16 absorbed MLA (G = 32): matrix-core token scoring + token_topk_kernel
    "mla_bf16": TieCase("mla", dict(batch=2, ctx_lo=3000, ctx_hi=4096, k_b=8, k_t=200, clusters=0, seed=7500),
                        5, 10, 120, 150),
    # the fused kernel with the cut ~45 octaves below the largest alpha (dominant
    # logits 31 above the tied group): the cut falls in the token top-k's
    # bottom first-pass bucket, which holds every key more than 32 octaves
    # below the upper bound and is refined with the keys above it excluded
    "gqa_bf16_fused_deep": TieCase("qwen3_gqa_48k", dict(batch=2, h_q=8, h_kv=2, ctx_lo=3000, ctx_hi=4096, k_b=8,
                                                         k_t=128, clusters=0, seed=7150), 5, 10, 100, 60,
                                   logit_a=40.0),
    "mla_bf16_70k": TieCase("mla", dict(batch=1, ctx_lo=70000, ctx_hi=70000, k_b=128, k_t=2048, clusters=0,
                                        seed=7600), 100, 60, 1500, 1200),
}

SEP_REL = 1e-3  # everything but the tied group lies farther than this from the cut score


def base_inputs(tc: TieCase):
    cfg = tc.cfg()
    d = synth.make_host(cfg, pad="nan")
    return cfg, d


def block_tie_inputs(tc: TieCase):
    """Inputs with n_hi dominant blocks and n_dup identical blocks per unit."""
    cfg, d = base_inputs(tc)
    hi, dup = synth.plant_tie_blocks(cfg, d["k"], d["ctx_lens"], tc.n_hi, tc.n_dup)
    return cfg, d, hi, dup


def token_tie_inputs(tc: TieCase, whole_context: bool = False):
    """Inputs with a given block list per unit and, inside it, n_a dominant
    tokens and n_b identical tokens per unit (anywhere in the context when
    whole_context)."""
    cfg, d = base_inputs(tc)
    blocks = None if whole_context else synth.draw_block_lists(cfg, d["ctx_lens"], cfg.k_b)
    sig = cfg.sigma
    pa, pb = synth.plant_tie_tokens(cfg, d["q"], d["k"], d["ctx_lens"], d["channels"], blocks, tc.n_a, tc.n_b,
                                    tc.logit_a / sig, tc.logit_b / sig)
    return cfg, d, blocks, pa, pb


def unit_arrays(cfg, d, s, g):
    q = synth.to_f64(d["q"], cfg.dtype)
    qg = q[s, g * cfg.group:(g + 1) * cfg.group]
    Ku = synth.to_f64(d["k"][s, g], cfg.dtype)
    Vu = Ku[:, :cfg.d_v] if cfg.mla else synth.to_f64(d["v"][s, g], cfg.dtype)
    return qg, Ku, Vu


def check_cut(scores_of_ids: dict, k: int, tied: set, what: str):
    """Precondition on the oracle's scores: the k-th largest score is shared
    exactly by the ids of `tied` (and by no other id), the cut takes some but
    not all of them, and every other score differs from it by more than
    SEP_REL relative."""
    ids = np.array(sorted(scores_of_ids))
    sc = np.array([scores_of_ids[i] for i in ids])
    order = np.lexsort((ids, -sc))
    kth = sc[order[k - 1]]
    eq = set(int(i) for i in ids[sc == kth])
    assert eq == set(int(x) for x in tied), f"{what}: the cut's tie group is not the planted group"
    taken = sum(1 for j in order[:k] if int(ids[j]) in eq)
    assert 0 < taken < len(eq), f"{what}: the cut does not split the tie group ({taken} of {len(eq)})"
    others = sc[sc != kth]
    assert np.all(np.abs(others - kth) > SEP_REL * abs(kth)), f"{what}: a near tie outside the planted group"
    return taken


def oracle_block_ties(tc: TieCase, cfg, d, hi, dup):
    """Oracle decode of every unit; asserts the block-cut precondition."""
    refs = {}
    for s in range(cfg.batch):
        n = int(d["ctx_lens"][s])
        for g in range(cfg.h_kv):
            qg, Ku, Vu = unit_arrays(cfg, d, s, g)
            r = O.decode_unit(qg, Ku, Vu, n, d["channels"][g], cfg.k_b, cfg.k_t, cfg.block, cfg.sigma)
            sc = r["block_scores"]
            check_cut({i: float(sc[i]) for i in range(len(sc))}, cfg.k_b, set(dup[s, g].tolist()),
                      f"blocks {(s, g)}")
            assert set(hi[s, g].tolist()) <= set(r["block_ids"].tolist())
            refs[(s, g)] = r
    return refs


def oracle_token_ties(tc: TieCase, cfg, d, blocks, pa, pb):
    """Oracle decode of every unit on the given block lists; asserts the
    token-cut precondition."""
    refs = {}
    for s in range(cfg.batch):
        n = int(d["ctx_lens"][s])
        for g in range(cfg.h_kv):
            qg, Ku, Vu = unit_arrays(cfg, d, s, g)
            if blocks is None:
                r = O.token_sparse_unit(qg, Ku, Vu, n, d["channels"][g], cfg.k_t, cfg.block, cfg.sigma)
            else:
                r = O.decode_unit(qg, Ku, Vu, n, d["channels"][g], cfg.k_b, cfg.k_t, cfg.block, cfg.sigma,
                                  block_ids=blocks[s, g])
            alpha = {int(t): float(a) for t, a in zip(r["cand"], r["alpha"])}
            check_cut(alpha, cfg.k_t, set(pb[s, g].tolist()), f"tokens {(s, g)}")
            assert set(pa[s, g].tolist()) <= set(r["token_ids"].tolist())
            refs[(s, g)] = r
    return refs


def zero_query(cfg, d):
    """The same inputs with every query entry zero: every block score and
    every approximate logit is 0, so both cuts tie over all candidates."""
    q = np.zeros_like(d["q"])
    return dict(d, q=q)


def oracle_all(cfg, d, **kw):
    refs = {}
    for s in range(cfg.batch):
        n = int(d["ctx_lens"][s])
        for g in range(cfg.h_kv):
            qg, Ku, Vu = unit_arrays(cfg, d, s, g)
            refs[(s, g)] = O.decode_unit(qg, Ku, Vu, n, d["channels"][g], cfg.k_b, cfg.k_t, cfg.block, cfg.sigma,
                                         **kw)
    return refs


def expected_zero_query(cfg, d, s):
    """With q = 0: blocks 0..K_b'-1 and the lowest K_t' candidate positions."""
    n = int(d["ctx_lens"][s])
    m = -(-n // cfg.block)
    # blocks 0..K_b'-1 hold the tokens 0..min(K_b*B, n)-1, all candidates
    return np.arange(min(cfg.k_b, m)), np.arange(min(cfg.k_t, cfg.k_b * cfg.block, n))
