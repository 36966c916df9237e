"""The tie layouts of tie_cases.py meet their preconditions on the oracle:
the planted group, and only it, straddles each cut with exactly equal
scores (CPU only; the GPU comparison is tests/test_gpu_ties.py)."""
import numpy as np
import pytest

import tie_cases as TC

SMALL = [n for n in TC.CASES if not n.endswith(("_96k", "_70k"))]


@pytest.mark.parametrize("name", SMALL)
def test_block_tie_layout(name):
    tc = TC.CASES[name]
    cfg, d, hi, dup = TC.block_tie_inputs(tc)
    refs = TC.oracle_block_ties(tc, cfg, d, hi, dup)
    for (s, g), r in refs.items():
        # the selected tied blocks are the lowest-numbered of the group
        taken = [b for b in dup[s, g] if b in set(r["block_ids"].tolist())]
        assert taken == sorted(dup[s, g])[:len(taken)]


@pytest.mark.parametrize("name", SMALL)
def test_token_tie_layout(name):
    tc = TC.CASES[name]
    cfg, d, blocks, pa, pb = TC.token_tie_inputs(tc)
    refs = TC.oracle_token_ties(tc, cfg, d, blocks, pa, pb)
    for (s, g), r in refs.items():
        taken = [t for t in pb[s, g] if t in set(r["token_ids"].tolist())]
        assert taken == sorted(pb[s, g])[:len(taken)] and len(taken) == cfg.k_t - tc.n_a


def test_token_tie_layout_whole_context():
    tc = TC.CASES["gqa_bf16_fused"]
    cfg, d, blocks, pa, pb = TC.token_tie_inputs(tc, whole_context=True)
    TC.oracle_token_ties(tc, cfg, d, None, pa, pb)


@pytest.mark.parametrize("name", ["gqa_f32", "mla_bf16"])
def test_zero_query_closed_form(name):
    """With q = 0 the oracle selects the lowest blocks and positions, and the
    output is the mean of the selected values (uniform weights)."""
    tc = TC.CASES[name]
    cfg, d = TC.base_inputs(tc)
    dz = TC.zero_query(cfg, d)
    for (s, g), r in TC.oracle_all(cfg, dz).items():
        blocks, toks = TC.expected_zero_query(cfg, dz, s)
        assert np.array_equal(r["block_ids"], blocks) and np.array_equal(r["token_ids"], toks)
        _, _, Vu = TC.unit_arrays(cfg, dz, s, g)
        np.testing.assert_allclose(r["out"], np.tile(Vu[toks].mean(axis=0), (cfg.group, 1)), rtol=1e-12,
                                   atol=1e-12)


def test_deep_cut_layout():
    """gqa_bf16_fused_deep puts the K_t-th largest alpha more than 32 octaves
    below the largest (so below the reach of the token top-k's spread first
    pass, whose buckets cover the 32 octaves under the upper bound), and the
    default cases put it within them."""
    for name, deep in (("gqa_bf16_fused_deep", True), ("gqa_bf16_fused", False)):
        tc = TC.CASES[name]
        cfg, d, blocks, pa, pb = TC.token_tie_inputs(tc)
        for (s, g), r in TC.oracle_token_ties(tc, cfg, d, blocks, pa, pb).items():
            a = np.sort(np.asarray(r["alpha"], dtype=np.float64))[::-1]
            octaves = np.log2(a[0] / a[cfg.k_t - 1])
            assert (octaves > 33.0) if deep else (octaves < 31.0), (name, (s, g), octaves)
