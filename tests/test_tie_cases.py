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
