"""Exact ties at the selection cuts, through the C ABI (Sec. 4.1 top-K_b and
top-K_t, ties to the lowest block id / token position).

The inputs of tie_cases.py put the K_b-th largest block score, or the K_t-th
largest approximate score, inside a group of byte-identical blocks or token
rows, and keep every other score far from the cut (checked on the oracle
before the GPU runs).  The GPU must then return exactly the oracle's ids:
the near-tie allowance of the other parity tests does not apply here.  A
zero query makes every score equal, so both cuts take the lowest ids.

Covered kernels: the fused bf16 selection (block top-k, token scoring and
token top-k in one work-group per unit, at small and 96k budgets),
block_topk_kernel, the vector-unit and matrix-core token scoring with
token_topk_kernel (fp32 GQA, bf16 G = 8, absorbed MLA), and the streaming
whole-context top-k of the token-level operator.
"""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import tie_cases as TC
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

NAMES = list(TC.CASES)
SMALL = [n for n in NAMES if not n.endswith(("_96k", "_70k"))]


def _case(cfg, d):
    return H.Case(cfg, backend="host", host=d).build_index()


def _ids(t, s, g):
    return H.valid_ids(t[s, g].cpu().numpy())


def _check_out(c, r, s, g, S, what):
    cfg = c.cfg
    qg = c.q_f64()[s, g * cfg.group:(g + 1) * cfg.group]
    Ku, Vu = c.unit_kv_f64(s, g)
    o, lse = O.sparse_attention(qg, Ku, Vu, S, cfg.sigma)
    G = cfg.group
    H.check_close(r["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), o, cfg.dtype, what + " out")
    H.check_close(r["lse"][s, g * G:(g + 1) * G].cpu().numpy(), lse, cfg.dtype, what + " lse")


@pytest.mark.parametrize("name", NAMES)
def test_block_cut_ties(name):
    tc = TC.CASES[name]
    cfg, d, hi, dup = TC.block_tie_inputs(tc)
    refs = TC.oracle_block_ties(tc, cfg, d, hi, dup)
    c = _case(cfg, d)
    ws = c.workspace()
    bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(c.layout, c.q, c.kmax, c.kmin, c.ctx, cfg.k_b, bids, None, ws)
    torch.cuda.synchronize()
    r = c.decode()
    for (s, g), ref in refs.items():
        what = f"{name} unit {(s, g)}"
        assert np.array_equal(_ids(bids, s, g), ref["block_ids"]), what + " tls_select_blocks"
        assert np.array_equal(_ids(r["bids"], s, g), ref["block_ids"]), what + " tls_sparse_decode blocks"
        H.check_selection(r["tids"][s, g].cpu().numpy(), ref["token_ids"], H.alpha_lookup(ref), what + " tokens")
        _check_out(c, r, s, g, _ids(r["tids"], s, g), what)
    assert tls.tls_check_device_error(ws) == 0 and tls.tls_check_device_error(r["ws"]) == 0


@pytest.mark.parametrize("name", SMALL)
def test_block_cut_ties_block_sparse(name):
    """The single-level block operator selects the same blocks."""
    tc = TC.CASES[name]
    cfg, d, hi, dup = TC.block_tie_inputs(tc)
    refs = TC.oracle_block_ties(tc, cfg, d, hi, dup)
    c = _case(cfg, d)
    ws = c.workspace()
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, c.kmax, c.kmin, None, None, None, cfg.k_b, cfg.k_t, None,
                          None, out, lse, bids, None, ws, mode=tls.MODE_BLOCK_SPARSE)
    torch.cuda.synchronize()
    r = dict(out=out, lse=lse)
    for (s, g), ref in refs.items():
        what = f"{name} block-sparse unit {(s, g)}"
        assert np.array_equal(_ids(bids, s, g), ref["block_ids"]), what
        _check_out(c, r, s, g, O.candidates(ref["block_ids"], int(c.ctx_host[s]), cfg.block), what)
    assert tls.tls_check_device_error(ws) == 0


@pytest.mark.parametrize("name", NAMES)
def test_token_cut_ties(name):
    tc = TC.CASES[name]
    cfg, d, blocks, pa, pb = TC.token_tie_inputs(tc)
    refs = TC.oracle_token_ties(tc, cfg, d, blocks, pa, pb)
    c = _case(cfg, d)
    M = torch.from_numpy(blocks).cuda()
    ws = c.workspace()
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    tls.tls_select_tokens(c.layout, c.q, c.codes, c.qparams, c.ch, M, cfg.k_b, c.ctx, cfg.k_t, tids, None, ws)
    torch.cuda.synchronize()
    r = c.decode(block_ids_in=M)
    for (s, g), ref in refs.items():
        what = f"{name} unit {(s, g)}"
        assert np.array_equal(_ids(tids, s, g), ref["token_ids"]), what + " tls_select_tokens"
        assert np.array_equal(_ids(r["tids"], s, g), ref["token_ids"]), what + " tls_sparse_decode tokens"
        _check_out(c, r, s, g, ref["token_ids"], what)
    assert tls.tls_check_device_error(ws) == 0 and tls.tls_check_device_error(r["ws"]) == 0


@pytest.mark.parametrize("name", ["gqa_bf16_fused", "gqa_f32", "mla_bf16"])
def test_token_cut_ties_token_sparse(name):
    """The token-level operator (every token a candidate) breaks the same
    ties with its streaming whole-context top-k."""
    tc = TC.CASES[name]
    cfg, d, _, pa, pb = TC.token_tie_inputs(tc, whole_context=True)
    refs = TC.oracle_token_ties(tc, cfg, d, None, pa, pb)
    c = _case(cfg, d)
    ws = c.workspace()
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, None, None, c.codes, c.qparams, c.ch, cfg.k_b, cfg.k_t,
                          None, None, out, lse, None, tids, ws, mode=tls.MODE_TOKEN_SPARSE)
    torch.cuda.synchronize()
    r = dict(out=out, lse=lse)
    for (s, g), ref in refs.items():
        what = f"{name} token-sparse unit {(s, g)}"
        assert np.array_equal(_ids(tids, s, g), ref["token_ids"]), what
        _check_out(c, r, s, g, ref["token_ids"], what)
    assert tls.tls_check_device_error(ws) == 0


@pytest.mark.parametrize("name", NAMES)
def test_zero_query_takes_lowest_ids(name):
    """q = 0: every block score and approximate score is equal, so the
    blocks are 0..K_b'-1 and the tokens the lowest K_t' positions; the output
    is the mean of their values."""
    tc = TC.CASES[name]
    cfg, d = TC.base_inputs(tc)
    dz = TC.zero_query(cfg, d)
    c = _case(cfg, dz)
    r = c.decode()
    for s in range(cfg.batch):
        blocks, toks = TC.expected_zero_query(cfg, dz, s)
        for g in range(cfg.h_kv):
            what = f"{name} zero query unit {(s, g)}"
            assert np.array_equal(_ids(r["bids"], s, g), blocks), what + " blocks"
            assert np.array_equal(_ids(r["tids"], s, g), toks), what + " tokens"
            _check_out(c, r, s, g, toks, what)
    assert tls.tls_check_device_error(r["ws"]) == 0
