"""The single-level operators of the library (block-sparse attention over
the top-K_b blocks, and dense attention over the whole context) against the
oracle through the C ABI: small cases on every unit, the full-size batched
and MLA workloads on sampled units."""
import numpy as np
import pytest
import torch

import synth
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

CASES = {
    "toy_f32": lambda: (synth.config("toy"), "host", None, None),
    "ragged_bf16": lambda: (synth.config("qwen3_gqa_48k").replace(batch=6, ctx_lo=0, ctx_hi=1000, clusters=1, k_b=6,
                                                                   k_t=96, seed=71),
                            "host", np.array([0, 1, 63, 65, 700, 1000], dtype=np.int32), None),
    "g8_f32": lambda: (synth.config("toy").replace(h_q=16, h_kv=2, ctx_lo=1500, ctx_hi=2100, batch=2, k_b=5,
                                                   k_t=200, seed=81), "host", None, None),
    "mla_small": lambda: (synth.config("mla").replace(batch=2, ctx_lo=2000, ctx_hi=3000, clusters=2, k_b=8,
                                                      k_t=200, seed=4100), "host", None, None),
    "batched_gqa": lambda: (synth.config("batched_gqa"), "device", None, 4),
    "mla": lambda: (synth.config("mla"), "device", None, 2),
}

_cache = {}


def get_case(name):
    if name in _cache:
        return _cache[name]
    _cache.clear()
    torch.cuda.empty_cache()
    cfg, backend, ctx, sample = CASES[name]()
    c = H.Case(cfg, backend=backend, pad="nan", ctx_lens=ctx).build_index()
    c.sample = c.units(sample)
    torch.cuda.synchronize()
    _cache[name] = c
    return c


def teardown_module(module):
    _cache.clear()
    torch.cuda.empty_cache()


def run_mode(c, mode, block_ids_in=None):
    import paper_2604_07815_amd as tls
    cfg = c.cfg
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    bids = tids = None
    if mode == tls.MODE_BLOCK_SPARSE and block_ids_in is None:
        bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    if mode == tls.MODE_TOKEN_SPARSE:
        tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    ws = c.workspace()
    tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch, cfg.k_b, cfg.k_t,
                          block_ids_in, None, out, lse, bids, tids, ws, mode=mode)
    torch.cuda.synchronize()
    assert tls.tls_check_device_error(ws) == 0
    return out, lse, bids if tids is None else tids


def _unit(c, s, g):
    cfg = c.cfg
    G = cfg.group
    qg = c.q_f64()[s, g * G:(g + 1) * G]
    Ku, Vu = c.unit_kv_f64(s, g)
    return qg, Ku, Vu, int(c.ctx_host[s])


@pytest.mark.parametrize("name", list(CASES))
def test_dense_mode(name):
    """Full attention over every valid token equals the oracle's."""
    import paper_2604_07815_amd as tls
    c = get_case(name)
    cfg = c.cfg
    G = cfg.group
    out, lse, _ = run_mode(c, tls.MODE_DENSE)
    for (s, g) in c.sample:
        qg, Ku, Vu, n = _unit(c, s, g)
        ref = O.dense_unit(qg, Ku, Vu, n, cfg.sigma)
        H.check_close(out[s, g * G:(g + 1) * G].float().cpu().numpy(), ref["out"], cfg.dtype, f"dense out {(s, g)}")
        H.check_close(lse[s, g * G:(g + 1) * G].cpu().numpy(), ref["lse"], cfg.dtype, f"dense lse {(s, g)}")


@pytest.mark.parametrize("name", list(CASES))
def test_block_sparse_mode(name):
    """Block-level selection alone: the top-K_b blocks (near-tie rule), then
    attention over every valid token of the GPU's blocks equals the
    oracle's; the same blocks given as input reproduce the output."""
    import paper_2604_07815_amd as tls
    c = get_case(name)
    cfg = c.cfg
    G = cfg.group
    out, lse, bids = run_mode(c, tls.MODE_BLOCK_SPARSE)
    for (s, g) in c.sample:
        qg, Ku, Vu, n = _unit(c, s, g)
        ref = O.block_sparse_unit(qg, Ku, Vu, n, cfg.k_b, cfg.block, cfg.sigma)
        H.check_selection(bids[s, g].cpu().numpy(), ref["block_ids"], lambda i: float(ref["block_scores"][i]),
                          f"blocks {(s, g)}")
        mine = H.valid_ids(bids[s, g].cpu().numpy())
        ref2 = O.block_sparse_unit(qg, Ku, Vu, n, cfg.k_b, cfg.block, cfg.sigma, block_ids=mine)
        H.check_close(out[s, g * G:(g + 1) * G].float().cpu().numpy(), ref2["out"], cfg.dtype, f"out {(s, g)}")
        H.check_close(lse[s, g * G:(g + 1) * G].cpu().numpy(), ref2["lse"], cfg.dtype, f"lse {(s, g)}")
    out2, lse2, _ = run_mode(c, tls.MODE_BLOCK_SPARSE, block_ids_in=bids)
    assert torch.equal(out2, out) and torch.equal(lse2.nan_to_num(0.0), lse.nan_to_num(0.0))


@pytest.mark.parametrize("name", list(CASES))
def test_token_sparse_mode(name):
    """Token-level selection alone: the top-K_t of the approximate score over
    every valid token (near-tie rule), then attention over the GPU's tokens
    equals the oracle's."""
    import paper_2604_07815_amd as tls
    c = get_case(name)
    cfg = c.cfg
    G = cfg.group
    out, lse, tids = run_mode(c, tls.MODE_TOKEN_SPARSE)
    for (s, g) in c.sample:
        qg, Ku, Vu, n = _unit(c, s, g)
        ref = O.token_sparse_unit(qg, Ku, Vu, n, c.ch_host[g], cfg.k_t, cfg.block, cfg.sigma)
        H.check_selection(tids[s, g].cpu().numpy(), ref["token_ids"], H.alpha_lookup(ref), f"tokens {(s, g)}")
        mine = H.valid_ids(tids[s, g].cpu().numpy())
        o, l = O.sparse_attention(qg, Ku, Vu, mine, cfg.sigma)
        H.check_close(out[s, g * G:(g + 1) * G].float().cpu().numpy(), o, cfg.dtype, f"out {(s, g)}")
        H.check_close(lse[s, g * G:(g + 1) * G].cpu().numpy(), l, cfg.dtype, f"lse {(s, g)}")
        planted = [int(p) + i for p in c.plant_starts[s, g] if p >= 0 for i in range(cfg.cluster_len)]
        assert set(planted) <= set(mine.tolist()), f"planted tokens missed in unit {(s, g)}"
