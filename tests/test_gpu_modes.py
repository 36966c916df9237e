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


DEGENERATE = {
    # fused selection (bf16, G = 4); lengths not multiples of the block size
    "gqa_bf16": lambda: synth.config("qwen3_gqa_48k").replace(batch=3, ctx_lo=2500, ctx_hi=4096, clusters=2,
                                                              k_b=8, k_t=512, seed=171),
    # separate scoring / normalisation / top-k kernels
    "toy_f32": lambda: synth.config("toy").replace(batch=2, ctx_lo=2500, ctx_hi=4096, k_b=8, k_t=512, seed=172),
    "mla_bf16": lambda: synth.config("mla").replace(batch=2, ctx_lo=2500, ctx_hi=4096, clusters=2, k_b=8, k_t=512,
                                                    seed=173),
}


def _two_level(c, k_b, k_t):
    import paper_2604_07815_amd as tls
    cfg = c.cfg
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    bids = torch.empty((cfg.batch, cfg.h_kv, k_b), dtype=torch.int32, device="cuda")
    tids = torch.empty((cfg.batch, cfg.h_kv, k_t), dtype=torch.int32, device="cuda")
    ws = c.workspace(k_b, k_t)
    tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch, k_b, k_t, None,
                          None, out, lse, bids, tids, ws)
    torch.cuda.synchronize()
    assert tls.tls_check_device_error(ws) == 0
    return out, lse, bids, tids


def _close(a, b, cfg, what):
    tol = dict(rtol=1e-5, atol=1e-5) if cfg.dtype == "f32" else dict(rtol=8e-3, atol=8e-3)
    np.testing.assert_allclose(a.float().cpu().numpy(), b.float().cpu().numpy(), err_msg=what, **tol)


@pytest.mark.parametrize("name", list(DEGENERATE))
def test_two_level_reduces_to_single_level(name):
    """The method's two degenerate settings, through the C ABI: with K_t =
    K_b * B every candidate is kept and the two-level operator is block-sparse
    attention over the same K_b blocks; with K_b = every block the candidates
    are every valid token and it is token-level selection over the whole
    context (selections equal up to the near-tie rule, then the same
    attention)."""
    import paper_2604_07815_amd as tls
    cfg = DEGENERATE[name]()
    c = H.Case(cfg, backend="host", pad="nan").build_index()
    G = cfg.group
    # (1) K_t = K_b * B
    out, lse, bids, tids = _two_level(c, cfg.k_b, cfg.k_b * cfg.block)
    bs_out, bs_lse, bs_bids = run_mode(c, tls.MODE_BLOCK_SPARSE)
    assert torch.equal(bids, bs_bids)
    for s in range(cfg.batch):
        n = int(c.ctx_host[s])
        for g in range(cfg.h_kv):
            blocks = sorted(b for b in bids[s, g].cpu().tolist() if b >= 0)
            want = [b * cfg.block + o for b in blocks for o in range(cfg.block) if b * cfg.block + o < n]
            got = tids[s, g].cpu().tolist()
            assert got[:len(want)] == want and all(t == -1 for t in got[len(want):]), f"unit {(s, g)}"
    _close(out, bs_out, cfg, "K_t = K_b*B: output against block-sparse attention")
    _close(lse, bs_lse, cfg, "K_t = K_b*B: lse against block-sparse attention")
    # (2) K_b = every block
    m_all = c.m_max
    out2, lse2, _, tids2 = _two_level(c, m_all, cfg.k_t)
    ts_out, ts_lse, ts_tids = run_mode(c, tls.MODE_TOKEN_SPARSE)
    for s in range(cfg.batch):
        n = int(c.ctx_host[s])
        for g in range(cfg.h_kv):
            qg, Ku, Vu, _ = _unit(c, s, g)
            ref = O.token_sparse_unit(qg, Ku, Vu, n, c.ch_host[g], cfg.k_t, cfg.block, cfg.sigma)
            H.check_selection(tids2[s, g].cpu().numpy(), ref["token_ids"], H.alpha_lookup(ref),
                              f"two-level, all blocks {(s, g)}")
            a, b = H.valid_ids(tids2[s, g].cpu().numpy()), H.valid_ids(ts_tids[s, g].cpu().numpy())
            if np.array_equal(a, b):
                _close(out2[s, g * G:(g + 1) * G], ts_out[s, g * G:(g + 1) * G], cfg, f"K_b = all: out {(s, g)}")
                _close(lse2[s, g * G:(g + 1) * G], ts_lse[s, g * G:(g + 1) * G], cfg, f"K_b = all: lse {(s, g)}")
            else:  # a near-tie swap on either side: both are valid selections
                H.check_selection(ts_tids[s, g].cpu().numpy(), ref["token_ids"], H.alpha_lookup(ref),
                                  f"token-sparse {(s, g)}")
