"""The lagged two-level operator (Sec. 4.2, one-step lag of the offloaded
tier) against the oracle, through the C ABI.

One call with TLS_MODE_LAGGED selects this step's blocks M_t from the query
(block_ids_out) while token selection and attention run over the previous
step's blocks M_{t-1} (block_ids_in).  Checked per unit: M_t against the
oracle's block selection, the tokens against the oracle's token stage over
M_{t-1}, the output against the oracle's attention over the GPU's tokens;
and the whole call against the two calls it stands for (tls_select_blocks,
then the two-level operator with the given blocks), which must agree bit
for bit.  Routes: the fused bf16 selection kernel, the fp32 stages and the
MLA stages; the full 96k workload on sampled units.
"""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import synth
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

CASES = {
    "toy_f32": lambda: (synth.config("toy"), "host", None, None),
    "ragged_bf16": lambda: (synth.config("qwen3_gqa_48k").replace(batch=6, ctx_lo=1, ctx_hi=1000, clusters=1,
                                                                   k_b=6, k_t=96, seed=71),
                            "host", np.array([1, 63, 64, 65, 700, 1000], dtype=np.int32), None),
    "mla_small": lambda: (synth.config("mla").replace(batch=2, ctx_lo=2000, ctx_hi=3000, clusters=2, k_b=8,
                                                      k_t=200, seed=4100), "host", None, None),
    "offload_gqa_96k": lambda: (synth.config("offload_gqa_96k"), "device", None, 32),
}


def previous_blocks(cfg, ctx, k_b, seed):
    """A seeded stand-in for the previous step's selection: min(k_b, m)
    distinct blocks per unit, ascending, -1 padded."""
    r = np.random.default_rng(seed)
    out = np.full((cfg.batch, cfg.h_kv, k_b), -1, dtype=np.int32)
    for s in range(cfg.batch):
        m = -(-int(ctx[s]) // cfg.block)
        for g in range(cfg.h_kv):
            k = min(k_b, m)
            out[s, g, :k] = np.sort(r.choice(m, size=k, replace=False))
    return out


def lagged_call(c, M_prev, ws):
    cfg = c.cfg
    dt = H.torch_dtype(cfg)
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dt, device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    M_t = torch.full((cfg.batch, cfg.h_kv, cfg.k_b), -7, dtype=torch.int32, device="cuda")
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch, cfg.k_b,
                          cfg.k_t, M_prev, None, out, lse, M_t, tids, ws, mode=tls.MODE_LAGGED)
    torch.cuda.synchronize()
    return dict(out=out, lse=lse, M_t=M_t, tids=tids)


_cache = {}


def get_case(name):
    if name not in _cache:
        _cache.clear()
        torch.cuda.empty_cache()
        cfg, backend, ctx, sample = CASES[name]()
        c = H.Case(cfg, backend=backend, pad="nan", ctx_lens=ctx).build_index()
        c.sample = c.units(sample)
        c.M_prev_host = previous_blocks(cfg, c.ctx_host, cfg.k_b, cfg.seed + 900)
        c.M_prev = torch.from_numpy(c.M_prev_host).cuda()
        c.ws = c.workspace()
        c.res = lagged_call(c, c.M_prev, c.ws)
        _cache[name] = c
    return _cache[name]


def teardown_module(module):
    _cache.clear()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", list(CASES))
def test_lagged_matches_oracle(name):
    c = get_case(name)
    cfg, G = c.cfg, c.cfg.group
    res = c.res
    assert tls.tls_check_device_error(c.ws) == 0
    for (s, g) in c.sample:
        n = int(c.ctx_host[s])
        # this step's blocks, from this step's query
        ref = c.oracle_unit(s, g)
        H.check_selection(res["M_t"][s, g].cpu().numpy(), ref["block_ids"],
                          lambda i: float(ref["block_scores"][i]), f"M_t unit {(s, g)}")
        # tokens and output over the previous step's blocks
        M_prev = c.M_prev_host[s, g]
        M_prev = M_prev[M_prev >= 0]
        tok = c.oracle_unit(s, g, block_ids=M_prev)
        H.check_selection(res["tids"][s, g].cpu().numpy(), tok["token_ids"], H.alpha_lookup(tok),
                          f"tokens unit {(s, g)}")
        S = H.valid_ids(res["tids"][s, g].cpu().numpy())
        cand = set(O.candidates(M_prev, n, cfg.block).tolist())
        assert set(S.tolist()) <= cand, f"unit {(s, g)}: a token outside the given blocks"
        qg = c.q_f64()[s, g * G:(g + 1) * G]
        Ku, Vu = c.unit_kv_f64(s, g)
        o_ref, lse_ref = O.sparse_attention(qg, Ku, Vu, S, cfg.sigma)
        H.check_close(res["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), o_ref, cfg.dtype, f"out {(s, g)}")
        H.check_close(res["lse"][s, g * G:(g + 1) * G].cpu().numpy(), lse_ref, cfg.dtype, f"lse {(s, g)}")


@pytest.mark.parametrize("name", list(CASES))
def test_lagged_equals_the_two_calls(name):
    """One lagged call gives, bit for bit, what tls_select_blocks followed by
    the two-level operator over the given blocks gives."""
    c = get_case(name)
    cfg = c.cfg
    M_t = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(c.layout, c.q, c.kmax, c.kmin, c.ctx, cfg.k_b, M_t, None, c.ws)
    two = c.decode(block_ids_in=c.M_prev, ws=c.ws)
    assert torch.equal(c.res["M_t"], M_t)
    assert torch.equal(c.res["tids"], two["tids"])
    assert torch.equal(c.res["out"], two["out"])
    assert torch.equal(c.res["lse"], two["lse"])


@pytest.mark.parametrize("name", ["toy_f32", "ragged_bf16", "mla_small"])
def test_lagged_over_a_pool(name):
    """The lagged call reading K/V through a block pool holding M_{t-1}
    (filled by tls_init_residency from the cache) gives, bit for bit, what
    it gives over the cache itself."""
    c = get_case(name)
    cfg = c.cfg
    units, B, n_slots = cfg.batch * cfg.h_kv, cfg.block, 2 * cfg.k_b
    dt = H.torch_dtype(cfg)
    pool_k = torch.full((units, n_slots, B, cfg.d_qk), float("nan"), dtype=dt, device="cuda")
    pool_v = None if cfg.mla else torch.full((units, n_slots, B, cfg.d_v), float("nan"), dtype=dt, device="cuda")
    slot_map = torch.empty((units, c.m_max), dtype=torch.int32, device="cuda")
    slot_owner = torch.empty((units, n_slots), dtype=torch.int32, device="cuda")
    tls.tls_init_residency(c.layout, c.k, c.v, c.ctx, c.M_prev, cfg.k_b, pool_k, pool_v, n_slots, slot_map,
                           slot_owner, c.ws)
    pooled = tls.KV(pool_k, pool_v, slot_map, n_slots)
    dtp = H.torch_dtype(cfg)
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dtp, device="cuda")
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
    M_t = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    tls.tls_sparse_decode(c.layout, c.q, pooled, c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch, cfg.k_b,
                          cfg.k_t, c.M_prev, None, out, lse, M_t, tids, c.ws, mode=tls.MODE_LAGGED)
    torch.cuda.synchronize()
    assert tls.tls_check_device_error(c.ws) == 0
    assert torch.equal(M_t, c.res["M_t"]) and torch.equal(tids, c.res["tids"])
    assert torch.equal(out, c.res["out"]) and torch.equal(lse, c.res["lse"])


def test_lagged_argument_rules():
    """The lagged operator needs both block lists, distinct, and no given tokens."""
    c = get_case("ragged_bf16")
    cfg = c.cfg
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=torch.bfloat16, device="cuda")
    M_t = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tids = torch.zeros((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")

    def call(bin_, bout, tin=None):
        tls.tls_sparse_decode(c.layout, c.q, c.kv(), c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch, cfg.k_b,
                              cfg.k_t, bin_, tin, out, None, bout, None, c.ws, mode=tls.MODE_LAGGED)

    for args in [(None, M_t), (c.M_prev, None), (c.M_prev, c.M_prev), (c.M_prev, M_t, tids)]:
        with pytest.raises(tls.TlsError) as e:
            call(*args)
        assert e.value.status == 1
