"""Prefill side of the hierarchical KV cache (Sec. 4.2, Fig. 2): the prefill
write-back fused with both index builds, the offload of the cache to pinned
host memory, and the initial residency chosen by the last prompt token's
query.

The fused call must leave the cache holding the prefill rows (rows past a
sequence's length untouched) and the indices equal to the oracle's block
summaries and INT4 token index of those rows, bit for bit, whether the prompt
arrives in one call or in chunks whose boundaries fall inside blocks.  The
residency must hold exactly the selected blocks, byte-identical to the cache,
and a decode step over the pool must equal one over the dense cache and the
oracle."""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import synth
from gpu_harness import Case, alpha_lookup, check_close, check_selection, torch_dtype, valid_ids
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

CASES = {
    "gqa_bf16": synth.config("qwen3_gqa_48k").replace(batch=3, ctx_lo=700, ctx_hi=1500, clusters=1, k_b=8,
                                                      k_t=128, seed=141),
    "gqa_f32": synth.config("toy").replace(batch=2, ctx_lo=500, ctx_hi=1000, clusters=1, k_b=6, k_t=100,
                                           seed=142),
    "mla_bf16": synth.config("mla").replace(batch=2, ctx_lo=600, ctx_hi=1100, clusters=1, k_b=6, k_t=100,
                                            seed=143),
    # V rows of 72 bytes (not a multiple of 16): the element-wise V copy
    "odd_dv_bf16": synth.config("toy").replace(dtype="bf16", batch=2, h_q=4, h_kv=2, d_v=36, ctx_lo=200, ctx_hi=333,
                                               clusters=1, k_b=2, k_t=32, seed=145),
    # 4 KB key rows: a block is staged in LDS in several passes of fewer rows
    "wide_f32": synth.config("toy").replace(batch=1, h_q=4, h_kv=2, d_qk=1024, d_v=64, d_c=64, ctx_lo=300,
                                            ctx_hi=300, clusters=1, k_b=2, k_t=32, seed=144),
}
SENTINEL = 7.0

_cases = {}


def get_case(name):
    if name not in _cases:
        _cases[name] = Case(CASES[name], backend="host", pad="nan")
    return _cases[name]


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _src(t, t0, t1):
    """Prefill output rows [t0, t1) in the token-major [b][S][H_kv][d] layout."""
    return t[:, :, t0:t1].transpose(1, 2).contiguous()


def _prefill(c, bounds):
    """Runs the fused prefill over consecutive token ranges, growing each
    sequence's length with the prompt (the realistic chunked flow)."""
    cfg = c.cfg
    dt = torch_dtype(cfg)
    K = torch.full(c.k.shape, SENTINEL, dtype=dt, device="cuda")
    V = None if cfg.mla else torch.full(c.v.shape, SENTINEL, dtype=dt, device="cuda")
    kmax = torch.full((cfg.batch, cfg.h_kv, c.m_max, cfg.d_qk), SENTINEL, dtype=dt, device="cuda")
    kmin = torch.full_like(kmax, SENTINEL)
    codes = torch.full((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 2), 0xAA, dtype=torch.uint8, device="cuda")
    qparams = torch.full((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 32, 2), SENTINEL, dtype=torch.float32,
                         device="cuda")
    ctx_full = torch.from_numpy(c.ctx_host).cuda()
    for (t0, t1) in bounds:
        ctx = torch.clamp(ctx_full, max=t1).to(torch.int32)
        tls.tls_prefill_kv(c.layout, _src(c.k, t0, t1), None if cfg.mla else _src(c.v, t0, t1), ctx, c.ch, t0, t1,
                           K, V, kmax, kmin, codes, qparams)
    torch.cuda.synchronize()
    return dict(K=K, V=V, kmax=kmax, kmin=kmin, codes=codes, qparams=qparams)


def _bounds(kind, T):
    if kind == "whole":
        return [(0, T)]
    # chunk edges inside blocks (and one chunk of a single token)
    edges = [0, 100, 101, 613, 1000, T]
    edges = sorted(set(min(e, T) for e in edges))
    return list(zip(edges[:-1], edges[1:]))


@pytest.mark.parametrize("kind", ["whole", "chunked"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_prefill_writes_cache_and_indices(name, kind):
    c = get_case(name)
    cfg = c.cfg
    r = _prefill(c, _bounds(kind, cfg.max_ctx))
    for s in range(cfg.batch):
        n = int(c.ctx_host[s])
        m = -(-n // cfg.block)
        for g in range(cfg.h_kv):
            what = f"{name}/{kind} unit {(s, g)}"
            assert torch.equal(_bits(r["K"][s, g, :n]), _bits(c.k[s, g, :n])), what + " K rows"
            assert bool((r["K"][s, g, n:] == SENTINEL).all()), what + " K rows past ctx_len written"
            if not cfg.mla:
                assert torch.equal(_bits(r["V"][s, g, :n]), _bits(c.v[s, g, :n])), what + " V rows"
                assert bool((r["V"][s, g, n:] == SENTINEL).all()), what + " V rows past ctx_len written"
            Ku, _ = c.unit_kv_f64(s, g)
            kmax, kmin = O.block_summaries(Ku, n, cfg.block)
            np.testing.assert_array_equal(synth.torch_to_f64(r["kmax"][s, g, :m]), kmax, err_msg=what + " kmax")
            np.testing.assert_array_equal(synth.torch_to_f64(r["kmin"][s, g, :m]), kmin, err_msg=what + " kmin")
            assert bool((r["kmax"][s, g, m:] == SENTINEL).all()), what + " blocks past the end written"
            codes, qp = O.token_index(Ku, n, c.ch_host[g])
            gc = r["codes"][s, g, :n].cpu().numpy()
            assert np.array_equal(gc, codes), f"{what} codes differ at {np.argwhere(gc != codes)[:5]}"
            np.testing.assert_array_equal(r["qparams"][s, g, :n].cpu().numpy(), qp, err_msg=what + " qparams")
            assert bool((r["codes"][s, g, n:] == 0xAA).all()), what + " token rows past ctx_len written"


@pytest.mark.parametrize("name", sorted(CASES))
def test_prefill_equals_separate_builders(name):
    """The fused call and the two standalone builders over the written cache
    give the same bytes."""
    c = get_case(name)
    cfg = c.cfg
    r = _prefill(c, _bounds("chunked", cfg.max_ctx))
    dt = torch_dtype(cfg)
    kmax = torch.full((cfg.batch, cfg.h_kv, c.m_max, cfg.d_qk), SENTINEL, dtype=dt, device="cuda")
    kmin = torch.full_like(kmax, SENTINEL)
    codes = torch.full_like(r["codes"], 0xAA)
    qparams = torch.full_like(r["qparams"], SENTINEL)
    tls.tls_build_block_index(c.layout, r["K"], c.ctx, 0, cfg.max_ctx, kmax, kmin)
    tls.tls_build_token_index(c.layout, r["K"], c.ctx, c.ch, 0, cfg.max_ctx, codes, qparams)
    torch.cuda.synchronize()
    assert torch.equal(_bits(kmax), _bits(r["kmax"]))
    assert torch.equal(_bits(kmin), _bits(r["kmin"]))
    assert torch.equal(codes, r["codes"])
    assert torch.equal(qparams.view(torch.int32), r["qparams"].view(torch.int32))


@pytest.mark.parametrize("name", ["gqa_bf16", "mla_bf16"])
def test_offload_copies_valid_rows(name):
    c = get_case(name)
    cfg = c.cfg
    r = _prefill(c, _bounds("whole", cfg.max_ctx))
    dt = torch_dtype(cfg)
    T = cfg.max_ctx
    for (t0, t1) in [(0, T), (130, 777)]:
        hk = torch.full(c.k.shape, SENTINEL, dtype=dt, pin_memory=True)
        hv = None if cfg.mla else torch.full(c.v.shape, SENTINEL, dtype=dt, pin_memory=True)
        tls.tls_offload_kv(c.layout, r["K"], r["V"], c.ctx, t0, t1, hk, hv)
        torch.cuda.synchronize()
        K = r["K"].cpu()
        V = None if cfg.mla else r["V"].cpu()
        for s in range(cfg.batch):
            hi = min(t1, int(c.ctx_host[s]))
            for g in range(cfg.h_kv):
                what = f"{name} [{t0},{t1}) unit {(s, g)}"
                if hi > t0:
                    assert torch.equal(_bits(hk[s, g, t0:hi]), _bits(K[s, g, t0:hi])), what
                    if V is not None:
                        assert torch.equal(_bits(hv[s, g, t0:hi]), _bits(V[s, g, t0:hi])), what
                assert bool((hk[s, g, :t0] == SENTINEL).all()), what + " rows before the range"
                assert bool((hk[s, g, max(hi, t0):] == SENTINEL).all()), what + " rows past the range"


@pytest.mark.parametrize("source", ["device", "host"])
@pytest.mark.parametrize("name", ["gqa_bf16", "gqa_f32", "mla_bf16"])
def test_initial_residency_from_last_query(name, source):
    """Prefill, select blocks with the last prompt token's query, offload, make
    the selection resident, then decode over the pool with that selection (the
    first step of the lagged schedule)."""
    c = get_case(name)
    cfg = c.cfg
    dt = torch_dtype(cfg)
    r = _prefill(c, _bounds("chunked", cfg.max_ctx))
    K, V = r["K"], r["V"]
    ws = c.workspace()
    M0 = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(c.layout, c.q, r["kmax"], r["kmin"], c.ctx, cfg.k_b, M0, None, ws)
    hk = torch.empty(c.k.shape, dtype=dt, pin_memory=True)
    hv = None if cfg.mla else torch.empty(c.v.shape, dtype=dt, pin_memory=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    tls.tls_offload_kv(c.layout, K, V, c.ctx, 0, cfg.max_ctx, hk, hv, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    units, B, n_slots = cfg.batch * cfg.h_kv, cfg.block, 2 * cfg.k_b
    pool_k = torch.full((units, n_slots, B, cfg.d_qk), float("nan"), dtype=dt, device="cuda")
    pool_v = None if cfg.mla else torch.full((units, n_slots, B, cfg.d_v), float("nan"), dtype=dt, device="cuda")
    slot_map = torch.full((units, c.m_max), 5, dtype=torch.int32, device="cuda")  # stale contents
    slot_owner = torch.full((units, n_slots), 3, dtype=torch.int32, device="cuda")
    src_k, src_v = (K, V) if source == "device" else (hk, hv)
    tls.tls_init_residency(c.layout, src_k, src_v, c.ctx, M0, cfg.k_b, pool_k, pool_v, n_slots, slot_map,
                           slot_owner, ws)
    torch.cuda.synchronize()
    smap, sown, M = slot_map.cpu().numpy(), slot_owner.cpu().numpy(), M0.cpu().numpy()
    pk = pool_k.cpu()
    Kc = K.cpu()
    for s in range(cfg.batch):
        n = int(c.ctx_host[s])
        for g in range(cfg.h_kv):
            u = s * cfg.h_kv + g
            what = f"{name}/{source} unit {(s, g)}"
            ids = valid_ids(M[s, g])
            expect = np.full(c.m_max, -1, dtype=np.int32)
            expect[ids] = np.arange(len(ids), dtype=np.int32)
            assert np.array_equal(smap[u], expect), what + " slot_map"
            owner = np.full(n_slots, -1, dtype=np.int32)
            owner[:len(ids)] = ids
            assert np.array_equal(sown[u], owner), what + " slot_owner"
            for k, b in enumerate(ids):
                rows = min(B, n - int(b) * B)
                assert torch.equal(_bits(pk[u, k, :rows]), _bits(Kc[s, g, int(b) * B:int(b) * B + rows])), what
    # decode over the pool with the lagged selection M0 == decode over the dense cache
    kv_pool = tls.KV(pool_k, pool_v, slot_map, n_slots)
    c2 = Case.__new__(Case)
    c2.__dict__.update(c.__dict__)
    c2.k, c2.v = K, V
    c2.kmax, c2.kmin, c2.codes, c2.qparams = r["kmax"], r["kmin"], r["codes"], r["qparams"]
    got = c2.decode(block_ids_in=M0, kv=kv_pool)
    ref = c2.decode(block_ids_in=M0)
    assert torch.equal(_bits(got["out"]), _bits(ref["out"]))
    assert torch.equal(got["lse"].view(torch.int32), ref["lse"].view(torch.int32))
    assert torch.equal(got["tids"], ref["tids"])
    G = cfg.group
    for s in range(cfg.batch):
        for g in range(cfg.h_kv):
            what = f"{name}/{source} decode unit {(s, g)}"
            ids = valid_ids(M[s, g])
            ora = c2.oracle_unit(s, g, block_ids=ids)
            sw = check_selection(got["tids"][s, g].cpu().numpy(), ora["token_ids"], alpha_lookup(ora),
                                 what + " tokens")
            if sw == 0:
                check_close(got["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), ora["out"], cfg.dtype,
                            what + " out")
    assert tls.tls_check_device_error(ws) == 0


def _boundary_rows(cfg, ch, rows, seed):
    """Key rows whose quantisation quotients sit on or next to rounding
    boundaries: per row a multiplier m and channel values m * v with v in
    {0, 15} (the range), the half-integers 0.5 .. 14.5 (exact ties when m is
    a power of two or 3), and 15 values one float32 ulp either side of a
    half-integer; the other channels are random."""
    r = np.random.default_rng(seed)
    mults = [1.0, 3.0, 0.1, 0.7, 1e-3, 2.0 ** -20, 37.25, 1.0 / 3.0]
    halves = np.arange(15, dtype=np.float32) + np.float32(0.5)
    out = r.standard_normal((rows, cfg.d_qk), dtype=np.float32)
    for t in range(rows):
        m = np.float32(mults[t % len(mults)])
        side = np.where(r.random(15) < 0.5, -np.inf, np.inf).astype(np.float32)
        nudged = np.nextafter(halves[r.permutation(15)], side)
        v = np.concatenate([np.float32([0.0, 15.0]), halves, nudged]).astype(np.float32)
        for grp in range(cfg.d_c // 32):
            cols = ch[grp * 32:(grp + 1) * 32]
            out[t, cols] = (m * v[r.permutation(32)]).astype(np.float32)
    return out


@pytest.mark.parametrize("name", ["gqa_bf16", "gqa_f32", "mla_bf16"])
def test_token_index_rounding_boundaries(name):
    """Codes equal the oracle's bit for bit where the quotient lies on or one
    ulp from a rounding boundary (the reciprocal shortcut must defer to the
    IEEE quotient there)."""
    base = get_case(name)
    c = Case.__new__(Case)
    c.__dict__.update(base.__dict__)
    c._unit_cache = {}
    cfg = c.cfg
    host_k = np.array(base.host["k"], copy=True)
    rows = 96
    for s in range(cfg.batch):
        for g in range(cfg.h_kv):
            x = _boundary_rows(cfg, c.ch_host[g], rows, seed=1000 * s + g)
            host_k[s, g, :rows] = synth._store(x, cfg.dtype)
    c.host = dict(base.host, k=host_k)
    c.k = synth.host_to_torch(host_k, cfg.dtype).cuda()
    r = _prefill(c, _bounds("chunked", cfg.max_ctx))
    codes_b = torch.full_like(r["codes"], 0xAA)
    qp_b = torch.full_like(r["qparams"], SENTINEL)
    tls.tls_build_token_index(c.layout, r["K"], c.ctx, c.ch, 0, cfg.max_ctx, codes_b, qp_b)
    torch.cuda.synchronize()
    assert torch.equal(codes_b, r["codes"])
    for s in range(cfg.batch):
        n = int(c.ctx_host[s])
        for g in range(cfg.h_kv):
            Ku, _ = c.unit_kv_f64(s, g)
            codes, qp = O.token_index(Ku, n, c.ch_host[g])
            gc = r["codes"][s, g, :n].cpu().numpy()
            assert np.array_equal(gc[:rows], codes[:rows]), (
                f"{name} unit {(s, g)}: codes differ at {np.argwhere(gc[:rows] != codes[:rows])[:5]}")
            assert np.array_equal(gc, codes)
            np.testing.assert_array_equal(r["qparams"][s, g, :n].cpu().numpy(), qp)
