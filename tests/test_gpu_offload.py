"""Offloaded KV tier on the GPU (Sec. 4.2): lagged selection and incremental
block transfer into an HBM pool, checked step by step against the oracle's
lagged schedule, which always reads the full K/V (offloading must not change
any result).

Per step t (t = 1..T), as in a serving loop:
  main stream: M_t = select_blocks(q_t)
  side stream: prefetch(new = M_t, live = M_{t-1})   (pinned host K/V -> pool)
  main stream: decode(q_t, pooled K/V, block_ids_in = M_{t-1})
  main stream waits for the prefetch before step t+1.
The pool starts filled with NaN, so reading a slot that was never filled, or
filled with the wrong block, poisons the output.
"""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import synth
from gpu_harness import Case, alpha_lookup, check_close, check_selection, torch_dtype, valid_ids
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

CASES = {
    # scaled-down shape of the 96k offloaded workload; ragged contexts
    "gqa_bf16": dict(batch=2, h_q=8, h_kv=2, ctx_lo=2900, ctx_hi=4096, k_b=8, k_t=128, clusters=2, steps=6),
    # no query drift: after the first step nothing is transferred
    "gqa_bf16_frozen": dict(batch=1, h_q=8, h_kv=2, ctx_lo=4096, ctx_hi=4096, k_b=8, k_t=128, clusters=2,
                            steps=3, rho=1.0),
}


def _run(name):
    cfg = synth.config("offload_gqa_96k").replace(**CASES[name])
    walk = synth.draw_query_walk(cfg)
    case = Case(cfg, backend="host", pad="nan", q_store=walk[0]).build_index()
    B, units, K_b = cfg.block, cfg.batch * cfg.h_kv, cfg.k_b
    n_slots = 2 * K_b
    dt = torch_dtype(cfg)
    host_k = torch.empty(case.k.shape, dtype=dt, pin_memory=True)
    host_k.copy_(case.k.cpu())
    host_v = torch.empty(case.v.shape, dtype=dt, pin_memory=True)
    host_v.copy_(case.v.cpu())
    pool_k = torch.full((units, n_slots, B, cfg.d_qk), float("nan"), dtype=dt, device="cuda")
    pool_v = torch.full((units, n_slots, B, cfg.d_v), float("nan"), dtype=dt, device="cuda")
    slot_map = torch.full((units, case.m_max), -1, dtype=torch.int32, device="cuda")
    slot_owner = torch.full((units, n_slots), -1, dtype=torch.int32, device="cuda")
    tcount = torch.zeros(units, dtype=torch.int32, device="cuda")
    ws = case.workspace()
    kv = tls.KV(pool_k, pool_v, slot_map, n_slots)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()

    qs = [synth.host_to_torch(walk[t], cfg.dtype).cuda() for t in range(walk.shape[0])]
    M_prev = torch.empty((cfg.batch, cfg.h_kv, K_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(case.layout, qs[0], case.kmax, case.kmin, case.ctx, K_b, M_prev, None, ws)
    tls.tls_prefetch_blocks(case.layout, host_k, host_v, case.ctx, M_prev, None, K_b, pool_k, pool_v, n_slots,
                            slot_map, slot_owner, tcount, ws)
    torch.cuda.synchronize()
    records = [dict(M=M_prev.cpu().numpy(), tcount=tcount.cpu().numpy(), slot_map=slot_map.cpu().numpy(),
                    slot_owner=slot_owner.cpu().numpy())]
    for t in range(1, walk.shape[0]):
        M_t = torch.empty_like(M_prev)
        tls.tls_select_blocks(case.layout, qs[t], case.kmax, case.kmin, case.ctx, K_b, M_t, None, ws)
        sel_done = torch.cuda.Event()
        sel_done.record(main)
        side.wait_event(sel_done)
        tls.tls_prefetch_blocks(case.layout, host_k, host_v, case.ctx, M_t, M_prev, K_b, pool_k, pool_v,
                                n_slots, slot_map, slot_owner, tcount, ws, stream=side)
        fetched = torch.cuda.Event()
        fetched.record(side)
        out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dt, device="cuda")
        lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
        tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
        tls.tls_sparse_decode(case.layout, qs[t], kv, case.ctx, case.kmax, case.kmin, case.codes, case.qparams,
                              case.ch, K_b, cfg.k_t, M_prev, None, out, lse, None, tids, ws)
        main.wait_event(fetched)
        torch.cuda.synchronize()
        records.append(dict(M=M_t.cpu().numpy(), lag=M_prev.cpu().numpy(), tids=tids.cpu().numpy(),
                            out=out.float().cpu().numpy(), lse=lse.cpu().numpy(), tcount=tcount.cpu().numpy(),
                            slot_map=slot_map.cpu().numpy(), slot_owner=slot_owner.cpu().numpy()))
        M_prev = M_t
    assert tls.tls_check_device_error(ws) == 0
    return cfg, case, walk, records, (host_k, host_v, pool_k, pool_v)


@pytest.mark.parametrize("name", sorted(CASES))
def test_offloaded_schedule_matches_oracle(name):
    cfg, case, walk, records, _ = _run(name)
    qs = synth.to_f64(walk, cfg.dtype)
    G, B = cfg.group, cfg.block
    for s in range(cfg.batch):
        n = int(case.ctx_host[s])
        for g in range(cfg.h_kv):
            u = s * cfg.h_kv + g
            Ku, Vu = case.unit_kv_f64(s, g)
            kmax, kmin = O.block_summaries(Ku, n, B)
            codes, qparams = O.token_index(Ku, n, case.ch_host[g])
            ref = O.lagged_decode(qs, synth.to_f64(case.host["k"], cfg.dtype),
                                  synth.to_f64(case.host["v"], cfg.dtype), n, case.ch_host[g], cfg.k_b,
                                  cfg.k_t, B, cfg.sigma, cfg.d_v, s=s, g=g)
            first = records[0]
            assert int(first["tcount"][u]) == len(valid_ids(first["M"][s, g]))
            for t, (prev, rec, st) in enumerate(zip(records[:-1], records[1:], ref), start=1):
                qg = qs[t, s, g * G:(g + 1) * G]
                what = f"{name} step {t} unit {(s, g)}"
                # M_t against the oracle's block selection of q_t
                ids, scores = O.select_blocks(qg, kmax, kmin, cfg.k_b)
                full = O.quest_scores(qg, kmax, kmin)
                check_selection(rec["M"][s, g], ids, lambda i: float(full[i]), what + " blocks")
                # transfers: T_t = M_t minus the resident set before the call, which
                # holds M_{t-1} (and whatever of M_{t-2} the pool still keeps)
                M_t = set(valid_ids(rec["M"][s, g]).tolist())
                lag = valid_ids(rec["lag"][s, g])
                before = set(int(x) for x in prev["slot_owner"][u] if x >= 0)
                assert before >= set(lag.tolist()), what
                assert int(rec["tcount"][u]) == len(M_t - before), what
                assert int(rec["tcount"][u]) <= len(M_t - set(lag.tolist())), what
                # after the call: M_t resident, only M_t and M_{t-1} kept, maps consistent
                smap, sown = rec["slot_map"][u], rec["slot_owner"][u]
                for b in M_t:
                    sl = int(smap[b])
                    assert 0 <= sl < 2 * cfg.k_b and int(sown[sl]) == b, what + f" block {b} not resident"
                owned = [int(x) for x in sown if x >= 0]
                assert len(owned) == len(set(owned)), what
                assert M_t <= set(owned) <= (M_t | set(lag.tolist())), what
                for sl, b in enumerate(sown):
                    if b >= 0:
                        assert int(smap[b]) == sl, what
                assert int((smap >= 0).sum()) == len(owned), what
                # S_t from the GPU's lagged block list, then attention on the GPU's S_t
                S_ref, alpha, cand = O.select_tokens(qg, case.ch_host[g], codes, qparams, lag, n, B, cfg.k_t,
                                                     cfg.sigma)
                res = dict(cand=cand, alpha=alpha)
                sw = check_selection(rec["tids"][s, g], S_ref, alpha_lookup(res), what + " tokens")
                S_gpu = valid_ids(rec["tids"][s, g])
                assert set(S_gpu.tolist()) <= set(O.candidates(lag, n, B).tolist())
                o, lse = O.sparse_attention(qg, Ku, Vu, S_gpu, cfg.sigma)
                check_close(rec["out"][s, g * G:(g + 1) * G], o, cfg.dtype, what + " out")
                check_close(rec["lse"][s, g * G:(g + 1) * G], lse, cfg.dtype, what + " lse")
                if sw == 0 and np.array_equal(lag, st["lag_block_ids"]):
                    assert np.array_equal(S_gpu, st["token_ids"]), what
                if cfg.rho == 1.0:
                    assert int(rec["tcount"][u]) == 0, what


def test_pool_holds_host_bytes():
    cfg, case, walk, records, (host_k, host_v, pool_k, pool_v) = _run("gqa_bf16")
    last = records[-1]
    B = cfg.block
    pk, pv = pool_k.cpu(), pool_v.cpu()
    for s in range(cfg.batch):
        n = int(case.ctx_host[s])
        for g in range(cfg.h_kv):
            u = s * cfg.h_kv + g
            for b in valid_ids(last["M"][s, g]):
                sl = int(last["slot_map"][u, b])
                rows = min(B, n - int(b) * B)
                src_k = host_k[s, g, int(b) * B:int(b) * B + rows]
                src_v = host_v[s, g, int(b) * B:int(b) * B + rows]
                assert torch.equal(pk[u, sl, :rows].view(torch.int16), src_k.view(torch.int16))
                assert torch.equal(pv[u, sl, :rows].view(torch.int16), src_v.view(torch.int16))


def test_offloaded_schedule_with_growing_context():
    """The 64-step offloaded workload lets the context grow (one token per
    sequence per step); here a scaled-down walk: before each step the new
    token is appended (host K/V row, pool row if its block is resident, block
    summary and token-index row), then the lagged step runs.  Every step is
    compared with the oracle's lagged schedule at the grown lengths, which
    reads the full K/V."""
    cfg = synth.config("offload_gqa_96k").replace(**CASES["gqa_bf16"])
    walk = synth.draw_query_walk(cfg)
    T = walk.shape[0] - 1
    case = Case(cfg, backend="host", pad="nan", q_store=walk[0])
    n_final = case.ctx_host.astype(np.int64)
    n0 = n_final - T
    B, units, K_b = cfg.block, cfg.batch * cfg.h_kv, cfg.k_b
    n_slots = 2 * K_b
    dt = torch_dtype(cfg)
    # host copy of the cache holds the prefill (rows < n0); the rest arrives by appends
    host_k = torch.empty(case.k.shape, dtype=dt, pin_memory=True)
    host_k.copy_(case.k.cpu())
    host_v = torch.empty(case.v.shape, dtype=dt, pin_memory=True)
    host_v.copy_(case.v.cpu())
    for s in range(cfg.batch):
        host_k[s, :, int(n0[s]):] = float("nan")
        host_v[s, :, int(n0[s]):] = float("nan")
    ctx = torch.from_numpy(n0.astype(np.int32)).cuda()
    kmax = torch.empty((cfg.batch, cfg.h_kv, case.m_max, cfg.d_qk), dtype=dt, device="cuda")
    kmin = torch.empty_like(kmax)
    codes = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 2), dtype=torch.uint8, device="cuda")
    qparams = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 32, 2), dtype=torch.float32, device="cuda")
    tls.tls_build_block_index(case.layout, case.k, ctx, 0, cfg.max_ctx, kmax, kmin)
    tls.tls_build_token_index(case.layout, case.k, ctx, case.ch, 0, cfg.max_ctx, codes, qparams)
    pool_k = torch.full((units, n_slots, B, cfg.d_qk), float("nan"), dtype=dt, device="cuda")
    pool_v = torch.full((units, n_slots, B, cfg.d_v), float("nan"), dtype=dt, device="cuda")
    slot_map = torch.empty((units, case.m_max), dtype=torch.int32, device="cuda")
    slot_owner = torch.empty((units, n_slots), dtype=torch.int32, device="cuda")
    ws = case.workspace()
    kv = tls.KV(pool_k, pool_v, slot_map, n_slots)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    qs = [synth.host_to_torch(walk[t], cfg.dtype).cuda() for t in range(T + 1)]
    M_prev = torch.empty((cfg.batch, cfg.h_kv, K_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(case.layout, qs[0], kmax, kmin, ctx, K_b, M_prev, None, ws)
    tls.tls_init_residency(case.layout, host_k, host_v, ctx, M_prev, K_b, pool_k, pool_v, n_slots, slot_map,
                           slot_owner, ws)
    torch.cuda.synchronize()
    records = []
    for t in range(1, T + 1):
        ctx += 1
        pos = (ctx - 1).long()
        idx = pos.view(-1, 1, 1, 1).expand(-1, cfg.h_kv, 1, cfg.d_qk)
        k_new = torch.gather(case.k, 2, idx).squeeze(2).contiguous()
        v_new = torch.gather(case.v, 2, idx[..., :cfg.d_v]).squeeze(2).contiguous()
        tls.tls_append_tokens(case.layout, k_new, v_new, ctx, case.ch, host_k, host_v, kmax, kmin, codes, qparams,
                              pool=kv)
        M_t = torch.empty_like(M_prev)
        tls.tls_select_blocks(case.layout, qs[t], kmax, kmin, ctx, K_b, M_t, None, ws)
        sel_done = torch.cuda.Event()
        sel_done.record(main)
        side.wait_event(sel_done)
        tls.tls_prefetch_blocks(case.layout, host_k, host_v, ctx, M_t, M_prev, K_b, pool_k, pool_v, n_slots,
                                slot_map, slot_owner, None, ws, stream=side)
        fetched = torch.cuda.Event()
        fetched.record(side)
        out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dt, device="cuda")
        tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
        tls.tls_sparse_decode(case.layout, qs[t], kv, ctx, kmax, kmin, codes, qparams, case.ch, K_b, cfg.k_t,
                              M_prev, None, out, None, None, tids, ws)
        main.wait_event(fetched)
        torch.cuda.synchronize()
        records.append(dict(M=M_t.cpu().numpy(), lag=M_prev.cpu().numpy(), tids=tids.cpu().numpy(),
                            out=out.float().cpu().numpy()))
        M_prev = M_t
    assert tls.tls_check_device_error(ws) == 0
    qf = synth.to_f64(walk, cfg.dtype)
    G = cfg.group
    for s in range(cfg.batch):
        n_steps = [int(n0[s]) + t for t in range(T + 1)]
        for g in range(cfg.h_kv):
            Ku, Vu = case.unit_kv_f64(s, g)
            ref = O.lagged_decode(qf, synth.to_f64(case.host["k"], cfg.dtype), synth.to_f64(case.host["v"], cfg.dtype),
                                  n_steps, case.ch_host[g], K_b, cfg.k_t, B, cfg.sigma, cfg.d_v, s=s, g=g)
            for t, (rec, st) in enumerate(zip(records, ref), start=1):
                what = f"growth step {t} unit {(s, g)}"
                qg = qf[t, s, g * G:(g + 1) * G]
                kmx, kmn = O.block_summaries(Ku, n_steps[t], B)
                full = O.quest_scores(qg, kmx, kmn)
                ids, _ = O.select_blocks(qg, kmx, kmn, K_b)
                check_selection(rec["M"][s, g], ids, lambda i: float(full[i]), what + " blocks")
                lag = valid_ids(rec["lag"][s, g])
                codes_o, qp_o = O.token_index(Ku, n_steps[t], case.ch_host[g])
                S_ref, alpha, cand = O.select_tokens(qg, case.ch_host[g], codes_o, qp_o, lag, n_steps[t], B,
                                                     cfg.k_t, cfg.sigma)
                sw = check_selection(rec["tids"][s, g], S_ref, alpha_lookup(dict(cand=cand, alpha=alpha)),
                                     what + " tokens")
                S_gpu = valid_ids(rec["tids"][s, g])
                assert S_gpu.max() < n_steps[t]
                o, _ = O.sparse_attention(qg, Ku, Vu, S_gpu, cfg.sigma)
                check_close(rec["out"][s, g * G:(g + 1) * G], o, cfg.dtype, what + " out")
                if sw == 0 and np.array_equal(lag, st["lag_block_ids"]):
                    assert np.array_equal(S_gpu, st["token_ids"]), what
