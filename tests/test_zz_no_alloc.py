"""tls_sparse_decode_noalloc (the decode step on the library's own scratch)
against tls_sparse_decode on a caller workspace, through the C ABI.

Both entry points run the same kernels in the same order, so every output
must be identical: selections, attention output and lse.  Each case makes
two calls in a row on the shared scratch, the second with a smaller input,
and covers the routes of the operator: the fused bf16 selection with the
whole-unit attention, the general selection stages (fp32, absorbed MLA)
with split attention and its merge, the single-level operators, the lagged
operator, and given token ids.  A request beyond the scratch is rejected before any launch, and
device-side error bits reach the caller's word.
"""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import synth

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")


def _cases(name):
    """(larger, smaller) workloads of one route."""
    if name == "gqa_bf16_fused":
        big = synth.config("qwen3_gqa_48k").replace(batch=4, ctx_lo=12000, ctx_hi=16384, k_b=64, k_t=1024,
                                                    clusters=4, seed=9100)
        small = big.replace(batch=2, ctx_lo=2000, ctx_hi=4096, k_b=8, k_t=128, clusters=1, seed=9101)
    elif name == "gqa_f32":
        big = synth.config("toy").replace(batch=3, ctx_lo=5000, ctx_hi=8192, k_b=16, k_t=512, seed=9200)
        small = big.replace(batch=1, ctx_lo=3000, ctx_hi=3000, k_b=8, k_t=128, seed=9201)
    elif name == "mla_bf16":
        big = synth.config("mla").replace(batch=3, ctx_lo=9000, ctx_hi=12000, k_b=64, k_t=1024, clusters=4,
                                          seed=9300)
        small = big.replace(batch=2, ctx_lo=2500, ctx_hi=3000, k_b=8, k_t=200, clusters=2, seed=9301)
    else:
        raise KeyError(name)
    return big, small


def _both(c, mode=tls.MODE_TWO_LEVEL, attn_splits=0, token_ids_in=None, block_ids_in=None):
    """The step through both entry points; returns (workspace run, scratch run)."""
    cfg = c.cfg
    runs = []
    for noalloc in (False, True):
        out = torch.full((cfg.batch, cfg.h_q, cfg.d_v), float("nan"), dtype=H.torch_dtype(cfg), device="cuda")
        lse = torch.full((cfg.batch, cfg.h_q), float("nan"), dtype=torch.float32, device="cuda")
        bids = tids = None
        sel_tokens = token_ids_in is None
        if mode == tls.MODE_LAGGED or (mode in (tls.MODE_TWO_LEVEL, tls.MODE_BLOCK_SPARSE) and sel_tokens
                                       and block_ids_in is None):
            bids = torch.full((cfg.batch, cfg.h_kv, cfg.k_b), -7, dtype=torch.int32, device="cuda")
        if mode in (tls.MODE_TWO_LEVEL, tls.MODE_TOKEN_SPARSE, tls.MODE_LAGGED) and sel_tokens:
            tids = torch.full((cfg.batch, cfg.h_kv, cfg.k_t), -7, dtype=torch.int32, device="cuda")
        idx = mode != tls.MODE_DENSE and sel_tokens
        args = (c.layout, c.q, c.kv(), c.ctx, c.kmax if idx else None, c.kmin if idx else None,
                c.codes if idx else None, c.qparams if idx else None, c.ch if idx else None, cfg.k_b, cfg.k_t,
                block_ids_in, token_ids_in, out, lse, bids, tids)
        if noalloc:
            derr = torch.zeros(1, dtype=torch.int32, device="cuda")
            tls.tls_sparse_decode_noalloc(*args, device_error=derr, attn_splits=attn_splits, mode=mode)
        else:
            ws = c.workspace()
            tls.tls_sparse_decode(*args, ws, attn_splits=attn_splits, mode=mode)
        torch.cuda.synchronize()
        err = int(derr.item()) if noalloc else tls.tls_check_device_error(ws)
        runs.append(dict(out=out, lse=lse, bids=bids, tids=tids, err=err))
    return runs


def _same(a, b, what):
    assert torch.equal(a["out"].view(torch.int16) if a["out"].dtype == torch.bfloat16 else a["out"],
                       b["out"].view(torch.int16) if b["out"].dtype == torch.bfloat16 else b["out"]), what + " out"
    assert torch.equal(a["lse"].nan_to_num(0.0, neginf=-1e30), b["lse"].nan_to_num(0.0, neginf=-1e30)), what + " lse"
    for k in ("bids", "tids"):
        if a[k] is not None:
            assert torch.equal(a[k], b[k]), f"{what} {k}"
    assert a["err"] == b["err"] == 0, what + " device error"


@pytest.mark.parametrize("name", ["gqa_bf16_fused", "gqa_f32", "mla_bf16"])
def test_noalloc_equals_workspace_decode(name):
    for i, cfg in enumerate(_cases(name)):
        c = H.Case(cfg, backend="host", pad="nan").build_index()
        ws_run, na_run = _both(c)
        _same(ws_run, na_run, f"{name} call {i}")
        # the scratch run is also the operator: sampled units against the oracle
        for (s, g) in c.units(2, seed=i):
            H.compare_unit(c, na_run, s, g)
        # split attention (partials and their merge in the scratch)
        a, b = _both(c, attn_splits=4)
        _same(a, b, f"{name} call {i} split")
        # the lagged operator (Sec. 4.2): tokens from a given previous selection
        a, b = _both(c, mode=tls.MODE_LAGGED, block_ids_in=ws_run["bids"])
        _same(a, b, f"{name} call {i} lagged")


def test_noalloc_routes_and_modes():
    big, small = _cases("gqa_bf16_fused")
    for i, cfg in enumerate((big, small)):
        c = H.Case(cfg, backend="host", pad="nan").build_index()
        for mode in (tls.MODE_BLOCK_SPARSE, tls.MODE_DENSE, tls.MODE_TOKEN_SPARSE):
            a, b = _both(c, mode=mode)
            _same(a, b, f"mode {mode} call {i}")
        own = _both(c)[0]
        a, b = _both(c, token_ids_in=own["tids"])
        _same(a, b, f"given tokens call {i}")
        a, b = _both(c, block_ids_in=own["bids"])
        _same(a, b, f"given blocks call {i}")


def test_noalloc_rejects_requests_beyond_its_scratch():
    """The token-level operator over 256 units of 65600 tokens needs 4 bytes
    per (unit, position) of scratch, 67.2 MB, more than the library's 64 MiB:
    the call fails before launching anything and leaves the outputs
    untouched.  (Every array has its full layout, so the request is valid in
    every other respect.)"""
    cfg = synth.config("offload_gqa_96k").replace(ctx_lo=65600, ctx_hi=65600)
    T, U = cfg.max_ctx, cfg.batch * cfg.h_kv
    assert U * T * 4 > 64 << 20
    L = tls.make_layout(cfg.batch, cfg.h_q, cfg.h_kv, cfg.d_qk, cfg.d_v, T, index_channels=cfg.d_c)
    dev = "cuda"
    q = torch.zeros((cfg.batch, cfg.h_q, cfg.d_qk), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((cfg.batch, cfg.h_kv, T, cfg.d_qk), dtype=torch.bfloat16, device=dev)
    v = torch.zeros((cfg.batch, cfg.h_kv, T, cfg.d_v), dtype=torch.bfloat16, device=dev)
    ctx = torch.full((cfg.batch,), T, dtype=torch.int32, device=dev)
    codes = torch.zeros((cfg.batch, cfg.h_kv, T, cfg.d_c // 2), dtype=torch.uint8, device=dev)
    qp = torch.zeros((cfg.batch, cfg.h_kv, T, cfg.d_c // 32, 2), dtype=torch.float32, device=dev)
    ch = torch.arange(cfg.d_c, dtype=torch.int32, device=dev).repeat(cfg.h_kv, 1).contiguous()
    out = torch.full((cfg.batch, cfg.h_q, cfg.d_v), 3.0, dtype=torch.bfloat16, device=dev)
    tids = torch.full((cfg.batch, cfg.h_kv, cfg.k_t), -7, dtype=torch.int32, device=dev)
    with pytest.raises(tls.TlsError) as e:
        tls.tls_sparse_decode_noalloc(L, q, tls.KV(k, v), ctx, None, None, codes, qp, ch, cfg.k_b, cfg.k_t, None,
                                      None, out, None, None, tids, mode=tls.MODE_TOKEN_SPARSE)
    assert e.value.status == 3  # TLS_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert torch.all(out == 3.0) and torch.all(tids == -7)
    del k, v, codes, qp
    torch.cuda.empty_cache()


def test_noalloc_reports_device_errors():
    """A given token id past ctx_len is skipped and flagged in the caller's
    error word, as tls_sparse_decode flags it in its workspace."""
    _, cfg = _cases("gqa_bf16_fused")
    c = H.Case(cfg, backend="host", pad="nan").build_index()
    bad = torch.zeros((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32)
    bad[...] = torch.arange(cfg.k_t, dtype=torch.int32)
    bad[..., -1] = int(c.ctx_host.max()) + 5  # ascending; the last id lies past every sequence
    bad = bad.cuda()
    a, b = _both(c, token_ids_in=bad)
    assert a["err"] == b["err"] == tls.DEVERR_TOKEN_ID
    assert torch.equal(a["out"].view(torch.int16), b["out"].view(torch.int16))
