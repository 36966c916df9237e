"""Incremental index maintenance during decode: appending one token per step
re-summarises the token's block and quantises its token-index row (the
builders' token range).  The maintained indices equal a full build bit for
bit, and a decode step at the grown length matches the oracle."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

CASES = {
    "gqa_bf16": lambda: synth.config("qwen3_gqa_48k").replace(batch=2, ctx_lo=1100, ctx_hi=1100, clusters=1, k_b=8,
                                                              k_t=128, seed=131),
    "gqa_f32": lambda: synth.config("toy").replace(batch=2, ctx_lo=1100, ctx_hi=1100, clusters=1, k_b=6, k_t=100,
                                                   seed=132),
    "mla_bf16": lambda: synth.config("mla").replace(batch=2, ctx_lo=1100, ctx_hi=1100, clusters=1, k_b=6, k_t=100,
                                                    seed=133),
}


@pytest.mark.parametrize("name", list(CASES))
def test_append_tokens_matches_full_build(name):
    import paper_2604_07815_amd as tls
    cfg = CASES[name]()
    final, start = 1100, 1000  # the appends cross the block boundaries at 1024 and 1088
    c = H.Case(cfg, backend="host", pad="nan", ctx_lens=np.array([final] * cfg.batch, dtype=np.int32))
    full = H.Case.__new__(H.Case)
    full.__dict__.update(c.__dict__)
    full.build_index()  # reference: one build at the final length
    ref = {k: getattr(full, k).clone() for k in ("kmax", "kmin", "codes", "qparams")}
    # incremental: build at `start`, then append one token at a time
    ctx = torch.full((cfg.batch,), start, dtype=torch.int32, device="cuda")
    c.ctx = ctx
    c.build_index()
    for t in range(start, final):
        ctx.fill_(t + 1)
        tls.tls_build_block_index(c.layout, c.k, ctx, t, t + 1, c.kmax, c.kmin)
        tls.tls_build_token_index(c.layout, c.k, ctx, c.ch, t, t + 1, c.codes, c.qparams)
    torch.cuda.synchronize()
    m = -(-final // cfg.block)
    assert torch.equal(c.kmax[:, :, :m], ref["kmax"][:, :, :m])
    assert torch.equal(c.kmin[:, :, :m], ref["kmin"][:, :, :m])
    assert torch.equal(c.codes[:, :, :final], ref["codes"][:, :, :final])
    assert torch.equal(c.qparams[:, :, :final], ref["qparams"][:, :, :final])
    # a decode step at the grown length on the maintained index
    r = c.decode()
    for (s, g) in c.units():
        H.compare_unit(c, r, s, g)
    assert tls.tls_check_device_error(r["ws"]) == 0
