"""Edge cases of the GPU path: dense mode, empty contexts, split invariance,
device-side error reporting."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")


def test_dense_mode_equals_dense_attention():
    """K_b = all blocks and K_t = all tokens: the operator is dense attention."""
    cfg = synth.config("toy")
    c = H.Case(cfg, backend="host").build_index()
    r = c.decode(k_b=64, k_t=4096)
    for (s, g) in c.units():
        ref = H.compare_unit(c, r, s, g, k_b=64, k_t=4096)
        assert len(ref["token_ids"]) == 4096


@pytest.mark.parametrize("splits", [0, 1])
def test_empty_and_tiny_contexts(splits):
    """splits=1 takes the whole-unit attention (one work-group per unit)."""
    cfg = synth.config("qwen3_gqa_48k").replace(batch=3, ctx_lo=0, ctx_hi=200, clusters=0, k_b=4, k_t=64, seed=5)
    c = H.Case(cfg, backend="host", ctx_lens=np.array([0, 1, 200], dtype=np.int32)).build_index()
    r = c.decode(attn_splits=splits)
    G = cfg.group
    # empty sequence: no ids, zero output, lse = -inf
    assert torch.all(r["bids"][0] == -1) and torch.all(r["tids"][0] == -1)
    assert torch.all(r["out"][0] == 0)
    assert torch.all(torch.isneginf(r["lse"][0]))
    for s in (1, 2):
        for g in range(cfg.h_kv):
            H.compare_unit(c, r, s, g)
    import paper_2604_07815_amd as tls
    assert tls.tls_check_device_error(r["ws"]) == 0


@pytest.mark.parametrize("splits", [1, 3, 16, 64, 100, 128])
def test_split_merge_invariance(splits):
    """LSE merge of split partials equals an unsplit computation."""
    cfg = synth.config("toy")
    c = H.Case(cfg, backend="host").build_index()
    base = c.decode(attn_splits=1)
    r = c.decode(attn_splits=splits)
    np.testing.assert_allclose(r["out"].cpu().numpy(), base["out"].cpu().numpy(), rtol=2e-6, atol=2e-6)
    np.testing.assert_allclose(r["lse"].cpu().numpy(), base["lse"].cpu().numpy(), rtol=2e-6, atol=2e-6)


@pytest.mark.parametrize("splits", [1, 2, 5, 64, 128])
def test_split_merge_invariance_bf16(splits):
    """bf16: one work-group per unit (splits=1, output written directly) and
    split partials merged by LSE agree to bf16 rounding, and each matches the
    oracle on the same token ids."""
    cfg = synth.config("qwen3_gqa_48k").replace(ctx_lo=3000, ctx_hi=3000, clusters=2, k_b=16, k_t=700)
    c = H.Case(cfg, backend="host").build_index()
    base = c.decode(attn_splits=1)
    r = c.decode(attn_splits=splits)
    np.testing.assert_allclose(r["out"].float().cpu().numpy(), base["out"].float().cpu().numpy(), rtol=8e-3,
                               atol=8e-3)
    np.testing.assert_allclose(r["lse"].cpu().numpy(), base["lse"].cpu().numpy(), rtol=1e-5, atol=1e-5)
    for (s, g) in c.units():
        ids = H.valid_ids(r["tids"][s, g].cpu().numpy())
        ref = c.oracle_unit(s, g, token_ids=ids)
        G = cfg.group
        H.check_close(r["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), ref["out"], cfg.dtype, "out")
        H.check_close(r["lse"][s, g * G:(g + 1) * G].cpu().numpy(), ref["lse"], cfg.dtype, "lse")


def test_out_of_range_token_id_sets_error_flag():
    import paper_2604_07815_amd as tls
    cfg = synth.config("toy").replace(ctx_lo=1000, ctx_hi=1000)
    c = H.Case(cfg, backend="host").build_index()
    ids = torch.full((1, cfg.h_kv, cfg.k_t), -1, dtype=torch.int32)
    ids[:, :, 0] = 5
    ids[:, :, 1] = 999
    ids[:, :, 2] = 1000  # == ctx_len: out of range, skipped
    r = c.decode(token_ids_in=ids.cuda())
    flags = tls.tls_check_device_error(r["ws"], clear=True)
    assert flags & tls.DEVERR_TOKEN_ID
    assert tls.tls_check_device_error(r["ws"]) == 0
    for g in range(cfg.h_kv):
        ref = c.oracle_unit(0, g, token_ids=np.array([5, 999]))
        G = cfg.group
        H.check_close(r["out"][0, g * G:(g + 1) * G].cpu().numpy(), ref["out"], cfg.dtype, "out")


@pytest.mark.parametrize("splits", [2, 3])
def test_wide_split_attention(splits):
    """Few units, long token lists: the split attention runs 12-wave
    work-groups writing partials; it matches the whole-unit result to bf16
    rounding and the oracle on the same token ids."""
    cfg = synth.config("qwen3_gqa_48k").replace(batch=2, ctx_lo=20000, ctx_hi=30000, clusters=4, k_b=64, k_t=2048,
                                               seed=91)
    c = H.Case(cfg, backend="host").build_index()
    base = c.decode(attn_splits=1)
    r = c.decode(attn_splits=splits)
    assert torch.equal(r["tids"], base["tids"])
    np.testing.assert_allclose(r["out"].float().cpu().numpy(), base["out"].float().cpu().numpy(), rtol=1e-2,
                               atol=1e-2)
    np.testing.assert_allclose(r["lse"].cpu().numpy(), base["lse"].cpu().numpy(), rtol=1e-5, atol=1e-5)
    G = cfg.group
    for (s, g) in c.units():
        ref = c.oracle_unit(s, g, token_ids=r["tids"][s, g].cpu().numpy()[r["tids"][s, g].cpu().numpy() >= 0])
        H.check_close(r["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), ref["out"], cfg.dtype, f"out {(s, g)}")
        H.check_close(r["lse"][s, g * G:(g + 1) * G].cpu().numpy(), ref["lse"], cfg.dtype, f"lse {(s, g)}")


@pytest.mark.parametrize("k_b,k_t", [(128, 2048), (192, 4096)])
def test_capacity_limits(k_b, k_t):
    """The largest shapes the library accepts: 131072 tokens (2048 blocks, the
    fused selection's block capacity) with 8192 candidates, and 12288
    candidates (K_b = 192, the general selection path's key capacity) with
    K_t = 4096; sampled units against the oracle."""
    import paper_2604_07815_amd as tls
    cfg = synth.config("qwen3_gqa_48k").replace(ctx_lo=131072, ctx_hi=131072, k_b=k_b, k_t=k_t, seed=97)
    c = H.Case(cfg, backend="device", pad="nan").build_index()
    r = c.decode()
    for (s, g) in c.units(3):
        H.compare_unit(c, r, s, g)
    assert tls.tls_check_device_error(r["ws"]) == 0
    with pytest.raises(tls.TlsError) as e:
        tls.tls_workspace_size(c.layout, k_b + 1 if k_b == 192 else 193, k_t)
    assert e.value.status == 2


@pytest.mark.parametrize("name,over", [
    # the MLA route: matrix-core scoring over many work-groups, alpha, top-K_t
    ("mla", dict(batch=2, ctx_lo=3000, ctx_hi=3000, clusters=2, k_b=13, k_t=300, seed=4101)),
    # the fused bf16 GQA selection (whole blocks per wave)
    ("qwen3_gqa_48k", dict(ctx_lo=3000, ctx_hi=3000, clusters=2, k_b=13, k_t=300, seed=4102)),
    # fp32 GQA: the vector-unit scoring kernel
    ("toy", dict(ctx_lo=3000, ctx_hi=3000, k_b=13, k_t=300, seed=4103)),
])
def test_given_blocks_with_empty_and_out_of_range_entries(name, over):
    """Token selection from a given block list (Sec. 4.1 fine stage) whose
    entries include -1 (empty), ids at and past the block count (skipped
    with TLS_DEVERR_BLOCK_ID) and the context's partial last block; with
    K_b = 13 the candidate count is not a multiple of a work-group's slots.
    Tokens against the oracle's selection from the valid blocks, then the
    output against the oracle's attention over the GPU's tokens."""
    import paper_2604_07815_amd as tls
    cfg = synth.config(name).replace(**over)
    c = H.Case(cfg, backend="host").build_index()
    n = 3000
    m = -(-n // cfg.block)
    rng = np.random.default_rng(cfg.seed)
    ids = np.full((cfg.batch, cfg.h_kv, cfg.k_b), -1, dtype=np.int32)
    valid = {}
    for (s, g) in c.units():
        v = np.append(np.sort(rng.choice(m - 1, 9, replace=False)), m - 1).astype(np.int32)
        valid[(s, g)] = v
        ids[s, g] = [v[0], v[1], v[2], -1, v[3], v[4], v[5], m, v[6], v[7], v[8], v[9], m + 5]
    r = c.decode(block_ids_in=torch.from_numpy(ids).cuda())
    flags = tls.tls_check_device_error(r["ws"], clear=True)
    assert flags & tls.DEVERR_BLOCK_ID
    assert (flags & ~tls.DEVERR_BLOCK_ID) == 0
    G = cfg.group
    for (s, g) in c.units():
        ref = c.oracle_unit(s, g, block_ids=valid[(s, g)])
        H.check_selection(r["tids"][s, g].cpu().numpy(), ref["token_ids"], H.alpha_lookup(ref),
                          f"tokens unit {(s, g)}")
        S = H.valid_ids(r["tids"][s, g].cpu().numpy())
        ref_s = c.oracle_unit(s, g, token_ids=S)
        H.check_close(r["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), ref_s["out"], cfg.dtype, "out")
        H.check_close(r["lse"][s, g * G:(g + 1) * G].cpu().numpy(), ref_s["lse"], cfg.dtype, "lse")


@pytest.mark.parametrize("name,over", [
    ("mla", dict(batch=2, ctx_lo=2500, ctx_hi=2500, clusters=2, k_b=8, k_t=200, seed=4104)),
    ("qwen3_gqa_48k", dict(ctx_lo=2500, ctx_hi=2500, clusters=2, k_b=8, k_t=200, seed=4105)),
    ("toy", dict(ctx_lo=2500, ctx_hi=2500, k_b=8, k_t=200, seed=4106)),
])
def test_out_of_range_channel_reads_channel_zero(name, over):
    """A channel id outside [0, d_qk) in C (Sec. 4.1 channel projection):
    the index build and the token scoring both read channel 0 at that
    position and the decode reports TLS_DEVERR_CHANNEL; the whole step then
    equals the oracle run with channel 0 in that position."""
    import paper_2604_07815_amd as tls
    cfg = synth.config(name).replace(**over)
    c = H.Case(cfg, backend="host")
    bad = c.ch_host.copy()
    bad[:, 5] = cfg.d_qk + 3
    bad[0, 17] = -2
    c.ch = torch.from_numpy(bad).cuda()
    fixed = c.ch_host.copy()
    fixed[:, 5] = 0
    fixed[0, 17] = 0
    c.ch_host = fixed
    c.build_index()
    r = c.decode()
    assert tls.tls_check_device_error(r["ws"], clear=True) == tls.DEVERR_CHANNEL
    for (s, g) in c.units():
        H.compare_unit(c, r, s, g)
