"""GPU path vs the CPU oracle, stage by stage, through the C ABI.

Small cases are compared on every unit; full-size workloads (the shapes the
benchmark times, same launch configuration) on sampled units.  Each stage is
fed the oracle's upstream result, so a legitimate near tie upstream cannot
cascade; the end-to-end test then runs the whole step on GPU selections.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

SMALL = {
    "toy_f32": lambda: (synth.config("toy"), "host", None),
    "ragged_bf16": lambda: (synth.config("qwen3_gqa_48k").replace(batch=6, ctx_lo=1, ctx_hi=1000, clusters=1,
                                                                   k_b=6, k_t=96, seed=71),
                            "host", np.array([1, 63, 64, 65, 700, 1000], dtype=np.int32)),
    "g8_f32": lambda: (synth.config("toy").replace(h_q=16, h_kv=2, ctx_lo=1500, ctx_hi=2100, batch=2, k_b=5,
                                                   k_t=200, seed=81), "host", None),
    "mla_small": lambda: (synth.config("mla").replace(batch=2, ctx_lo=2000, ctx_hi=3000, clusters=2, k_b=8,
                                                      k_t=200, seed=4100), "host", None),
}
FULL = {
    "qwen3_gqa_48k": (synth.config("qwen3_gqa_48k"), None),   # all 8 units
    "batched_gqa": (synth.config("batched_gqa"), 32),          # 32 of 128 units
    "mla": (synth.config("mla"), None),                        # all 8 units
    "offload_gqa_96k": (synth.config("offload_gqa_96k"), 32),  # 32 of 256 units
}
ALL = list(SMALL) + list(FULL)

_cache = {}


def get_case(name):
    if name in _cache:
        return _cache[name]
    if name in FULL:  # keep at most one full-size workload resident
        for k in [k for k in _cache if k in FULL]:
            del _cache[k]
        torch.cuda.empty_cache()
        cfg, sample = FULL[name]
        c = H.Case(cfg, backend="device", pad="nan").build_index()
        c.sample = c.units(sample)
    else:
        cfg, backend, ctx = SMALL[name]()
        c = H.Case(cfg, backend=backend, pad="nan", ctx_lens=ctx).build_index()
        c.sample = c.units()
    torch.cuda.synchronize()
    c.oracle = {u: c.oracle_unit(*u) for u in c.sample}
    _cache[name] = c
    return c


def teardown_module(module):
    _cache.clear()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ALL)
def test_index_bit_exact(name):
    """Block summaries and INT4 token index equal the oracle's exactly."""
    c = get_case(name)
    cfg = c.cfg
    for (s, g) in c.sample:
        n = int(c.ctx_host[s])
        Ku, _ = c.unit_kv_f64(s, g)
        kmax, kmin = O.block_summaries(Ku, n, cfg.block)
        m = kmax.shape[0]
        np.testing.assert_array_equal(synth.torch_to_f64(c.kmax[s, g, :m]), kmax, err_msg=f"kmax {(s, g)}")
        np.testing.assert_array_equal(synth.torch_to_f64(c.kmin[s, g, :m]), kmin, err_msg=f"kmin {(s, g)}")
        codes, qp = c.oracle_index(s, g)
        gc = c.codes[s, g, :n].cpu().numpy()
        assert np.array_equal(gc, codes), f"codes differ in unit {(s, g)}: {np.argwhere(gc != codes)[:5]}"
        np.testing.assert_array_equal(c.qparams[s, g, :n].cpu().numpy(), qp, err_msg=f"qparams {(s, g)}")


@pytest.mark.parametrize("name", ALL)
def test_select_blocks(name):
    """Top-K_b block ids (near-tie rule) and the block scores themselves."""
    c = get_case(name)
    cfg = c.cfg
    ws = c.workspace()
    bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    scores = torch.empty((cfg.batch, cfg.h_kv, c.m_max), dtype=torch.float32, device="cuda")
    import paper_2604_07815_amd as tls
    tls.tls_select_blocks(c.layout, c.q, c.kmax, c.kmin, c.ctx, cfg.k_b, bids, scores, ws)
    torch.cuda.synchronize()
    for (s, g) in c.sample:
        ref = c.oracle[(s, g)]
        m = len(ref["block_scores"])
        got = scores[s, g].cpu().numpy()
        scale = max(1.0, float(np.abs(ref["block_scores"]).max())) if m else 1.0
        np.testing.assert_allclose(got[:m], ref["block_scores"], rtol=1e-5, atol=1e-5 * scale)
        assert np.all(np.isneginf(got[m:]))
        H.check_selection(bids[s, g].cpu().numpy(), ref["block_ids"], lambda i: float(ref["block_scores"][i]),
                          f"blocks {(s, g)}")
    assert tls.tls_check_device_error(ws) == 0


def _ids_tensor(c, rows, width, fill_from=None):
    cfg = c.cfg
    t = torch.full((cfg.batch, cfg.h_kv, width), -1, dtype=torch.int32)
    if fill_from is not None:
        t.copy_(fill_from.cpu())
    for (s, g), ids in rows.items():
        t[s, g] = -1
        t[s, g, :len(ids)] = torch.from_numpy(np.asarray(ids, dtype=np.int32))
    return t.cuda()


@pytest.mark.parametrize("name", ALL)
def test_select_tokens(name):
    """Given the oracle's block selection: top-K_t token ids (near-tie rule)
    and the approximate scores of the selected tokens."""
    c = get_case(name)
    cfg = c.cfg
    import paper_2604_07815_amd as tls
    ws = c.workspace()
    own = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
    tls.tls_select_blocks(c.layout, c.q, c.kmax, c.kmin, c.ctx, cfg.k_b, own, None, ws)
    bids = _ids_tensor(c, {u: c.oracle[u]["block_ids"] for u in c.sample}, cfg.k_b, fill_from=own)
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")
    tsc = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.float32, device="cuda")
    tls.tls_select_tokens(c.layout, c.q, c.codes, c.qparams, c.ch, bids, cfg.k_b, c.ctx, cfg.k_t, tids, tsc, ws)
    torch.cuda.synchronize()
    for (s, g) in c.sample:
        ref = c.oracle[(s, g)]
        alpha = H.alpha_lookup(ref)
        got = tids[s, g].cpu().numpy()
        H.check_selection(got, ref["token_ids"], alpha, f"tokens {(s, g)}")
        k = int((got >= 0).sum())
        np.testing.assert_allclose(tsc[s, g, :k].cpu().numpy(), [alpha(t) for t in got[:k]], rtol=1e-4,
                                   atol=1e-9)
    assert tls.tls_check_device_error(ws) == 0


@pytest.mark.parametrize("name", ALL)
def test_attention_given_ids(name):
    """Given the oracle's token selection: output and log-sum-exp."""
    c = get_case(name)
    cfg = c.cfg
    own = c.decode()["tids"]
    tids = _ids_tensor(c, {u: c.oracle[u]["token_ids"] for u in c.sample}, cfg.k_t, fill_from=own)
    r = c.decode(token_ids_in=tids)
    G = cfg.group
    for (s, g) in c.sample:
        ref = c.oracle[(s, g)]
        H.check_close(r["out"][s, g * G:(g + 1) * G].float().cpu().numpy(), ref["out"], cfg.dtype, f"out {(s, g)}")
        H.check_close(r["lse"][s, g * G:(g + 1) * G].cpu().numpy(), ref["lse"], cfg.dtype, f"lse {(s, g)}")


@pytest.mark.parametrize("name", ALL)
def test_decode_end_to_end(name):
    """The whole step on GPU selections, compared unit by unit; planted
    tokens recovered; bit-identical on a second run."""
    c = get_case(name)
    cfg = c.cfg
    r = c.decode()
    for (s, g) in c.sample:
        H.compare_unit(c, r, s, g)
        st = c.plant_starts[s, g]
        planted = [int(p) + i for p in st if p >= 0 for i in range(cfg.cluster_len)]
        got = set(r["tids"][s, g].cpu().numpy().tolist())
        assert set(planted) <= got, f"planted tokens missed in unit {(s, g)}"
    r2 = c.decode()
    assert torch.equal(r["out"], r2["out"]) and torch.equal(r["tids"], r2["tids"])
    assert torch.equal(r["lse"].nan_to_num(0.0), r2["lse"].nan_to_num(0.0))
    import paper_2604_07815_amd as tls
    assert tls.tls_check_device_error(r["ws"]) == 0
