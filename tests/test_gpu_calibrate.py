"""Channel calibration on the GPU (Sec. 4.1: the importance of every score
dimension over a calibration set, then the top-d_c channels per KV group)
against the oracle.  The per-channel maxima are exact and must match bit for
bit; scores are float32 sums of exact products (float64 in the oracle); the
channel sets must agree up to near ties of the oracle's scores."""
import numpy as np
import pytest
import torch

import paper_2604_07815_amd as tls
import synth
from gpu_harness import check_selection
from oracle import tls_oracle as O

pytestmark = pytest.mark.gpu

CASES = {
    "gqa_bf16": (synth.config("qwen3_gqa_48k"), 3000),     # 32/8 heads, d = 128, d_c = 32
    "gqa_f32": (synth.config("toy"), 1000),                # 8/2 heads, fp32
    "mla_bf16": (synth.config("mla"), 700),                # 32/1 heads, d = 576, d_c = 128
    "one_row": (synth.config("qwen3_gqa_48k"), 1),
}


def _layout(cfg):
    return tls.make_layout(1, cfg.h_q, cfg.h_kv, cfg.d_qk, cfg.d_v, 64, index_channels=cfg.d_c,
                           dtype=tls.DTYPE_BF16 if cfg.dtype == "bf16" else tls.DTYPE_F32, mla_shared_kv=cfg.mla)


def _run(cfg, q, k, batches=1):
    L = _layout(cfg)
    qa = torch.full((cfg.h_q, cfg.d_qk), 5.0, device="cuda")   # stale contents: accumulate=0 must clear them
    ka = torch.full((cfg.h_kv, cfg.d_qk), 5.0, device="cuda")
    qt = synth.host_to_torch(q, cfg.dtype).cuda()
    kt = synth.host_to_torch(k, cfg.dtype).cuda()
    edges = np.linspace(0, q.shape[0], batches + 1).astype(int)
    for i in range(batches):
        a, b = edges[i], edges[i + 1]
        tls.tls_calibrate_absmax(L, qt[a:b] if b > a else None, kt[a:b] if b > a else None, qa, ka,
                                 accumulate=i > 0)
    ch = torch.empty((cfg.h_kv, cfg.d_c), dtype=torch.int32, device="cuda")
    sc = torch.empty((cfg.h_kv, cfg.d_qk), dtype=torch.float32, device="cuda")
    tls.tls_calibrate_channels(L, qa, ka, ch, sc)
    torch.cuda.synchronize()
    return qa.cpu().numpy(), ka.cpu().numpy(), ch.cpu().numpy(), sc.cpu().numpy()


@pytest.mark.parametrize("name", sorted(CASES))
def test_calibration_matches_oracle(name):
    cfg, n = CASES[name]
    q, k, outliers = synth.draw_calibration(cfg, n)
    qa, ka, ch, sc = _run(cfg, q, k)
    och, osc, oqa, oka = O.calibrate_channels(synth.to_f64(q, cfg.dtype), synth.to_f64(k, cfg.dtype), cfg.group,
                                              cfg.d_c)
    np.testing.assert_array_equal(qa.astype(np.float64), oqa)
    np.testing.assert_array_equal(ka.astype(np.float64), oka)
    np.testing.assert_allclose(sc, osc, rtol=2e-6, atol=0)
    for g in range(cfg.h_kv):
        check_selection(ch[g], och[g], lambda i: float(osc[g][i]), f"{name} channels of KV head {g}", rel=1e-5)
        if n >= 500:  # the planted outlier channels are found
            assert set(outliers[g].tolist()) <= set(ch[g].tolist())


@pytest.mark.parametrize("batches", [2, 5])
def test_calibration_batches_equal_one_pass(batches):
    cfg, n = CASES["gqa_bf16"]
    q, k, _ = synth.draw_calibration(cfg, n)
    one = _run(cfg, q, k)
    many = _run(cfg, q, k, batches=batches)
    for a, b in zip(one, many):
        assert np.array_equal(a, b)


def test_empty_calibration_set():
    cfg, _ = CASES["gqa_bf16"]
    q, k, _ = synth.draw_calibration(cfg, 0)
    qa, ka, ch, sc = _run(cfg, q, k)
    assert np.all(qa == 0) and np.all(ka == 0) and np.all(sc == 0)
    np.testing.assert_array_equal(ch, np.tile(np.arange(cfg.d_c), (cfg.h_kv, 1)))


def test_calibrated_channels_drive_the_token_index():
    """Channels from the GPU calibration feed the token-index build and a
    decode step, which still matches the oracle on those channels."""
    from gpu_harness import Case, compare_unit
    cfg = synth.config("qwen3_gqa_48k").replace(ctx_lo=3000, ctx_hi=3000, clusters=2, k_b=8, k_t=128)
    q, k, _ = synth.draw_calibration(cfg, 2048)
    _, _, ch, _ = _run(cfg, q, k)
    c = Case(cfg, backend="host", pad="nan")
    c.ch_host = ch.astype(np.int32)
    c.ch = torch.from_numpy(c.ch_host).cuda()
    c.build_index()
    r = c.decode()
    for (s, g) in c.units():
        compare_unit(c, r, s, g)
