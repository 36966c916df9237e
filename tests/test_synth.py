"""The seeded generator: deterministic, padded as asked, planted rows in place."""
import numpy as np

import synth


def test_bf16_round_trip_and_rne():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5, 3.0e38, np.inf], dtype=np.float32)
    b = synth.f32_to_bf16_bits(x)
    back = synth.bf16_bits_to_f32(b)
    assert back[0] == 1.0
    assert back[1] == 1.0            # exactly halfway between 1 and 1+2^-7 -> even (1.0)
    assert back[2] == 1.0078125      # above halfway -> up
    assert back[3] == -2.5 and np.isinf(back[5])


def test_deterministic_and_padded():
    cfg = synth.config("toy").replace(ctx_lo=300, ctx_hi=500, batch=3, h_q=4, h_kv=2,
                                      clusters=1, d_qk=64, d_v=32, d_c=32)
    a = synth.make_host(cfg, pad="nan")
    b = synth.make_host(cfg, pad="nan")
    for key in ("q", "k", "v", "ctx_lens", "channels", "plant_starts"):
        np.testing.assert_array_equal(a[key], b[key])
    for s, n in enumerate(a["ctx_lens"]):
        assert np.all(np.isnan(a["k"][s, :, n:])) and np.all(np.isfinite(a["k"][s, :, :n]))
    for s in range(cfg.batch):
        for h in range(cfg.h_kv):
            st = a["plant_starts"][s, h, 0]
            assert np.all(a["k"][s, h, st:st + 8] == a["planted_key"][s, h])
    assert np.all(np.diff(a["channels"], axis=1) > 0)


def test_query_walk_locality():
    cfg = synth.config("toy").replace(steps=4, rho=0.95)
    w = synth.to_f64(synth.draw_query_walk(cfg), cfg.dtype)
    assert w.shape[0] == 5
    c = [np.corrcoef(w[t].ravel(), w[t + 1].ravel())[0, 1] for t in range(4)]
    assert min(c) > 0.9
