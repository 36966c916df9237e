"""Seeded random shapes through the whole two-level step (C ABI) against the
oracle: group sizes 1-8, head dims 64 and 128, both dtypes, index widths 32
and 64 channels, ragged lengths (including lengths shorter than K_b blocks
and not multiples of the block size), budgets K_b and K_t drawn per case, and
the attention split count drawn as well.  Every unit of every case is
compared (selections bit for bit up to the near-tie rule, outputs within
the dtype's tolerance).  The absorbed-latent layout (576-dim scores, 512-dim
values) gets its own draws: 16 or 32 heads, 64 or 128 index channels."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

N_CASES = 20
N_MLA = 6


def _draw(i):
    r = np.random.Generator(np.random.PCG64(7700 + i))
    G = int(r.choice([1, 2, 4, 8]))
    h_kv = int(r.choice([1, 2, 3]))
    d = int(r.choice([64, 128]))
    d_c = int(r.choice([32, 64]))
    dtype = "bf16" if i % 3 != 2 else "f32"
    batch = int(r.integers(1, 4))
    ctx_hi = int(r.integers(300, 2600))
    ctx_lo = int(r.integers(1, ctx_hi + 1))
    k_b = int(r.integers(1, 12))
    k_t = int(r.integers(1, k_b * 64 + 1))
    splits = int(r.choice([0, 1, 2, 5]))
    cfg = synth.config("toy").replace(batch=batch, h_q=G * h_kv, h_kv=h_kv, d_qk=d, d_v=d, dtype=dtype,
                                      ctx_lo=ctx_lo, ctx_hi=ctx_hi, d_c=d_c, k_b=k_b, k_t=k_t, clusters=1,
                                      seed=7800 + i)
    return cfg, splits


def _draw_mla(i):
    r = np.random.Generator(np.random.PCG64(7900 + i))
    h_q = int(r.choice([16, 32]))
    d_c = int(r.choice([64, 128]))
    batch = int(r.integers(1, 4))
    ctx_hi = int(r.integers(300, 2600))
    ctx_lo = int(r.integers(1, ctx_hi + 1))
    k_b = int(r.integers(1, 12))
    k_t = int(r.integers(1, k_b * 64 + 1))
    splits = int(r.choice([0, 1, 3]))
    cfg = synth.config("mla").replace(batch=batch, h_q=h_q, ctx_lo=ctx_lo, ctx_hi=ctx_hi, d_c=d_c, k_b=k_b, k_t=k_t,
                                      clusters=1, seed=8000 + i)
    return cfg, splits


CASES = [("gqa", i) for i in range(N_CASES)] + [("mla", i) for i in range(N_MLA)]


@pytest.mark.parametrize("kind,i", CASES)
def test_random_shape_end_to_end(kind, i):
    import paper_2604_07815_amd as tls
    cfg, splits = _draw(i) if kind == "gqa" else _draw_mla(i)
    c = H.Case(cfg, backend="host", pad="nan").build_index()
    r = c.decode(attn_splits=splits)
    for (s, g) in c.units():
        H.compare_unit(c, r, s, g)
    assert tls.tls_check_device_error(r["ws"]) == 0
