"""Seeded synthetic inputs for two-level sparse decode attention.

This module only draws data: queries, keys, values, context lengths, channel
sets and planted high-affinity token positions, with the shapes and value
distributions of the decode workloads (Qwen3-8B-shaped GQA, absorbed-MLA
shaped latents).  It holds none of the operator's arithmetic, so both the CPU
oracle and the GPU path can consume the very same bits without sharing code.

Two back-ends draw the large key/value arrays:

* ``make_host``   - numpy PCG64 on the host (small cases and CPU-only tests);
* ``make_device`` - a seeded ``torch.Generator`` on the GPU (full-size cases);
  the oracle then reads the same bits copied back to the host.

Everything small (queries, context lengths, channel sets, planted positions,
AR(1) query walks) is always drawn on the host with numpy, so both back-ends
agree on it bit for bit.

bf16 data is carried on the host as ``uint16`` bit patterns produced by
round-to-nearest-even from float32.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

__all__ = [
    "DecodeConfig", "CONFIGS", "config", "f32_to_bf16_bits", "bf16_bits_to_f32",
    "to_f64", "draw_ctx_lens", "draw_channels", "draw_plant_starts",
    "draw_queries", "draw_query_walk", "planted_key", "make_host", "make_device",
    "plant_tie_blocks", "plant_tie_tokens", "draw_block_lists",
]


# ----------------------------------------------------------------------------
# bf16 bit conversion (plain IEEE data plumbing)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern (uint16), round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    nan = np.isnan(x)
    rounded = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    if nan.any():
        rounded = np.where(nan, np.uint16(0x7FC0), rounded)
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of a stored array ('f32' floats or 'bf16' bits)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _store(x32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    return np.ascontiguousarray(x32, dtype=np.float32)


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class DecodeConfig:
    name: str
    batch: int
    h_q: int
    h_kv: int
    d_qk: int
    d_v: int
    mla: bool            # absorbed-latent layout: one shared KV row, V = K[:, :d_v]
    dtype: str           # 'f32' | 'bf16'
    ctx_lo: int          # per-sequence context length drawn uniformly in [ctx_lo, ctx_hi]
    ctx_hi: int
    d_c: int             # token-index channels
    k_b: int
    k_t: int
    clusters: int        # planted clusters per (sequence, KV head)
    cluster_len: int = 8
    block: int = 64
    q_std: float = 1.0
    seed: int = 0
    steps: int = 1       # decode steps (AR(1) query walk when > 1)
    rho: float = 0.95

    @property
    def group(self) -> int:
        return self.h_q // self.h_kv

    @property
    def max_ctx(self) -> int:
        return self.ctx_hi

    @property
    def sigma(self) -> float:
        return 1.0 / math.sqrt(self.d_qk)

    def replace(self, **kw) -> "DecodeConfig":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    # toy GQA decode step, fp32; two clusters of 8 planted tokens per KV head
    "toy": DecodeConfig("toy", 1, 8, 2, 128, 128, False, "f32", 4096, 4096,
                        32, 8, 128, clusters=2, seed=1000),
    # Qwen3-8B-shaped GQA layer, one decode step, 48k context
    "qwen3_gqa_48k": DecodeConfig("qwen3_gqa_48k", 1, 32, 8, 128, 128, False, "bf16",
                                  49152, 49152, 32, 128, 2048, clusters=32, seed=2000),
    # batched GQA decode, lengths uniform in [48k, 96k]
    "batched_gqa": DecodeConfig("batched_gqa", 16, 32, 8, 128, 128, False, "bf16",
                                49152, 98304, 32, 128, 2048, clusters=32, seed=3000),
    # absorbed MLA decode: 576-dim score rows (512 latent + 64 rope), value = latent
    "mla": DecodeConfig("mla", 8, 32, 1, 576, 512, True, "bf16", 65536, 65536,
                        128, 128, 2048, clusters=32, q_std=1.0 / 24.0, seed=4000),
    # host-offloaded GQA, 96k context, 64 decode steps with an AR(1) query walk
    "offload_gqa_96k": DecodeConfig("offload_gqa_96k", 32, 32, 8, 128, 128, False, "bf16",
                                    98304, 98304, 32, 128, 2048, clusters=32,
                                    seed=5000, steps=64, rho=0.95),
}


def config(name: str, **overrides) -> DecodeConfig:
    cfg = CONFIGS[name]
    return cfg.replace(**overrides) if overrides else cfg


# ----------------------------------------------------------------------------
# Small draws (always host numpy, shared by both back-ends)
# ----------------------------------------------------------------------------

def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def draw_ctx_lens(cfg: DecodeConfig) -> np.ndarray:
    if cfg.ctx_lo == cfg.ctx_hi:
        return np.full(cfg.batch, cfg.ctx_hi, dtype=np.int32)
    r = _rng(cfg.seed + 100)
    return r.integers(cfg.ctx_lo, cfg.ctx_hi + 1, size=cfg.batch).astype(np.int32)


def draw_channels(cfg: DecodeConfig) -> np.ndarray:
    """Seeded random d_c-subset of the score dimensions, ascending, per KV head.

    Stands in for calibrated channels: with i.i.d. synthetic activations every
    channel has the same expected importance, so a calibration pass would rank
    them at random anyway."""
    r = _rng(cfg.seed + 900)
    out = np.empty((cfg.h_kv, cfg.d_c), dtype=np.int32)
    for h in range(cfg.h_kv):
        out[h] = np.sort(r.choice(cfg.d_qk, size=cfg.d_c, replace=False))
    return out


def draw_calibration(cfg: DecodeConfig, n_cal: int, seed_offset: int = 950):
    """Seeded calibration activations for the channel-importance pass, in
    storage form: q [n_cal][h_q][d_qk], k [n_cal][h_kv][d_qk].

    Unlike the decode workloads, channels differ in scale, as in trained
    models: every (head, channel) has a log-normal scale exp(0.5 z), and each
    KV head has d_c/4 outlier channels, scaled by 6 in its keys and in the
    queries of its group.  Returns (q, k, outliers [h_kv][d_c/4])."""
    r = _rng(cfg.seed + seed_offset)
    G, d = cfg.group, cfg.d_qk
    k_scale = np.exp(0.5 * r.standard_normal((cfg.h_kv, d)))
    q_scale = np.exp(0.5 * r.standard_normal((cfg.h_q, d))) * cfg.q_std
    outliers = np.stack([np.sort(r.choice(d, size=cfg.d_c // 4, replace=False)) for _ in range(cfg.h_kv)])
    for g in range(cfg.h_kv):
        k_scale[g, outliers[g]] *= 6.0
        q_scale[g * G:(g + 1) * G, outliers[g]] *= 6.0
    q = r.standard_normal((n_cal, cfg.h_q, d), dtype=np.float32) * q_scale.astype(np.float32)
    k = r.standard_normal((n_cal, cfg.h_kv, d), dtype=np.float32) * k_scale.astype(np.float32)
    return _store(q.astype(np.float32), cfg.dtype), _store(k.astype(np.float32), cfg.dtype), outliers.astype(np.int32)


def draw_plant_starts(cfg: DecodeConfig, ctx_lens: np.ndarray) -> np.ndarray:
    """Start positions of non-overlapping planted clusters, [batch][h_kv][clusters].

    Stars-and-bars: sorted uniform draws in [0, n - L*c] shifted by L*i give
    uniformly placed, non-overlapping clusters of length L."""
    r = _rng(cfg.seed + 700)
    c, L = cfg.clusters, cfg.cluster_len
    out = np.zeros((cfg.batch, cfg.h_kv, c), dtype=np.int64)
    for s in range(cfg.batch):
        n = int(ctx_lens[s])
        for h in range(cfg.h_kv):
            if c == 0 or n < L * c:
                out[s, h] = -1
                continue
            base = np.sort(r.integers(0, n - L * c + 1, size=c))
            out[s, h] = base + L * np.arange(c)
    return out


def draw_queries(cfg: DecodeConfig) -> np.ndarray:
    """q [batch][h_q][d_qk] in storage form (float32 or bf16 bits)."""
    r = _rng(cfg.seed + 1)
    q = r.standard_normal((cfg.batch, cfg.h_q, cfg.d_qk), dtype=np.float32)
    q *= np.float32(cfg.q_std)
    return _store(q, cfg.dtype)


def draw_query_walk(cfg: DecodeConfig, steps: Optional[int] = None) -> np.ndarray:
    """AR(1) query walk q_t = rho q_{t-1} + sqrt(1-rho^2) eps_t, t = 0..steps.

    Returns [steps+1][batch][h_q][d_qk] in storage form; the float32 state is
    carried between steps and rounded to the storage type per step."""
    steps = cfg.steps if steps is None else steps
    r0 = _rng(cfg.seed + 1)
    state = r0.standard_normal((cfg.batch, cfg.h_q, cfg.d_qk), dtype=np.float32)
    state *= np.float32(cfg.q_std)
    rho = np.float32(cfg.rho)
    nz = np.float32(math.sqrt(1.0 - cfg.rho * cfg.rho) * cfg.q_std)
    out = [_store(state, cfg.dtype)]
    for t in range(1, steps + 1):
        eps = _rng(cfg.seed + 500 + t).standard_normal(state.shape, dtype=np.float32)
        state = rho * state + nz * eps
        out.append(_store(state, cfg.dtype))
    return np.stack(out)


def planted_key(cfg: DecodeConfig, q_store: np.ndarray) -> np.ndarray:
    """Planted key per (sequence, KV head): 4*sqrt(d_qk) times the unit mean
    query direction of the group, [batch][h_kv][d_qk] in storage form."""
    q = to_f64(q_store, cfg.dtype).reshape(cfg.batch, cfg.h_kv, cfg.group, cfg.d_qk)
    mean = q.mean(axis=2)
    norm = np.linalg.norm(mean, axis=-1, keepdims=True)
    norm[norm == 0] = 1.0
    key = 4.0 * math.sqrt(cfg.d_qk) * mean / norm
    return _store(key.astype(np.float32), cfg.dtype)


def _seq_seed(cfg: DecodeConfig, s: int) -> int:
    return cfg.seed + 1 + 17 * (s + 1)


# ----------------------------------------------------------------------------
# Full input sets
# ----------------------------------------------------------------------------

def make_host(cfg: DecodeConfig, pad: str = "nan", q_store: Optional[np.ndarray] = None,
              ctx_lens: Optional[np.ndarray] = None) -> dict:
    """All inputs on the host (numpy).  Keys/values beyond a sequence's length
    are filled with NaN (pad='nan', so a stray read poisons the result) or 0.

    Returns dict(q, k, v, ctx_lens, channels, plant_starts, planted_key);
    k is [b][h_kv][max_ctx][d_qk]; v is [b][h_kv][max_ctx][d_v] or None (MLA).
    `ctx_lens` overrides the drawn context lengths."""
    ctx = draw_ctx_lens(cfg) if ctx_lens is None else np.asarray(ctx_lens, dtype=np.int32)
    ch = draw_channels(cfg)
    q = draw_queries(cfg) if q_store is None else q_store
    starts = draw_plant_starts(cfg, ctx)
    pk = planted_key(cfg, q)
    fill = np.float32(np.nan if pad == "nan" else 0.0)
    T = cfg.max_ctx
    k32 = np.full((cfg.batch, cfg.h_kv, T, cfg.d_qk), fill, dtype=np.float32)
    v32 = None if cfg.mla else np.full((cfg.batch, cfg.h_kv, T, cfg.d_v), fill, dtype=np.float32)
    for s in range(cfg.batch):
        n = int(ctx[s])
        r = _rng(_seq_seed(cfg, s))
        k32[s, :, :n] = r.standard_normal((cfg.h_kv, n, cfg.d_qk), dtype=np.float32)
        if v32 is not None:
            v32[s, :, :n] = r.standard_normal((cfg.h_kv, n, cfg.d_v), dtype=np.float32)
    k = _store(k32, cfg.dtype)
    del k32
    v = None if v32 is None else _store(v32, cfg.dtype)
    for s in range(cfg.batch):
        for h in range(cfg.h_kv):
            for st in starts[s, h]:
                if st >= 0:
                    k[s, h, st:st + cfg.cluster_len] = pk[s, h]
    return dict(q=q, k=k, v=v, ctx_lens=ctx, channels=ch, plant_starts=starts,
                planted_key=pk)


def make_device(cfg: DecodeConfig, device="cuda", pad: str = "zero",
                q_store: Optional[np.ndarray] = None, ctx_lens: Optional[np.ndarray] = None) -> dict:
    """All inputs as torch tensors on `device`; the large K/V arrays are drawn
    with a seeded torch.Generator there (one generator per sequence)."""
    import torch

    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    ctx = draw_ctx_lens(cfg) if ctx_lens is None else np.asarray(ctx_lens, dtype=np.int32)
    ch = draw_channels(cfg)
    q = draw_queries(cfg) if q_store is None else q_store
    starts = draw_plant_starts(cfg, ctx)
    pk = planted_key(cfg, q)
    fill = float("nan") if pad == "nan" else 0.0
    T = cfg.max_ctx
    k = torch.empty((cfg.batch, cfg.h_kv, T, cfg.d_qk), dtype=tdt, device=device)
    v = None if cfg.mla else torch.empty((cfg.batch, cfg.h_kv, T, cfg.d_v), dtype=tdt, device=device)
    g = torch.Generator(device=device)
    for s in range(cfg.batch):
        n = int(ctx[s])
        g.manual_seed(_seq_seed(cfg, s))
        k[s, :, :n] = torch.randn((cfg.h_kv, n, cfg.d_qk), generator=g, device=device,
                                  dtype=torch.float32).to(tdt)
        k[s, :, n:] = fill
        if v is not None:
            v[s, :, :n] = torch.randn((cfg.h_kv, n, cfg.d_v), generator=g, device=device,
                                      dtype=torch.float32).to(tdt)
            v[s, :, n:] = fill
    pk_t = host_to_torch(pk, cfg.dtype).to(device)
    for s in range(cfg.batch):
        for h in range(cfg.h_kv):
            for st in starts[s, h]:
                if st >= 0:
                    k[s, h, st:st + cfg.cluster_len] = pk_t[s, h]
    return dict(q=host_to_torch(q, cfg.dtype).to(device), k=k, v=v,
                ctx_lens=torch.from_numpy(ctx).to(device),
                channels=torch.from_numpy(ch).to(device),
                plant_starts=starts, planted_key=pk, q_host=q,
                ctx_host=ctx, channels_host=ch)


# ----------------------------------------------------------------------------
# Inputs with exact ties at the selection cuts
# ----------------------------------------------------------------------------

def plant_tie_blocks(cfg: DecodeConfig, k: np.ndarray, ctx_lens: np.ndarray, n_hi: int, n_dup: int,
                     hi_scale: float = 5.0, dup_scale: float = 3.0, seed_offset: int = 800):
    """Per (sequence, KV head): n_hi blocks whose rows are the drawn rows
    times hi_scale, and n_dup blocks that are byte-identical copies of one
    block whose rows are the drawn rows times dup_scale, at seeded distinct
    positions among the sequence's full blocks.  Identical blocks have
    identical summaries, so any block budget between n_hi and n_hi + n_dup
    cuts through a group of exactly equal block scores.

    k: storage-form [b][h_kv][T][d] (modified in place).  Returns
    (hi [b][h_kv][n_hi], dup [b][h_kv][n_dup]), ascending block ids."""
    r = _rng(cfg.seed + seed_offset)
    B = cfg.block
    hi = np.zeros((cfg.batch, cfg.h_kv, n_hi), dtype=np.int64)
    dup = np.zeros((cfg.batch, cfg.h_kv, n_dup), dtype=np.int64)
    for s in range(cfg.batch):
        full = int(ctx_lens[s]) // B
        assert full >= n_hi + n_dup, "not enough full blocks for the tie layout"
        for g in range(cfg.h_kv):
            pick = r.choice(full, size=n_hi + n_dup, replace=False)
            hi[s, g] = np.sort(pick[:n_hi])
            dup[s, g] = np.sort(pick[n_hi:])
            rows = k[s, g]
            for b in hi[s, g]:
                x = to_f64(rows[b * B:(b + 1) * B], cfg.dtype) * hi_scale
                rows[b * B:(b + 1) * B] = _store(x.astype(np.float32), cfg.dtype)
            t0 = int(dup[s, g, 0])
            tmpl = _store((to_f64(rows[t0 * B:(t0 + 1) * B], cfg.dtype) * dup_scale).astype(np.float32), cfg.dtype)
            for b in dup[s, g]:
                rows[b * B:(b + 1) * B] = tmpl
    return hi, dup


def draw_block_lists(cfg: DecodeConfig, ctx_lens: np.ndarray, k_b: int, seed_offset: int = 820) -> np.ndarray:
    """A seeded ascending list of k_b distinct blocks per (sequence, KV head),
    [b][h_kv][k_b] (a given block selection for the token stage)."""
    r = _rng(cfg.seed + seed_offset)
    out = np.zeros((cfg.batch, cfg.h_kv, k_b), dtype=np.int32)
    for s in range(cfg.batch):
        m = -(-int(ctx_lens[s]) // cfg.block)
        for g in range(cfg.h_kv):
            out[s, g] = np.sort(r.choice(m, size=k_b, replace=False))
    return out


def plant_tie_tokens(cfg: DecodeConfig, q_store: np.ndarray, k: np.ndarray, ctx_lens: np.ndarray,
                     channels: np.ndarray, blocks: Optional[np.ndarray], n_a: int, n_b: int, dot_a: float,
                     dot_b: float, seed_offset: int = 850):
    """Per (sequence, KV head): n_a tokens with the key dot_a * w and n_b
    tokens with the key dot_b * w, where w is the least-norm vector on the
    channels of the head's index set C (zero elsewhere) whose dot product
    with every query of the group is 1, so that every head sees them with
    the dot products dot_a and dot_b (up to the storage rounding).  Positions are
    seeded, distinct, valid tokens of `blocks[s][g]` (every block when None).
    Rows of one kind are byte-identical, so a token budget between n_a and
    n_a + n_b cuts through a group of exactly equal approximate scores.

    k: storage-form [b][h_kv][T][d] (modified in place).  Returns
    (pos_a [b][h_kv][n_a], pos_b [b][h_kv][n_b]), ascending positions."""
    r = _rng(cfg.seed + seed_offset)
    B = cfg.block
    q = to_f64(q_store, cfg.dtype).reshape(cfg.batch, cfg.h_kv, cfg.group, cfg.d_qk)
    pa = np.zeros((cfg.batch, cfg.h_kv, n_a), dtype=np.int64)
    pb = np.zeros((cfg.batch, cfg.h_kv, n_b), dtype=np.int64)
    for s in range(cfg.batch):
        n = int(ctx_lens[s])
        for g in range(cfg.h_kv):
            if blocks is None:
                cand = np.arange(n)
            else:
                cand = np.array([b * B + o for b in blocks[s, g] if b >= 0 for o in range(B) if b * B + o < n])
            pick = r.choice(cand, size=n_a + n_b, replace=False)
            pa[s, g] = np.sort(pick[:n_a])
            pb[s, g] = np.sort(pick[n_a:])
            w = np.zeros(cfg.d_qk)
            C = channels[g]
            w[C] = np.linalg.pinv(q[s, g][:, C]) @ np.ones(cfg.group)
            rows = k[s, g]
            rows[pa[s, g]] = _store((dot_a * w).astype(np.float32), cfg.dtype)
            rows[pb[s, g]] = _store((dot_b * w).astype(np.float32), cfg.dtype)
    return pa, pb


def host_to_torch(arr: np.ndarray, dtype: str):
    """Storage-form numpy array -> CPU torch tensor of the storage dtype."""
    import torch

    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))


def torch_to_f64(t) -> np.ndarray:
    """Exact float64 values of a torch tensor (any device)."""
    import torch

    return t.detach().to("cpu").to(torch.float64).numpy()
