"""The decode step captured in a HIP graph (torch.cuda.CUDAGraph).

No call on the decode path allocates, copies through the host or clears
memory with a memset node, so a serving loop can capture a step once and
replay it.  Each replay must recompute the whole step from its inputs: the
tests interleave eager calls that reuse the same workspace with different
queries, change the captured query buffer between replays, and compare every
replay with an eager call bit for bit (the kernels are deterministic: no
floating-point atomics, fixed-order reductions)."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

H = pytest.importorskip("gpu_harness")

CASES = {
    # fused two-level selection (bf16, G = 4), default attention splits
    "gqa_bf16": (lambda: synth.config("batched_gqa").replace(batch=2, ctx_lo=5000, ctx_hi=9000, k_b=32, k_t=512,
                                                             clusters=2, seed=301), 0),
    # one 12-wave work-group per unit writes the output (no partials, no merge)
    "gqa_bf16_whole": (lambda: synth.config("batched_gqa").replace(batch=2, ctx_lo=5000, ctx_hi=9000, k_b=32,
                                                                   k_t=512, clusters=2, seed=302), 1),
    "mla_bf16": (lambda: synth.config("mla").replace(batch=2, ctx_lo=4096, ctx_hi=4096, k_b=16, k_t=256,
                                                     clusters=2, seed=303), 0),
    # fp32: separate scoring, normalisation and top-k kernels
    "toy_f32": (lambda: synth.config("toy").replace(batch=2, seed=304), 0),
}


def _bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    return t


class _Step:
    """Static buffers of one decode call (what a captured graph reads and writes)."""

    def __init__(self, c, splits, ws):
        cfg = c.cfg
        self.c, self.splits, self.ws = c, splits, ws
        self.q = c.q.clone()
        self.out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda")
        self.lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda")
        self.bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda")
        self.tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda")

    def __call__(self):
        import paper_2604_07815_amd as tls
        c, cfg = self.c, self.c.cfg
        tls.tls_sparse_decode(c.layout, self.q, c.kv(), c.ctx, c.kmax, c.kmin, c.codes, c.qparams, c.ch,
                              cfg.k_b, cfg.k_t, None, None, self.out, self.lse, self.bids, self.tids, self.ws,
                              attn_splits=self.splits)

    def results(self):
        return [t.clone() for t in (self.out, self.lse, self.bids, self.tids)]


def _assert_same(got, ref, what):
    for name, g, r in zip(("out", "lse", "block_ids", "token_ids"), got, ref):
        assert torch.equal(_bits(g), _bits(r)), f"{what}: {name} differs from the eager call"


@pytest.mark.parametrize("name", list(CASES))
def test_decode_step_graph_replay(name):
    import paper_2604_07815_amd as tls
    make, splits = CASES[name]
    cfg = make()
    c = H.Case(cfg, backend="host", pad="nan").build_index()
    ws = c.workspace()
    qa = c.q.clone()
    qb = torch.flip(c.q, dims=[-1]).contiguous()  # a second query: other blocks and tokens win
    # eager references on the graph's own buffers and workspace
    st = _Step(c, splits, ws)
    ref = {}
    for key, qv in (("a", qa), ("b", qb)):
        st.q.copy_(qv)
        st()
        torch.cuda.synchronize()
        ref[key] = st.results()
    assert not torch.equal(ref["a"][3], ref["b"][3]), "the two queries should select different tokens"
    # the oracle agrees with the eager call (query a)
    st.q.copy_(qa)
    r = dict(out=ref["a"][0], lse=ref["a"][1], bids=ref["a"][2], tids=ref["a"][3], ws=ws)
    for (s, g) in list(c.units())[:3]:
        H.compare_unit(c, r, s, g)
    # capture (after a warm-up on a side stream, as torch requires)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        st()
    # an eager step with its own outputs, sharing the workspace
    other = _Step(c, splits, ws)
    for rep, key in enumerate(("a", "b", "a", "b", "b")):
        st.q.copy_(qa if key == "a" else qb)
        other.q.copy_(qb if key == "a" else qa)
        for t in (st.out, st.lse):
            t.fill_(float("nan"))
        st.tids.fill_(-7)
        st.bids.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        _assert_same(st.results(), ref[key], f"replay {rep} (query {key})")
        other()  # eager work on the same workspace between replays
        torch.cuda.synchronize()
        _assert_same(other.results(), ref["b" if key == "a" else "a"], f"eager call after replay {rep}")
    assert tls.tls_check_device_error(ws) == 0


@pytest.mark.parametrize("name", ["gqa_bf16", "mla_bf16"])
def test_serving_loop_graph_replay(name):
    """One captured serving step, replayed T times: advance the lengths by one,
    append the new token (cache row, block summary, token-index row), decode.
    Every replay equals the same sequence of eager calls on a copy of the state."""
    import paper_2604_07815_amd as tls
    make, splits = CASES[name]
    start, T = 6000, 5
    cfg = make().replace(ctx_lo=start + T, ctx_hi=start + T)
    c = H.Case(cfg, backend="host", pad="nan").build_index()
    new_k = [c.k[:, :, start + t].contiguous() for t in range(T)]
    new_v = [None if cfg.mla else c.v[:, :, start + t].contiguous() for t in range(T)]

    def state():
        K = c.k.clone()
        K[:, :, start:] = 0
        V = None
        if not cfg.mla:
            V = c.v.clone()
            V[:, :, start:] = 0
        ctx = torch.full((cfg.batch,), start, dtype=torch.int32, device="cuda")
        # zero-filled: the builders leave rows past the current lengths untouched
        kmax = torch.zeros_like(c.kmax)
        kmin = torch.zeros_like(c.kmin)
        codes = torch.zeros_like(c.codes)
        qparams = torch.zeros_like(c.qparams)
        tls.tls_build_block_index(c.layout, K, ctx, 0, cfg.max_ctx, kmax, kmin)
        tls.tls_build_token_index(c.layout, K, ctx, c.ch, 0, cfg.max_ctx, codes, qparams)
        return dict(K=K, V=V, ctx=ctx, kmax=kmax, kmin=kmin, codes=codes, qparams=qparams, ws=c.workspace(),
                    k_new=torch.empty_like(new_k[0]), v_new=None if cfg.mla else torch.empty_like(new_v[0]),
                    out=torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=H.torch_dtype(cfg), device="cuda"),
                    lse=torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device="cuda"),
                    bids=torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device="cuda"),
                    tids=torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device="cuda"))

    def serve(S):
        S["ctx"].add_(1)
        tls.tls_append_tokens(c.layout, S["k_new"], S["v_new"], S["ctx"], c.ch, S["K"], S["V"], S["kmax"],
                              S["kmin"], S["codes"], S["qparams"])
        tls.tls_sparse_decode(c.layout, c.q, tls.KV(S["K"], S["V"]), S["ctx"], S["kmax"], S["kmin"], S["codes"],
                              S["qparams"], c.ch, cfg.k_b, cfg.k_t, None, None, S["out"], S["lse"], S["bids"], S["tids"],
                              S["ws"], attn_splits=splits)

    E, G = state(), state()
    torch.cuda.synchronize()
    # capture G's step; the warm-up runs on a throw-away copy so G stays at `start`
    W = state()
    W["k_new"].copy_(new_k[0])
    if W["v_new"] is not None:
        W["v_new"].copy_(new_v[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        serve(W)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    del W
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        serve(G)
    for t in range(T):
        for S in (E, G):
            S["k_new"].copy_(new_k[t])
            if S["v_new"] is not None:
                S["v_new"].copy_(new_v[t])
        serve(E)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(G["ctx"][0]) == start + t + 1
        for key in ("out", "lse", "bids", "tids", "kmax", "kmin", "codes", "qparams", "K"):
            assert torch.equal(_bits(G[key]), _bits(E[key])), f"step {t}: {key} differs from the eager loop"
        if not cfg.mla:
            assert torch.equal(_bits(G["V"]), _bits(E["V"])), f"step {t}: V differs from the eager loop"
    assert tls.tls_check_device_error(G["ws"]) == 0
    assert tls.tls_check_device_error(E["ws"]) == 0
    # after the last append the state holds the case's full context: the oracle agrees
    r = dict(out=G["out"], lse=G["lse"], bids=G["bids"], tids=G["tids"], ws=G["ws"])
    for (s, g) in list(c.units())[:3]:
        H.compare_unit(c, r, s, g)
