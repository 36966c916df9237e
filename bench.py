"""Benchmark of the two-level sparse decode step on one MI355X.

One step = one tls_sparse_decode call over the whole batch: block scoring,
top-K_b, token scoring over the selected blocks, top-K_t, and attention over
the gathered K/V (the index build is prefill and is timed separately).
Inputs are synthetic, generated on the GPU and resident in HBM before the
timed region.  Several byte-identical copies of the layer are rotated so the
256 MB Infinity Cache cannot serve a step from the previous one.

Prints ONE JSON line (see README/DESIGN for the fields).
"""
from __future__ import annotations

import argparse
import ctypes
import gc
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "two-level sparse decode µs/layer-step at 96k ctx + achieved HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0
STAGES = ["block_score", "block_topk", "token_score", "token_norm", "token_topk", "attention", "merge"]

WORKLOADS = {
    # 96k-context GQA decode of the offloaded-KV workload shape, K/V resident in HBM
    "gqa_b32_ctx96k": ("offload_gqa_96k", dict()),
    "gqa_b16_ctx48k_96k": ("batched_gqa", dict()),
    "gqa_b1_ctx48k": ("qwen3_gqa_48k", dict()),
    "mla_b8_ctx64k": ("mla", dict()),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="gqa_b32_ctx96k", choices=sorted(WORKLOADS))
    ap.add_argument("--copies", type=int, default=0, help="layer copies rotated (0: auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-modes", action="store_true", help="skip timing the single-level operators")
    ap.add_argument("--offload", action="store_true",
                    help="also run the offloaded-KV schedule of the 96k workload (full K/V in pinned host memory, "
                         "lagged selection, side-stream prefetch over PCIe) for a non-default --workload "
                         "(the default workload always reports it under 'workloads')")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the batched 48k-96k step and the offloaded schedule reported under 'workloads'")
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + steps of the decode only (for rocprofv3), print nothing else")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="with --profile-only: first copy a 1 GiB buffer three times (the known-size "
                         "reference for the PMC byte counters)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc csv runs (FETCH_SIZE, WRITE_SIZE) of "
                         "'--profile-only --calibrate-copy' into the committed traffic summary, then exit")
    return ap.parse_args()


# ----------------------------------------------------------------------------
# raw HIP events (the library records them on the stream it launches on)
# ----------------------------------------------------------------------------
class HipEvents:
    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            out.append(e.value)
        return out

    def elapsed_ms(self, a, b):
        self.hip.hipEventSynchronize(ctypes.c_void_p(b))
        t = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(t), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(t.value)

    def destroy(self, evs):
        for e in evs:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))

    def stream_wait(self, stream, e):
        """Makes `stream` (a torch stream) wait for event `e`."""
        if self.hip.hipStreamWaitEvent(ctypes.c_void_p(stream.cuda_stream), ctypes.c_void_p(e), 0) != 0:
            raise RuntimeError("hipStreamWaitEvent failed")


def algorithmic_bytes(cfg, ctx, bids, e):
    """Bytes the step must move: all block-summary rows, the token-index rows
    of the candidates, the gathered K/V rows of the selected tokens, q and out."""
    import numpy as np
    B = cfg.block
    blk = 0
    tok = 0
    kv = 0
    idx_row = cfg.d_c // 2 + 8 * (cfg.d_c // 32)
    kv_row = cfg.d_qk * e if cfg.mla else (cfg.d_qk + cfg.d_v) * e
    bids = bids.reshape(cfg.batch, cfg.h_kv, -1)
    for s in range(cfg.batch):
        n = int(ctx[s])
        m = -(-n // B)
        for g in range(cfg.h_kv):
            sel = bids[s, g][bids[s, g] >= 0]
            cand = int(sum(min(B, n - int(b) * B) for b in sel))
            blk += m * 2 * cfg.d_qk * e
            tok += cand * idx_row
            kv += min(cfg.k_t, cand) * kv_row
    qo = cfg.batch * cfg.h_q * (cfg.d_qk + cfg.d_v) * e
    return dict(block_index=blk, token_index=tok, gathered_kv=kv, q_out=qo, total=blk + tok + kv + qo)


# Inputs of the CPU baseline, set in the parent before the worker pool is
# forked, so that every worker reads them without a copy through a pipe.
_CPU = {}


def cpu_baseline(units, cores):
    """Time the oracle's decode step (as it stands) on the given units, one
    task per unit on `cores` forked worker processes.  Each worker builds its
    unit's float64 inputs and the prefill-side indices untimed, then times
    decode_unit alone.  Returns (per-unit decode seconds, per-unit index
    build seconds, wall seconds of the pool)."""
    import concurrent.futures
    import multiprocessing as mp
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with concurrent.futures.ProcessPoolExecutor(max_workers=cores, mp_context=ctx,
                                                initializer=_cpu_worker_init) as ex:
        res = list(ex.map(_cpu_unit_timed, units, chunksize=max(1, len(units) // (4 * cores))))
    wall = time.perf_counter() - t0
    return [r[0] for r in res], [r[1] for r in res], wall, [r[2] for r in res]


def _cpu_worker_init():
    try:
        import threadpoolctl
        threadpoolctl.threadpool_limits(1)
    except Exception:
        pass


def _cpu_unit_inputs(u):
    import synth
    D = _CPU
    cfg = D["cfg"]
    s, g = divmod(u, cfg.h_kv)
    n = int(D["ctx"][s])
    qg = synth.to_f64(D["q"], cfg.dtype)[s, g * cfg.group:(g + 1) * cfg.group]
    Ku = synth.to_f64(D["k"][s, g, :n], cfg.dtype)
    Vu = Ku[:, :cfg.d_v] if cfg.mla else synth.to_f64(D["v"][s, g, :n], cfg.dtype)
    return cfg, qg, Ku, Vu, n, D["channels"][g]


def _cpu_unit_timed(u):
    from oracle import tls_oracle as O
    cfg, qg, Ku, Vu, n, ch = _cpu_unit_inputs(u)
    t0 = time.perf_counter()
    summ = O.block_summaries(Ku, n, cfg.block)
    index = O.token_index(Ku, n, ch)
    t_index = time.perf_counter() - t0
    t0 = time.perf_counter()
    res = O.decode_unit(qg, Ku, Vu, n, ch, cfg.k_b, cfg.k_t, cfg.block, cfg.sigma, index=index, summaries=summ)
    t_dec = time.perf_counter() - t0
    gpu = _CPU.get("gpu")
    return t_dec, t_index, (_unit_parity(O, u, cfg, qg, Ku, Vu, n, ch, index, res, gpu) if gpu else None)


def _unit_parity(O, u, cfg, qg, Ku, Vu, n, ch, index, res, gpu):
    """The GPU step's result for unit u against the oracle's, by the
    selection rule of the parity tests: equal id sets except ids whose oracle
    score lies within 1e-3 relative of the oracle's k-th score; a block swap
    is followed by the oracle's token stage on the GPU's blocks, any swap by
    the oracle's attention on the GPU's tokens; the output within the dtype's
    tolerance.  (After the timed decode; not part of the baseline.)"""
    import numpy as np
    s, g = divmod(u, cfg.h_kv)
    rel = 1e-3
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-5

    def ids(row):
        k = int((row >= 0).sum())
        ok = bool(np.all(row[:k] >= 0) and np.all(row[k:] == -1) and np.all(np.diff(row[:k]) > 0))
        return row[:k], ok

    def swaps(got, want, score):
        gs, ws = set(int(x) for x in got), set(int(x) for x in want)
        diff = gs ^ ws
        if len(gs) != len(ws):
            return len(diff), False
        if not diff:
            return 0, True
        kth = min(score(i) for i in ws)
        return len(diff) // 2, all(abs(score(i) - kth) <= rel * abs(kth) for i in diff)

    M, ok_m = ids(gpu["bids"][s, g])
    S, ok_s = ids(gpu["tids"][s, g])
    sb, ok_b = swaps(M, res["block_ids"], lambda i: float(res["block_scores"][i]))
    tok = res
    if sb:
        S_ref, alpha, cand = O.select_tokens(qg, ch, index[0], index[1], M, n, cfg.block, cfg.k_t, cfg.sigma)
        tok = dict(token_ids=S_ref, alpha=alpha, cand=cand)
    pos = {int(t): i for i, t in enumerate(tok["cand"])}
    if not all(int(t) in pos for t in S):
        st, ok_t = len(S), False
    else:
        st, ok_t = swaps(S, tok["token_ids"], lambda t: float(tok["alpha"][pos[int(t)]]))
    o_ref, lse_ref = (O.sparse_attention(qg, Ku, Vu, S, cfg.sigma) if (sb or st) else (res["out"], res["lse"]))
    G = cfg.group
    o = gpu["out"][s, g * G:(g + 1) * G].astype(np.float64)
    lse = gpu["lse"][s, g * G:(g + 1) * G].astype(np.float64)
    err_o = float(np.max(np.abs(o - o_ref))) if o.size else 0.0
    fin = np.isfinite(lse_ref)
    err_l = float(np.max(np.abs(lse[fin] - lse_ref[fin]))) if fin.any() else 0.0
    within = bool(np.all(np.abs(o - o_ref) <= tol + tol * np.abs(o_ref)) and
                  np.all(np.abs(lse[fin] - lse_ref[fin]) <= tol + tol * np.abs(lse_ref[fin])) and
                  np.array_equal(np.isfinite(lse), fin))
    want = set(int(x) for x in res["token_ids"])
    recall = len(want & set(int(x) for x in S)) / len(want) if want else 1.0
    return dict(block_swaps=sb, token_swaps=st, ok=bool(ok_m and ok_s and ok_b and ok_t and within),
                err_out=err_o, err_lse=err_l, recall=recall)


ATTN_SOURCES = ["attention_gqa.hip", "attn_gqa_mfma.hpp", "attn_common.hpp", "common.hpp", "kernels.hpp"]
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "attention_gqa_b32_ctx96k_traffic.json")
COPY_BYTES = 1 << 30


def attention_source_hash():
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2604_07815_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def pmc_summary(fetch_dir, write_dir):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the attention
    kernel and of the 1 GiB reference copy, from the csv output of two
    rocprofv3 --pmc runs of the same command; the copy (the dispatches that
    write 1 GiB, found in the WRITE_SIZE run; the same dispatch ids in the
    FETCH_SIZE run) converts counter KiB to bytes."""
    import csv
    import glob

    def dispatches(d, counter):
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit(f"no counter_collection.csv under {d}")
        vals, names = {}, {}
        for f in files:
            for row in csv.DictReader(open(f)):
                if row.get("Counter_Name") != counter:
                    continue
                i = int(row["Dispatch_Id"])
                vals[i] = vals.get(i, 0.0) + float(row["Counter_Value"])
                names[i] = row["Kernel_Name"]
        return vals, names

    wv, wn = dispatches(write_dir, "WRITE_SIZE")
    fv, fn = dispatches(fetch_dir, "FETCH_SIZE")
    true_kib = COPY_BYTES / 1024
    ref = [i for i, v in wv.items() if "copy" in wn[i].lower() and abs(v - true_kib) < 0.01 * true_kib]
    if not ref or any(i not in fv or fn[i] != wn[i] for i in ref):
        raise SystemExit(f"reference copies not found consistently ({len(ref)})")
    out = {}
    for counter, vals, names in (("FETCH_SIZE", fv, fn), ("WRITE_SIZE", wv, wn)):
        attn = [v for i, v in vals.items() if "attn_gqa_mfma_kernel" in names[i]]
        copy_kib = sum(vals[i] for i in ref) / len(ref)
        attn_kib = sum(attn) / len(attn)
        scale = true_kib / copy_kib
        out[counter] = {"attention_kib_per_dispatch": round(attn_kib, 1), "reference_copy_kib": round(copy_kib, 1),
                        "reference_true_kib": true_kib, "scale": round(scale, 4),
                        "attention_bytes_per_launch": round(attn_kib * 1024 * scale), "dispatches": len(attn)}
    traffic = out["FETCH_SIZE"]["attention_bytes_per_launch"] + out["WRITE_SIZE"]["attention_bytes_per_launch"]
    rec = {"kernel": "attn_gqa_mfma_kernel<128, 4, 12, 176, true>", "workload": "gqa_b32_ctx96k",
           "kernel_src_sha256": attention_source_hash(), "traffic_bytes_per_launch": traffic,
           "counters": out}
    json.dump(rec, open(TRAFFIC_JSON, "w"), indent=1)
    print(json.dumps(rec))


def traffic_from_profiles(kernel_src_hash):
    """HBM traffic per launch of the dominant kernel from committed PMC runs,
    valid only while the kernel source is unchanged."""
    p = TRAFFIC_JSON
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("kernel_src_sha256") != kernel_src_hash:
        return None
    return d.get("traffic_bytes_per_launch")


def cpu_baseline_record(cfg, d, np, torch, gpu=None):
    """The oracle's decode step (block scores, top-K_b, token scores over the
    candidates, top-K_t, attention; float64 NumPy, prebuilt indices) over
    every (sequence, KV head) unit of the workload's step, on the host
    cores: the value is the summed per-unit decode time divided by the
    worker count (the step's time with the units spread evenly).  With
    `gpu` (host copies of one GPU step's out, lse, block and token ids on
    the same inputs), each worker also compares its unit with the GPU's
    after timing it; returns (baseline record, parity record or None)."""
    def host(t):
        if t is None:
            return None
        return t.view(torch.int16).cpu().numpy().view(np.uint16) if cfg.dtype == "bf16" else t.cpu().numpy()
    _CPU.update(cfg=cfg, q=d["q_host"], k=host(d["k"]), v=host(d["v"]), ctx=d["ctx_host"],
                channels=d["channels_host"], gpu=gpu)
    units = list(range(cfg.batch * cfg.h_kv))
    cores = max(1, min(16, len(os.sched_getaffinity(0)), len(units)))
    dec, idx, wall, par = cpu_baseline(units, cores)
    # one unit on one core in this process, nothing else running
    _CPU["gpu"] = None
    one = min(_cpu_unit_timed(units[0])[0] for _ in range(3))
    _CPU.clear()
    parity = None
    if gpu is not None:
        parity = {
            "units": len(par),
            "all_within_rule": all(p["ok"] for p in par),
            "units_with_block_swap": sum(p["block_swaps"] > 0 for p in par),
            "units_with_token_swap": sum(p["token_swaps"] > 0 for p in par),
            "max_abs_err_out": float(f"{max(p['err_out'] for p in par):.3g}"),
            "max_abs_err_lse": float(f"{max(p['err_lse'] for p in par):.3g}"),
            "token_recall_min": round(min(p["recall"] for p in par), 5),
            "token_recall_mean": round(float(np.mean([p["recall"] for p in par])), 5),
            "rule": "every unit of one GPU step against the oracle on the same inputs: block and token id sets "
                    "equal except near ties (oracle score within 1e-3 relative of its k-th), a swap followed "
                    "by the oracle's later stages on the GPU's selection; out and lse within "
                    + ("2e-2" if cfg.dtype == "bf16" else "1e-5") + " abs+rel; recall = |S_gpu & S_oracle| / |S_oracle|",
        }
    value_s = sum(dec) / cores
    ratio = value_s / (one * len(units) / cores)
    if not 0.5 <= ratio <= 2.0:
        print(f"bench.py: cpu_baseline is {ratio:.2f}x the single-core estimate", file=sys.stderr)
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": round(value_s * 1e6, 1), "unit": "µs/layer-step", "cores": cores, "kind": "oracle",
        "sample": f"all {len(units)} (sequence, KV head) units of one step: the float64 NumPy oracle's decode_unit "
                  f"on prebuilt indices, one task per unit on {cores} forked worker processes (inputs inherited, "
                  f"not pickled); value = summed per-unit decode time / {cores}",
        "cpu_model": cpu_model,
        "unit_decode_s_mean": round(float(np.mean(dec)), 5),
        "single_core_s_per_unit": round(one, 5),
        "value_vs_single_core_estimate": round(ratio, 3),
        "index_build_s_per_unit": round(float(np.mean(idx)), 4),
        "pool_wall_s": round(wall, 2),
    }, parity


def prefill_timing(tls, torch, cfg, layout, d, L, e, reps=3):
    """Prefill-side calls on the full workload, HIP events on the launch
    stream, median of `reps` after one warm call: the two index builders over
    the resident K, and the fused prefill (K/V rows from the token-major
    prefill output into the cache, both indices from the same read).  The
    fused call rewrites the cache with the bytes it already holds."""
    import numpy as np
    ctx, ch, T = d["ctx_lens"], d["channels"], cfg.max_ctx
    n_tok = int(d["ctx_host"].astype(np.int64).sum()) * cfg.h_kv
    m_tok = int(sum(-(-int(n) // cfg.block) for n in d["ctx_host"])) * cfg.h_kv
    idx_out = m_tok * 2 * cfg.d_qk * e + n_tok * (cfg.d_c // 2 + 8 * (cfg.d_c // 32))
    row_kv = cfg.d_qk * e + (0 if cfg.mla else cfg.d_v * e)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(f):
        f()
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            start.record()
            f()
            stop.record()
            torch.cuda.synchronize()
            ts.append(start.elapsed_time(stop))
        return float(np.median(ts))

    def build():
        tls.tls_build_block_index(layout, L["k"], ctx, 0, T, L["kmax"], L["kmin"])
        tls.tls_build_token_index(layout, L["k"], ctx, ch, 0, T, L["codes"], L["qparams"])

    build_ms = timed(build)
    k_src = L["k"].transpose(1, 2).contiguous()
    v_src = None if cfg.mla else L["v"].transpose(1, 2).contiguous()

    def fused():
        tls.tls_prefill_kv(layout, k_src, v_src, ctx, ch, 0, T, L["k"], L["v"], L["kmax"], L["kmin"], L["codes"],
                           L["qparams"])

    fused_ms = timed(fused)
    del k_src, v_src
    torch.cuda.empty_cache()
    build_bytes = 2 * n_tok * cfg.d_qk * e + idx_out       # each builder reads K once
    fused_bytes = 2 * n_tok * row_kv + idx_out             # prefill rows in, cache rows out, indices out
    return {
        "index_build_ms": round(build_ms, 3),
        "index_build_GBps": round(build_bytes / (build_ms * 1e-3) / 1e9, 1),
        "prefill_kv_ms": round(fused_ms, 3),
        "prefill_kv_GBps": round(fused_bytes / (fused_ms * 1e-3) / 1e9, 1),
        "note": "index_build = tls_build_block_index + tls_build_token_index over the whole context (K read by "
                "each); prefill_kv = tls_prefill_kv: K/V rows from the token-major prefill output written to the "
                "cache and both indices built from the same read; bytes = reads + writes of valid rows",
    }


def calibration_timing(tls, torch, cfg, layout, dev, n_cal=16384, reps=5):
    """The channel-calibration pass (Sec. 4.1) over n_cal token rows of the
    workload's head shapes (random activations generated on the GPU; the
    paper does not state the size of its calibration set): the per-channel
    maxima over all query and key heads, then the scores and top-d_c
    channels.  HIP events on the launch stream, median of `reps`."""
    import numpy as np
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    g = torch.Generator(device=dev).manual_seed(cfg.seed + 950)
    q = torch.randn((n_cal, cfg.h_q, cfg.d_qk), generator=g, device=dev).to(dt)
    k = torch.randn((n_cal, cfg.h_kv, cfg.d_qk), generator=g, device=dev).to(dt)
    qa = torch.empty((cfg.h_q, cfg.d_qk), dtype=torch.float32, device=dev)
    ka = torch.empty((cfg.h_kv, cfg.d_qk), dtype=torch.float32, device=dev)
    ch = torch.empty((cfg.h_kv, cfg.d_c), dtype=torch.int32, device=dev)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(f):
        f()
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            a.record()
            f()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    absmax_ms = timed(lambda: tls.tls_calibrate_absmax(layout, q, k, qa, ka))
    select_ms = timed(lambda: tls.tls_calibrate_channels(layout, qa, ka, ch))
    nbytes = n_cal * (cfg.h_q + cfg.h_kv) * cfg.d_qk * q.element_size()
    return {"n_cal_rows": n_cal, "absmax_ms": round(absmax_ms, 3),
            "absmax_GBps": round(nbytes / (absmax_ms * 1e-3) / 1e9, 1), "select_us": round(select_ms * 1e3, 1)}


def offload_schedule(tls, synth, torch, np):
    """The offloaded KV tier of the 96k workload (Sec. 4.2), as a serving loop:
    K/V of every sequence in pinned host memory, block and token indices and
    a pool of 2*K_b block slots per unit in HBM.  Per step t of the AR(1)
    query walk, one lagged decode call on the main stream selects M_t from
    q_t and, in the same call, selects tokens from M_{t-1} and attends over
    the pool; once M_t is complete (the call's stage event after token
    selection) the side stream brings T_t = M_t minus the resident set into
    the pool over PCIe, overlapping the call's attention; the main stream
    waits for the transfer before step t+1.  Reported per step (median over
    the walk): step wall time, decode time, transfer time and bytes."""
    cfg = synth.config("offload_gqa_96k")
    dev = torch.device("cuda", 0)
    walk = synth.draw_query_walk(cfg)
    d = synth.make_device(cfg, device=dev, pad="zero", q_store=walk[0])
    dt = torch.bfloat16
    layout = tls.make_layout(cfg.batch, cfg.h_q, cfg.h_kv, cfg.d_qk, cfg.d_v, cfg.max_ctx, index_channels=cfg.d_c,
                             block_size=cfg.block, dtype=tls.DTYPE_BF16)
    m_max = -(-cfg.max_ctx // cfg.block)
    kmax = torch.empty((cfg.batch, cfg.h_kv, m_max, cfg.d_qk), dtype=dt, device=dev)
    kmin = torch.empty_like(kmax)
    codes = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 2), dtype=torch.uint8, device=dev)
    qparams = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 32, 2), dtype=torch.float32, device=dev)
    ctx, ch = d["ctx_lens"], d["channels"]
    B, units, K_b = cfg.block, cfg.batch * cfg.h_kv, cfg.k_b
    n_slots = 2 * K_b
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    ws = tls.alloc_workspace(layout, K_b, cfg.k_t, device=dev)
    qs = [synth.host_to_torch(walk[t], cfg.dtype).to(dev) for t in range(walk.shape[0])]
    M = [torch.empty((cfg.batch, cfg.h_kv, K_b), dtype=torch.int32, device=dev) for _ in range(2)]
    # prefill flow (Fig. 2): the prompt's K/V rows (token-major) go to the HBM
    # cache with both indices built on the way; the final prompt query selects
    # the initial residency; the cache is offloaded to pinned host memory on a
    # side stream, and the HBM cache is then released
    # the context grows by one token per sequence per step (from n - T to n):
    # the rows the walk appends are kept aside; the prompt is the rest
    T_steps = walk.shape[0] - 1
    n0 = cfg.max_ctx - T_steps
    k_future = d["k"][:, :, n0:].contiguous()
    v_future = d["v"][:, :, n0:].contiguous()
    ctx = torch.full_like(ctx, n0)
    k_src = d["k"][:, :, :n0].transpose(1, 2).contiguous()
    v_src = d["v"][:, :, :n0].transpose(1, 2).contiguous()
    K, V = d.pop("k"), d.pop("v")
    p0, p1 = ev(), ev()
    p0.record(main)
    tls.tls_prefill_kv(layout, k_src, v_src, ctx, ch, 0, n0, K, V, kmax, kmin, codes, qparams)
    p1.record(main)
    del k_src, v_src
    host_k = torch.empty(K.shape, dtype=dt, pin_memory=True)
    host_v = torch.empty(V.shape, dtype=dt, pin_memory=True)
    pool_k = torch.zeros((units, n_slots, B, cfg.d_qk), dtype=dt, device=dev)
    pool_v = torch.zeros((units, n_slots, B, cfg.d_v), dtype=dt, device=dev)
    slot_map = torch.empty((units, m_max), dtype=torch.int32, device=dev)
    slot_owner = torch.empty((units, n_slots), dtype=torch.int32, device=dev)
    tcount = torch.zeros(units, dtype=torch.int32, device=dev)
    o0, o1, r0, r1 = ev(), ev(), ev(), ev()
    tls.tls_select_blocks(layout, qs[0], kmax, kmin, ctx, K_b, M[0], None, ws)
    r0.record(main)
    tls.tls_init_residency(layout, K, V, ctx, M[0], K_b, pool_k, pool_v, n_slots, slot_map, slot_owner, ws)
    r1.record(main)
    # the offload starts once the residency copy is done: copy work-groups that
    # share a compute unit with work-groups stalled on PCIe stores slow down
    side.wait_stream(main)
    o0.record(side)
    tls.tls_offload_kv(layout, K, V, ctx, 0, cfg.max_ctx, host_k, host_v, stream=side)
    o1.record(side)
    torch.cuda.synchronize()
    kv_bytes = 2 * cfg.batch * cfg.h_kv * n0 * cfg.d_qk * K.element_size()  # the rows offloaded
    prefill_rec = dict(prefill_kv_ms=p0.elapsed_time(p1), offload_ms=o0.elapsed_time(o1),
                       residency_ms=r0.elapsed_time(r1))
    del K, V, d
    torch.cuda.empty_cache()
    kv = tls.KV(pool_k, pool_v, slot_map, n_slots)
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dt, device=dev)
    hev = HipEvents()
    sev = hev.create(tls.NUM_STAGE_EVENTS)
    rec = []
    for t in range(1, walk.shape[0]):
        M_prev, M_t = M[(t - 1) % 2], M[t % 2]
        e0, e_app, e_dec, e1, p0, p1 = ev(), ev(), ev(), ev(), ev(), ev()
        k_new, v_new = k_future[:, :, t - 1].contiguous(), v_future[:, :, t - 1].contiguous()
        e0.record(main)
        ctx += 1  # the token generated by the previous step joins the context
        tls.tls_append_tokens(layout, k_new, v_new, ctx, ch, host_k, host_v, kmax, kmin, codes, qparams, pool=kv)
        e_app.record(main)
        tls.tls_sparse_decode(layout, qs[t], kv, ctx, kmax, kmin, codes, qparams, ch, K_b, cfg.k_t, M_prev, None,
                              out, None, M_t, None, ws, stage_events=sev, mode=tls.MODE_LAGGED)
        e_dec.record(main)
        hev.stream_wait(side, sev[5])  # M_t is complete after the call's token selection
        p0.record(side)
        tls.tls_prefetch_blocks(layout, host_k, host_v, ctx, M_t, M_prev, K_b, pool_k, pool_v, n_slots, slot_map,
                                slot_owner, tcount, ws, stream=side)
        p1.record(side)
        main.wait_event(p1)
        e1.record(main)
        e1.synchronize()
        moved = int(tcount.sum().item())
        rec.append(dict(wall=e0.elapsed_time(e1) * 1e3, append=e0.elapsed_time(e_app) * 1e3,
                        select=hev.elapsed_ms(sev[0], sev[5]) * 1e3, decode=e_app.elapsed_time(e_dec) * 1e3,
                        xfer=p0.elapsed_time(p1) * 1e3, blocks=moved))
    hev.destroy(sev)
    # the same lagged decode call (block selection of M_t, token selection
    # from the resident blocks of M_{t-1} and attention over the pool) with no
    # transfer running
    M_last = M[(walk.shape[0] - 1) % 2]
    M_tmp = torch.empty_like(M_last)

    def quiet_call():
        tls.tls_sparse_decode(layout, qs[-1], kv, ctx, kmax, kmin, codes, qparams, ch, K_b, cfg.k_t, M_last, None,
                              out, None, M_tmp, None, ws, mode=tls.MODE_LAGGED)

    for _ in range(10):  # untimed warm-up, as for the headline steps
        quiet_call()
    n_quiet = 100
    q0, q1 = ev(), ev()
    torch.cuda.synchronize()
    q0.record(main)
    for _ in range(n_quiet):
        quiet_call()
    q1.record(main)
    torch.cuda.synchronize()
    quiet_us = q0.elapsed_time(q1) * 1e3 / n_quiet
    ctx_now = ctx.cpu().numpy()
    step_bytes = algorithmic_bytes(cfg, ctx_now, M_last.cpu().numpy(), 2)["total"]
    err = tls.tls_check_device_error(ws)
    block_bytes = B * (cfg.d_qk + cfg.d_v) * 2
    med = lambda k: float(np.median([r[k] for r in rec]))  # noqa: E731
    blocks = float(np.mean([r["blocks"] for r in rec]))
    xfer_bytes = blocks * block_bytes
    return {
        "workload": "offload_gqa_96k: b=32, 32/8 heads, d=128, bf16, K_b=128, K_t=2048, "
                    f"{len(rec)} steps of an AR(1) query walk (rho={cfg.rho}) with the context growing from {n0} to "
                    f"{n0 + len(rec)} tokens (one appended per sequence per step: host row, pool row when resident, "
                    f"block summary, token-index row); K/V {2 * host_k.numel() * 2 / 1e9:.1f} GB "
                    f"in pinned host memory, pool of {n_slots} slots per unit in HBM",
        "step_wall_us_median": round(med("wall"), 1),
        "append_us_median": round(med("append"), 1),
        "selection_us_median": round(med("select"), 1),
        "decode_call_with_transfer_us_median": round(med("decode"), 1),
        "decode_call_no_transfer_us": round(quiet_us, 1),
        "decode_call_no_transfer_frac_of_peak_hbm": round(step_bytes / (quiet_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
        "transfer_us_median": round(med("xfer"), 1),
        "blocks_moved_per_step_mean": round(blocks, 1),
        "block_repeat_rate": round(1.0 - blocks / (units * K_b), 4),
        "transfer_MB_per_step_mean": round(xfer_bytes / 1e6, 1),
        "pcie_GBps": round(xfer_bytes / (med("xfer") * 1e-6) / 1e9, 1),
        "prefill_flow": {
            "prefill_kv_ms": round(prefill_rec["prefill_kv_ms"], 2),
            "offload_ms": round(prefill_rec["offload_ms"], 1),
            "offload_GBps": round(kv_bytes / (prefill_rec["offload_ms"] * 1e-3) / 1e9, 1),
            "initial_residency_ms": round(prefill_rec["residency_ms"], 3),
            "note": "tls_prefill_kv (write-back + both indices), then the final prompt query's blocks made "
                    "resident from HBM (tls_init_residency), then tls_offload_kv copies the whole cache to pinned "
                    "host memory on a side stream",
        },
        "device_error_flags": err,
    }


def setup_decode(tls, synth, torch, workload, copies_arg=0):
    """One workload's decode inputs on the GPU: device-generated q, K/V, the
    prefill-built block and token indices, and `copies` byte-identical copies
    of the layer at distinct addresses, rotated so that one rotation touches
    at least eight times the 256 MiB Infinity Cache (within a 64 GB budget).
    `step(i)` runs the decode over copy i mod copies."""
    import types
    cfg_name, over = WORKLOADS[workload]
    cfg = synth.config(cfg_name, **over)
    dev = torch.device("cuda", 0)
    e = 2 if cfg.dtype == "bf16" else 4
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d = synth.make_device(cfg, device=dev, pad="zero")
    layout = tls.make_layout(cfg.batch, cfg.h_q, cfg.h_kv, cfg.d_qk, cfg.d_v, cfg.max_ctx,
                             index_channels=cfg.d_c, block_size=cfg.block,
                             dtype=tls.DTYPE_BF16 if cfg.dtype == "bf16" else tls.DTYPE_F32,
                             mla_shared_kv=cfg.mla)
    m_max = -(-cfg.max_ctx // cfg.block)
    kmax = torch.empty((cfg.batch, cfg.h_kv, m_max, cfg.d_qk), dtype=dt, device=dev)
    kmin = torch.empty_like(kmax)
    codes = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 2), dtype=torch.uint8, device=dev)
    qparams = torch.empty((cfg.batch, cfg.h_kv, cfg.max_ctx, cfg.d_c // 32, 2), dtype=torch.float32, device=dev)
    tls.tls_build_block_index(layout, d["k"], d["ctx_lens"], 0, cfg.max_ctx, kmax, kmin)
    tls.tls_build_token_index(layout, d["k"], d["ctx_lens"], d["channels"], 0, cfg.max_ctx, codes, qparams)
    torch.cuda.synchronize()
    layer = dict(q=d["q"], k=d["k"], v=d["v"], kmax=kmax, kmin=kmin, codes=codes, qparams=qparams)
    per_layer = sum(t.numel() * t.element_size() for t in layer.values() if t is not None)
    # touched bytes per step (upper estimate)
    m_hi = -(-int(d["ctx_host"].max()) // cfg.block)
    units = cfg.batch * cfg.h_kv
    touched = units * (m_hi * 2 * cfg.d_qk * e + cfg.k_b * cfg.block * 24 + cfg.k_t * (cfg.d_qk + cfg.d_v) * e)
    copies = copies_arg or int(min(64, max(2, math.ceil(8 * 2 ** 28 / touched)), max(2, 64e9 // per_layer)))
    layers = [layer] + [{k: (None if t is None else t.clone()) for k, t in layer.items()} for _ in range(copies - 1)]
    ctx_t, ch_t = d["ctx_lens"], d["channels"]
    ws = tls.alloc_workspace(layout, cfg.k_b, cfg.k_t, device=dev)
    out = torch.empty((cfg.batch, cfg.h_q, cfg.d_v), dtype=dt, device=dev)
    lse = torch.empty((cfg.batch, cfg.h_q), dtype=torch.float32, device=dev)
    bids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_b), dtype=torch.int32, device=dev)
    tids = torch.empty((cfg.batch, cfg.h_kv, cfg.k_t), dtype=torch.int32, device=dev)

    def step(i, events=None):
        L = layers[i % len(layers)]
        tls.tls_sparse_decode(layout, L["q"], tls.KV(L["k"], L["v"]), ctx_t, L["kmax"], L["kmin"], L["codes"],
                              L["qparams"], ch_t, cfg.k_b, cfg.k_t, None, None, out, lse, bids, tids, ws,
                              stage_events=events)

    def step_args(i):
        L = layers[i % len(layers)]
        return tls.sparse_decode_args(layout, L["q"], tls.KV(L["k"], L["v"]), ctx_t, L["kmax"], L["kmin"],
                                      L["codes"], L["qparams"], ch_t, cfg.k_b, cfg.k_t, None, None, out, lse, bids,
                                      tids, ws)

    return types.SimpleNamespace(cfg=cfg, d=d, layout=layout, layers=layers, copies=copies, e=e, dev=dev, dt=dt,
                                 ctx_t=ctx_t, ch_t=ch_t, ws=ws, out=out, lse=lse, bids=bids, tids=tids, step=step,
                                 step_args=step_args)


def host_call_us(tls, torch, s, n=48):
    """Host time per decode call: `n` back-to-back calls issued with no wait
    (the GPU runs behind them), timed on the host clock.  `binding`: through
    the Python binding (argument checks and marshalling included); `c_abi`:
    the C entry point alone, its arguments marshalled once beforehand."""
    prepared = [s.step_args(i) for i in range(n)]
    fn = tls.lib().tls_sparse_decode

    def run(f):
        best = float("inf")
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(n):
                f(i)
            t1 = time.perf_counter()
            torch.cuda.synchronize()
            best = min(best, (t1 - t0) * 1e6 / n)
        return round(best, 2)

    def raw(i):
        if fn(*prepared[i][0]) != 0:
            raise RuntimeError("tls_sparse_decode failed")

    return {"binding": run(s.step), "c_abi": run(raw), "calls": n,
            "method": "best of 3 runs of back-to-back calls, host clock, no wait between calls"}


def secondary_workload(tls, synth, torch, np, workload, steps, warmup):
    """µs per step and the fraction of peak HBM bandwidth of another
    workload's decode step (same timing as the headline: torch events around
    `steps` back-to-back steps over the rotated layer copies), plus the
    median of steps that each follow an untimed 1 GiB scratch write."""
    W = setup_decode(tls, synth, torch, workload)
    for i in range(warmup):
        W.step(i)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(steps):
        W.step(i)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / steps
    flush = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=W.dev)
    ts = []
    for i in range(min(steps, 30)):
        flush.fill_(float(i))
        a.record()
        W.step(i)
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b) * 1e3)
    del flush
    err = tls.tls_check_device_error(W.ws)
    nb = algorithmic_bytes(W.cfg, W.d["ctx_host"], W.bids.cpu().numpy(), W.e)
    gbps = nb["total"] / (us * 1e-6) / 1e9
    cfg = W.cfg
    rec = {
        "config": {"batch": cfg.batch, "h_q": cfg.h_q, "h_kv": cfg.h_kv, "d_qk": cfg.d_qk, "d_v": cfg.d_v,
                   "ctx_min": int(W.d["ctx_host"].min()), "ctx_max": int(W.d["ctx_host"].max()), "k_b": cfg.k_b,
                   "k_t": cfg.k_t, "dtype": cfg.dtype, "layer_copies_rotated": W.copies},
        "us_per_step": round(us, 2), "achieved_GBps": round(gbps, 1),
        "step_frac_of_peak_hbm": round(gbps / PEAK_HBM_GBPS, 4),
        "step_us_after_1GiB_flush_median": round(float(np.median(ts)), 2),
        "algorithmic_bytes_per_step": nb["total"], "device_error_flags": err,
    }
    del W
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary)
        return
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (asked for --gpus {args.gpus}); "
              "the operator shards by (sequence, KV head) without cross-GPU exchange, "
              "so per-GPU throughput is the single-GPU figure", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2604_07815_amd as tls
    import synth

    torch.cuda.init()
    W = setup_decode(tls, synth, torch, args.workload, args.copies)
    cfg, d, layout, layers, copies, e = W.cfg, W.d, W.layout, W.layers, W.copies, W.e
    dev, dt, ctx_t, ch_t, ws, out, lse, bids, tids, step = (W.dev, W.dt, W.ctx_t, W.ch_t, W.ws, W.out, W.lse,
                                                            W.bids, W.tids, W.step)
    layer = layers[0]

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    if args.profile_only:
        if args.calibrate_copy:
            src_b = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
            dst_b = torch.empty_like(src_b)
            for _ in range(3):
                dst_b.copy_(src_b)
            torch.cuda.synchronize()
            del src_b, dst_b
        for i in range(args.steps):
            step(i)
        torch.cuda.synchronize()
        print(json.dumps({"profile_only": True, "workload": args.workload, "steps": args.steps}), flush=True)
        return

    # ---- timed region (clean: no stage markers) ---------------------------------
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(i)
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps

    # ---- per-step distribution: 200 steps, each bracketed by events; then the same
    # with a 1 GiB scratch write between steps (untimed) so no step can find its
    # data in the 256 MB Infinity Cache -----------------------------------------------
    def step_distribution(n, flush=None):
        pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        torch.cuda.synchronize()
        for i in range(n):
            if flush is not None:
                flush.fill_(float(i))
            pairs[i][0].record()
            step(i)
            pairs[i][1].record()
        torch.cuda.synchronize()
        ts = np.array([a.elapsed_time(b) * 1e3 for a, b in pairs])
        return {"n": n, "median_us": round(float(np.median(ts)), 2), "p10_us": round(float(np.percentile(ts, 10)), 2),
                "p90_us": round(float(np.percentile(ts, 90)), 2)}

    dist = step_distribution(200)
    flush_buf = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dist_flush = step_distribution(50, flush_buf)
    del flush_buf

    # ---- the same steps replayed from a HIP graph: one capture of a rotation over
    # the layer copies, as a serving loop that captures its step would run it ------
    def graph_replay_us():
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for i in range(len(layers)):
                step(i)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(len(layers)):
                step(i)
        reps = max(1, args.steps // len(layers))
        graph.replay()
        torch.cuda.synchronize()
        start.record()
        for _ in range(reps):
            graph.replay()
        stop.record()
        torch.cuda.synchronize()
        return round(start.elapsed_time(stop) * 1e3 / (reps * len(layers)), 2)

    graph_us = graph_replay_us()
    host_us = host_call_us(tls, torch, W)

    # ---- per-stage timing with HIP events on the launch stream --------------------
    hev = HipEvents()
    evs = [hev.create(tls.NUM_STAGE_EVENTS) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(i, events=evs[i])
    torch.cuda.synchronize()
    stage_ms = np.zeros(len(STAGES))
    for i in range(args.steps):
        for j in range(len(STAGES)):
            stage_ms[j] += hev.elapsed_ms(evs[i][j], evs[i][j + 1])
    stage_ms /= args.steps
    marked_ms = sum(hev.elapsed_ms(evs[i][0], evs[i][-1]) for i in range(args.steps)) / args.steps
    for ev in evs:
        hev.destroy(ev)

    # ---- the dominant kernel alone: back-to-back attention launches -------------
    # (token ids given: the call runs the attention stage only); torch's events
    # are recorded on its current stream, the stream the library launches on
    tids_sel = tids.clone()
    attn_out = torch.empty_like(out)

    def attn_only(i):
        L = layers[i % len(layers)]
        tls.tls_sparse_decode(layout, L["q"], tls.KV(L["k"], L["v"]), ctx_t, None, None, None, None, None,
                              cfg.k_b, cfg.k_t, None, tids_sel, attn_out, None, None, None, ws)

    for i in range(args.warmup):
        attn_only(i)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        attn_only(i)
    stop.record()
    torch.cuda.synchronize()
    attn_ms = start.elapsed_time(stop) / args.steps

    # ---- the single-level operators on the same workload (the paper's baselines) ----
    modes = {}
    if not args.no_modes:
        def time_mode(mode, k_b, steps):
            def f(i):
                L = layers[i % len(layers)]
                tls.tls_sparse_decode(layout, L["q"], tls.KV(L["k"], L["v"]), ctx_t, L["kmax"], L["kmin"], L["codes"],
                                      L["qparams"], ch_t, k_b, cfg.k_t, None, None, attn_out, None, None, None, ws,
                                      mode=mode)
            for i in range(2):
                f(i)
            torch.cuda.synchronize()
            start.record()
            for i in range(steps):
                f(i)
            stop.record()
            torch.cuda.synchronize()
            return start.elapsed_time(stop) / steps * 1e3
        ms = max(4, min(args.steps, 20))
        modes["two_level_us"] = round(ms_per_step * 1e3, 2)
        modes["block_sparse_same_blocks_us"] = round(time_mode(tls.MODE_BLOCK_SPARSE, cfg.k_b, ms), 2)
        kb_eq = max(1, cfg.k_t // cfg.block)
        modes["block_sparse_same_tokens_us"] = round(time_mode(tls.MODE_BLOCK_SPARSE, kb_eq, ms), 2)
        modes["token_sparse_us"] = round(time_mode(tls.MODE_TOKEN_SPARSE, cfg.k_b, ms), 2)
        modes["dense_us"] = round(time_mode(tls.MODE_DENSE, cfg.k_b, ms), 2)
        modes["speedup_vs_dense"] = round(modes["dense_us"] / modes["two_level_us"], 2)
        modes["speedup_vs_token_sparse"] = round(modes["token_sparse_us"] / modes["two_level_us"], 2)
        modes["note"] = (f"same inputs; block-sparse attends every token of the top-{cfg.k_b} blocks "
                         f"({cfg.k_b * cfg.block} tokens) or of the top-{kb_eq} blocks ({kb_eq * cfg.block} tokens, "
                         f"the two-level token budget); token-sparse selects the top-{cfg.k_t} tokens of the "
                         f"whole context by the same approximate score; dense attends all ctx_len tokens")

    # ---- prefill side (off the per-step clock): index build, fused write-back ----
    prefill = None if args.profile_only else prefill_timing(tls, torch, cfg, layout, d, layers[0], e)
    calibration = calibration_timing(tls, torch, cfg, layout, dev)

    err = tls.tls_check_device_error(ws)
    nb = algorithmic_bytes(cfg, d["ctx_host"], bids.cpu().numpy(), e)
    us = ms_per_step * 1e3
    gbps = nb["total"] / (ms_per_step * 1e-3) / 1e9

    attn_bytes = nb["gathered_kv"] + cfg.batch * cfg.h_q * (cfg.d_qk + cfg.d_v) * e  # + q read, out written
    attn_gbps = attn_bytes / (attn_ms * 1e-3) / 1e9
    traffic = traffic_from_profiles(attention_source_hash()) if args.workload == "gqa_b32_ctx96k" else None

    result = {
        "metric": METRIC,
        "value": round(us, 2),
        "unit": "µs/layer-step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": args.workload, "batch": cfg.batch, "h_q": cfg.h_q, "h_kv": cfg.h_kv,
            "d_qk": cfg.d_qk, "d_v": cfg.d_v, "ctx_min": int(d["ctx_host"].min()),
            "ctx_max": int(d["ctx_host"].max()), "block": cfg.block, "k_b": cfg.k_b, "k_t": cfg.k_t,
            "d_c": cfg.d_c, "kv": "hbm-resident", "layer_copies_rotated": copies,
        },
        "achieved_GBps": round(gbps, 1),
        "step_frac_of_peak_hbm": round(gbps / PEAK_HBM_GBPS, 4),
        "algorithmic_bytes_per_step": nb,
        "step_us_distribution": dist,
        "step_us_after_1GiB_flush": dist_flush,
        "step_us_graph_replay": graph_us,
        "host_us_per_call": host_us,
        "stage_us": {k: round(float(v) * 1e3, 2) for k, v in zip(STAGES, stage_ms)},
        "stage_marked_step_us": round(marked_ms * 1e3, 2),
        "prefill": prefill,
        "calibration": calibration,
        "device_error_flags": err,
        "operators": modes or None,
        "roofline": {
            "kernel": "attn_mla_mfma_kernel" if cfg.mla else
                      ("attn_gqa_mfma_kernel" if cfg.dtype == "bf16" else "attn_gqa_kernel"),
            "bound": "hbm", "achieved": round(attn_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(attn_gbps / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "bytes_per_launch": attn_bytes, "avg_launch_us": round(attn_ms * 1e3, 2),
            "timing": f"{args.steps} back-to-back launches of the attention stage alone on the step's token ids, "
                      "HIP events on the launch stream",
        },
    }

    # ---- CPU baseline: the oracle's decode step over every unit of the step -------
    if not args.no_cpu_baseline:
        # one more step on the resident layer: its outputs are checked against
        # the oracle unit by unit inside the baseline leg
        step(0)
        torch.cuda.synchronize()
        gpu = dict(out=out.float().cpu().numpy(), lse=lse.cpu().numpy(), bids=bids.cpu().numpy(),
                   tids=tids.cpu().numpy())
        result["cpu_baseline"], result["parity"] = cpu_baseline_record(cfg, d, np, torch, gpu)
    # ---- the other legs of the 60 % gate: the batched 48k-96k step and the
    # offloaded 96k workload's decode over the HBM pool (with and without the
    # PCIe transfer running), reported beside the headline -----------------------
    if (args.workload == "gqa_b32_ctx96k" and not args.no_workloads) or args.offload:
        del layers, layer, d, step, W
        gc.collect()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        workloads = {}
        if args.workload != "gqa_b16_ctx48k_96k":
            workloads["gqa_b16_ctx48k_96k"] = secondary_workload(tls, synth, torch, np, "gqa_b16_ctx48k_96k",
                                                                 args.steps, args.warmup)
        workloads["offload_gqa_b32_ctx96k"] = offload_schedule(tls, synth, torch, np)
        result["workloads"] = workloads
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
