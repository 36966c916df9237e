"""Two-level sparse decode attention on MI355X (gfx950): Python binding.

Thin ctypes binding of ``libtls.so`` (see include/tls.h for the contract).
Every function has the name of the C entry point it wraps and only
marshals arguments: torch tensors are passed by ``data_ptr()`` and the
stream defaults to torch's current stream.  All computation happens in the
library's HIP kernels; importing this package fails loudly when the library
has not been built (``python paper_2604_07815_amd/build.py``).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

__all__ = [
    "TlsError", "Layout", "KvView", "KV", "DecodeOpts", "NUM_STAGE_EVENTS", "LIB_PATH",
    "tls_version", "tls_status_string", "tls_workspace_size", "tls_workspace_init",
    "tls_build_block_index", "tls_build_token_index", "tls_select_blocks", "tls_select_tokens",
    "tls_sparse_decode", "tls_sparse_decode_noalloc", "tls_prefetch_blocks", "tls_check_device_error",
    "tls_prefill_kv", "tls_offload_kv", "tls_init_residency", "tls_calibrate_absmax", "tls_calibrate_channels",
    "tls_append_tokens", "sparse_decode_args", "lib", "make_layout", "alloc_workspace", "DTYPE_F32", "DTYPE_BF16",
    "EXPORTED_SYMBOLS",
    "MODE_TWO_LEVEL", "MODE_BLOCK_SPARSE", "MODE_DENSE", "MODE_TOKEN_SPARSE", "MODE_LAGGED",
    "DEVERR_CTX_LEN", "DEVERR_BLOCK_ID", "DEVERR_TOKEN_ID", "DEVERR_SLOT", "DEVERR_POOL_FULL", "DEVERR_CHANNEL",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtls.so")

OK, INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP_ERROR = 0, 1, 2, 3, 4
DTYPE_F32, DTYPE_BF16 = 0, 1
MODE_TWO_LEVEL, MODE_BLOCK_SPARSE, MODE_DENSE, MODE_TOKEN_SPARSE, MODE_LAGGED = 0, 1, 2, 3, 4
NUM_STAGE_EVENTS = 8
DEVERR_CTX_LEN, DEVERR_BLOCK_ID, DEVERR_TOKEN_ID, DEVERR_SLOT, DEVERR_POOL_FULL, DEVERR_CHANNEL = 1, 2, 4, 8, 16, 32

EXPORTED_SYMBOLS = [
    "tls_version", "tls_status_string", "tls_workspace_size", "tls_workspace_init",
    "tls_build_block_index", "tls_build_token_index", "tls_select_blocks", "tls_select_tokens",
    "tls_sparse_decode", "tls_prefetch_blocks", "tls_check_device_error", "tls_prefill_kv",
    "tls_offload_kv", "tls_init_residency", "tls_calibrate_absmax", "tls_calibrate_channels", "tls_append_tokens",
    "tls_sparse_decode_noalloc",
]


class TlsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {tls_status_string(status)} ({status})")


class Layout(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim_qk", ctypes.c_int32),
        ("head_dim_v", ctypes.c_int32), ("block_size", ctypes.c_int32),
        ("index_channels", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("mla_shared_kv", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
    ]


class KvView(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("slot_map", ctypes.c_void_p), ("n_slots", ctypes.c_int64)]


class DecodeOpts(ctypes.Structure):
    _fields_ = [("attn_splits", ctypes.c_int32), ("mode", ctypes.c_int32), ("reserved", ctypes.c_int32 * 6),
                ("stage_events", ctypes.c_void_p)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2604_07815_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    LP = ctypes.POINTER(Layout)
    sig = {
        "tls_version": (ctypes.c_char_p, []),
        "tls_status_string": (ctypes.c_char_p, [I32]),
        "tls_workspace_size": (I32, [LP, I32, I32, ctypes.POINTER(SZ)]),
        "tls_workspace_init": (I32, [P, SZ, P]),
        "tls_build_block_index": (I32, [LP, P, P, I32, I32, P, P, P]),
        "tls_build_token_index": (I32, [LP, P, P, P, I32, I32, P, P, P]),
        "tls_prefill_kv": (I32, [LP, P, P, P, P, I32, I32, P, P, P, P, P, P, P]),
        "tls_select_blocks": (I32, [LP, P, P, P, P, I32, P, P, P, SZ, P]),
        "tls_select_tokens": (I32, [LP, P, P, P, P, P, I32, P, I32, P, P, P, SZ, P]),
        "tls_sparse_decode": (I32, [LP, P, ctypes.POINTER(KvView), P, P, P, P, P, P, I32, I32, P, P,
                                    P, P, P, P, P, SZ, ctypes.POINTER(DecodeOpts), P]),
        "tls_sparse_decode_noalloc": (I32, [LP, P, ctypes.POINTER(KvView), P, P, P, P, P, P, I32, I32, P, P,
                                            P, P, P, P, P, ctypes.POINTER(DecodeOpts), P]),
        "tls_prefetch_blocks": (I32, [LP, P, P, P, P, P, I32, P, P, I64, P, P, P, P, SZ, P]),
        "tls_offload_kv": (I32, [LP, P, P, P, I32, I32, P, P, P]),
        "tls_append_tokens": (I32, [LP, P, P, P, P, P, P, P, P, P, P, ctypes.POINTER(KvView), P]),
        "tls_calibrate_absmax": (I32, [LP, P, P, I32, P, P, I32, P]),
        "tls_calibrate_channels": (I32, [LP, P, P, P, P, P]),
        "tls_init_residency": (I32, [LP, P, P, P, P, I32, P, P, I64, P, P, P, SZ, P]),
        "tls_check_device_error": (I32, [P, SZ, I32, ctypes.POINTER(I32), P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib() -> ctypes.CDLL:
    """The loaded libtls.so (its C entry points with their ctypes signatures)."""
    return _lib


# ----------------------------------------------------------------------------
# marshalling helpers
# ----------------------------------------------------------------------------

def _ptr(t: Optional[torch.Tensor], what: str, device: bool = True):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what}: expected a torch.Tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what}: tensor must be contiguous")
    if device and not t.is_cuda:
        raise ValueError(f"{what}: tensor must live on the GPU")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    return ctypes.c_void_p(handle)


def _check(status: int, where: str) -> None:
    if status != OK:
        raise TlsError(status, where)


def make_layout(batch, num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, max_ctx,
                index_channels=32, block_size=64, dtype=DTYPE_BF16, mla_shared_kv=False,
                softmax_scale: float = 0.0) -> Layout:
    if isinstance(dtype, torch.dtype):
        dtype = DTYPE_BF16 if dtype == torch.bfloat16 else DTYPE_F32
    return Layout(int(batch), int(num_q_heads), int(num_kv_heads), int(head_dim_qk), int(head_dim_v),
                  int(block_size), int(index_channels), int(max_ctx), int(dtype),
                  1 if mla_shared_kv else 0, float(softmax_scale))


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ----------------------------------------------------------------------------

def tls_version() -> str:
    return _lib.tls_version().decode()


def tls_status_string(status: int) -> str:
    return _lib.tls_status_string(int(status)).decode()


def tls_workspace_size(layout: Layout, K_b: int, K_t: int) -> int:
    out = ctypes.c_size_t(0)
    _check(_lib.tls_workspace_size(ctypes.byref(layout), K_b, K_t, ctypes.byref(out)), "tls_workspace_size")
    return int(out.value)


def tls_workspace_init(ws: torch.Tensor, stream=None) -> None:
    _check(_lib.tls_workspace_init(_ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)),
           "tls_workspace_init")


def alloc_workspace(layout: Layout, K_b: int, K_t: int, device="cuda", stream=None) -> torch.Tensor:
    """Allocate (torch) and initialise a workspace for these budgets."""
    ws = torch.empty(tls_workspace_size(layout, K_b, K_t), dtype=torch.uint8, device=device)
    tls_workspace_init(ws, stream)
    return ws


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def tls_build_block_index(layout, K, ctx_lens, tok_begin, tok_end, kmax, kmin, stream=None) -> None:
    _check(_lib.tls_build_block_index(ctypes.byref(layout), _ptr(K, "K"), _ptr(ctx_lens, "ctx_lens"),
                                      int(tok_begin), int(tok_end), _ptr(kmax, "kmax"), _ptr(kmin, "kmin"),
                                      _stream(stream)), "tls_build_block_index")


def tls_build_token_index(layout, K, ctx_lens, channels, tok_begin, tok_end, codes, qparams,
                          stream=None) -> None:
    _check(_lib.tls_build_token_index(ctypes.byref(layout), _ptr(K, "K"), _ptr(ctx_lens, "ctx_lens"),
                                      _ptr(channels, "channels"), int(tok_begin), int(tok_end),
                                      _ptr(codes, "codes"), _ptr(qparams, "qparams"), _stream(stream)),
           "tls_build_token_index")


def tls_calibrate_absmax(layout, q_cal, k_cal, q_absmax, k_absmax, accumulate: bool = False, stream=None) -> None:
    """Running max |x| per (head, channel) over calibration rows q_cal [N][H_q][d], k_cal [N][H_kv][d]."""
    n = 0 if q_cal is None else int(q_cal.shape[0])
    if k_cal is not None and int(k_cal.shape[0]) != n:
        raise ValueError("q_cal and k_cal must hold the same number of rows")
    _check(_lib.tls_calibrate_absmax(ctypes.byref(layout), _ptr(q_cal, "q_cal") if n else None,
                                     _ptr(k_cal, "k_cal") if n else None, n, _ptr(q_absmax, "q_absmax"),
                                     _ptr(k_absmax, "k_absmax"), 1 if accumulate else 0, _stream(stream)),
           "tls_calibrate_absmax")


def tls_calibrate_channels(layout, q_absmax, k_absmax, channels, scores=None, stream=None) -> None:
    """Channel importance and the top-d_c channels per KV head (ascending)."""
    _check(_lib.tls_calibrate_channels(ctypes.byref(layout), _ptr(q_absmax, "q_absmax"), _ptr(k_absmax, "k_absmax"),
                                       _ptr(channels, "channels"), _ptr(scores, "scores"), _stream(stream)),
           "tls_calibrate_channels")


def tls_prefill_kv(layout, k_src, v_src, ctx_lens, channels, tok_begin, tok_end, K, V, kmax, kmin, codes,
                   qparams, stream=None) -> None:
    """Prefill write-back of rows [tok_begin, tok_end) fused with both index builds."""
    _check(_lib.tls_prefill_kv(ctypes.byref(layout), _ptr(k_src, "k_src"), _ptr(v_src, "v_src"),
                               _ptr(ctx_lens, "ctx_lens"), _ptr(channels, "channels"), int(tok_begin),
                               int(tok_end), _ptr(K, "K"), _ptr(V, "V"), _ptr(kmax, "kmax"), _ptr(kmin, "kmin"),
                               _ptr(codes, "codes"), _ptr(qparams, "qparams"), _stream(stream)),
           "tls_prefill_kv")


def tls_select_blocks(layout, q, kmax, kmin, ctx_lens, K_b, block_ids, block_scores, ws, stream=None) -> None:
    _check(_lib.tls_select_blocks(ctypes.byref(layout), _ptr(q, "q"), _ptr(kmax, "kmax"), _ptr(kmin, "kmin"),
                                  _ptr(ctx_lens, "ctx_lens"), int(K_b), _ptr(block_ids, "block_ids"),
                                  _ptr(block_scores, "block_scores"), _ptr(ws, "ws"), _nbytes(ws),
                                  _stream(stream)), "tls_select_blocks")


def tls_select_tokens(layout, q, codes, qparams, channels, block_ids, K_b, ctx_lens, K_t, token_ids,
                      token_scores, ws, stream=None) -> None:
    _check(_lib.tls_select_tokens(ctypes.byref(layout), _ptr(q, "q"), _ptr(codes, "codes"),
                                  _ptr(qparams, "qparams"), _ptr(channels, "channels"),
                                  _ptr(block_ids, "block_ids"), int(K_b), _ptr(ctx_lens, "ctx_lens"), int(K_t),
                                  _ptr(token_ids, "token_ids"), _ptr(token_scores, "token_scores"),
                                  _ptr(ws, "ws"), _nbytes(ws), _stream(stream)), "tls_select_tokens")


@dataclass
class KV:
    """K/V source of the attention stage: dense arrays, or the block pool."""
    k: torch.Tensor
    v: Optional[torch.Tensor] = None
    slot_map: Optional[torch.Tensor] = None
    n_slots: int = 0

    def as_struct(self) -> KvView:
        return KvView(_ptr(self.k, "kv.k"), _ptr(self.v, "kv.v"), _ptr(self.slot_map, "kv.slot_map"),
                      int(self.n_slots))


def tls_sparse_decode(layout, q, kv: KV, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t,
                      block_ids_in, token_ids_in, out, lse, block_ids_out, token_ids_out, ws,
                      attn_splits: int = 0, stage_events: Optional[Sequence[int]] = None,
                      mode: int = MODE_TWO_LEVEL, stream=None) -> None:
    """One decode step.  stage_events: NUM_STAGE_EVENTS raw hipEvent_t handles;
    mode: MODE_TWO_LEVEL, MODE_LAGGED (tokens from block_ids_in, this step's
    block selection to block_ids_out), or one of the single-level baselines."""
    args, keep = sparse_decode_args(layout, q, kv, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t,
                                     block_ids_in, token_ids_in, out, lse, block_ids_out, token_ids_out, ws,
                                     attn_splits, stage_events, mode, stream)
    _check(_lib.tls_sparse_decode(*args), "tls_sparse_decode")
    del keep


def sparse_decode_args(layout, q, kv: KV, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t,
                       block_ids_in, token_ids_in, out, lse, block_ids_out, token_ids_out, ws,
                       attn_splits: int = 0, stage_events: Optional[Sequence[int]] = None,
                       mode: int = MODE_TWO_LEVEL, stream=None):
    """The marshalled argument tuple of tls_sparse_decode, and the ctypes
    objects it points into (keep them alive while the tuple is used).  A
    caller that repeats one call can marshal it once and call
    `lib().tls_sparse_decode(*args)` (returns the TLS_* status)."""
    opts, ev_arr = _decode_opts(attn_splits, stage_events, mode)
    view = kv.as_struct()
    args = (ctypes.byref(layout), _ptr(q, "q"), ctypes.byref(view), _ptr(ctx_lens, "ctx_lens"),
            _ptr(kmax, "kmax"), _ptr(kmin, "kmin"), _ptr(codes, "codes"), _ptr(qparams, "qparams"),
            _ptr(channels, "channels"), int(K_b), int(K_t), _ptr(block_ids_in, "block_ids_in"),
            _ptr(token_ids_in, "token_ids_in"), _ptr(out, "out"), _ptr(lse, "lse"),
            _ptr(block_ids_out, "block_ids_out"), _ptr(token_ids_out, "token_ids_out"), _ptr(ws, "ws"),
            _nbytes(ws), ctypes.byref(opts), _stream(stream))
    return args, (opts, ev_arr, view, layout)


def _decode_opts(attn_splits, stage_events, mode):
    opts = DecodeOpts()
    opts.attn_splits = int(attn_splits)
    opts.mode = int(mode)
    ev_arr = None
    if stage_events is not None:
        if len(stage_events) != NUM_STAGE_EVENTS:
            raise ValueError(f"stage_events must hold {NUM_STAGE_EVENTS} events")
        ev_arr = (ctypes.c_void_p * NUM_STAGE_EVENTS)(*[ctypes.c_void_p(int(e)) for e in stage_events])
        opts.stage_events = ctypes.cast(ev_arr, ctypes.c_void_p)
    return opts, ev_arr


def tls_sparse_decode_noalloc(layout, q, kv: KV, ctx_lens, kmax, kmin, codes, qparams, channels, K_b, K_t,
                              block_ids_in, token_ids_in, out, lse, block_ids_out, token_ids_out,
                              device_error: Optional[torch.Tensor] = None, attn_splits: int = 0,
                              stage_events: Optional[Sequence[int]] = None, mode: int = MODE_TWO_LEVEL,
                              stream=None) -> None:
    """tls_sparse_decode on the library's own scratch (no workspace, no
    allocation).  device_error: optional one-element int32 GPU tensor that
    receives the device-side error bits (zero it first)."""
    opts, ev_arr = _decode_opts(attn_splits, stage_events, mode)
    view = kv.as_struct()
    _check(_lib.tls_sparse_decode_noalloc(
        ctypes.byref(layout), _ptr(q, "q"), ctypes.byref(view), _ptr(ctx_lens, "ctx_lens"),
        _ptr(kmax, "kmax"), _ptr(kmin, "kmin"), _ptr(codes, "codes"), _ptr(qparams, "qparams"),
        _ptr(channels, "channels"), int(K_b), int(K_t), _ptr(block_ids_in, "block_ids_in"),
        _ptr(token_ids_in, "token_ids_in"), _ptr(out, "out"), _ptr(lse, "lse"),
        _ptr(block_ids_out, "block_ids_out"), _ptr(token_ids_out, "token_ids_out"),
        _ptr(device_error, "device_error"), ctypes.byref(opts), _stream(stream)), "tls_sparse_decode_noalloc")
    del ev_arr


def tls_prefetch_blocks(layout, host_k, host_v, ctx_lens, block_ids_new, block_ids_live, K_b, pool_k, pool_v,
                        n_slots, slot_map, slot_owner, transfer_count, ws, stream=None) -> None:
    """Incremental block transfer; host_k/host_v are pinned CPU tensors."""
    for t, name in ((host_k, "host_k"), (host_v, "host_v")):
        if t is not None and (t.is_cuda or not t.is_pinned()):
            raise ValueError(f"{name}: must be a pinned host tensor")
    _check(_lib.tls_prefetch_blocks(
        ctypes.byref(layout), _ptr(host_k, "host_k", device=False), _ptr(host_v, "host_v", device=False),
        _ptr(ctx_lens, "ctx_lens"), _ptr(block_ids_new, "block_ids_new"),
        _ptr(block_ids_live, "block_ids_live"), int(K_b), _ptr(pool_k, "pool_k"), _ptr(pool_v, "pool_v"),
        int(n_slots), _ptr(slot_map, "slot_map"), _ptr(slot_owner, "slot_owner"),
        _ptr(transfer_count, "transfer_count"), _ptr(ws, "ws"), _nbytes(ws), _stream(stream)),
        "tls_prefetch_blocks")


def tls_append_tokens(layout, k_new, v_new, ctx_lens, channels, K, V, kmax, kmin, codes, qparams,
                      pool: Optional["KV"] = None, stream=None) -> None:
    """Append the token at ctx_lens - 1 of every sequence: cache row (K/V on the GPU or pinned host tensors),
    incremental block summary, token-index row, and the pool row when pool (a pooled KV view) holds its block."""
    def cache(t, name):
        return None if t is None else (_ptr(t, name) if t.is_cuda else _pinned(t, name))
    view = pool.as_struct() if pool is not None else None
    _check(_lib.tls_append_tokens(ctypes.byref(layout), _ptr(k_new, "k_new"), _ptr(v_new, "v_new"),
                                  _ptr(ctx_lens, "ctx_lens"), _ptr(channels, "channels"), cache(K, "K"),
                                  cache(V, "V"), _ptr(kmax, "kmax"), _ptr(kmin, "kmin"), _ptr(codes, "codes"),
                                  _ptr(qparams, "qparams"), ctypes.byref(view) if view is not None else None,
                                  _stream(stream)), "tls_append_tokens")


def _pinned(t, name):
    if t is not None and (t.is_cuda or not t.is_pinned()):
        raise ValueError(f"{name}: must be a pinned host tensor")
    return _ptr(t, name, device=False)


def tls_offload_kv(layout, K, V, ctx_lens, tok_begin, tok_end, host_k, host_v, stream=None) -> None:
    """Device -> pinned host copy of the cache rows [tok_begin, tok_end)."""
    _check(_lib.tls_offload_kv(ctypes.byref(layout), _ptr(K, "K"), _ptr(V, "V"), _ptr(ctx_lens, "ctx_lens"),
                               int(tok_begin), int(tok_end), _pinned(host_k, "host_k"), _pinned(host_v, "host_v"),
                               _stream(stream)), "tls_offload_kv")


def tls_init_residency(layout, src_k, src_v, ctx_lens, block_ids, K_b, pool_k, pool_v, n_slots, slot_map,
                       slot_owner, ws, stream=None) -> None:
    """Empty the pool and make block_ids resident; src_k/src_v: GPU tensors or pinned host tensors."""
    def src(t, name):
        return None if t is None else (_ptr(t, name) if t.is_cuda else _pinned(t, name))
    _check(_lib.tls_init_residency(
        ctypes.byref(layout), src(src_k, "src_k"), src(src_v, "src_v"), _ptr(ctx_lens, "ctx_lens"),
        _ptr(block_ids, "block_ids"), int(K_b), _ptr(pool_k, "pool_k"), _ptr(pool_v, "pool_v"), int(n_slots),
        _ptr(slot_map, "slot_map"), _ptr(slot_owner, "slot_owner"), _ptr(ws, "ws"), _nbytes(ws),
        _stream(stream)), "tls_init_residency")


def tls_check_device_error(ws, clear: bool = False, stream=None) -> int:
    flags = ctypes.c_int32(0)
    _check(_lib.tls_check_device_error(_ptr(ws, "ws"), _nbytes(ws), 1 if clear else 0, ctypes.byref(flags),
                                       _stream(stream)), "tls_check_device_error")
    return int(flags.value)
