"""The C-ABI library loads, exports every symbol include/tls.h declares, and
its host-side validation rejects bad arguments before any GPU work (these
calls never reach the device, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tls.h")
LIB = os.path.join(ROOT, "paper_2604_07815_amd", "libtls.so")


@pytest.fixture(scope="module")
def tls():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    import paper_2604_07815_amd as t
    return t


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:tls_status|const char\*)\s+(tls_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["tls_build_block_index", "tls_build_token_index", "tls_select_blocks", "tls_select_tokens",
              "tls_sparse_decode", "tls_prefetch_blocks", "tls_workspace_size", "tls_check_device_error",
              "tls_prefill_kv", "tls_offload_kv", "tls_init_residency", "tls_calibrate_absmax",
              "tls_calibrate_channels", "tls_append_tokens"]:
        assert n in names, n


def test_library_exports_every_declared_symbol(tls):
    lib = ctypes.CDLL(LIB)
    for n in declared_functions():
        assert hasattr(lib, n), f"libtls.so does not export {n}"
    assert set(declared_functions()) == set(tls.EXPORTED_SYMBOLS)
    # the binding wraps every entry point under its C name and exports it
    for n in tls.EXPORTED_SYMBOLS:
        assert callable(getattr(tls, n, None)) and n in tls.__all__, n


def test_version_and_status_strings(tls):
    assert "gfx950" in tls.tls_version()
    assert tls.tls_status_string(0) == "TLS_OK"
    assert tls.tls_status_string(3) == "TLS_ERR_WORKSPACE_TOO_SMALL"


def _layout(tls, **kw):
    base = dict(batch=2, num_q_heads=32, num_kv_heads=8, head_dim_qk=128, head_dim_v=128, max_ctx=4096,
                index_channels=32, block_size=64, dtype=tls.DTYPE_BF16)
    base.update(kw)
    return tls.make_layout(**base)


def test_workspace_size_is_host_only_and_grows_with_budgets(tls):
    a = tls.tls_workspace_size(_layout(tls), 8, 128)
    b = tls.tls_workspace_size(_layout(tls), 128, 2048)
    assert 0 < a < b


@pytest.mark.parametrize("kw,code", [
    (dict(num_q_heads=30), 1),           # H_q not a multiple of H_kv
    (dict(index_channels=48), 1),        # d_c not a multiple of 32
    (dict(index_channels=256), 1),       # d_c > d_qk
    (dict(dtype=7), 1),                  # unknown dtype
    (dict(block_size=32), 2),            # only B = 64 is compiled
    (dict(max_ctx=64 * 20000), 2),       # more blocks than the top-k capacity
    (dict(head_dim_qk=100, head_dim_v=100), 2),
])
def test_bad_layouts(tls, kw, code):
    with pytest.raises(tls.TlsError) as e:
        tls.tls_workspace_size(_layout(tls, **kw), 8, 128)
    assert e.value.status == code


def test_bad_budgets(tls):
    for kb, kt, code in [(0, 128, 1), (8, 0, 1), (300, 128, 2)]:
        with pytest.raises(tls.TlsError) as e:
            tls.tls_workspace_size(_layout(tls), kb, kt)
        assert e.value.status == code


def _raw(tls):
    return tls._lib


def test_null_pointers_are_rejected_before_launch(tls):
    lib = _raw(tls)
    L = _layout(tls)
    dummy = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    null = None
    # missing K
    assert lib.tls_build_block_index(ctypes.byref(L), null, dummy, 0, 64, dummy, dummy, null) == 1
    # tok_end beyond max_ctx
    assert lib.tls_build_block_index(ctypes.byref(L), dummy, dummy, 0, 5000, dummy, dummy, null) == 1
    # workspace too small
    assert lib.tls_select_blocks(ctypes.byref(L), dummy, dummy, dummy, dummy, 8, dummy, null, dummy, 16,
                                 null) == 3
    # GQA decode without V
    kv = tls.KvView(dummy.value, None, None, 0)
    opts = tls.DecodeOpts()
    st = lib.tls_sparse_decode(ctypes.byref(L), dummy, ctypes.byref(kv), dummy, dummy, dummy, dummy, dummy,
                               dummy, 8, 128, null, null, dummy, null, null, null, dummy, 1 << 40,
                               ctypes.byref(opts), null)
    assert st == 1
    # reserved option fields must be zero
    kv = tls.KvView(dummy.value, dummy.value, None, 0)
    opts.reserved[2] = 5
    st = lib.tls_sparse_decode(ctypes.byref(L), dummy, ctypes.byref(kv), dummy, dummy, dummy, dummy, dummy,
                               dummy, 8, 128, null, null, dummy, null, null, null, dummy, 1 << 40,
                               ctypes.byref(opts), null)
    assert st == 1
    # MLA layout must not pass V
    Lm = _layout(tls, num_kv_heads=1, head_dim_qk=576, head_dim_v=512, index_channels=128, mla_shared_kv=True)
    opts.reserved[2] = 0
    st = lib.tls_sparse_decode(ctypes.byref(Lm), dummy, ctypes.byref(kv), dummy, dummy, dummy, dummy, dummy,
                               dummy, 8, 128, null, null, dummy, null, null, null, dummy, 1 << 40,
                               ctypes.byref(opts), null)
    assert st == 1
    # pool too small for the live + new sets
    st = lib.tls_prefetch_blocks(ctypes.byref(L), dummy, dummy, dummy, dummy, dummy, 8, dummy, dummy, 10,
                                 dummy, dummy, null, dummy, 1 << 40, null)
    assert st == 1


def test_prefill_calls_are_validated_before_launch(tls):
    """The prefill-side entry points reject bad arguments on the host (none of
    these calls reaches the device)."""
    lib = _raw(tls)
    L = _layout(tls)
    Lm = _layout(tls, num_kv_heads=1, head_dim_qk=576, head_dim_v=512, index_channels=128, mla_shared_kv=True)
    d = ctypes.c_void_p(0x1000)
    null = None
    ok_args = [d, d, d, d, 0, 64, d, d, d, d, d, d]
    assert lib.tls_prefill_kv(ctypes.byref(L), *([null] + ok_args[1:]), null) == 1   # no k_src
    assert lib.tls_prefill_kv(ctypes.byref(L), *(ok_args[:1] + [null] + ok_args[2:]), null) == 1  # GQA without v_src
    bad_range = list(ok_args)
    bad_range[4], bad_range[5] = 100, 50
    assert lib.tls_prefill_kv(ctypes.byref(L), *bad_range, null) == 1                # tok_end < tok_begin
    bad_range[4], bad_range[5] = 0, 4097
    assert lib.tls_prefill_kv(ctypes.byref(L), *bad_range, null) == 1                # past max_ctx
    assert lib.tls_prefill_kv(ctypes.byref(Lm), *ok_args, null) == 1                 # MLA passes no V
    # an empty range is a no-op that succeeds without touching anything
    empty = list(ok_args)
    empty[4] = empty[5] = 64
    assert lib.tls_prefill_kv(ctypes.byref(L), *empty, null) == 0
    # offload: host arrays must be pinned host memory (a device-looking pointer is not)
    assert lib.tls_offload_kv(ctypes.byref(L), d, d, d, 0, 64, null, d, null) == 1
    assert lib.tls_offload_kv(ctypes.byref(L), d, null, d, 0, 64, d, d, null) == 1
    assert lib.tls_offload_kv(ctypes.byref(Lm), d, d, d, 0, 64, d, null, null) == 1
    # residency: budget, pool size and workspace checks
    assert lib.tls_init_residency(ctypes.byref(L), d, d, d, d, 0, d, d, 16, d, d, d, 1 << 40, null) == 1
    assert lib.tls_init_residency(ctypes.byref(L), d, d, d, d, 8, d, d, 4, d, d, d, 1 << 40, null) == 1
    assert lib.tls_init_residency(ctypes.byref(L), d, d, d, d, 8, d, d, 16, d, d, null, 1 << 40, null) == 1
    assert lib.tls_init_residency(ctypes.byref(Lm), d, d, d, d, 8, d, d, 16, d, d, d, 1 << 40, null) == 1


def test_append_is_validated_before_launch(tls):
    lib = _raw(tls)
    L = _layout(tls)
    Lm = _layout(tls, num_kv_heads=1, head_dim_qk=576, head_dim_v=512, index_channels=128, mla_shared_kv=True)
    d = ctypes.c_void_p(0x1000)
    null = None
    args = [d, d, d, d, d, d, d, d, d, d]
    assert lib.tls_append_tokens(ctypes.byref(L), *([null] + args[1:]), null, null) == 1      # no k_new
    assert lib.tls_append_tokens(ctypes.byref(L), *(args[:1] + [null] + args[2:]), null, null) == 1  # GQA, no v_new
    assert lib.tls_append_tokens(ctypes.byref(Lm), *args, null, null) == 1                    # MLA passes no V
    bad_pool = tls.KvView(d.value, d.value, None, 16)                                         # pool without slot map
    assert lib.tls_append_tokens(ctypes.byref(L), *args, ctypes.byref(bad_pool), null) == 1
    no_slots = tls.KvView(d.value, d.value, d.value, 0)
    assert lib.tls_append_tokens(ctypes.byref(L), *args, ctypes.byref(no_slots), null) == 1


def test_calibration_calls_are_validated_before_launch(tls):
    lib = _raw(tls)
    L = _layout(tls)
    d = ctypes.c_void_p(0x1000)
    null = None
    assert lib.tls_calibrate_absmax(ctypes.byref(L), d, d, -1, d, d, 0, null) == 1     # negative row count
    assert lib.tls_calibrate_absmax(ctypes.byref(L), null, d, 16, d, d, 0, null) == 1   # rows without q
    assert lib.tls_calibrate_absmax(ctypes.byref(L), d, d, 16, null, d, 0, null) == 1   # no output
    assert lib.tls_calibrate_absmax(ctypes.byref(L), d, d, 16, d, d, 2, null) == 1      # accumulate not 0/1
    assert lib.tls_calibrate_channels(ctypes.byref(L), d, d, null, null, null) == 1     # no channel output
    assert lib.tls_calibrate_channels(ctypes.byref(_layout(tls, num_q_heads=30)), d, d, d, null, null) == 1


def test_decode_modes_are_validated_before_launch(tls):
    """Unknown operator modes and id arguments the single-level operators do
    not take are rejected on the host."""
    lib = _raw(tls)
    L = _layout(tls)
    dummy = ctypes.c_void_p(0x1000)
    null = None
    kv = tls.KvView(dummy.value, dummy.value, None, 0)

    def call(mode, bids_in=None, tids_in=None, bids_out=None, tids_out=None):
        opts = tls.DecodeOpts()
        opts.mode = mode
        return lib.tls_sparse_decode(ctypes.byref(L), dummy, ctypes.byref(kv), dummy, dummy, dummy, dummy, dummy,
                                     dummy, 8, 128, bids_in, tids_in, dummy, null, bids_out, tids_out, dummy,
                                     1 << 40, ctypes.byref(opts), null)

    assert call(4) == 1 and call(-1) == 1
    assert call(tls.MODE_TOKEN_SPARSE, bids_in=dummy) == 1
    assert call(tls.MODE_TOKEN_SPARSE, tids_in=dummy) == 1
    assert call(tls.MODE_TOKEN_SPARSE, bids_out=dummy) == 1
    assert call(tls.MODE_DENSE, tids_in=dummy) == 1
    assert call(tls.MODE_DENSE, bids_in=dummy) == 1
    assert call(tls.MODE_DENSE, bids_out=dummy) == 1
    assert call(tls.MODE_BLOCK_SPARSE, tids_in=dummy) == 1
    assert call(tls.MODE_BLOCK_SPARSE, tids_out=dummy) == 1
    # the lagged operator: both block lists, distinct, no given tokens
    other = ctypes.c_void_p(0x100000)
    assert call(5) == 1
    assert call(tls.MODE_LAGGED) == 1
    assert call(tls.MODE_LAGGED, bids_in=dummy) == 1
    assert call(tls.MODE_LAGGED, bids_out=dummy) == 1
    assert call(tls.MODE_LAGGED, bids_in=dummy, bids_out=dummy) == 1
    assert call(tls.MODE_LAGGED, bids_in=dummy, bids_out=ctypes.c_void_p(0x1000 + 4)) == 1  # overlapping
    assert call(tls.MODE_LAGGED, bids_in=dummy, bids_out=other, tids_in=dummy) == 1
