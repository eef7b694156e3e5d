"""The C ABI on the host: the library loads, exports every entry point that
include/vd.h declares, and rejects bad arguments before touching the GPU
(these calls return before any HIP call, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2609_23314_amd import vd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vd.h")

FAKE_V = 0x7F0000000000   # never dereferenced: validation fails first
FAKE_K = 0x7F0000100000


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:vd_status|size_t|const char \*)\s*(vd_\w+)\s*\(",
                                 text, flags=re.M)))


def test_header_declares_the_five_calls():
    names = declared_functions()
    for f in ("vd_score", "vd_select_topn", "vd_compact", "vd_evict_step", "vd_geometry"):
        assert f in names
    assert set(names) == set(vd.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(vd.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert not hasattr(lib, "vd_debug_take_error_word")   # the release build has no checks


def test_debug_library_exports_every_declared_symbol():
    from paper_2609_23314_amd import build as lib_build
    lib = ctypes.CDLL(lib_build.DEBUG_LIB)
    for name in declared_functions() + ["vd_debug_take_error_word"]:
        assert hasattr(lib, name), name
    lib.vd_debug_take_error_word.argtypes = [ctypes.c_void_p]
    assert lib.vd_debug_take_error_word(None) == vd.VD_ERR_INVALID_ARG


def good_desc(**kw):
    d = vd.VdCacheDesc()
    d.k, d.v = FAKE_K, FAKE_V
    d.dtype = vd.VD_DTYPE_BF16
    d.num_seqs, d.num_layers, d.num_kv_heads, d.num_q_heads = 2, 3, 4, 16
    d.head_dim, d.capacity = 128, 100
    d.stride_slot = 128
    d.stride_head = 100 * 128
    d.stride_layer = 4 * 100 * 128
    d.stride_seq = 3 * 4 * 100 * 128
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def call_step(d, n=(50, 60), N=(40, 40), variant=0, rs=None, **kw):
    lib = vd.load()
    S = max(int(d.num_seqs), 1)
    n_arr = (ctypes.c_int32 * S)(*(list(n) + [0] * S)[:S])
    N_arr = (ctypes.c_int32 * S)(*(list(N) + [1] * S)[:S])
    return lib.vd_evict_step(ctypes.byref(d), n_arr, N_arr, variant, rs, None, None, None, None,
                             0, None)


@pytest.mark.parametrize("field,value,status", [
    ("v", None, vd.VD_ERR_INVALID_ARG),
    ("dtype", 7, vd.VD_ERR_INVALID_ARG),
    ("num_seqs", 0, vd.VD_ERR_INVALID_ARG),
    ("num_layers", -1, vd.VD_ERR_INVALID_ARG),
    ("num_q_heads", 6, vd.VD_ERR_INVALID_ARG),      # not a multiple of the KV heads
    ("head_dim", 96, vd.VD_ERR_UNSUPPORTED),
    ("head_dim", 0, vd.VD_ERR_INVALID_ARG),
    ("capacity", 0, vd.VD_ERR_INVALID_ARG),
    ("capacity", vd.MAX_CAPACITY + 1, vd.VD_ERR_UNSUPPORTED),
    ("stride_slot", 64, vd.VD_ERR_INVALID_ARG),     # rows would overlap
    ("stride_slot", 132, vd.VD_ERR_INVALID_ARG),    # rows not 16-byte aligned
    ("stride_head", -128, vd.VD_ERR_INVALID_ARG),
    ("v", FAKE_V + 8, vd.VD_ERR_INVALID_ARG),       # misaligned base
    ("k", FAKE_V, vd.VD_ERR_INVALID_ARG),           # k aliases v
])
def test_descriptor_rejected(field, value, status):
    assert call_step(good_desc(**{field: value})) == status


def n_arr_2():
    return (ctypes.c_int32 * 2)(5, 5)


def test_counts_rejected():
    d = good_desc()
    assert call_step(d, n=(101, 5)) == vd.VD_ERR_INVALID_ARG    # n > capacity
    assert call_step(d, n=(-1, 5)) == vd.VD_ERR_INVALID_ARG
    assert call_step(d, N=(0, 5)) == vd.VD_ERR_INVALID_ARG      # budget < 1
    assert call_step(d, variant=7) == vd.VD_ERR_INVALID_ARG
    assert call_step(d, variant=6) == vd.VD_ERR_INVALID_ARG          # FastCAOTE: decode step only
    nok = good_desc()
    nok.k = None
    for key_variant in (3, 4, 5):                                     # key-side scores need K
        assert call_step(nok, variant=key_variant) == vd.VD_ERR_INVALID_ARG
        assert vd.load().vd_score(ctypes.byref(nok), n_arr_2(), key_variant, FAKE_V, None,
                                  None) == vd.VD_ERR_INVALID_ARG
    assert call_step(d, rs=ctypes.c_void_p(0x1004)) == vd.VD_ERR_INVALID_ARG  # misaligned state
    lib = vd.load()
    n_arr = (ctypes.c_int32 * 2)(5, 5)
    assert lib.vd_evict_step(ctypes.byref(d), n_arr, None, 0, None, None, None, None, None, 0,
                             None) == vd.VD_ERR_INVALID_ARG     # budget missing
    assert lib.vd_score(ctypes.byref(d), n_arr, 0, None, None, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_select_topn(ctypes.byref(d), None, n_arr, n_arr, None, None) == \
        vd.VD_ERR_INVALID_ARG
    assert lib.vd_compact(ctypes.byref(d), None, n_arr, n_arr, None, None) == \
        vd.VD_ERR_INVALID_ARG
    assert lib.vd_evict_step(None, n_arr, n_arr, 0, None, None, None, None, None, 0, None) == \
        vd.VD_ERR_INVALID_ARG


def test_status_strings_and_workspace():
    lib = vd.load()
    for s in range(5):
        assert lib.vd_status_string(s)
    assert lib.vd_evict_step_workspace_size(ctypes.byref(good_desc())) == 0


def test_stream_read_rejects_bad_arguments():
    lib = vd.load()
    good = 0x7F0000000000   # never dereferenced: validation fails first
    assert lib.vd_stream_read(None, 16, good, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_stream_read(good + 4, 16, good, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_stream_read(good, 24, good, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_stream_read(good, 0, good, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_stream_read(good, 16, None, None) == vd.VD_ERR_INVALID_ARG


def test_geometry_rejects_bad_arguments():
    lib = vd.load()
    n_arr = (ctypes.c_int32 * 2)(5, 5)
    out = ctypes.c_void_p(0x7F0000000000)
    sums = ctypes.c_void_p(0x7F0000200000)
    d = good_desc()
    d.k = None                                   # K is required
    assert lib.vd_geometry(ctypes.byref(d), n_arr, None, None, out, None) == vd.VD_ERR_INVALID_ARG
    d = good_desc()
    assert lib.vd_geometry(ctypes.byref(d), None, None, None, out, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_geometry(ctypes.byref(d), (ctypes.c_int32 * 2)(101, 5), None, None, out,
                           None) == vd.VD_ERR_INVALID_ARG            # n > capacity
    assert lib.vd_geometry(ctypes.byref(d), n_arr, None, None, None, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_geometry(ctypes.byref(d), n_arr, None, None, ctypes.c_void_p(0x7F0000000004),
                           None) == vd.VD_ERR_INVALID_ARG            # misaligned out
    assert lib.vd_geometry(ctypes.byref(d), n_arr, sums, None, out,
                           None) == vd.VD_ERR_INVALID_ARG            # one sum without the other
    assert lib.vd_geometry(ctypes.byref(d), n_arr, None, sums, out, None) == vd.VD_ERR_INVALID_ARG
    assert lib.vd_geometry(ctypes.byref(d), n_arr, sums, ctypes.c_void_p(0x7F0000200004), out,
                           None) == vd.VD_ERR_INVALID_ARG            # misaligned sum
    assert lib.vd_geometry(ctypes.byref(good_desc(head_dim=96)), n_arr, None, None, out,
                           None) == vd.VD_ERR_UNSUPPORTED


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(vd, "_lib", None)
    monkeypatch.setattr(vd, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        vd.load()


def call_decode(d, n=(50, 60), N=(49, 59), variant=0, q=FAKE_V, scale=0.1, rs=FAKE_V,
                pos=None, out=FAKE_V, ws=FAKE_V, ws_bytes=1 << 40):
    lib = vd.load()
    S = max(int(d.num_seqs), 1)
    n_arr = (ctypes.c_int32 * S)(*(list(n) + [0] * S)[:S])
    N_arr = None if N is None else (ctypes.c_int32 * S)(*(list(N) + [1] * S)[:S])
    return lib.vd_decode_attention_evict(ctypes.byref(d), q, scale, n_arr, N_arr, variant, rs, pos,
                                         out, ws, ws_bytes, None)


def decode_desc(**kw):
    return good_desc(**{"num_q_heads": 16, **kw})   # 4 KV heads, G = 4 by default


def test_decode_attention_rejections():
    """Every rejection path of vd_decode_attention_evict returns before any HIP
    call (the pointers are never dereferenced)."""
    d = decode_desc()
    bad_ptr = ctypes.c_void_p(FAKE_V + 4)
    assert call_decode(d, n=(51, 60)) == vd.VD_ERR_UNSUPPORTED        # n > N + 1
    # a budget of INT32_MAX passes the one-token check without overflow (q is
    # null so that validation still fails before any launch)
    assert call_decode(d, N=(2**31 - 1, 59), q=None) == vd.VD_ERR_INVALID_ARG
    assert call_decode(decode_desc(num_q_heads=12)) == vd.VD_ERR_UNSUPPORTED   # G = 3
    assert call_decode(decode_desc(num_q_heads=32)) == vd.VD_ERR_UNSUPPORTED   # G = 8
    assert call_decode(d, variant=1) == vd.VD_ERR_INVALID_ARG          # Dir is not a decode score
    assert call_decode(d, variant=7) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, scale=float("inf")) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, scale=float("nan")) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, rs=None) == vd.VD_ERR_INVALID_ARG            # state required
    assert call_decode(d, rs=bad_ptr) == vd.VD_ERR_INVALID_ARG         # misaligned state
    assert call_decode(d, q=None) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, out=None) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, q=ctypes.c_void_p(FAKE_V + 2)) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, pos=ctypes.c_void_p(FAKE_V + 2)) == vd.VD_ERR_INVALID_ARG
    assert call_decode(d, N=None) == vd.VD_ERR_INVALID_ARG             # budget missing
    assert call_decode(d, N=(0, 59)) == vd.VD_ERR_INVALID_ARG          # budget < 1
    assert call_decode(d, n=(101, 60)) == vd.VD_ERR_INVALID_ARG        # n > capacity
    assert call_decode(d, ws=None) == vd.VD_ERR_WORKSPACE
    assert call_decode(d, ws=ctypes.c_void_p(FAKE_V + 8)) == vd.VD_ERR_WORKSPACE  # misaligned
    need = vd.load().vd_decode_attention_workspace_size(ctypes.byref(d), 0)
    assert need > 0
    assert call_decode(d, ws_bytes=need - 1) == vd.VD_ERR_WORKSPACE    # short
    nok = decode_desc()
    nok.k = None
    assert call_decode(nok) == vd.VD_ERR_INVALID_ARG                   # K required


def test_decode_attention_workspace_sizes():
    lib = vd.load()
    d = decode_desc()
    l2 = lib.vd_decode_attention_workspace_size(ctypes.byref(d), 0)
    assert l2 > 0
    assert lib.vd_decode_attention_workspace_size(ctypes.byref(d), 1) == 0      # not a decode score
    assert lib.vd_decode_attention_workspace_size(ctypes.byref(good_desc(head_dim=96)), 0) == 0
