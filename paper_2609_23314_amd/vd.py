"""Python binding of ``libvd.so`` (argument marshalling only).

The names follow the C ABI in ``include/vd.h``.  Tensors are torch tensors on
the GPU: torch supplies device memory and the stream, every step of the pass
runs in the library's HIP kernels.  There is no fallback: if the library is
missing or a call is rejected, an exception is raised.

Cache tensors ``k`` and ``v`` are 5-D views ``[seq, layer, kv_head, slot,
head_dim]`` with any strides whose last one is 1 (a per-layer ``[seq, slot,
kv_head, head_dim]`` cache is ``x.permute(0, 2, 1, 3).unsqueeze(1)``).
Per-unit arrays are ``[seq, layer, kv_head, ...]`` contiguous, i.e. unit
``u = (s * layers + l) * kv_heads + h``.
"""
import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvd.so")

VD_OK, VD_ERR_INVALID_ARG, VD_ERR_UNSUPPORTED, VD_ERR_WORKSPACE, VD_ERR_HIP = range(5)
VD_DTYPE_BF16, VD_DTYPE_F32 = 0, 1
VARIANTS = {"l2": 0, "dir": 1, "norm": 2, "key_l2": 3, "key_dir": 4, "key_norm": 5,
            "fastcaote": 6}
MAX_CAPACITY = 16384

EXPORTS = ("vd_score", "vd_select_topn", "vd_compact", "vd_evict_step",
           "vd_evict_step_workspace_size", "vd_status_string", "vd_stream_read",
           "vd_geometry", "vd_decode_attention_evict", "vd_decode_attention_workspace_size",
           "vd_decode_attention_evict_noalloc", "vd_decode_attention_noalloc_max_bytes")


class VdError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: {msg} (status {status})")
        self.status = status


class VdCacheDesc(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("dtype", ctypes.c_int32), ("num_seqs", ctypes.c_int32),
        ("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("capacity", ctypes.c_int32),
        ("stride_seq", ctypes.c_int64), ("stride_layer", ctypes.c_int64),
        ("stride_head", ctypes.c_int64), ("stride_slot", ctypes.c_int64),
    ]


_lib = None


def load():
    """Loads ``libvd.so``; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_23314_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(VdCacheDesc)
    lib.vd_score.argtypes = [D, P, I32, P, P, P]
    lib.vd_select_topn.argtypes = [D, P, P, P, P, P]
    lib.vd_compact.argtypes = [D, P, P, P, P, P]
    lib.vd_evict_step.argtypes = [D, P, P, I32, P, P, P, P, P, SZ, P]
    for f in ("vd_score", "vd_select_topn", "vd_compact", "vd_evict_step"):
        getattr(lib, f).restype = ctypes.c_int
    lib.vd_evict_step_workspace_size.argtypes = [D]
    lib.vd_evict_step_workspace_size.restype = ctypes.c_size_t
    lib.vd_status_string.argtypes = [ctypes.c_int]
    lib.vd_status_string.restype = ctypes.c_char_p
    lib.vd_stream_read.argtypes = [P, SZ, P, P]
    lib.vd_stream_read.restype = ctypes.c_int
    lib.vd_geometry.argtypes = [D, P, P, P, P, P]
    lib.vd_geometry.restype = ctypes.c_int
    lib.vd_decode_attention_evict.argtypes = [D, P, ctypes.c_float, P, P, I32, P, P, P, P, SZ, P]
    lib.vd_decode_attention_evict.restype = ctypes.c_int
    lib.vd_decode_attention_workspace_size.argtypes = [D, I32]
    lib.vd_decode_attention_evict_noalloc.argtypes = [D, P, ctypes.c_float, P, P, I32, P, P, P, P]
    lib.vd_decode_attention_evict_noalloc.restype = ctypes.c_int
    lib.vd_decode_attention_noalloc_max_bytes.argtypes = []
    lib.vd_decode_attention_noalloc_max_bytes.restype = ctypes.c_size_t
    lib.vd_decode_attention_workspace_size.restype = ctypes.c_size_t
    _lib = lib
    return lib


def _check(fn, status):
    if status != VD_OK:
        raise VdError(fn, status, load().vd_status_string(status).decode())


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return VD_DTYPE_BF16
    if t.dtype == torch.float32:
        return VD_DTYPE_F32
    raise TypeError(f"cache dtype must be bfloat16 or float32, got {t.dtype}")


def cache_desc(v, k=None, num_q_heads=None) -> VdCacheDesc:
    """Descriptor of a 5-D ``[seq, layer, kv_head, slot, head_dim]`` cache view."""
    if v.dim() != 5:
        raise ValueError("v must be a 5-D [seq, layer, kv_head, slot, head_dim] view")
    if v.stride(4) != 1:
        raise ValueError("the head_dim stride must be 1")
    if k is not None and (k.shape != v.shape or k.stride() != v.stride() or k.dtype != v.dtype):
        raise ValueError("k must match v in shape, strides and dtype")
    S, L, H, C, Dh = v.shape
    d = VdCacheDesc()
    d.k = k.data_ptr() if k is not None else None
    d.v = v.data_ptr()
    d.dtype = _dtype_code(v)
    d.num_seqs, d.num_layers, d.num_kv_heads = S, L, H
    d.num_q_heads = H if num_q_heads is None else int(num_q_heads)
    d.head_dim, d.capacity = Dh, C
    d.stride_seq, d.stride_layer, d.stride_head, d.stride_slot = v.stride()[:4]
    return d


def _host_i32(x, S, name):
    t = torch.as_tensor(x, dtype=torch.int32).reshape(-1).cpu().contiguous()
    if t.numel() != S:
        raise ValueError(f"{name} must have one entry per sequence ({S})")
    return t


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(dev, stream):
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    return s.cuda_stream


def _units(v):
    S, L, H = v.shape[:3]
    return S * L * H


def _need(t, name, dtype, numel, dev):
    if t.dtype != dtype or not t.is_contiguous() or t.numel() < numel or t.device != dev:
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of >= {numel} "
                         f"elements on {dev}")


def vd_score(v, n_valid, variant="l2", scores=None, mean_out=None, *, k=None,
             num_q_heads=None, stream=None):
    """Mean and scores of every unit; returns (scores [U, cap] f32, mean_out or None)."""
    U, C, Dh = _units(v), v.shape[3], v.shape[4]
    desc = cache_desc(v, k, num_q_heads)
    n_h = _host_i32(n_valid, v.shape[0], "n_valid")
    if scores is None:
        scores = torch.empty((U, C), dtype=torch.float32, device=v.device)
    _need(scores, "scores", torch.float32, U * C, v.device)
    if mean_out is not None:
        _need(mean_out, "mean_out", torch.float32, U * Dh, v.device)
    _check("vd_score", load().vd_score(ctypes.byref(desc), _ptr(n_h), VARIANTS[variant],
                                       _ptr(scores), _ptr(mean_out), _stream(v.device, stream)))
    return scores, mean_out


def vd_select_topn(v, scores, n_valid, budget, keep_mask=None, *, stream=None):
    """Keep mask (uint8 [U, cap]) of the N highest scores of every unit."""
    U, C = _units(v), v.shape[3]
    desc = cache_desc(v)
    n_h = _host_i32(n_valid, v.shape[0], "n_valid")
    b_h = _host_i32(budget, v.shape[0], "budget")
    _need(scores, "scores", torch.float32, U * C, v.device)
    if keep_mask is None:
        keep_mask = torch.empty((U, C), dtype=torch.uint8, device=v.device)
    _need(keep_mask, "keep_mask", torch.uint8, U * C, v.device)
    _check("vd_select_topn", load().vd_select_topn(ctypes.byref(desc), _ptr(scores), _ptr(n_h),
                                                   _ptr(b_h), _ptr(keep_mask),
                                                   _stream(v.device, stream)))
    return keep_mask


def vd_compact(k, v, keep_mask, n_valid, budget, pos=None, *, stream=None):
    """Slot-reuse gather of K, V (and pos) from a keep mask, in place."""
    U, C = _units(v), v.shape[3]
    desc = cache_desc(v, k)
    n_h = _host_i32(n_valid, v.shape[0], "n_valid")
    b_h = _host_i32(budget, v.shape[0], "budget")
    _need(keep_mask, "keep_mask", torch.uint8, U * C, v.device)
    if pos is not None:
        _need(pos, "pos", torch.int32, U * C, v.device)
    _check("vd_compact", load().vd_compact(ctypes.byref(desc), _ptr(keep_mask), _ptr(n_h),
                                           _ptr(b_h), _ptr(pos), _stream(v.device, stream)))


def vd_evict_step_workspace_size(v, k=None):
    desc = cache_desc(v, k)
    return int(load().vd_evict_step_workspace_size(ctypes.byref(desc)))


def vd_evict_step(k, v, n_valid, budget, variant="l2", running_sum=None, pos=None,
                  scores_out=None, keep_out=None, workspace=None, *, num_q_heads=None,
                  stream=None):
    """One eviction pass over every unit, in place (see ``vd_evict_step`` in vd.h)."""
    U, C, Dh = _units(v), v.shape[3], v.shape[4]
    desc = cache_desc(v, k, num_q_heads)
    n_h = _host_i32(n_valid, v.shape[0], "n_valid")
    b_h = _host_i32(budget, v.shape[0], "budget")
    if running_sum is not None:
        _need(running_sum, "running_sum", torch.float64, U * (Dh + 1), v.device)
    if pos is not None:
        _need(pos, "pos", torch.int32, U * C, v.device)
    if scores_out is not None:
        _need(scores_out, "scores_out", torch.float32, U * C, v.device)
    if keep_out is not None:
        _need(keep_out, "keep_out", torch.uint8, U * C, v.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vd_evict_step", load().vd_evict_step(
        ctypes.byref(desc), _ptr(n_h), _ptr(b_h), VARIANTS[variant], _ptr(running_sum),
        _ptr(pos), _ptr(scores_out), _ptr(keep_out), _ptr(workspace), ws_bytes,
        _stream(v.device, stream)))


def vd_geometry(k, v, n_valid, out=None, *, k_sum=None, v_sum=None, stream=None):
    """Key and value geometry of every unit (see ``vd_geometry`` in vd.h):
    float64 [U, 5] = sigma_K, sigma_V, mean ||k - k_bar||, mean ||v - v_bar||,
    bos-cosim.  k_sum / v_sum: optional float64 [U, D + 1] column sums and
    row counts (both or neither)."""
    U, Dh = _units(v), v.shape[4]
    if k is None:
        raise ValueError("vd_geometry needs k")
    desc = cache_desc(v, k)
    n_h = _host_i32(n_valid, v.shape[0], "n_valid")
    if out is None:
        out = torch.empty((U, 5), dtype=torch.float64, device=v.device)
    _need(out, "out", torch.float64, U * 5, v.device)
    for t, nm in ((k_sum, "k_sum"), (v_sum, "v_sum")):
        if t is not None:
            _need(t, nm, torch.float64, U * (Dh + 1), v.device)
    _check("vd_geometry", load().vd_geometry(ctypes.byref(desc), _ptr(n_h), _ptr(k_sum),
                                             _ptr(v_sum), _ptr(out), _stream(v.device, stream)))
    return out


def vd_decode_attention_workspace_size(k, v, num_q_heads, variant="l2"):
    desc = cache_desc(v, k, num_q_heads)
    return int(load().vd_decode_attention_workspace_size(ctypes.byref(desc), VARIANTS[variant]))


def _decode_args(k, v, q, n_valid, budget, running_sum, pos, out):
    if k is None:
        raise ValueError("the fused decode step needs k")
    S, L, H, C, Dh = v.shape
    if q.dim() != 4 or q.shape[0] != S or q.shape[1] != L or q.shape[3] != Dh:
        raise ValueError("q must be [S, L, Hq, D] matching the cache")
    U = _units(v)
    desc = cache_desc(v, k, q.shape[2])
    n_h = _host_i32(n_valid, S, "n_valid")
    b_h = _host_i32(budget, S, "budget")
    _need(q, "q", torch.float32, q.numel(), v.device)
    _need(running_sum, "running_sum", torch.float64, U * (Dh + 1), v.device)
    if pos is not None:
        _need(pos, "pos", torch.int32, U * C, v.device)
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=v.device)
    _need(out, "out", torch.float32, q.numel(), v.device)
    return desc, n_h, b_h, out


def vd_decode_attention_evict(k, v, q, n_valid, budget, running_sum, scale=None, pos=None,
                              out=None, workspace=None, *, variant="l2", stream=None):
    """One decode step fused with its eviction (see ``vd_decode_attention_evict``
    in vd.h): q is float32 [S, L, Hq, D]; returns the attention output (float32,
    q's shape).  K, V, pos and the running sum are updated in place.  variant is
    "l2" (ValueDiff) or "fastcaote"."""
    desc, n_h, b_h, out = _decode_args(k, v, q, n_valid, budget, running_sum, pos, out)
    ws_need = int(load().vd_decode_attention_workspace_size(ctypes.byref(desc), VARIANTS[variant]))
    if workspace is None:
        workspace = torch.zeros(max(ws_need, 16), dtype=torch.uint8, device=v.device)
    ws_bytes = workspace.numel() * workspace.element_size()
    sc = float(v.shape[4]) ** -0.5 if scale is None else float(scale)
    _check("vd_decode_attention_evict", load().vd_decode_attention_evict(
        ctypes.byref(desc), _ptr(q), sc, _ptr(n_h), _ptr(b_h), VARIANTS[variant],
        _ptr(running_sum), _ptr(pos), _ptr(out), _ptr(workspace), ws_bytes,
        _stream(v.device, stream)))
    return out


def vd_decode_attention_evict_noalloc(k, v, q, n_valid, budget, running_sum, out, scale=None,
                                      pos=None, *, variant="l2", stream=None):
    """The fused decode step without a workspace (see
    ``vd_decode_attention_evict_noalloc`` in vd.h): the library's static device
    scratch holds the split partials.  ``out`` is required (float32, q's
    shape); nothing is allocated here."""
    if out is None:
        raise ValueError("out is required: the allocation-free call allocates nothing")
    desc, n_h, b_h, out = _decode_args(k, v, q, n_valid, budget, running_sum, pos, out)
    sc = float(v.shape[4]) ** -0.5 if scale is None else float(scale)
    _check("vd_decode_attention_evict_noalloc", load().vd_decode_attention_evict_noalloc(
        ctypes.byref(desc), _ptr(q), sc, _ptr(n_h), _ptr(b_h), VARIANTS[variant],
        _ptr(running_sum), _ptr(pos), _ptr(out), _stream(v.device, stream)))
    return out


def vd_decode_attention_noalloc_max_bytes():
    return int(load().vd_decode_attention_noalloc_max_bytes())


def vd_stream_read(buf, sink, *, stream=None):
    """One streaming read of the whole of ``buf`` (a measurement aid: the
    practical HBM read ceiling next to the pass); ``sink`` is a device int32
    tensor of at least one element."""
    if not buf.is_contiguous() or sink.dtype != torch.int32 or sink.device != buf.device:
        raise ValueError("buf must be contiguous and sink an int32 tensor on the same device")
    _check("vd_stream_read", load().vd_stream_read(_ptr(buf), buf.numel() * buf.element_size(),
                                                   _ptr(sink), _stream(buf.device, stream)))
