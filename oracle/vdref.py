"""ctypes front end of the C oracle (TEST INFRASTRUCTURE ONLY).

Arrays are numpy: bfloat16 data travels as its raw ``uint16`` bit patterns,
fp32 data as ``float32``.  Scores and means come back in float64.

``Oracle(path)`` wraps one build of ``vdref.c``; the module-level functions use
the default build ``oracle/libvdref.so``.  (The pin tests also load mutated
builds through ``Oracle`` to show that the pins catch plausible mistakes.)
"""
import ctypes
import os

import numpy as np

BF16 = 0
F32 = 1
L2 = 0
DIR = 1
NORM = 2
KEY_L2 = 3
KEY_DIR = 4
KEY_NORM = 5
VARIANTS = {"l2": L2, "dir": DIR, "norm": NORM, "key_l2": KEY_L2, "key_dir": KEY_DIR,
            "key_norm": KEY_NORM}

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvdref.so")

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int


def _dtype_tag(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return F32
    raise TypeError(f"oracle takes uint16 (bf16 bits) or float32, got {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _need_contig(a, name):
    if a is not None and not a.flags.c_contiguous:
        raise ValueError(f"{name} must be C-contiguous")


def _variant(v):
    return VARIANTS[v] if isinstance(v, str) else int(v)


class Oracle:
    def __init__(self, path: str = LIB_PATH):
        lib = ctypes.CDLL(path)
        lib.vdref_decode_elem.argtypes = [_p, _i32, _i64]
        lib.vdref_decode_elem.restype = ctypes.c_double
        lib.vdref_mean.argtypes = [_p, _i32, _i64, _i32, _i64, _p]
        lib.vdref_score.argtypes = [_p, _i32, _i64, _i32, _i64, _i32, _p, _p]
        lib.vdref_select_topn.argtypes = [_p, _i64, _i64, _p]
        lib.vdref_select_smallest.argtypes = [_p, _i64, _i64, _p]
        lib.vdref_fastcaote_scores.argtypes = [_p, _i32, _p, _p, _i32, _i64, _i32, _i64,
                                               ctypes.c_double, _p]
        lib.vdref_compact.argtypes = [_p, _p, _i32, _i64, _i64, _i32, _i64, _p, _p]
        lib.vdref_evict_step.argtypes = [_p, _p, _i32, _i64, _i64, _i32, _p, _p, _i32,
                                         _p, _p, _p, _p, _i32]
        lib.vdref_geometry.argtypes = [_p, _p, _i32, _i64, _i32, _i64, _p]
        lib.vdref_attention.argtypes = [_p, _p, _p, _i32, _i64, _i32, _i64, ctypes.c_double, _p]
        for f in ("vdref_mean", "vdref_score", "vdref_select_topn", "vdref_compact",
                  "vdref_evict_step", "vdref_geometry", "vdref_attention",
                  "vdref_select_smallest", "vdref_fastcaote_scores"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def decode_elems(self, rows: np.ndarray) -> np.ndarray:
        """Element values (float64) as the oracle reads them."""
        flat = np.ascontiguousarray(rows).reshape(-1)
        tag = _dtype_tag(flat)
        return np.array([self.lib.vdref_decode_elem(_ptr(flat), tag, i)
                         for i in range(flat.size)])

    def mean(self, v: np.ndarray) -> np.ndarray:
        """Mean of the n rows of ``v`` ([n, d])."""
        v = np.ascontiguousarray(v)
        n, d = v.shape
        out = np.empty(d, np.float64)
        if self.lib.vdref_mean(_ptr(v), _dtype_tag(v), n, d, d, _ptr(out)):
            raise ValueError("vdref_mean rejected its arguments")
        return out

    def score(self, v: np.ndarray, variant="l2"):
        """(scores [n], mean [d]) of the rows of ``v`` ([n, d]): the value rows
        for a value-side variant, the key rows for a key-side one."""
        v = np.ascontiguousarray(v)
        n, d = v.shape
        s = np.empty(n, np.float64)
        m = np.empty(d, np.float64)
        if self.lib.vdref_score(_ptr(v), _dtype_tag(v), n, d, d, _variant(variant),
                                _ptr(s), _ptr(m)):
            raise ValueError("vdref_score rejected its arguments")
        return s, m

    def select_topn(self, scores: np.ndarray, N: int) -> np.ndarray:
        """Keep mask (uint8 [n]) of the N highest scores, ties to the lower index."""
        scores = np.ascontiguousarray(scores, dtype=np.float64)
        n = scores.shape[0]
        keep = np.empty(n, np.uint8)
        if self.lib.vdref_select_topn(_ptr(scores), n, N, _ptr(keep)):
            raise ValueError("vdref_select_topn rejected its arguments")
        return keep

    def select_smallest(self, scores: np.ndarray, N: int) -> np.ndarray:
        """Keep mask (uint8 [n]) of the N lowest scores, ties to the lower index."""
        scores = np.ascontiguousarray(scores, dtype=np.float64)
        n = scores.shape[0]
        keep = np.empty(n, np.uint8)
        if self.lib.vdref_select_smallest(_ptr(scores), n, N, _ptr(keep)):
            raise ValueError("vdref_select_smallest rejected its arguments")
        return keep

    def fastcaote_scores(self, q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         scale: float) -> np.ndarray:
        """FastCAOTE scores (float64 [n]) of one decode step: q [G, d] (the
        query rows of the KV head, any float dtype, taken as fp64), k and v
        [n, d]."""
        k, v = np.ascontiguousarray(k), np.ascontiguousarray(v)
        q = np.ascontiguousarray(np.atleast_2d(q), dtype=np.float64)
        if k.shape != v.shape or k.dtype != v.dtype or q.shape[1] != v.shape[1]:
            raise ValueError("q [G, d], k and v [n, d] of one dtype")
        n, d = v.shape
        out = np.empty(n, np.float64)
        if self.lib.vdref_fastcaote_scores(_ptr(q), q.shape[0], _ptr(k), _ptr(v), _dtype_tag(v),
                                           n, d, d, float(scale), _ptr(out)):
            raise ValueError("vdref_fastcaote_scores rejected its arguments")
        return out

    def compact(self, k, v, n: int, N: int, keep: np.ndarray, pos=None):
        """Slot-reuse gather, in place, on [>=n, d] arrays ``k`` and ``v``."""
        ref = v if v is not None else k
        for a, nm in ((k, "k"), (v, "v"), (pos, "pos")):
            _need_contig(a, nm)
        keep = np.ascontiguousarray(keep, dtype=np.uint8)
        d = ref.shape[-1]
        if self.lib.vdref_compact(_ptr(k), _ptr(v), _dtype_tag(ref), n, N, d, d,
                                  _ptr(keep), _ptr(pos)):
            raise ValueError("vdref_compact rejected its arguments")

    def geometry(self, k: np.ndarray, v: np.ndarray) -> np.ndarray:
        """[sigma_K, sigma_V, mean ||k - k_bar||, mean ||v - v_bar||, bos-cosim]
        of the n rows of ``k`` and ``v`` ([n, d] each)."""
        k, v = np.ascontiguousarray(k), np.ascontiguousarray(v)
        if k.shape != v.shape or k.dtype != v.dtype:
            raise ValueError("k and v must share shape and dtype")
        n, d = v.shape
        out = np.empty(5, np.float64)
        if self.lib.vdref_geometry(_ptr(k), _ptr(v), _dtype_tag(v), n, d, d, _ptr(out)):
            raise ValueError("vdref_geometry rejected its arguments")
        return out

    def attention(self, q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
        """softmax(scale * q . k_j) weighted sum of the rows v_j: q [d] (any
        float dtype, taken as fp64), k and v [n, d]; returns float64 [d]."""
        k, v = np.ascontiguousarray(k), np.ascontiguousarray(v)
        q = np.ascontiguousarray(q, dtype=np.float64)
        if k.shape != v.shape or k.dtype != v.dtype or q.shape != (v.shape[1],):
            raise ValueError("q [d], k and v [n, d] of one dtype")
        n, d = v.shape
        out = np.empty(d, np.float64)
        if self.lib.vdref_attention(_ptr(q), _ptr(k), _ptr(v), _dtype_tag(v), n, d, d,
                                    float(scale), _ptr(out)):
            raise ValueError("vdref_attention rejected its arguments")
        return out

    def evict_step(self, k, v, n_unit, N_unit, variant="l2", pos=None, nthreads=0):
        """One eviction pass over U units, in place.

        k, v    : [U, cap, d] C-contiguous (uint16 bf16 bits or float32); k may be None
        n_unit  : [U] cached tokens per unit (the appended block included)
        N_unit  : [U] budget per unit
        pos     : optional int32 [U, cap] payload moved with the rows
        returns : (scores f64 [U, cap], keep u8 [U, cap], mean f64 [U, d]);
                  entries at or beyond a unit's n are left zero.
        """
        for a, nm in ((k, "k"), (v, "v"), (pos, "pos")):
            _need_contig(a, nm)
        U, cap, d = v.shape
        if k is not None and (k.shape != v.shape or k.dtype != v.dtype):
            raise ValueError("k and v must share shape and dtype")
        n_unit = np.ascontiguousarray(n_unit, dtype=np.int32).reshape(U)
        N_unit = np.ascontiguousarray(N_unit, dtype=np.int32).reshape(U)
        scores = np.zeros((U, cap), np.float64)
        keep = np.zeros((U, cap), np.uint8)
        means = np.zeros((U, d), np.float64)
        if self.lib.vdref_evict_step(_ptr(k), _ptr(v), _dtype_tag(v), U, cap, d,
                                     _ptr(n_unit), _ptr(N_unit), _variant(variant),
                                     _ptr(scores), _ptr(keep), _ptr(means), _ptr(pos),
                                     int(nthreads)):
            raise ValueError("vdref_evict_step rejected its arguments")
        return scores, keep, means


_default = None


def load() -> Oracle:
    """The default oracle build, compiled with gcc first if it is missing."""
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _build
            _build.build()
        _default = Oracle(LIB_PATH)
    return _default


def decode_elems(rows):
    return load().decode_elems(rows)


def mean(v):
    return load().mean(v)


def score(v, variant="l2"):
    return load().score(v, variant)


def select_topn(scores, N):
    return load().select_topn(scores, N)


def compact(k, v, n, N, keep, pos=None):
    return load().compact(k, v, n, N, keep, pos)


def evict_step(k, v, n_unit, N_unit, variant="l2", pos=None, nthreads=0):
    return load().evict_step(k, v, n_unit, N_unit, variant, pos, nthreads)


def geometry(k, v):
    return load().geometry(k, v)


def select_smallest(scores, N):
    return load().select_smallest(scores, N)


def fastcaote_scores(q, k, v, scale):
    return load().fastcaote_scores(q, k, v, scale)


def attention(q, k, v, scale):
    return load().attention(q, k, v, scale)
