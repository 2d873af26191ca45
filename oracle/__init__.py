"""CPU oracle for the KVLink hot path (arXiv 2502.16002).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It never imports the GPU
package and the GPU package never imports it.

Thin numpy wrappers over ``libkvlink_oracle.so`` (plain C, double precision,
long-double RoPE angles).  Every function follows a passage of the paper:

* :func:`layout`, :func:`allowed`, :func:`full_mask` -- the concatenated
  sequence with link tokens and its attention map (Sec. 2.3, Fig. 2).
* :func:`rope`, :func:`reencode` -- RoPE and the positional re-encoding of
  cached keys (Sec. 2.2).
* :func:`attend`, :func:`attend_probs` -- attention of the link and query tokens
  over the concatenated sequence (Sec. 2.3, last paragraph).
"""
import ctypes
import os

import numpy as np

from . import build as _build

KIND_DOC, KIND_LINK, KIND_QUERY = 0, 1, 2

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        ip = ctypes.POINTER(ctypes.c_int)
        dp = ctypes.POINTER(ctypes.c_double)
        llp = ctypes.POINTER(ctypes.c_longlong)
        i, d, ll = ctypes.c_int, ctypes.c_double, ctypes.c_longlong
        lib.kvo_num_threads.restype = i
        lib.kvo_layout.argtypes = [i, ip, ip, i, ip, ip, ip]
        lib.kvo_layout.restype = i
        lib.kvo_allowed.argtypes = [ip, ip, i, i]
        lib.kvo_allowed.restype = i
        lib.kvo_full_mask.argtypes = [i, ip, ip, ctypes.POINTER(ctypes.c_ubyte)]
        lib.kvo_rope.argtypes = [dp, i, ll, d]
        lib.kvo_reencode.argtypes = [dp, dp, ll, i, ll, d]
        lib.kvo_reencode.restype = i
        lib.kvo_attend.argtypes = [i, ip, ip, i, llp, i, i, i, d, d,
                                   dp, dp, dp, dp, dp, i, ip, dp, dp]
        lib.kvo_attend.restype = i
        lib.kvo_attend_probs.argtypes = [i, ip, ip, i, llp, i, i, i, d, d,
                                         dp, dp, dp, i, i, dp]
        lib.kvo_attend_probs.restype = i
        _lib = lib
    return _lib


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct)) if a is not None else None


def num_threads():
    return _load().kvo_num_threads()


def layout(doc_len, link_count, n_query):
    """Per global position: (kind, seg, idx) int32 arrays (Sec. 2.3)."""
    lib = _load()
    dl, lc = _i32(doc_len), _i32(link_count)
    T = lib.kvo_layout(len(dl), _ptr(dl, ctypes.c_int), _ptr(lc, ctypes.c_int), int(n_query),
                       None, None, None)
    if T < 0:
        raise ValueError("invalid layout")
    kind, seg, idx = (np.zeros(T, np.int32) for _ in range(3))
    lib.kvo_layout(len(dl), _ptr(dl, ctypes.c_int), _ptr(lc, ctypes.c_int), int(n_query),
                   _ptr(kind, ctypes.c_int), _ptr(seg, ctypes.c_int), _ptr(idx, ctypes.c_int))
    return kind, seg, idx


def allowed(kind, seg, a, b):
    kind, seg = _i32(kind), _i32(seg)
    return bool(_load().kvo_allowed(_ptr(kind, ctypes.c_int), _ptr(seg, ctypes.c_int), a, b))


def full_mask(kind, seg):
    kind, seg = _i32(kind), _i32(seg)
    T = len(kind)
    m = np.zeros((T, T), np.uint8)
    _load().kvo_full_mask(T, _ptr(kind, ctypes.c_int), _ptr(seg, ctypes.c_int),
                          _ptr(m, ctypes.c_ubyte))
    return m.astype(bool)


def rope(x, pos, theta):
    """R_pos x for one vector x of even length d (Sec. 2.2)."""
    y = _f64(x).copy()
    _load().kvo_rope(_ptr(y, ctypes.c_double), y.shape[-1], int(pos), float(theta))
    return y


def reencode(k, delta, theta):
    """R_delta applied to every length-d vector along the last axis of k."""
    k = _f64(k)
    out = np.empty_like(k)
    d = k.shape[-1]
    rc = _load().kvo_reencode(_ptr(k, ctypes.c_double), _ptr(out, ctypes.c_double),
                              k.size // d, d, int(delta), float(theta))
    if rc:
        raise ValueError("invalid head_dim")
    return out


def attend(doc_len, link_count, n_query, q_new, k_new, v_new, k_cached, v_cached,
           theta, scale, rows=None, src_pos0=None):
    """Attention output and LSE of the new tokens of one request, one layer.

    k_cached, v_cached: [H_kv, T_c, d] (documents back to back);
    q_new: [n_new, H_q, d]; k_new, v_new: [n_new, H_kv, d] (pre-RoPE).
    Returns (out [n_rows, H_q, d], lse [n_rows, H_q]).
    """
    lib = _load()
    dl, lc = _i32(doc_len), _i32(link_count)
    q, kn, vn = _f64(q_new), _f64(k_new), _f64(v_new)
    kc, vc = _f64(k_cached), _f64(v_cached)
    n_new, hq, d = q.shape
    hkv = kn.shape[1]
    r = None if rows is None else _i32(rows)
    nr = n_new if r is None else len(r)
    sp = None if src_pos0 is None else np.ascontiguousarray(np.asarray(src_pos0, np.int64))
    out = np.zeros((nr, hq, d), np.float64)
    lse = np.zeros((nr, hq), np.float64)
    rc = lib.kvo_attend(len(dl), _ptr(dl, ctypes.c_int), _ptr(lc, ctypes.c_int), int(n_query),
                        _ptr(sp, ctypes.c_longlong), hq, hkv, d, float(theta), float(scale),
                        _ptr(kc, ctypes.c_double), _ptr(vc, ctypes.c_double),
                        _ptr(q, ctypes.c_double), _ptr(kn, ctypes.c_double),
                        _ptr(vn, ctypes.c_double), nr, _ptr(r, ctypes.c_int),
                        _ptr(out, ctypes.c_double), _ptr(lse, ctypes.c_double))
    if rc:
        raise ValueError("invalid attention input")
    return out, lse


def attend_probs(doc_len, link_count, n_query, q_new, k_new, k_cached, theta, scale,
                 row, head, src_pos0=None):
    """Softmax row (length T, zeros where masked) of one new token and head."""
    lib = _load()
    dl, lc = _i32(doc_len), _i32(link_count)
    q, kn, kc = _f64(q_new), _f64(k_new), _f64(k_cached)
    n_new, hq, d = q.shape
    hkv = kn.shape[1]
    T = lib.kvo_layout(len(dl), _ptr(dl, ctypes.c_int), _ptr(lc, ctypes.c_int), int(n_query),
                       None, None, None)
    sp = None if src_pos0 is None else np.ascontiguousarray(np.asarray(src_pos0, np.int64))
    probs = np.zeros(max(T, 1), np.float64)
    rc = lib.kvo_attend_probs(len(dl), _ptr(dl, ctypes.c_int), _ptr(lc, ctypes.c_int),
                              int(n_query), _ptr(sp, ctypes.c_longlong), hq, hkv, d,
                              float(theta), float(scale), _ptr(kc, ctypes.c_double),
                              _ptr(q, ctypes.c_double), _ptr(kn, ctypes.c_double),
                              int(row), int(head), _ptr(probs, ctypes.c_double))
    if rc < 0:
        raise ValueError("invalid attention input")
    return probs[:T]
