"""CPU oracle for the 3LC compression path (paper Sections 3.1-3.3).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP library: the arithmetic lives in ``tlc_ref.c`` (plain C, one thread,
the paper's step order); this module only marshals numpy arrays through
ctypes.

Every wrapper takes and returns host numpy arrays.
"""
import ctypes
import os

import numpy as np

from . import build as _build

OK = 0
E_INVALID = -1
E_CAPACITY = -2
E_NONFINITE = -3
E_CORRUPT = -4

_lib = None


def lib():
    """Load (building first if needed) the oracle shared library.
    TLC_REF_LIBRARY may name a build of a changed copy of tlc_ref.c: the
    mutation test plants mistakes that way and runs the pins against them."""
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("TLC_REF_LIBRARY")
    if not path:
        path = _build.LIB
        src = os.path.join(_build.HERE, "tlc_ref.c")
        if (not os.path.exists(_build.LIB)
                or os.path.getmtime(_build.LIB) < os.path.getmtime(src)):
            _build.build()
    L = ctypes.CDLL(path)
    c_sz, c_f, c_i = ctypes.c_size_t, ctypes.c_float, ctypes.c_int
    vp = ctypes.c_void_p
    L.tlc_ref_quartic_len.argtypes = [c_sz]
    L.tlc_ref_quartic_len.restype = c_sz
    L.tlc_ref_accumulate.argtypes = [vp, vp, c_sz, vp]
    L.tlc_ref_accumulate.restype = None
    L.tlc_ref_absmax_scale.argtypes = [vp, c_sz, c_f, ctypes.POINTER(c_f)]
    L.tlc_ref_absmax_scale.restype = c_i
    L.tlc_ref_quantize.argtypes = [vp, c_sz, c_f, vp, vp]
    L.tlc_ref_quantize.restype = None
    L.tlc_ref_dequantize.argtypes = [vp, c_sz, c_f, vp, c_i]
    L.tlc_ref_dequantize.restype = None
    L.tlc_ref_quartic_encode.argtypes = [vp, c_sz, vp]
    L.tlc_ref_quartic_encode.restype = None
    L.tlc_ref_quartic_decode.argtypes = [vp, c_sz, vp]
    L.tlc_ref_quartic_decode.restype = None
    L.tlc_ref_zre_encode.argtypes = [vp, c_sz, vp]
    L.tlc_ref_zre_encode.restype = c_sz
    L.tlc_ref_zre_decode.argtypes = [vp, c_sz, vp, c_sz]
    L.tlc_ref_zre_decode.restype = c_i
    L.tlc_ref_compress.argtypes = [vp, vp, c_sz, c_f, vp, c_sz,
                                   ctypes.POINTER(c_sz), ctypes.POINTER(c_f)]
    L.tlc_ref_compress.restype = c_i
    L.tlc_ref_compress_in_place.argtypes = [vp, vp, c_sz, c_f, vp, c_sz,
                                            ctypes.POINTER(c_sz), ctypes.POINTER(c_f)]
    L.tlc_ref_compress_in_place.restype = c_i
    L.tlc_ref_decompress.argtypes = [vp, c_sz, c_f, c_sz, vp, c_i]
    L.tlc_ref_decompress.restype = c_i
    L.tlc_ref_philox4x32_10.argtypes = [vp, vp, vp]
    L.tlc_ref_philox4x32_10.restype = None
    L.tlc_ref_compress_nozre.argtypes = [vp, vp, c_sz, c_f, vp, c_sz,
                                         ctypes.POINTER(c_sz), ctypes.POINTER(c_f), c_i]
    L.tlc_ref_compress_nozre.restype = c_i
    u64 = ctypes.c_uint64
    L.tlc_ref_compress_stochastic.argtypes = [vp, c_sz, c_f, u64, u64, vp, c_sz,
                                              ctypes.POINTER(c_sz), ctypes.POINTER(c_f)]
    L.tlc_ref_compress_stochastic.restype = c_i
    L.tlc_ref_int8_step.argtypes = [c_f]
    L.tlc_ref_int8_step.restype = c_f
    L.tlc_ref_int8_quantize.argtypes = [vp, c_sz, c_f, vp, vp]
    L.tlc_ref_int8_quantize.restype = None
    L.tlc_ref_compress_int8.argtypes = [vp, vp, c_sz, c_f, vp, c_sz,
                                        ctypes.POINTER(c_sz), ctypes.POINTER(c_f), c_i]
    L.tlc_ref_compress_int8.restype = c_i
    L.tlc_ref_decompress_int8.argtypes = [vp, c_sz, c_f, c_sz, vp, c_i]
    L.tlc_ref_decompress_int8.restype = c_i
    _lib = L
    return L


def _ptr(a):
    return a.ctypes.data if a.size else None


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def quartic_len(n):
    return int(lib().tlc_ref_quartic_len(n))


def accumulate(x, r):
    x, r = _f32(x), _f32(r)
    acc = np.empty_like(x)
    lib().tlc_ref_accumulate(_ptr(x), _ptr(r), x.size, _ptr(acc))
    return acc


def absmax_scale(acc, s):
    """Return (status, M)."""
    acc = _f32(acc)
    M = ctypes.c_float(0.0)
    st = lib().tlc_ref_absmax_scale(_ptr(acc), acc.size, s, ctypes.byref(M))
    return st, M.value


def quantize(acc, M):
    """Return (q int8, residual float32)."""
    acc = _f32(acc)
    q = np.empty(acc.size, dtype=np.int8)
    r = np.empty_like(acc)
    lib().tlc_ref_quantize(_ptr(acc), acc.size, M, _ptr(q), _ptr(r))
    return q, r


def dequantize(q, M, out=None, accumulate=False):
    q = np.ascontiguousarray(q, dtype=np.int8)
    if out is None:
        out = np.empty(q.size, dtype=np.float32)
    lib().tlc_ref_dequantize(_ptr(q), q.size, M, _ptr(out), int(accumulate))
    return out


def quartic_encode(q):
    q = np.ascontiguousarray(q, dtype=np.int8)
    Q = np.empty(quartic_len(q.size), dtype=np.uint8)
    lib().tlc_ref_quartic_encode(_ptr(q), q.size, _ptr(Q))
    return Q


def quartic_decode(Q, n):
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    assert Q.size == quartic_len(n)
    q = np.empty(n, dtype=np.int8)
    lib().tlc_ref_quartic_decode(_ptr(Q), n, _ptr(q))
    return q


def zre_encode(Q):
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    out = np.empty(Q.size, dtype=np.uint8)
    c = lib().tlc_ref_zre_encode(_ptr(Q), Q.size, _ptr(out))
    return out[:c].copy()


def zre_decode(C, m):
    """Return (status, Q)."""
    C = np.ascontiguousarray(C, dtype=np.uint8)
    Q = np.empty(m, dtype=np.uint8)
    st = lib().tlc_ref_zre_decode(_ptr(C), C.size, _ptr(Q), m)
    return st, Q


def compress(x, r, s, cap=None, in_place=False):
    """Encode x with error buffer r (updated in place, float32 contiguous).
    in_place: tlc_ref_compress_in_place (on NaN/Inf r keeps x + r).

    Return (status, bytes uint8[len], M).
    """
    x = _f32(x)
    assert r.dtype == np.float32 and r.flags.c_contiguous and r.size == x.size
    n = x.size
    m = quartic_len(n)
    if cap is None:
        cap = m
    out = np.zeros(max(cap, 1), dtype=np.uint8)
    ln = ctypes.c_size_t(0)
    M = ctypes.c_float(0.0)
    fn = lib().tlc_ref_compress_in_place if in_place else lib().tlc_ref_compress
    st = fn(_ptr(x), _ptr(r), n, s, out.ctypes.data, cap, ctypes.byref(ln), ctypes.byref(M))
    return st, out[:ln.value].copy(), M.value


def decompress(C, M, n, out=None, accumulate=False):
    """Decode into out (float32, created as zeros if None).  Return (status, out)."""
    C = np.ascontiguousarray(C, dtype=np.uint8)
    if out is None:
        out = np.zeros(n, dtype=np.float32)
    assert out.dtype == np.float32 and out.flags.c_contiguous and out.size == n
    st = lib().tlc_ref_decompress(_ptr(C), C.size, M, n, _ptr(out),
                                  int(accumulate))
    return st, out


def philox4x32_10(ctr, key):
    """Four 32-bit words of Philox4x32-10 for a 4-word counter and 2-word key."""
    c = np.array(ctr, dtype=np.uint32)
    k = np.array(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().tlc_ref_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return [int(v) for v in out]


def compress_nozre(x, r, s, in_place=False):
    """Quantize + quartic encode without zero-run encoding; r updated in place.
    Return (status, bytes, M)."""
    x = _f32(x)
    assert r.dtype == np.float32 and r.flags.c_contiguous and r.size == x.size
    m = quartic_len(x.size)
    out = np.zeros(max(m, 1), dtype=np.uint8)
    ln = ctypes.c_size_t(0)
    M = ctypes.c_float(0.0)
    st = lib().tlc_ref_compress_nozre(_ptr(x), _ptr(r), x.size, s, out.ctypes.data, m,
                                      ctypes.byref(ln), ctypes.byref(M), int(in_place))
    return st, out[:ln.value].copy(), M.value


def compress_stochastic(x, s, seed, step):
    """Stochastic 3-value quantization + quartic encoding.  Return (status,
    bytes, M)."""
    x = _f32(x)
    m = quartic_len(x.size)
    out = np.zeros(max(m, 1), dtype=np.uint8)
    ln = ctypes.c_size_t(0)
    M = ctypes.c_float(0.0)
    st = lib().tlc_ref_compress_stochastic(_ptr(x), x.size, s, seed, step, out.ctypes.data,
                                           m, ctypes.byref(ln), ctypes.byref(M))
    return st, out[:ln.value].copy(), M.value


def int8_step(M):
    """The 8-bit comparator's quantization step fl(M / 127)."""
    return lib().tlc_ref_int8_step(M)


def int8_quantize(acc, M, residual=True):
    """8-bit codes of acc at scale M.  Return (q int8, residual or None)."""
    acc = _f32(acc)
    q = np.zeros(acc.size, dtype=np.int8)
    res = np.zeros(acc.size, dtype=np.float32) if residual else None
    lib().tlc_ref_int8_quantize(_ptr(acc), acc.size, M, _ptr(q),
                                _ptr(res) if residual else None)
    return q, res


def compress_int8(x, r, s, in_place=False):
    """8-bit encode; r (float32, updated in place) or None for no error
    feedback.  Return (status, bytes, M)."""
    x = _f32(x)
    if r is not None:
        assert r.dtype == np.float32 and r.flags.c_contiguous and r.size == x.size
    out = np.zeros(max(x.size, 1), dtype=np.uint8)
    ln = ctypes.c_size_t(0)
    M = ctypes.c_float(0.0)
    st = lib().tlc_ref_compress_int8(_ptr(x), _ptr(r) if r is not None else None, x.size, s,
                                     out.ctypes.data, x.size, ctypes.byref(ln), ctypes.byref(M),
                                     int(in_place))
    return st, out[:ln.value].copy(), M.value


def decompress_int8(C, M, n, out=None, accumulate=False):
    """8-bit decode into out (float32, zeros if None).  Return (status, out)."""
    C = np.ascontiguousarray(C, dtype=np.uint8)
    if out is None:
        out = np.zeros(n, dtype=np.float32)
    assert out.dtype == np.float32 and out.flags.c_contiguous and out.size == n
    st = lib().tlc_ref_decompress_int8(_ptr(C), C.size, M, n, _ptr(out), int(accumulate))
    return st, out
