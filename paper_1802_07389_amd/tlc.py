"""ctypes binding of ``libtlc.so`` (declared in ``include/tlc.h``).

Argument marshalling only: every step of encode and decode runs in the HIP
kernels of the library.  The functions keep the C names; ``Context`` wraps
them for torch tensors (torch provides device memory and the stream, nothing
else).  Importing this module raises ImportError when the library has not
been built -- there is no fallback.
"""
import ctypes
import os

import torch  # load torch's HIP runtime first so libtlc binds to the same one

_HERE = os.path.dirname(os.path.abspath(__file__))
# TLC_LIBRARY may name another build of this same library (the look-back
# stress build libtlc_delay.so, which the stress test loads this way).
LIB_PATH = os.environ.get("TLC_LIBRARY") or os.path.join(_HERE, "libtlc.so")

TLC_OK = 0
TLC_E_INVALID = -1
TLC_E_CAPACITY = -2
TLC_E_NONFINITE = -3
TLC_E_CORRUPT = -4
TLC_E_DEVICE = -5

TLC_MAX_N = 4294967295
TLC_MAX_TENSORS = 65536

TLC_KERNEL_ABSMAX = 0
TLC_KERNEL_QUANT_ENCODE = 1
TLC_KERNEL_ZRE_INDEX = 2
TLC_KERNEL_EXPAND_DEQUANT = 3
TLC_KERNEL_ABSMAX_BATCH = 4
TLC_KERNEL_QUANT_ENCODE_BATCH = 5
TLC_KERNEL_ZRE_INDEX_BATCH = 6
TLC_KERNEL_EXPAND_DEQUANT_BATCH = 7
TLC_KERNEL_EXPAND_SUM = 8
TLC_KERNEL_QUANT_PACK = 9
TLC_KERNEL_INT8_QUANT = 10
TLC_KERNEL_INT8_DEQUANT = 11
TLC_KERNEL_ZRE_CHUNKS = 12
TLC_KERNEL_ZRE_COMPACT = 13
TLC_KERNEL_QUANT_ENCODE_CHAINED = 14
TLC_KERNEL_ABSMAX_CHECK = 15
TLC_KERNEL_ABSMAX_CHECK_BATCH = 16
TLC_KERNEL_ACCUM_QUANTIZE = 17
TLC_KERNEL_COUNT = 18

TLC_OPT_IN_PLACE_FEEDBACK = 1

TLC_NOALLOC_MAX_N = 8388608
TLC_ENC_EPOCH_MAX = 8388607
TLC_DEC_EPOCH_MAX = 67108863

TLC_MODE_3LC = 0
TLC_MODE_NO_ZRE = 1
TLC_MODE_STOCHASTIC = 2
TLC_MODE_INT8 = 3

EXPORTS = (
    "tlc_max_compressed_bytes", "tlc_ctx_create", "tlc_ctx_create_batch",
    "tlc_ctx_destroy", "tlc_compress", "tlc_compress_ex", "tlc_compress_batch",
    "tlc_decompress", "tlc_decompress_ex",
    "tlc_decompress_batch", "tlc_decompress_sum", "tlc_sync",
    "tlc_last_error_string", "tlc_profile_enable", "tlc_profile_mask", "tlc_profile_get",
    "tlc_profile_reset", "tlc_kernel_name", "tlc_ctx_set_options",
    "tlc_compress_noalloc", "tlc_ctx_set_epochs",
)


class tlc_result(ctypes.Structure):
    """struct tlc_result of tlc.h (written to device memory by
    tlc_compress_noalloc; this layout reads a host copy of it)."""
    _fields_ = [("status", ctypes.c_int32), ("bytes_len", ctypes.c_uint32),
                ("scale", ctypes.c_float), ("reserved", ctypes.c_uint32)]


class TLCError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{msg} (status {code})")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built: run `python -m paper_1802_07389_amd.build` "
            "or __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    sz, vp, i, f = ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    L.tlc_max_compressed_bytes.argtypes = [sz]
    L.tlc_max_compressed_bytes.restype = sz
    L.tlc_ctx_create.argtypes = [ctypes.POINTER(vp), sz, vp]
    L.tlc_ctx_create.restype = i
    L.tlc_ctx_create_batch.argtypes = [ctypes.POINTER(vp), sz, sz, vp]
    L.tlc_ctx_create_batch.restype = i
    P = ctypes.POINTER
    L.tlc_compress_batch.argtypes = [vp, sz, P(vp), P(vp), P(sz), P(f), P(vp), P(sz),
                                     P(sz), P(f), P(i)]
    L.tlc_compress_batch.restype = i
    L.tlc_decompress_batch.argtypes = [vp, sz, P(vp), P(sz), P(f), P(sz), P(vp), i]
    L.tlc_decompress_batch.restype = i
    L.tlc_decompress_sum.argtypes = [vp, sz, P(vp), P(sz), P(f), sz, vp, i]
    L.tlc_decompress_sum.restype = i
    L.tlc_compress_ex.argtypes = [vp, i, vp, vp, sz, f, ctypes.c_uint64, ctypes.c_uint64, vp,
                                  sz, P(sz), P(f)]
    L.tlc_compress_ex.restype = i
    L.tlc_ctx_destroy.argtypes = [vp]
    L.tlc_ctx_destroy.restype = i
    L.tlc_compress.argtypes = [vp, vp, vp, sz, f, vp, sz, ctypes.POINTER(sz),
                               ctypes.POINTER(f)]
    L.tlc_compress.restype = i
    L.tlc_decompress.argtypes = [vp, vp, sz, f, sz, vp, i]
    L.tlc_decompress.restype = i
    L.tlc_decompress_ex.argtypes = [vp, i, vp, sz, f, sz, vp, i]
    L.tlc_decompress_ex.restype = i
    L.tlc_sync.argtypes = [vp]
    L.tlc_sync.restype = i
    L.tlc_last_error_string.argtypes = []
    L.tlc_last_error_string.restype = ctypes.c_char_p
    L.tlc_profile_enable.argtypes = [vp, i]
    L.tlc_profile_enable.restype = i
    L.tlc_profile_mask.argtypes = [vp, ctypes.c_uint32]
    L.tlc_profile_mask.restype = i
    L.tlc_profile_get.argtypes = [vp, i, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_uint64)]
    L.tlc_profile_get.restype = i
    L.tlc_profile_reset.argtypes = [vp]
    L.tlc_profile_reset.restype = i
    L.tlc_ctx_set_options.argtypes = [vp, ctypes.c_uint32]
    L.tlc_ctx_set_options.restype = i
    L.tlc_kernel_name.argtypes = [i]
    L.tlc_kernel_name.restype = ctypes.c_char_p
    L.tlc_compress_noalloc.argtypes = [vp, vp, sz, f, vp, sz, vp, vp]
    L.tlc_compress_noalloc.restype = i
    L.tlc_ctx_set_epochs.argtypes = [vp, ctypes.c_uint32, ctypes.c_uint32]
    L.tlc_ctx_set_epochs.restype = i
    return L


lib = _load()


# ----------------------------------------------------------------- C names
def tlc_max_compressed_bytes(n):
    return int(lib.tlc_max_compressed_bytes(n))


def tlc_last_error_string():
    return lib.tlc_last_error_string().decode()


def _check(st):
    if st != TLC_OK:
        raise TLCError(st, tlc_last_error_string())
    return st


def tlc_ctx_create(max_n, hip_stream):
    """Return a context handle (int) bound to ``hip_stream`` (int or None)."""
    h = ctypes.c_void_p()
    _check(lib.tlc_ctx_create(ctypes.byref(h), max_n, hip_stream))
    return h.value


def tlc_ctx_create_batch(max_n, max_tensors, hip_stream):
    """Return a context handle for batched calls."""
    h = ctypes.c_void_p()
    _check(lib.tlc_ctx_create_batch(ctypes.byref(h), max_n, max_tensors, hip_stream))
    return h.value


def _arr(ctype, values):
    return (ctype * len(values))(*values)


def tlc_compress_batch(ctx, tensors, residuals, ns, s, bytes_, caps):
    """Device pointer lists in; returns (status, bytes_len list, scales list,
    per-tensor status list)."""
    k = len(tensors)
    lens = (ctypes.c_size_t * k)()
    scales = (ctypes.c_float * k)()
    stat = (ctypes.c_int * k)()
    st = lib.tlc_compress_batch(
        ctx, k, _arr(ctypes.c_void_p, tensors), _arr(ctypes.c_void_p, residuals),
        _arr(ctypes.c_size_t, ns), _arr(ctypes.c_float, s), _arr(ctypes.c_void_p, bytes_),
        _arr(ctypes.c_size_t, caps), lens, scales, stat)
    return st, list(lens), list(scales), list(stat)


def tlc_decompress_batch(ctx, bytes_, bytes_len, scales, ns, outs, accumulate):
    k = len(bytes_)
    return lib.tlc_decompress_batch(
        ctx, k, _arr(ctypes.c_void_p, bytes_), _arr(ctypes.c_size_t, bytes_len),
        _arr(ctypes.c_float, scales), _arr(ctypes.c_size_t, ns), _arr(ctypes.c_void_p, outs),
        int(bool(accumulate)))


def tlc_decompress_sum(ctx, bytes_, bytes_len, scales, n, out, accumulate):
    k = len(bytes_)
    return lib.tlc_decompress_sum(
        ctx, k, _arr(ctypes.c_void_p, bytes_), _arr(ctypes.c_size_t, bytes_len),
        _arr(ctypes.c_float, scales), n, out, int(bool(accumulate)))


def tlc_ctx_destroy(ctx):
    return lib.tlc_ctx_destroy(ctx)


def tlc_compress(ctx, tensor, residual, n, s, bytes_, bytes_cap):
    """Device pointers in; returns (status, bytes_len, scale)."""
    ln = ctypes.c_size_t(0)
    sc = ctypes.c_float(0.0)
    st = lib.tlc_compress(ctx, tensor, residual, n, s, bytes_, bytes_cap,
                          ctypes.byref(ln), ctypes.byref(sc))
    return st, ln.value, sc.value


def tlc_compress_ex(ctx, mode, tensor, residual, n, s, seed, step, bytes_, bytes_cap):
    """Device pointers in; returns (status, bytes_len, scale)."""
    ln = ctypes.c_size_t(0)
    sc = ctypes.c_float(0.0)
    st = lib.tlc_compress_ex(ctx, mode, tensor, residual, n, s, seed, step, bytes_, bytes_cap,
                             ctypes.byref(ln), ctypes.byref(sc))
    return st, ln.value, sc.value


def tlc_decompress(ctx, bytes_, bytes_len, scale, n, out, accumulate):
    return lib.tlc_decompress(ctx, bytes_, bytes_len, scale, n, out,
                              int(bool(accumulate)))


def tlc_decompress_ex(ctx, mode, bytes_, bytes_len, scale, n, out, accumulate):
    return lib.tlc_decompress_ex(ctx, mode, bytes_, bytes_len, scale, n, out,
                                 int(bool(accumulate)))


def tlc_sync(ctx):
    return lib.tlc_sync(ctx)


def tlc_compress_noalloc(tensor, residual, n, s, bytes_, bytes_cap, result, hip_stream):
    """Device pointers in (result: device address of a 16-byte tlc_result);
    returns the status of the call (the encode's own status is in *result)."""
    return lib.tlc_compress_noalloc(tensor, residual, n, s, bytes_, bytes_cap, result,
                                    hip_stream)


def tlc_ctx_set_epochs(ctx, enc_epoch, dec_epoch):
    return lib.tlc_ctx_set_epochs(ctx, int(enc_epoch), int(dec_epoch))


def tlc_profile_enable(ctx, on):
    return lib.tlc_profile_enable(ctx, int(bool(on)))


def tlc_profile_mask(ctx, mask):
    return lib.tlc_profile_mask(ctx, int(mask) & 0xffffffff)


def tlc_profile_get(ctx, kernel):
    """Return (status, total_ms, launches)."""
    ms = ctypes.c_double(0.0)
    cnt = ctypes.c_uint64(0)
    st = lib.tlc_profile_get(ctx, kernel, ctypes.byref(ms), ctypes.byref(cnt))
    return st, ms.value, cnt.value


def tlc_profile_reset(ctx):
    return lib.tlc_profile_reset(ctx)


def tlc_ctx_set_options(ctx, options):
    return lib.tlc_ctx_set_options(ctx, int(options) & 0xffffffff)


def tlc_kernel_name(kernel):
    r = lib.tlc_kernel_name(kernel)
    return r.decode() if r is not None else None


# ----------------------------------------------------------------- torch
def _dev_f32(t, name):
    if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")
    return t.data_ptr()


def _dev_u8(t, name):
    if not (t.is_cuda and t.dtype == torch.uint8 and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous uint8 GPU tensor")
    return t.data_ptr()


class Context:
    """One compression context (one tensor, one direction) on one stream."""

    def __init__(self, max_n, stream=None, device=None, max_tensors=1, options=0):
        self.device = torch.device(device) if device is not None else torch.device(
            "cuda", torch.cuda.current_device())
        with torch.cuda.device(self.device):
            self.stream = stream if stream is not None else torch.cuda.current_stream()
            self.max_n = int(max_n)
            self.max_tensors = int(max_tensors)
            self.handle = tlc_ctx_create_batch(self.max_n, self.max_tensors,
                                               self.stream.cuda_stream)
        if options:
            self.set_options(options)

    def set_options(self, options):
        """TLC_OPT_* flags (0: the default error policy)."""
        _check(tlc_ctx_set_options(self.handle, options))

    def close(self):
        if getattr(self, "handle", None):
            tlc_ctx_destroy(self.handle)
            self.handle = None

    __del__ = close

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def max_compressed_bytes(self, n):
        return tlc_max_compressed_bytes(n)

    def compress(self, tensor, residual, s, out=None):
        """Encode; returns (bytes view uint8[len], scale).  residual is updated."""
        n = tensor.numel()
        if residual.numel() != n:
            raise ValueError("tensor and residual sizes differ")
        cap = tlc_max_compressed_bytes(n)
        if out is None:
            out = torch.empty(max(cap, 1), dtype=torch.uint8, device=self.device)
        st, ln, sc = tlc_compress(self.handle, _dev_f32(tensor, "tensor"),
                                  _dev_f32(residual, "residual"), n, float(s),
                                  _dev_u8(out, "out"), out.numel())
        _check(st)
        return out[:ln], sc

    def decompress(self, data, scale, n, out, accumulate=False):
        """Decode into out (async; check with sync())."""
        if out.numel() != n:
            raise ValueError("out has the wrong size")
        ptr = _dev_u8(data, "data") if data.numel() else None
        _check(tlc_decompress(self.handle, ptr, data.numel(), float(scale), n,
                              _dev_f32(out, "out"), accumulate))

    def compress_mode(self, mode, tensor, residual, s, seed=0, step=0, out=None):
        """Encode with TLC_MODE_NO_ZRE, TLC_MODE_STOCHASTIC or TLC_MODE_INT8
        (residual may be None for the stochastic mode, and for the 8-bit mode
        without error feedback).  Returns (bytes view, scale)."""
        n = tensor.numel()
        cap = n if mode == TLC_MODE_INT8 else tlc_max_compressed_bytes(n)
        if out is None:
            out = torch.empty(max(cap, 1), dtype=torch.uint8, device=self.device)
        rp = _dev_f32(residual, "residual") if residual is not None else None
        st, ln, sc = tlc_compress_ex(self.handle, mode, _dev_f32(tensor, "tensor"), rp, n,
                                     float(s), int(seed), int(step), _dev_u8(out, "out"),
                                     out.numel())
        _check(st)
        return out[:ln], sc

    def compress_batch(self, tensors, residuals, s, outs=None):
        """Encode a list of tensors in one pass.  Returns a list of
        (bytes view, scale); raises TLCError if any tensor is refused (the
        others are still encoded: see per-tensor status via the C call)."""
        if outs is None:
            outs = [torch.empty(max(tlc_max_compressed_bytes(t.numel()), 1),
                                dtype=torch.uint8, device=self.device) for t in tensors]
        ss = list(s) if isinstance(s, (list, tuple)) else [float(s)] * len(tensors)
        st, lens, scales, _ = tlc_compress_batch(
            self.handle, [_dev_f32(t, "tensor") for t in tensors],
            [_dev_f32(r, "residual") for r in residuals], [t.numel() for t in tensors], ss,
            [_dev_u8(o, "out") for o in outs], [o.numel() for o in outs])
        _check(st)
        return [(o[:ln], sc) for o, ln, sc in zip(outs, lens, scales)]

    def decompress_mode(self, mode, data, scale, out, accumulate=False):
        """Decode a stream of any mode into out (async)."""
        _check(tlc_decompress_ex(self.handle, mode, _dev_u8(data, "data") if data.numel() else None,
                                 data.numel(), float(scale), out.numel(),
                                 _dev_f32(out, "out") if out.numel() else None, accumulate))

    def decompress_batch(self, datas, scales, outs, accumulate=False):
        """Decode a list of streams into a list of outputs (async)."""
        _check(tlc_decompress_batch(
            self.handle, [_dev_u8(d, "data") if d.numel() else None for d in datas],
            [d.numel() for d in datas], [float(x) for x in scales],
            [o.numel() for o in outs], [_dev_f32(o, "out") for o in outs], accumulate))

    def decompress_sum(self, datas, scales, out, accumulate=False):
        """Decode streams of one tensor and add them into out in order (async)."""
        _check(tlc_decompress_sum(
            self.handle, [_dev_u8(d, "data") if d.numel() else None for d in datas],
            [d.numel() for d in datas], [float(x) for x in scales], out.numel(),
            _dev_f32(out, "out"), accumulate))

    def sync(self):
        _check(tlc_sync(self.handle))

    # per-kernel event timing
    def profile(self, on=True, kernels=None):
        """Enable or disable per-kernel event timing; `kernels` (a list of
        TLC_KERNEL_* ids) limits it to those kernels (default: all)."""
        mask = 0xffffffff if kernels is None else sum(1 << k for k in kernels)
        _check(tlc_profile_mask(self.handle, mask))
        _check(tlc_profile_enable(self.handle, on))

    def profile_reset(self):
        _check(tlc_profile_reset(self.handle))

    def profile_get(self, kernel):
        st, ms, cnt = tlc_profile_get(self.handle, kernel)
        _check(st)
        return ms, cnt
