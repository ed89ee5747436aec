"""Helpers for GPU parity tests: move numpy inputs through the C ABI.

Every function here calls the HIP library through ``paper_1802_07389_amd.tlc``
(ctypes over libtlc.so) and returns host numpy arrays for comparison with
the CPU oracle.
"""
import sys

import numpy as np
import torch

from paper_1802_07389_amd import tlc


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def to_dev(a, offset=0):
    """Copy a float32 numpy array to the GPU; ``offset`` > 0 places it that
    many elements into a larger buffer (to test unaligned pointers)."""
    a = np.ascontiguousarray(a)
    if offset == 0:
        return torch.from_numpy(a).cuda()
    buf = torch.empty(a.size + offset, dtype=torch.from_numpy(a[:0]).dtype, device="cuda")
    view = buf[offset:]
    view.copy_(torch.from_numpy(a))
    return view


def gpu_compress(ctx, x, r, s, offset=0, r_offset=None):
    """Return (status, bytes np.uint8, scale, residual np.float32).  The
    residual sits r_offset elements into its buffer (default: offset)."""
    n = x.size
    xd = to_dev(x, offset)
    rd = to_dev(r, offset if r_offset is None else r_offset)
    cap = max(tlc.tlc_max_compressed_bytes(n), 1)
    out = torch.full((cap,), 0xAB, dtype=torch.uint8, device="cuda")
    st, ln, sc = tlc.tlc_compress(ctx.handle, xd.data_ptr() if n else None,
                                  rd.data_ptr() if n else None, n, float(s),
                                  out.data_ptr(), cap)
    torch.cuda.synchronize()
    return st, out[:ln].cpu().numpy(), sc, rd.cpu().numpy()


def gpu_decompress(ctx, C, scale, n, out0=None, accumulate=False, offset=0):
    """Return (status from tlc_sync, out np.float32)."""
    if out0 is None:
        out0 = np.zeros(n, np.float32)
    od = to_dev(out0, offset)
    Cd = torch.from_numpy(np.ascontiguousarray(C, np.uint8)).cuda()
    st = tlc.tlc_decompress(ctx.handle, Cd.data_ptr() if C.size else None, C.size,
                            float(scale), n, od.data_ptr() if n else None, accumulate)
    if st != tlc.TLC_OK:
        return st, od.cpu().numpy()
    st = tlc.tlc_sync(ctx.handle)
    return st, od.cpu().numpy()
