"""GPU parity of the 8-bit integer comparator (TLC_MODE_INT8 through
tlc_compress_ex / tlc_decompress_ex) against the CPU oracle.  Bar:
bit-exact codes, scale, residual and decoded fp32 values."""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

pytestmark = pytest.mark.gpu

F32 = np.float32
TINY = F32(2.0 ** -149)


def G():
    import gpuutil
    return gpuutil


@pytest.fixture(scope="module")
def ctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=workloads.C4_N)
    yield c
    c.close()


def gpu_int8(ctx, x, r, s, offset=0):
    """Return (status, bytes, scale, residual or None)."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = x.size
    xd = g.to_dev(x, offset)
    rd = g.to_dev(r, offset) if r is not None else None
    buf = torch.full((max(n, 1) + offset,), 0xAB, dtype=torch.uint8, device="cuda")
    out = buf[offset:]
    st, ln, sc = tlc.tlc_compress_ex(ctx.handle, tlc.TLC_MODE_INT8,
                                     xd.data_ptr() if n else None,
                                     rd.data_ptr() if (rd is not None and n) else None, n,
                                     float(s), 0, 0, out.data_ptr(), max(n, 1))
    torch.cuda.synchronize()
    return st, out[:ln].cpu().numpy(), sc, (rd.cpu().numpy() if rd is not None else None)


def gpu_int8_decode(ctx, C, M, n, out0, accumulate, offset=0):
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    od = g.to_dev(out0, offset)
    cb = torch.zeros(C.size + offset, dtype=torch.uint8, device="cuda")
    cd = cb[offset:]
    cd.copy_(torch.from_numpy(np.ascontiguousarray(C)))
    st = tlc.tlc_decompress_ex(ctx.handle, tlc.TLC_MODE_INT8, cd.data_ptr() if C.size else None,
                               C.size, float(M), n, od.data_ptr() if n else None, accumulate)
    if st == 0:
        st = tlc.tlc_sync(ctx.handle)
    return st, od.cpu().numpy()


def check(ctx, x, r, s, offset=0, tag=""):
    g = G()
    r_ref = r.copy() if r is not None else None
    st_ref, C_ref, M_ref = oracle.compress_int8(x, r_ref, s)
    st, C, M, r_gpu = gpu_int8(ctx, x, r, s, offset)
    assert st == st_ref, (tag, st, st_ref)
    if st != 0:
        return
    assert M == M_ref and np.array_equal(C, C_ref), tag
    if r is not None:
        assert np.array_equal(g.bits(r_gpu), g.bits(r_ref)), tag
    n = x.size
    for acc in (False, True):
        out0 = workloads.normal([970, n], n)
        st, out = gpu_int8_decode(ctx, C_ref, M_ref, n, out0.copy(), acc, offset)
        st_ref, out_ref = oracle.decompress_int8(C_ref, M_ref, n, out0.copy(), acc)
        assert st == st_ref == 0
        assert np.array_equal(g.bits(out), g.bits(out_ref)), (tag, acc)


SIZES = [1, 3, 4, 5, 1023, 1024, 16384, 16385, 100003, 1 << 20]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("offset", [0, 1])
def test_int8_parity(ctx, n, offset):
    x = workloads.normal([971, n], n, 1e-3)
    r = workloads.normal([972, n], n, 1e-5)
    for s in (1.0, 1.75):
        check(ctx, x, r, s, offset, tag=f"feedback n={n} s={s}")
        check(ctx, x, None, s, offset, tag=f"plain n={n} s={s}")


def test_int8_special_scales(ctx):
    # subnormal step: M / D = 190 is clamped to 127; D == 0 quantizes to 0
    check(ctx, np.array([190, -190, 3, 0], F32) * TINY, np.zeros(4, F32), 1.0, tag="clamp")
    check(ctx, np.array([63, -5, 1], F32) * TINY, np.zeros(3, F32), 1.0, tag="zero step")
    check(ctx, np.zeros(5000, F32), np.zeros(5000, F32), 1.0, tag="zeros")
    acc = (np.arange(-127 * 4, 127 * 4 + 1) / 4.0).astype(F32)  # ties at M = 127
    check(ctx, acc, None, 1.0, tag="ties")
    check(ctx, acc, np.zeros_like(acc), 1.0, tag="ties feedback")
    # sums of -0.0 (tensor -0.0, residual -0.0) keep -0.0 as their residual
    x = np.array([1.0, -0.0, -0.0, 0.5, 0.0] * 1000, F32)
    r = np.array([0.0, -0.0, 0.0, 0.0, -0.0] * 1000, F32)
    check(ctx, x, r, 1.0, tag="signed zeros")
    check(ctx, x, r, 1.0, offset=1, tag="signed zeros, unaligned")


def test_int8_c4_size(ctx):
    """2^28 values with error feedback, two steps: every code and residual."""
    g = G()
    n = workloads.C4_N
    r = np.zeros(n, F32)
    import torch
    from paper_1802_07389_amd import tlc
    rd = torch.zeros(n, device="cuda")
    out = torch.empty(n, dtype=torch.uint8, device="cuda")
    for step in range(2):
        x = workloads.c4_tensor(step)
        st_ref, C_ref, M_ref = oracle.compress_int8(x, r, workloads.C4_S)
        xd = torch.from_numpy(x).cuda()
        C, M = ctx.compress_mode(tlc.TLC_MODE_INT8, xd, rd, workloads.C4_S, out=out)
        assert st_ref == 0 and M == M_ref
        assert np.array_equal(C.cpu().numpy(), C_ref), step
        assert np.array_equal(g.bits(rd.cpu().numpy()), g.bits(r)), step
        del xd
        g.log(f"int8 C4 step {step} ok")


def test_int8_errors(ctx):
    import torch
    from paper_1802_07389_amd import tlc
    x = workloads.normal([973], 1000)
    x[10] = np.nan
    r = workloads.normal([974], 1000, 1e-3)
    st, C, M, r_gpu = gpu_int8(ctx, x, r, 1.0)
    assert st == tlc.TLC_E_NONFINITE and C.size == 0
    assert np.array_equal(G().bits(r_gpu), G().bits(r))  # untouched
    ctx.set_options(tlc.TLC_OPT_IN_PLACE_FEEDBACK)
    try:
        r_ref = r.copy()
        assert oracle.compress_int8(x, r_ref, 1.0, in_place=True)[0] == oracle.E_NONFINITE
        st, C, M, r_gpu = gpu_int8(ctx, x, r, 1.0)
        assert st == tlc.TLC_E_NONFINITE and C.size == 0
        assert np.array_equal(G().bits(r_gpu), G().bits(r_ref))  # x + r
    finally:
        ctx.set_options(0)
    xd = torch.zeros(100, device="cuda")
    o = torch.zeros(100, dtype=torch.uint8, device="cuda")
    st, ln, sc = tlc.tlc_compress_ex(ctx.handle, tlc.TLC_MODE_INT8, xd.data_ptr(), None, 100,
                                     1.0, 0, 0, o.data_ptr(), 99)
    assert st == tlc.TLC_E_CAPACITY
    out0 = workloads.normal([975], 100)
    st, out = gpu_int8_decode(ctx, np.zeros(99, np.uint8), 1.0, 100, out0.copy(), True)
    assert st == tlc.TLC_E_CORRUPT and np.array_equal(out, out0)
    st = tlc.tlc_decompress_ex(ctx.handle, 9, o.data_ptr(), 100, 1.0, 100, xd.data_ptr(), 0)
    assert st == tlc.TLC_E_INVALID
    assert tlc.tlc_sync(ctx.handle) == tlc.TLC_OK


def test_decompress_ex_forwards_3lc(ctx):
    """tlc_decompress_ex with the 3LC mode is tlc_decompress."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = 50003
    x = workloads.runs_tensor([976], n)
    st, C, M = oracle.compress(x, np.zeros(n, F32), 1.5)
    out0 = workloads.normal([977], n)
    od = torch.from_numpy(out0.copy()).cuda()
    ctx.decompress_mode(tlc.TLC_MODE_3LC, torch.from_numpy(C).cuda(), M, od, accumulate=True)
    ctx.sync()
    st, out_ref = oracle.decompress(C, M, n, out0.copy(), True)
    assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(out_ref))
