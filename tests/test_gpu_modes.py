"""GPU parity of the comparison encodings (tlc_compress_ex): quartic encoding
without zero-run encoding and stochastic 3-value quantization with Philox
words.  Bar: bit-exact bytes, scale and residual; decoded through
tlc_decompress."""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

pytestmark = pytest.mark.gpu

F32 = np.float32


def G():
    import gpuutil
    return gpuutil


@pytest.fixture(scope="module")
def ctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=workloads.C4_N)
    yield c
    c.close()


def gpu_mode(ctx, mode, x, r, s, seed=0, step=0, offset=0):
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = x.size
    xd = g.to_dev(x, offset)
    rd = g.to_dev(r, offset) if r is not None else None
    cap = max(tlc.tlc_max_compressed_bytes(n), 1)
    out = torch.full((cap,), 0xAB, dtype=torch.uint8, device="cuda")
    st, ln, sc = tlc.tlc_compress_ex(ctx.handle, mode, xd.data_ptr(),
                                     rd.data_ptr() if rd is not None else None, n, float(s),
                                     seed, step, out.data_ptr(), cap)
    torch.cuda.synchronize()
    return st, out[:ln].cpu().numpy(), sc, (rd.cpu().numpy() if rd is not None else None)


SIZES = [1, 7, 40, 4096 * 5, 4096 * 5 + 3, 100003, 1 << 20]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("offset", [0, 1])
def test_nozre_parity(ctx, n, offset):
    from paper_1802_07389_amd import tlc
    g = G()
    x = workloads.runs_tensor([900, n], n)
    r = workloads.normal([901, n], n, 1e-4)
    for s in (1.0, 1.75):
        r_ref = r.copy()
        st_ref, Q_ref, M_ref = oracle.compress_nozre(x, r_ref, s)
        st, Q, M, r_gpu = gpu_mode(ctx, tlc.TLC_MODE_NO_ZRE, x, r, s, offset=offset)
        assert st == st_ref == 0 and M == M_ref
        assert np.array_equal(Q, Q_ref), (n, s)
        assert np.array_equal(g.bits(r_gpu), g.bits(r_ref)), (n, s)
        out0 = workloads.normal([902, n], n)
        st, out = g.gpu_decompress(ctx, Q, M, n, out0.copy(), accumulate=True)
        st_ref, out_ref = oracle.decompress(Q_ref, M_ref, n, out0.copy(), accumulate=True)
        assert st == 0 and np.array_equal(g.bits(out), g.bits(out_ref))


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("offset", [0, 2])
def test_stochastic_parity(ctx, n, offset):
    from paper_1802_07389_amd import tlc
    g = G()
    x = workloads.normal([910, n], n, 1e-3)
    for seed, step, s in [(0, 0, 1.0), (0x123456789ABCDEF, 77, 1.0), (5, 1 << 40, 1.5)]:
        st_ref, Q_ref, M_ref = oracle.compress_stochastic(x, s, seed, step)
        st, Q, M, _ = gpu_mode(ctx, tlc.TLC_MODE_STOCHASTIC, x, None, s, seed, step, offset)
        assert st == st_ref == 0 and M == M_ref
        assert np.array_equal(Q, Q_ref), (n, seed, step)
        st, out = g.gpu_decompress(ctx, Q, M, n)
        st_ref, out_ref = oracle.decompress(Q_ref, M_ref, n)
        assert st == 0 and np.array_equal(g.bits(out), g.bits(out_ref))


def test_stochastic_c4_size(ctx):
    """A 2^28-value stochastic encode: bytes and scale match the oracle."""
    from paper_1802_07389_amd import tlc
    x = workloads.c4_tensor(0)
    st_ref, Q_ref, M_ref = oracle.compress_stochastic(x, 1.0, 99, 1)
    st, Q, M, _ = gpu_mode(ctx, tlc.TLC_MODE_STOCHASTIC, x, None, 1.0, 99, 1)
    assert st == 0 and M == M_ref and np.array_equal(Q, Q_ref)


def test_modes_reject_bad_input(ctx):
    from paper_1802_07389_amd import tlc
    x = workloads.normal([920], 1000)
    x[3] = np.nan
    st, Q, M, _ = gpu_mode(ctx, tlc.TLC_MODE_STOCHASTIC, x, None, 1.0)
    assert st == tlc.TLC_E_NONFINITE and Q.size == 0
    r = workloads.normal([922], 1000, 1e-3)
    r_ref = r.copy()
    assert oracle.compress_nozre(x, r_ref, 1.0)[0] == oracle.E_NONFINITE
    st, Q, M, r_gpu = gpu_mode(ctx, tlc.TLC_MODE_NO_ZRE, x, r.copy(), 1.0)
    assert st == tlc.TLC_E_NONFINITE and Q.size == 0
    assert np.array_equal(r_gpu.view(np.uint32), r_ref.view(np.uint32))  # untouched
    ctx.set_options(tlc.TLC_OPT_IN_PLACE_FEEDBACK)
    try:
        r_ref = r.copy()
        assert oracle.compress_nozre(x, r_ref, 1.0, in_place=True)[0] == oracle.E_NONFINITE
        st, Q, M, r_gpu = gpu_mode(ctx, tlc.TLC_MODE_NO_ZRE, x, r.copy(), 1.0)
        assert st == tlc.TLC_E_NONFINITE and Q.size == 0
        assert np.array_equal(r_gpu.view(np.uint32), r_ref.view(np.uint32))  # x + r
    finally:
        ctx.set_options(0)
    st, *_ = gpu_mode(ctx, 7, workloads.normal([921], 10), np.zeros(10, F32), 1.0)
    assert st == tlc.TLC_E_INVALID
