"""Accumulating decodes add M*q into every aggregate value, on every
decode path, bit for bit as in the oracle (reading A13: -0.0 + M*0 gives
+0.0).  The decoder stores only the sums whose bits differ from what is
there, so the aggregates here hold -0.0 (which must turn into +0.0),
infinities, subnormals and ordinary values both where q = 0 and where
q != 0.  (No NaNs: an add need not keep a NaN's payload.)"""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

pytestmark = pytest.mark.gpu

F32 = np.float32
SPECIAL = np.array([0x80000000, 0x7F800000, 0xFF800000, 0x00000001, 0x80000001, 0x00800000,
                    0x80000000, 0x80000000], np.uint32)


def G():
    import gpuutil
    return gpuutil


def sparse_case(seed, n, spikes=300):
    """x: zeros with spikes (q != 0 only there); out0: specials where x = 0,
    -0.0 at half the spikes."""
    rng = np.random.default_rng(seed)
    P = np.unique(rng.integers(0, n, spikes))
    x = np.zeros(n, F32)
    x[P] = rng.choice(np.array([1.0, -1.0, 0.75, -0.6], F32), P.size)
    out0 = workloads.normal([seed, 1], n, 1.0)
    zero = np.ones(n, bool)
    zero[P] = False
    idx = np.flatnonzero(zero)
    pick = idx[rng.integers(0, idx.size, min(idx.size, 4000))]
    out0.view(np.uint32)[pick] = SPECIAL[rng.integers(0, SPECIAL.size, pick.size)]
    neg0 = P[::2]  # -0.0 meeting non-zero updates too
    out0[neg0] = -0.0
    return x, out0


def encode(x, s=1.0):
    st, C, M = oracle.compress(x, np.zeros(x.size, F32), s)
    assert st == 0
    return C, M


@pytest.fixture(scope="module")
def ctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=1 << 27, max_tensors=8)
    yield c
    c.close()


# n: m % 4 == 0 (float4 path), m % 4 != 0 (aligned cells off the grid); the
# offset puts out off the 16-byte grid (scalar path)
@pytest.mark.parametrize("n,offset", [(5 * 4096 * 3 + 20, 0), (5 * 4096 * 3 + 7, 0),
                                      (5 * 4096 * 3 + 20, 1), (3, 0)])
def test_single_stream(ctx, n, offset):
    g = G()
    x, out0 = sparse_case(900 + n % 97 + offset, n, spikes=min(300, n))
    C, M = encode(x)
    st_ref, ref = oracle.decompress(C, M, n, out0.copy(), accumulate=True)
    st, out = g.gpu_decompress(ctx, C, M, n, out0.copy(), accumulate=True, offset=offset)
    assert st == st_ref == 0
    assert np.array_equal(g.bits(out), g.bits(ref)), (n, offset)


@pytest.mark.parametrize("every", [10, 17, 60])
def test_single_stream_literal_density(ctx, every):
    """Non-zero quartic bytes at two offsets every `every` bytes: ranges
    from many to few stored float4s."""
    g = G()
    n = 5 * 4096 * 3 + 20
    m = -(-n // 5)
    x, out0 = sparse_case(940 + every, n, spikes=0)
    x[:m:every] = 1.0  # partition 0: q = 1 (s = 1: M = 1)
    x[3 * m + 5:4 * m:every] = -1.0
    zero = x == 0
    out0[~zero] = workloads.normal([941, every], int((~zero).sum()), 1.0)
    out0[np.flatnonzero(~zero)[::5]] = -0.0
    C, M = encode(x)
    st_ref, ref = oracle.decompress(C, M, n, out0.copy(), accumulate=True)
    st, out = g.gpu_decompress(ctx, C, M, n, out0.copy(), accumulate=True)
    assert st == st_ref == 0
    assert np.array_equal(g.bits(out), g.bits(ref)), every


def test_single_stream_large(ctx):
    """2^27 values: the decode of outputs of 512 MiB and more (nontemporal
    sweep, with the stores of unchanged float4s skipped)."""
    g = G()
    n = 1 << 27
    x, out0 = sparse_case(910, n, spikes=20000)
    C, M = encode(x, 1.5)
    st_ref, ref = oracle.decompress(C, M, n, out0.copy(), accumulate=True)
    st, out = g.gpu_decompress(ctx, C, M, n, out0, accumulate=True)
    assert st == st_ref == 0
    assert np.array_equal(g.bits(out), g.bits(ref))


def test_batch_and_sum(ctx):
    import torch
    g = G()
    sizes = [5 * 4096 + 20, 5 * 4096 * 2 + 7, 1001]
    cases = [sparse_case(920 + i, n) for i, n in enumerate(sizes)]
    pays = [encode(x) for x, _ in cases]
    outs = [torch.from_numpy(o.copy()).cuda() for _, o in cases]
    ctx.decompress_batch([torch.from_numpy(C).cuda() for C, _ in pays], [M for _, M in pays],
                         outs, accumulate=True)
    ctx.sync()
    for i, (C, M) in enumerate(pays):
        st, ref = oracle.decompress(C, M, sizes[i], cases[i][1].copy(), accumulate=True)
        assert np.array_equal(g.bits(outs[i].cpu().numpy()), g.bits(ref)), i
    # two streams of one tensor into one aggregate
    n = sizes[1]
    x0, out0 = cases[1]
    x1 = np.zeros(n, F32)
    x1[np.flatnonzero(x0)[::3]] = 0.5  # partly the same positions, partly new
    x1[7] = -1.0
    streams = [encode(x0), encode(x1)]
    for acc in (False, True):
        ref = out0.copy()
        for p, (C, M) in enumerate(streams):
            st, ref = oracle.decompress(C, M, n, ref, accumulate=(acc or p > 0))
        od = torch.from_numpy(out0.copy()).cuda()
        ctx.decompress_sum([torch.from_numpy(C).cuda() for C, _ in streams],
                           [M for _, M in streams], od, accumulate=acc)
        ctx.sync()
        assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(ref)), acc


def test_int8_dense(ctx):
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = 3 * 4096 + 5
    x, out0 = sparse_case(930, n)
    st, C, M = oracle.compress_int8(x, None, 1.0)
    assert st == 0
    st, ref = oracle.decompress_int8(C, M, n, out0.copy(), True)
    od = torch.from_numpy(out0.copy()).cuda()
    cd = torch.from_numpy(C).cuda()
    assert tlc.tlc_decompress_ex(ctx.handle, tlc.TLC_MODE_INT8, cd.data_ptr(), n, M, n,
                                 od.data_ptr(), 1) == 0
    assert tlc.tlc_sync(ctx.handle) == 0
    assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(ref))
