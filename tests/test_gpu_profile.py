"""Per-kernel event timing (tlc_profile_*): the launchers' kernels record
the event pair themselves, the first kernel the start and the last the end.
Timed and untimed calls give the same results; the mask selects kernels;
reset clears the counts."""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

pytestmark = pytest.mark.gpu

F32 = np.float32


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


@pytest.fixture(scope="module")
def ctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=1 << 24)
    yield c
    c.close()


def round_trip(ctx, x, r, out0, s):
    import torch
    xd = torch.from_numpy(x).cuda()
    rd = torch.from_numpy(r.copy()).cuda()
    C, M = ctx.compress(xd, rd, s)
    od = torch.from_numpy(out0.copy()).cuda()
    ctx.decompress(C, M, x.size, od, accumulate=True)
    ctx.sync()
    return C.cpu().numpy(), M, rd.cpu().numpy(), od.cpu().numpy()


def test_every_kernel_of_a_round_trip_is_timed(ctx):
    from paper_1802_07389_amd import tlc
    n = 1 << 24  # 820 tiles: the three-pass encoder (chunk scans are two kernels)
    x = workloads.normal([61, 0], n, 1e-3)
    r = workloads.normal([61, 1], n, 1e-4)
    out0 = workloads.normal([61, 2], n, 1e-3)
    plain = round_trip(ctx, x, r, out0, 1.75)
    ctx.profile(True)
    ctx.profile_reset()
    timed = round_trip(ctx, x, r, out0, 1.75)
    ctx.profile(False)
    for a, b in zip(plain, timed):
        if isinstance(a, np.ndarray):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
        else:
            assert a == b
    used = [tlc.TLC_KERNEL_ABSMAX_CHECK, tlc.TLC_KERNEL_ACCUM_QUANTIZE,
            tlc.TLC_KERNEL_QUANT_ENCODE, tlc.TLC_KERNEL_ZRE_CHUNKS, tlc.TLC_KERNEL_ZRE_COMPACT,
            tlc.TLC_KERNEL_ZRE_INDEX, tlc.TLC_KERNEL_EXPAND_DEQUANT]
    for k in range(tlc.TLC_KERNEL_COUNT):
        ms, cnt = ctx.profile_get(k)
        if k in used:
            assert cnt == 1 and 0.0 < ms < 100.0, (k, ms, cnt)
        else:
            assert cnt == 0 and ms == 0.0, (k, ms, cnt)
    # the bit-exact stream and residual against the oracle as well
    r_ref = r.copy()
    st, C_ref, M_ref = oracle.compress(x, r_ref, 1.75)
    assert st == 0 and timed[1] == M_ref and np.array_equal(timed[0], C_ref)
    assert np.array_equal(bits(timed[2]), bits(r_ref))


def test_mask_and_reset(ctx):
    from paper_1802_07389_amd import tlc
    n = 1 << 21
    x = workloads.normal([62, 0], n, 1e-3)
    r = np.zeros(n, F32)
    out0 = np.zeros(n, F32)
    ctx.profile(True, kernels=[tlc.TLC_KERNEL_EXPAND_DEQUANT])
    ctx.profile_reset()
    for _ in range(3):
        round_trip(ctx, x, r, out0, 1.0)
    ctx.profile(False)
    ms, cnt = ctx.profile_get(tlc.TLC_KERNEL_EXPAND_DEQUANT)
    assert cnt == 3 and ms > 0.0
    for k in range(tlc.TLC_KERNEL_COUNT):
        if k != tlc.TLC_KERNEL_EXPAND_DEQUANT:
            assert ctx.profile_get(k) == (0.0, 0), k
    ctx.profile_reset()
    assert ctx.profile_get(tlc.TLC_KERNEL_EXPAND_DEQUANT) == (0.0, 0)
    # untimed launches after profiling leave no timings behind
    round_trip(ctx, x, r, out0, 1.0)
    assert ctx.profile_get(tlc.TLC_KERNEL_EXPAND_DEQUANT) == (0.0, 0)
