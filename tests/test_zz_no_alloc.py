"""tlc_compress_noalloc (the encode without a context, scratch in a static
device array) against tlc_compress and the CPU oracle, through the C ABI.
Bar: stream bytes, scale and residual bit-exact, on calls in a row whose
sizes shrink (the shared scratch keeps the previous call's contents)."""
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
    c = tlc.Context(max_n=tlc.TLC_NOALLOC_MAX_N)
    yield c
    c.close()


def noalloc(x, r, s, offset=0):
    """Run tlc_compress_noalloc on copies of x and r; return (call status,
    tlc_result, stream bytes, residual)."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = x.size
    xd = g.to_dev(x, offset)
    rd = g.to_dev(r, offset)
    cap = max(tlc.tlc_max_compressed_bytes(n), 1)
    out = torch.full((cap,), 0xAB, dtype=torch.uint8, device="cuda")
    res = torch.full((4,), -7, dtype=torch.int32, device="cuda")  # one tlc_result
    st = tlc.tlc_compress_noalloc(xd.data_ptr() if n else None, rd.data_ptr() if n else None,
                                  n, float(s), out.data_ptr(), cap, res.data_ptr(),
                                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    result = tlc.tlc_result.from_buffer_copy(res.cpu().numpy().tobytes())
    return st, result, out.cpu().numpy()[:result.bytes_len], rd.cpu().numpy()


def check_same_as_compress(ctx, x, r, s, offset=0, tag=""):
    g = G()
    st, res, C, r_new = noalloc(x, r, s, offset)
    assert st == 0 and res.status == 0 and res.reserved == 0, (tag, st, res.status)
    st2, C2, M2, r2 = g.gpu_compress(ctx, x, r.copy(), s, offset)
    assert st2 == 0, tag
    assert res.bytes_len == C2.size and res.scale == M2, (tag, res.bytes_len, C2.size)
    assert np.array_equal(C, C2), tag
    assert np.array_equal(g.bits(r_new), g.bits(r2)), tag
    r_ref = r.copy()
    st3, C3, M3 = oracle.compress(x, r_ref, s)
    assert st3 == 0 and M3 == res.scale and np.array_equal(C, C3), tag
    assert np.array_equal(g.bits(r_new), g.bits(r_ref)), tag
    G().log(f"{tag}: n={x.size} len={res.bytes_len} ok")


def test_two_calls_second_smaller(ctx):
    """Two calls in a row, the second on a smaller tensor, each equal to
    tlc_compress on the same inputs (and to the oracle)."""
    n1 = (1 << 20) + 3
    x1 = workloads.normal([80, 1], n1, 1e-3)
    r1 = workloads.normal([80, 2], n1, 1e-4)
    check_same_as_compress(ctx, x1, r1, 1.5, tag="first call")
    n2 = 77_777
    x2 = workloads.runs_tensor([80, 3], n2)
    r2 = np.zeros(n2, F32)
    check_same_as_compress(ctx, x2, r2, 1.75, tag="second call, smaller")


def test_sizes_alignment_and_the_limit(ctx):
    """Every size class of the chained path, unaligned pointers, and the
    largest accepted n; one value more is refused before anything runs."""
    from paper_1802_07389_amd import tlc
    for n, off in [(1, 0), (7, 0), (5 * 4096 + 3, 0), (5 * 4096 * 3 + 7, 1),
                   (tlc.TLC_NOALLOC_MAX_N, 0), (12_345, 3)]:
        x = workloads.normal([81, n], n, 1e-3)
        r = workloads.normal([82, n], n, 1e-5)
        check_same_as_compress(ctx, x, r, 1.0, off, tag=f"n={n} offset={off}")
    import torch
    n = tlc.TLC_NOALLOC_MAX_N + 1
    x = torch.zeros(n, device="cuda")
    r = torch.zeros(n, device="cuda")
    out = torch.zeros(tlc.tlc_max_compressed_bytes(n), dtype=torch.uint8, device="cuda")
    res = torch.zeros(4, dtype=torch.int32, device="cuda")
    st = tlc.tlc_compress_noalloc(x.data_ptr(), r.data_ptr(), n, 1.5, out.data_ptr(),
                                  out.numel(), res.data_ptr(), None)
    assert st == tlc.TLC_E_INVALID and "TLC_NOALLOC_MAX_N" in tlc.tlc_last_error_string()


def test_nonfinite_then_good_call(ctx):
    """NaN in the sum: status TLC_E_NONFINITE, residual and bytes left as they
    were; the next call (which clears the shared scratch) is exact again."""
    from paper_1802_07389_amd import tlc
    n = 300_001
    x = workloads.normal([83, 0], n, 1e-3)
    x[123_456] = np.nan
    r = workloads.normal([83, 1], n, 1e-4)
    st, res, C, r_new = noalloc(x, r, 1.5)
    assert st == 0 and res.status == tlc.TLC_E_NONFINITE and res.bytes_len == 0
    assert res.scale == 0.0
    assert np.array_equal(G().bits(r_new), G().bits(r))
    x[123_456] = 0.0
    check_same_as_compress(ctx, x, r, 1.5, tag="after the NaN call")


def test_empty_and_argument_errors(ctx):
    import torch
    from paper_1802_07389_amd import tlc
    st, res, C, _ = noalloc(np.zeros(0, F32), np.zeros(0, F32), 1.5)
    assert st == 0 and res.status == 0 and res.bytes_len == 0 and res.scale == 0.0
    x = torch.zeros(100, device="cuda")
    r = torch.zeros(100, device="cuda")
    out = torch.zeros(20, dtype=torch.uint8, device="cuda")
    res = torch.zeros(4, dtype=torch.int32, device="cuda")
    P = lambda t: t.data_ptr()
    assert tlc.tlc_compress_noalloc(P(x), P(r), 100, 2.0, P(out), 20, P(res),
                                    None) == tlc.TLC_E_INVALID
    assert tlc.tlc_compress_noalloc(P(x), P(r), 100, 1.5, P(out), 19, P(res),
                                    None) == tlc.TLC_E_CAPACITY
    assert tlc.tlc_compress_noalloc(P(x), P(r), 100, 1.5, P(out), 20, None,
                                    None) == tlc.TLC_E_INVALID
    assert tlc.tlc_compress_noalloc(P(x), P(x), 100, 1.5, P(out), 20, P(res),
                                    None) == tlc.TLC_E_INVALID
    assert tlc.tlc_compress_noalloc(P(x), P(r), 100, 1.5, P(out), 20, P(r) + 8,
                                    None) == tlc.TLC_E_INVALID
