"""The largest tensor the C ABI accepts: n = TLC_MAX_N = 2^32 - 1 values
(m = 858,993,459 quartic bytes; 16 GiB per fp32 buffer).  Sparse input so
the host side stays cheap: zeros with spikes at the five partition starts,
quartic-tile edges and the last value.  Bar: the whole stream byte for
byte, M, and the whole residual and decoded output bit for bit (compared
in chunks of 2^28 values, so a -0.0/+0.0 flip anywhere fails)."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

F32 = np.float32


def spike_positions(n, m):
    pos = set()
    for k in range(5):
        for d in range(-3, 4):
            pos.add(k * m + d)
    for t in (1, 2, 209715, 209716 - 1):  # quartic-tile edges (4096 bytes)
        for k in range(5):
            for d in (-1, 0, 1):
                pos.add(k * m + 4096 * t + d)
    pos.update([n - 1, n - 2, n - 5, 2 ** 31 - 1, 2 ** 31, 2 ** 32 - 6])
    rng = np.random.default_rng(123)
    pos.update(int(v) for v in rng.integers(0, n, 2000))
    return np.array(sorted(p for p in pos if 0 <= p < n), dtype=np.int64)


def same_bits(a, b, chunk=1 << 28):
    """Index of the first value whose bits differ, or -1."""
    assert a.size == b.size
    for i in range(0, a.size, chunk):
        d = np.flatnonzero(a[i:i + chunk].view(np.uint32) != b[i:i + chunk].view(np.uint32))
        if d.size:
            return i + int(d[0])
    return -1


def test_max_n_round_trip():
    import torch
    from paper_1802_07389_amd import tlc
    import gpuutil as g
    n = tlc.TLC_MAX_N
    m = tlc.tlc_max_compressed_bytes(n)
    assert m == 858993459
    P = spike_positions(n, m)
    x = np.zeros(n, F32)
    vals = np.where(np.arange(P.size) % 3 == 0, F32(0.3), F32(1.0))
    vals = np.where(np.arange(P.size) % 2 == 0, vals, -vals).astype(F32)
    x[P] = vals
    g.log(f"max n: {n} values, {P.size} spikes")
    ctx = tlc.Context(max_n=n)
    try:
        xd = torch.from_numpy(x).cuda()
        rd = torch.zeros(n, dtype=torch.float32, device="cuda")
        C, M = ctx.compress(xd, rd, 1.75)
        C = C.cpu().numpy()
        g.log(f"gpu encode done: {C.size} bytes, M = {M}")
        del xd
        r_ref = np.zeros(n, F32)
        st, C_ref, M_ref = oracle.compress(x, r_ref, 1.75)
        g.log("oracle encode done")
        assert st == 0 and M == M_ref == F32(1.75)
        assert C.size == C_ref.size and np.array_equal(C, C_ref)
        r_gpu = rd.cpu().numpy()
        del rd
        i = same_bits(r_gpu, r_ref)
        assert i < 0, (i, r_gpu[i], r_ref[i])
        del r_gpu, r_ref
        g.log("stream and the whole residual match")

        od = torch.zeros(n, dtype=torch.float32, device="cuda")
        ctx.decompress(torch.from_numpy(C_ref).cuda(), M_ref, n, od, accumulate=True)
        ctx.sync()
        out = od.cpu().numpy()
        del od
        st, out_ref = oracle.decompress(C_ref, M_ref, n, np.zeros(n, F32), accumulate=True)
        assert st == 0
        i = same_bits(out, out_ref)
        assert i < 0, (i, out[i], out_ref[i])
        g.log("the whole decoded output matches")
    finally:
        ctx.close()
