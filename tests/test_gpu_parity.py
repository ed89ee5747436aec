"""GPU parity: the HIP path through the C ABI against the CPU oracle.

The bar is bit-exactness: the compressed byte stream byte for byte, the
scale M, the residual and the decoded fp32 output to 0 ULP (the method's
fp32 operations are fixed and every product in it is exact).
"""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

pytestmark = pytest.mark.gpu

F32 = np.float32


@pytest.fixture(scope="module")
def ctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=workloads.C4_N)
    yield c
    c.close()


def G():
    import gpuutil
    return gpuutil


def check_encode_decode(ctx, x, r, s, out0=None, accumulate=False, offset=0, tag=""):
    """Encode and decode x on both sides; assert bit equality; return the
    oracle's (bytes, M, residual, decoded)."""
    g = G()
    r_ref = r.copy()
    st_ref, C_ref, M_ref = oracle.compress(x, r_ref, s)
    st, C, M, r_gpu = g.gpu_compress(ctx, x, r, s, offset=offset)
    assert st == st_ref, (tag, st, st_ref)
    if st != 0:
        return None
    assert np.array_equal(g.bits(np.array([M])), g.bits(np.array([M_ref]))), (tag, M, M_ref)
    assert C.size == C_ref.size, (tag, C.size, C_ref.size)
    if not np.array_equal(C, C_ref):
        i = int(np.flatnonzero(C != C_ref)[0])
        raise AssertionError(f"{tag}: byte {i} differs: gpu {C[i]} oracle {C_ref[i]}")
    if not np.array_equal(g.bits(r_gpu), g.bits(r_ref)):
        i = int(np.flatnonzero(g.bits(r_gpu) != g.bits(r_ref))[0])
        raise AssertionError(f"{tag}: residual {i} differs: {r_gpu[i]!r} vs {r_ref[i]!r}")
    n = x.size
    if out0 is None:
        out0 = np.zeros(n, F32)
    st_ref, out_ref = oracle.decompress(C_ref, M_ref, n, out0.copy(), accumulate)
    st, out = g.gpu_decompress(ctx, C_ref, M_ref, n, out0.copy(), accumulate, offset=offset)
    assert st == st_ref == 0, (tag, st, st_ref)
    if not np.array_equal(g.bits(out), g.bits(out_ref)):
        i = int(np.flatnonzero(g.bits(out) != g.bits(out_ref))[0])
        raise AssertionError(f"{tag}: decoded {i} differs: {out[i]!r} vs {out_ref[i]!r}")
    return C_ref, M_ref, r_ref, out_ref


# ------------------------------------------------------------------ small cases
def test_worked_examples_on_gpu(ctx):
    import json, os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "worked_examples.json")))
    for case in gold["cases"]:
        if "x" not in case:
            continue
        x = np.array(case["x"], F32)
        r = np.array(case["r"], F32)
        st, C, M, r_gpu = G().gpu_compress(ctx, x, r, case["s"])
        assert st == 0 and C.tolist() == case["bytes"] and M == case["scale"], case["name"]
        assert r_gpu.tolist() == case["residual"], case["name"]
        st, out = G().gpu_decompress(ctx, C, M, x.size)
        assert st == 0 and out.tolist() == case["decoded"], case["name"]


@pytest.mark.parametrize("s", [1.0, 1.5, 1.9])
def test_tiny_sizes(ctx, s):
    for n in range(1, 41):
        x = workloads.normal([10, n], n, 1.0)
        r = workloads.normal([11, n], n, 0.3)
        check_encode_decode(ctx, x, r, s, tag=f"n={n}")
        check_encode_decode(ctx, x, r, s, out0=workloads.normal([12, n], n),
                            accumulate=True, tag=f"acc n={n}")


def test_empty_tensor(ctx):
    from paper_1802_07389_amd import tlc
    st, C, M, _ = G().gpu_compress(ctx, np.zeros(0, F32), np.zeros(0, F32), 1.0)
    assert st == 0 and C.size == 0 and M == 0.0
    assert tlc.tlc_decompress(ctx.handle, None, 0, 0.0, 0, None, 0) == 0


# sizes around the 4096-byte zero-run tile and the vector/scalar paths
EDGE_N = [5 * 4096 - 1, 5 * 4096, 5 * 4096 + 1, 5 * 4096 * 2 + 7, 5 * 4096 * 3 - 5,
          4 * 5 * 1000, 4 * 5 * 1000 + 3, 65537, 1000003]


@pytest.mark.parametrize("n", EDGE_N)
def test_tile_edges_dense_and_sparse(ctx, n):
    for s, sigma_scale in [(1.0, 1.0), (1.9, 1.0)]:
        x = workloads.normal([20, n], n, sigma_scale)
        check_encode_decode(ctx, x, np.zeros(n, F32), s, tag=f"dense n={n} s={s}")
    x = workloads.runs_tensor([21, n], n)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.5, tag=f"runs n={n}")


@pytest.mark.parametrize("n", [7, 70, 71, 5 * 14 * 4096, 5 * 14 * 4096 + 3, 2 ** 20, 3 * 10 ** 6])
def test_all_zero_tensors(ctx, n):
    """Zero runs spanning many tiles; the 280x ceiling (Section 3.3)."""
    x = np.zeros(n, F32)
    res = check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"zeros n={n}")
    C = res[0]
    if n % 70 == 0:
        assert 4 * n / C.size == 280


@pytest.mark.parametrize("m", [8191, 8192, 8193, 2 * 8192 - 1, 2 * 8192 + 1, 3 * 8192 + 5,
                               16383, 16384, 16385, 2 * 16384 + 1, 200 * 4096 + 7,
                               300 * 4096 + 1])
def test_index_scan_tile_edges(ctx, m):
    """Streams ending at and around the tiles of the zero-run index scan:
    8192 bytes when the scan runs in the first blocks of the decode's
    single launch (small streams), 16384 in its own launch (the last two
    sizes, with more than 256 blocks in all).  All-ones tensors quantize to q = 1 everywhere (M = 1 at
    s = 1), so every quartic byte is 242 and the stream is exactly m bytes,
    with range starts on tile edges; then zero groups turn random spans of
    bytes into 121, whose run codes land across the edges."""
    n = 5 * m
    x = np.ones(n, F32)
    res = check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"ones m={m}")
    assert res[0].size == m
    rng = np.random.default_rng([31, m])
    for trial in range(3):
        x = np.ones(n, F32)
        for j0 in rng.integers(0, m, size=60):
            span = np.arange(j0, min(m, j0 + int(rng.integers(1, 60))))
            for k in range(5):
                x[k * m + span] = F32(0.0)
        check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"ones+runs m={m} {trial}")


def test_long_runs_with_sparse_spikes(ctx):
    """Runs of every length mod 14 ending exactly at and across tile edges."""
    rng = np.random.default_rng(30)
    n = 5 * 4096 * 6
    m = n // 5
    for trial in range(8):
        x = np.zeros(n, F32)
        # non-zero groups at chosen quartic positions j (partition 0)
        js = np.unique(np.concatenate([
            np.arange(4096 - 20, 4096 + 20, int(rng.integers(1, 15))),
            rng.integers(0, m, size=int(rng.integers(1, 30)))]))
        x[js] = F32(1.0)
        check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"spikes {trial}")


# m = ceil(n/5) with m % 4 = 1, 2, 3 spanning several 4096-byte tiles and a
# ragged tail: every partition but p0 starts off the float4 grid
SHIFT_N = [5 * (4 * 4096 + 1), 5 * (4 * 4096 + 2) - 3, 5 * (4 * 4096 + 3) - 1,
           5 * (3 * 4096 + 1001) - 4, 5 * 4097 + 2]


@pytest.mark.parametrize("n", SHIFT_N)
@pytest.mark.parametrize("offset", [0, 4])
def test_partitions_off_float4_grid(ctx, n, offset):
    """16-byte aligned tensors whose partition boundaries k*m are not."""
    assert ((n + 4) // 5) % 4 != 0
    x = workloads.runs_tensor([45, n], n)
    r = workloads.normal([46, n], n, 1e-4)
    check_encode_decode(ctx, x, r, 1.75, out0=workloads.normal([47, n], n), accumulate=True,
                        offset=offset, tag=f"shift n={n}")
    x = workloads.normal([48, n], n, 1.0)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, offset=offset, tag=f"shift dense n={n}")


# tensors of 520 encoder tiles and more take the three-pass encoder (each
# tile encoded into its own slot, then the tile summaries scanned and the
# stream compacted); the patterns below stress its tile boundaries.  The
# last two have m % 4 = 0 and n % 4 = 3 or 1: the float4 path with a
# partial last float4, whose values the max pass quantizes one by one.
THREE_PASS_N = [5 * 4096 * 520, 5 * 4096 * 520 + 13, 5 * (4096 * 531 + 2) - 1,
                5 * 4096 * 520 - 1, 5 * 4096 * 520 - 3]


@pytest.mark.parametrize("n", THREE_PASS_N)
def test_three_pass_encoder_patterns(ctx, n):
    m = (n + 4) // 5
    g = G()
    check_encode_decode(ctx, np.zeros(n, F32), np.zeros(n, F32), 1.0, tag=f"zeros n={n}")
    # non-zero groups just before, at and after tile edges, and runs of every
    # length mod 14 ending at a tile edge
    rng = np.random.default_rng(n % 1000)
    x = np.zeros(n, F32)
    js = [4096 * t + d for t in range(1, m // 4096, 37) for d in (-15, -14, -13, -1, 0, 1)]
    js += [4096 * 7 - 14 * k - r for k in range(3) for r in range(14)]
    js += list(rng.integers(0, m, 300))
    js = np.unique([j for j in js if 0 <= j < m])
    x[js] = F32(1.0)
    x[4 * m + (js[js < n - 4 * m] if n - 4 * m > 0 else js[:0])] = F32(-1.0)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"edge spikes n={n}")
    x = workloads.runs_tensor([50, n], n)
    r = workloads.normal([51, n], n, 1e-4)
    check_encode_decode(ctx, x, r, 1.5, out0=workloads.normal([52, n], n), accumulate=True,
                        tag=f"runs n={n}")
    check_encode_decode(ctx, x, r, 1.5, offset=1, tag=f"runs unaligned n={n}")
    x = workloads.normal([53, n], n, 1.0)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"dense n={n}")
    g.log(f"three-pass patterns n={n} ok")


# at least 8192 encode tiles (the first pass then runs two waves per tile,
# 32 quartic bytes per thread): m % 4 = 1, 3 and 2, partial last tiles,
# padding of 2 and 4 values and none
TWO_WAVE_N = [5 * (4096 * 8192 + 1) - 2, 5 * (4096 * 8200 + 3) - 4, 5 * (4096 * 8192 + 2)]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("n", TWO_WAVE_N)
def test_first_pass_two_waves_per_tile(ctx, n):
    m = (n + 4) // 5
    g = G()
    # non-zero groups at tile edges and at the edges of each thread's two
    # 16-byte halves, in every partition
    rng = np.random.default_rng(n % 997)
    x = np.zeros(n, F32)
    js = [4096 * t + d for t in range(0, m // 4096, 97) for d in (0, 15, 16, 17, 31, 32, 4095)]
    js += list(rng.integers(0, m, 2000))
    js = np.unique([j for j in js if 0 <= j < m])
    for k in range(5):
        e = k * m + js
        x[e[e < n]] = F32(1.0 if k % 2 else -1.0)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.0, tag=f"two-wave spikes n={n}")
    x = workloads.runs_tensor([54, n], n)
    r = workloads.normal([55, n], n, 1e-4)
    check_encode_decode(ctx, x, r, 1.5, out0=workloads.normal([56, n], n), accumulate=True,
                        tag=f"two-wave runs n={n}")
    g.log(f"two-wave first pass n={n} ok")


@pytest.mark.parametrize("offset", [1, 2, 3])
def test_unaligned_pointers(ctx, offset):
    """Tensors that are not 16-byte aligned take the scalar kernels."""
    n = 5 * 4096 + 20
    x = workloads.normal([40, offset], n)
    r = workloads.normal([41, offset], n, 1e-4)
    check_encode_decode(ctx, x, r, 1.75, out0=workloads.normal([42], n), accumulate=True,
                        offset=offset, tag=f"offset {offset}")


@pytest.mark.parametrize("n", [5 * 4096 * 3 + 20, 5 * 4096 * 3 + 7, THREE_PASS_N[0],
                               THREE_PASS_N[2]])
@pytest.mark.parametrize("x_off,r_off", [(1, 0), (0, 3)])
def test_mixed_alignment(ctx, n, x_off, r_off):
    """Only one of tensor and residual 16-byte aligned: the accumulation
    takes its scalar loop, the quantizer the path the buffer allows."""
    g = G()
    x = workloads.normal([43, n, x_off], n)
    r = workloads.normal([44, n, r_off], n, 1e-4)
    r_ref = r.copy()
    st_ref, C_ref, M_ref = oracle.compress(x, r_ref, 1.5)
    st, C, M, r_gpu = g.gpu_compress(ctx, x, r, 1.5, offset=x_off, r_offset=r_off)
    assert st == st_ref == 0 and M == M_ref
    assert np.array_equal(C, C_ref)
    assert np.array_equal(g.bits(r_gpu), g.bits(r_ref))


def test_threshold_boundaries(ctx):
    """Values on both sides of the q = +-1 decision (M/2 and its rounding)."""
    for M_target in [1.0, 3.0, 1.2345678, 7.1e-39, 3 * 2.0 ** -140, 1.0e30]:
        M = F32(M_target)
        half = np.float64(M) * (0.5 + 2.0 ** -25)
        c = F32(half)
        cand = [c]
        for _ in range(4):
            cand.append(np.nextafter(cand[-1], F32(np.inf)))
        d = c
        for _ in range(4):
            d = np.nextafter(d, F32(0))
            cand.append(d)
        vals = np.array(cand + [F32(M / 2)], F32)
        x = np.concatenate([[M], vals, -vals, [F32(0.0), F32(-0.0)]]).astype(F32)
        check_encode_decode(ctx, x, np.zeros_like(x), 1.0, tag=f"M={M_target}")


@pytest.mark.parametrize("M_target", [1.0, 1.2345678, 3 * 2.0 ** -140])
def test_float4_skip_bound_edges(ctx, M_target):
    """Large tensors on the float4 path: by default the max pass decides
    every q against U itself (after the check pass has given M); with the
    in-place option it leaves a bound per float4 (top 16 bits of the
    largest |acc|) and the quantizer skips float4s whose bound is below U's
    top 16 bits.  Plant values at U, one ulp either side, and at both ends
    of U's top-half bucket among small values, in every partition and at
    tile edges; both policies, two steps each."""
    from paper_1802_07389_amd import tlc
    for opts in (0, tlc.TLC_OPT_IN_PLACE_FEEDBACK):
        ctx.set_options(opts)
        try:
            _skip_bound_edges(ctx, M_target)
        finally:
            ctx.set_options(0)


def _skip_bound_edges(ctx, M_target):
    g = G()
    n = THREE_PASS_N[0]
    m = -(-n // 5)
    assert m % 4 == 0
    M = F32(M_target)
    half = np.float64(M) * (0.5 + 2.0 ** -25)
    U = F32(half)
    if np.float64(U) <= half:
        U = np.nextafter(U, F32(np.inf))
    ub = int(np.array([U], F32).view(np.uint32)[0])
    edges = [ub, ub - 1, ub + 1, ub & ~0xFFFF, (ub & ~0xFFFF) - 1, ub | 0xFFFF,
             ((ub >> 16) + 1) << 16, ((ub >> 16) - 1) << 16 | 0xFFFF]
    # (for a subnormal U the top half is 0 and nothing may be skipped)
    mb = int(np.array([M], F32).view(np.uint32)[0])
    vals = np.array([e for e in edges if 0 < e < mb], np.uint32).view(F32)
    assert vals.size >= 3 and (vals < M).all()
    x = (workloads.normal([45], n, 1.0) * (M * F32(1e-3))).astype(F32)
    rng = np.random.default_rng(46)
    pos = set(int(p) for p in rng.integers(0, n, 400))
    for k in range(5):
        for t in (0, 1, 37, m // 4096 - 1):
            for d in (0, 1, 3, 4, 4095):
                pos.add(k * m + t * 4096 + d)
    pos = sorted(p for p in pos if 0 <= p < n)
    for i, p in enumerate(pos):
        x[p] = vals[i % len(vals)] * (1 if i % 3 else -1)
    x[n // 2 + 1] = M  # the largest |acc|: s = 1 gives exactly M
    r = np.zeros(n, F32)
    r_ref = r.copy()
    st_ref, C_ref, M_ref = oracle.compress(x, r_ref, 1.0)
    assert st_ref == 0 and M_ref == M
    st, C, Mg, r_gpu = g.gpu_compress(ctx, x, r, 1.0)
    assert st == 0 and Mg == M_ref
    assert np.array_equal(C, C_ref)
    assert np.array_equal(g.bits(r_gpu), g.bits(r_ref))
    # a second step on the returned residual (acc = x + r)
    st_ref, C_ref, M_ref = oracle.compress(x, r_ref, 1.0)
    st, C, Mg, r_gpu2 = g.gpu_compress(ctx, x, r_gpu, 1.0)
    assert st == st_ref == 0 and Mg == M_ref and np.array_equal(C, C_ref)
    assert np.array_equal(g.bits(r_gpu2), g.bits(r_ref))


def test_subnormals(ctx):
    x = (workloads.normal([50], 50000, 1.0) * F32(2.0 ** -130)).astype(F32)
    check_encode_decode(ctx, x, np.zeros_like(x), 1.0, tag="subnormal")
    check_encode_decode(ctx, x, np.zeros_like(x), 1.75, tag="subnormal s=1.75")


def test_negative_zero_accumulate(ctx):
    """Dense Eq. 3: -0.0 + M*0 = +0.0 on both sides."""
    n = 4096
    x = workloads.normal([60], n, 1.0)
    out0 = np.full(n, -0.0, F32)
    check_encode_decode(ctx, x, np.zeros(n, F32), 1.9, out0=out0, accumulate=True, tag="-0")


@pytest.mark.parametrize("scale", [-0.0, 0.0, 3.5])
def test_decode_signed_zero_scales(ctx, scale):
    """Eq. 3 takes M*q literally: a scale of -0.0 (accepted, as -0.0 >= 0)
    gives M*0 = -0.0, so -0.0 + M*0 stays -0.0, and +0.0 + M*0 is +0.0.
    Streams of random quartic bytes (q = -1, 0, 1 mixed, zero runs
    included) decoded into outputs that mix -0.0, +0.0 and other values,
    on the float4 path (m % 4 = 0, the last group in the padding), the
    shifted path (m % 4 = 2) and unaligned outputs."""
    g = G()
    rng = np.random.default_rng([61, int(np.signbit(scale)), int(scale)])
    for n, offset in [(5 * 4096 * 4, 0), (5 * 4096 * 4 - 3, 0), (61447, 0), (61447, 1)]:
        m = oracle.quartic_len(n)
        Q = rng.integers(0, 243, m, dtype=np.uint8)
        Q[rng.random(m) < 0.6] = 121
        C = oracle.zre_encode(Q)
        out0 = rng.standard_normal(n).astype(F32)
        pick = rng.random(n)
        out0[pick < 0.3] = -0.0
        out0[(pick >= 0.3) & (pick < 0.5)] = 0.0
        for acc in (False, True):
            tag = f"scale={scale!r} n={n} offset={offset} acc={acc}"
            g.log(tag)
            st_ref, out_ref = oracle.decompress(C, scale, n, out0.copy(), acc)
            st, out = g.gpu_decompress(ctx, C, scale, n, out0.copy(), acc, offset=offset)
            assert st == st_ref == 0, (tag, st, st_ref)
            if not np.array_equal(g.bits(out), g.bits(out_ref)):
                i = int(np.flatnonzero(g.bits(out) != g.bits(out_ref))[0])
                raise AssertionError(f"{tag}: decoded {i} differs: {out[i]!r} vs {out_ref[i]!r}")


# ------------------------------------------------------------------ error paths
def test_nonfinite_leaves_residual_and_bytes(ctx):
    """NaN/Inf: no byte is written and the residual is left as it was
    (reading A4), on the chained (small) and three-pass (large) encoders;
    with TLC_OPT_IN_PLACE_FEEDBACK it holds the step-1 sum x + r, as in
    the oracle's in-place variant."""
    import torch
    from paper_1802_07389_amd import tlc
    for opts in (0, tlc.TLC_OPT_IN_PLACE_FEEDBACK):
        ctx.set_options(opts)
        try:
            for n in (100_000, THREE_PASS_N[0], THREE_PASS_N[1]):
                for pos, bad in [(0, np.nan), (n - 1, np.inf), (4321, -np.inf)]:
                    x = workloads.normal([70, pos], n)
                    x[pos] = bad
                    r = workloads.normal([71, pos], n)
                    r_ref = r.copy()
                    st_ref, _, _ = oracle.compress(x, r_ref, 1.0, in_place=bool(opts))
                    xd, rd = torch.from_numpy(x).cuda(), torch.from_numpy(r).cuda()
                    out = torch.full((n // 5 + 1,), 7, dtype=torch.uint8, device="cuda")
                    st, ln, sc = tlc.tlc_compress(ctx.handle, xd.data_ptr(), rd.data_ptr(), n,
                                                  1.0, out.data_ptr(), out.numel())
                    assert st == st_ref == tlc.TLC_E_NONFINITE and ln == 0
                    assert np.array_equal(G().bits(rd.cpu().numpy()), G().bits(r_ref)), opts
                    assert bool((out == 7).all())
            # overflow of max * s: every sum is finite
            x = np.array([3.0e38, 1.0, 2.0, 3.0, 4.0], F32)
            r0 = np.array([-0.0, 0.5, 0.0, -1.0, 2.0], F32)
            r_ref = r0.copy()
            assert oracle.compress(x, r_ref, 1.5, in_place=bool(opts))[0] == oracle.E_NONFINITE
            st, _, _, r_gpu = G().gpu_compress(ctx, x, r0.copy(), 1.5)
            assert st == tlc.TLC_E_NONFINITE
            assert np.array_equal(G().bits(r_gpu), G().bits(r_ref)), opts
        finally:
            ctx.set_options(0)
    # the context still works afterwards
    check_encode_decode(ctx, workloads.normal([72], 1000), np.zeros(1000, F32), 1.0)


@pytest.mark.parametrize("n", [100_003, THREE_PASS_N[0], THREE_PASS_N[1], THREE_PASS_N[3]])
def test_in_place_option_same_results(ctx, n):
    """On finite input the in-place option changes no byte or residual."""
    from paper_1802_07389_amd import tlc
    x = workloads.normal([73, n], n, 1.0)
    r = workloads.normal([74, n], n, 1e-2)
    ctx.set_options(tlc.TLC_OPT_IN_PLACE_FEEDBACK)
    try:
        check_encode_decode(ctx, x, r, 1.5, out0=workloads.normal([75], n), accumulate=True,
                            tag=f"in place n={n}")
    finally:
        ctx.set_options(0)


def test_invalid_arguments(ctx):
    import torch
    from paper_1802_07389_amd import tlc
    n = 1000
    xd = torch.zeros(n, device="cuda")
    rd = torch.zeros(n, device="cuda")
    out = torch.zeros(n, dtype=torch.uint8, device="cuda")
    for s in (0.5, 2.0, float("nan")):
        assert tlc.tlc_compress(ctx.handle, xd.data_ptr(), rd.data_ptr(), n, s,
                                out.data_ptr(), n)[0] == tlc.TLC_E_INVALID
    assert tlc.tlc_compress(ctx.handle, xd.data_ptr(), rd.data_ptr(), n, 1.0,
                            out.data_ptr(), n // 5 - 1)[0] == tlc.TLC_E_CAPACITY
    assert tlc.tlc_compress(ctx.handle, xd.data_ptr(), xd.data_ptr(), n, 1.0,
                            out.data_ptr(), n)[0] == tlc.TLC_E_INVALID
    assert tlc.tlc_compress(ctx.handle, xd.data_ptr(), rd.data_ptr(), ctx.max_n + 1, 1.0,
                            out.data_ptr(), n)[0] == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress(ctx.handle, out.data_ptr(), 10, float("inf"), n,
                              xd.data_ptr(), 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress(ctx.handle, out.data_ptr(), 10, -1.0, n,
                              xd.data_ptr(), 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress(ctx.handle, out.data_ptr(), n // 5 + 1, 1.0, n,
                              xd.data_ptr(), 0) == tlc.TLC_E_CORRUPT
    assert tlc.tlc_decompress(ctx.handle, out.data_ptr(), 0, 1.0, n,
                              xd.data_ptr(), 0) == tlc.TLC_E_CORRUPT
    # a stream that lies inside its own output is refused before any launch
    inside = xd.data_ptr() + 4 * (n - 10)
    assert tlc.tlc_decompress(ctx.handle, inside, 40, 1.0, n,
                              xd.data_ptr(), 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress_ex(ctx.handle, tlc.TLC_MODE_INT8, xd.data_ptr(), n, 1.0, n,
                                 xd.data_ptr(), 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress_batch(ctx.handle, [inside], [40], [1.0], [n],
                                    [xd.data_ptr()], 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_decompress_sum(ctx.handle, [out.data_ptr(), inside], [40, 40],
                                  [1.0, 1.0], n, xd.data_ptr(), 0) == tlc.TLC_E_INVALID
    assert tlc.tlc_sync(ctx.handle) == tlc.TLC_OK


def test_corrupt_streams_leave_out_unchanged(ctx):
    from paper_1802_07389_amd import tlc
    n = 5 * 4096 * 3 + 11
    x = workloads.runs_tensor([80], n)
    st, C, M = oracle.compress(x, np.zeros(n, F32), 1.5)
    out0 = workloads.normal([81], n)
    bad_streams = [C[:-1], np.append(C, C[-1:]), C.copy()]
    bad_streams[2][len(C) // 2] = 255 if C[len(C) // 2] != 255 else 7
    for k, bad in enumerate(bad_streams):
        assert oracle.decompress(bad, M, n, out0.copy(), True)[0] == oracle.E_CORRUPT
        st, out = G().gpu_decompress(ctx, bad, M, n, out0.copy(), accumulate=True)
        assert st == tlc.TLC_E_CORRUPT, k
        assert np.array_equal(G().bits(out), G().bits(out0)), k
    # sticky status is cleared by tlc_sync; a good stream decodes afterwards
    st, out = G().gpu_decompress(ctx, C, M, n, out0.copy(), accumulate=True)
    assert st == tlc.TLC_OK


def test_repeated_calls_are_deterministic(ctx):
    """The look-back scans give identical bytes on every run."""
    n = 5 * 4096 * 40 + 3
    x = workloads.runs_tensor([90], n)
    first = None
    for rep in range(25):
        st, C, M, r = G().gpu_compress(ctx, x, np.zeros(n, F32), 1.5)
        assert st == 0
        if first is None:
            first = (C, M, r)
            st_ref, C_ref, M_ref = oracle.compress(x, np.zeros(n, F32), 1.5)
            assert np.array_equal(C, C_ref)
        else:
            assert np.array_equal(C, first[0]) and M == first[1]
            assert np.array_equal(G().bits(r), G().bits(first[2]))


# ------------------------------------------------------------------ configs
def test_c1_single_tensor_round_trip(ctx):
    """2^20 values ~ N(0, 1e-3), seed 0, zero residual, s = 1; acc = 0 and 1."""
    x = workloads.c1_tensor()
    r = np.zeros_like(x)
    check_encode_decode(ctx, x, r, workloads.C1_S, tag="C1")
    check_encode_decode(ctx, x, r, workloads.C1_S, out0=np.zeros_like(x), accumulate=True,
                        tag="C1 acc")


def test_c2_resnet110_ten_steps(ctx):
    """335 ResNet-110 tensors, s = 1.75, residual carried over 10 steps."""
    g = G()
    sizes = workloads.c2_sizes()
    res_gpu = [np.zeros(n, F32) for n in sizes]
    res_ref = [np.zeros(n, F32) for n in sizes]
    for step in range(workloads.C2_STEPS):
        for t, n in enumerate(sizes):
            x = workloads.c2_gradient(step, t, n)
            st_ref, C_ref, M_ref = oracle.compress(x, res_ref[t], workloads.C2_S)
            st, C, M, r = g.gpu_compress(ctx, x, res_gpu[t], workloads.C2_S)
            assert st == st_ref == 0
            assert M == M_ref and np.array_equal(C, C_ref), (step, t)
            assert np.array_equal(g.bits(r), g.bits(res_ref[t])), (step, t)
            res_gpu[t] = r
            if t % 37 == 0 or step == workloads.C2_STEPS - 1:
                st, out = g.gpu_decompress(ctx, C, M, n)
                st_ref, out_ref = oracle.decompress(C_ref, M_ref, n)
                assert st == 0 and np.array_equal(g.bits(out), g.bits(out_ref)), (step, t)
        g.log(f"C2 step {step} ok")


@pytest.mark.timeout(600)
def test_c3_runs_sweep_s(ctx):
    """64M Laplace values, 70% zeros in geometric runs; s in {1.0, 1.5, 1.9}."""
    x = workloads.c3_tensor()
    for s in workloads.C3_S:
        check_encode_decode(ctx, x, np.zeros_like(x), s, tag=f"C3 s={s}")
        G().log(f"C3 s={s} ok")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("n", [(1 << 27) + 3, 134_217_738])
def test_large_accumulate_nontemporal(ctx, n):
    """Outputs of 512 MiB and more decode with the nontemporal partition
    sweep.  Streams of synthetic quartic bytes: sparse ranges (~1.5 %
    non-121 bytes) and 10 % dense ranges (half the bytes random), decoded
    with accumulate into an output of -0.0, +0.0 and normal values (dense
    Eq. 3: -0.0 + M*0 = +0.0); m % 4 = 3 (shifted cells) and m % 4 = 0, both
    with values in the padding's partition.  A truncated and an extended
    stream must leave the output untouched."""
    from paper_1802_07389_amd import tlc
    g = G()
    rng = np.random.default_rng([62, n])
    m = oracle.quartic_len(n)
    Q = np.full(m, 121, np.uint8)
    hit = rng.random(m) < 0.015
    dense_ranges = rng.random(-(-m // 4096)) < 0.1
    hit |= np.repeat(dense_ranges, 4096)[:m] & (rng.random(m) < 0.5)
    Q[hit] = rng.integers(0, 243, int(hit.sum()), dtype=np.uint8)
    C = oracle.zre_encode(Q)
    out0 = rng.standard_normal(n).astype(F32)
    pick = rng.random(n)
    out0[pick < 0.2] = -0.0
    out0[(pick >= 0.2) & (pick < 0.3)] = 0.0
    M = np.float32(2.5e-3)
    g.log(f"nontemporal accumulate n={n} m%4={m % 4} len={C.size}")
    st_ref, out_ref = oracle.decompress(C, M, n, out0.copy(), True)
    st, out = g.gpu_decompress(ctx, C, M, n, out0.copy(), True)
    assert st == st_ref == 0, (st, st_ref)
    if not np.array_equal(g.bits(out), g.bits(out_ref)):
        i = int(np.flatnonzero(g.bits(out) != g.bits(out_ref))[0])
        raise AssertionError(f"decoded {i} differs: {out[i]!r} vs {out_ref[i]!r}")
    del out, out_ref
    for bad in (C[:-1], np.append(C, C[-1:])):
        st, out = g.gpu_decompress(ctx, bad, M, n, out0.copy(), True)
        assert st == tlc.TLC_E_CORRUPT
        assert np.array_equal(g.bits(out), g.bits(out0))


@pytest.mark.timeout(900)
def test_c4_256m_five_steps(ctx):
    """2^28 values, s = 1.75, residual carried over 5 steps; every payload
    decoded with accumulate into a persistent model buffer."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = workloads.C4_N
    r_ref = np.zeros(n, F32)
    model_ref = np.zeros(n, F32)
    rd = torch.zeros(n, device="cuda")
    model = torch.zeros(n, device="cuda")
    out = torch.empty(tlc.tlc_max_compressed_bytes(n), dtype=torch.uint8, device="cuda")
    for step in range(workloads.C4_STEPS):
        x = workloads.c4_tensor(step)
        xd = torch.from_numpy(x).cuda()
        C, M = ctx.compress(xd, rd, workloads.C4_S, out=out)
        ctx.decompress(C, M, n, model, accumulate=True)
        ctx.sync()
        st, C_ref, M_ref = oracle.compress(x, r_ref, workloads.C4_S)
        assert st == 0 and M == M_ref
        assert np.array_equal(C.cpu().numpy(), C_ref), step
        assert np.array_equal(g.bits(rd.cpu().numpy()), g.bits(r_ref)), step
        st, model_ref = oracle.decompress(C_ref, M_ref, n, model_ref, accumulate=True)
        assert np.array_equal(g.bits(model.cpu().numpy()), g.bits(model_ref)), step
        g.log(f"C4 step {step} ok: len={C_ref.size} ratio={4 * n / (C_ref.size + 4):.1f}")
        del xd


@pytest.mark.timeout(900)
def test_c5_aggregation_and_reencode(ctx):
    """16 payloads of 25.6M values decoded into one fp32 sum, then re-encoded."""
    import torch
    g = G()
    n = workloads.C5_N
    sum_ref = np.zeros(n, F32)
    sumd = torch.zeros(n, device="cuda")
    payloads = []
    for p in range(workloads.C5_PAYLOADS):
        x = workloads.c5_tensor(p)
        st, C, M, r = g.gpu_compress(ctx, x, np.zeros(n, F32), workloads.C5_S)
        r_ref = np.zeros(n, F32)
        st_ref, C_ref, M_ref = oracle.compress(x, r_ref, workloads.C5_S)
        assert st == st_ref == 0 and M == M_ref and np.array_equal(C, C_ref), p
        assert np.array_equal(g.bits(r), g.bits(r_ref)), p
        payloads.append((torch.from_numpy(C).cuda(), M, C_ref))
    for Cd, M, C_ref in payloads:
        ctx.decompress(Cd, M, n, sumd, accumulate=True)
        oracle.decompress(C_ref, M, n, sum_ref, accumulate=True)
    ctx.sync()
    assert np.array_equal(g.bits(sumd.cpu().numpy()), g.bits(sum_ref))
    g.log("C5 aggregate ok")
    res = check_encode_decode(ctx, sum_ref, np.zeros(n, F32), workloads.C5_S, tag="C5 re-encode")
    g.log(f"C5 re-encode ok: len={res[0].size}")


# ------------------------------------------------------------------ seeded shapes
def _seeded_cases(count=40, seed=20261202):
    """(index, kind, n, offset, s, accumulate) draws: n log-uniform up to 3M
    values, every tenth past the three-pass threshold (512 tiles of 4096
    quartic bytes); offsets 0-4 values (alignment); s in [1, 2) as fp32."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        kind = ("normal", "runs", "spikes", "wide")[i % 4]
        if i % 10 == 9:
            n = int(5 * 4096 * 512 + rng.integers(0, 5 * 4096 * 4))
        else:
            n = int(np.exp(rng.uniform(0.0, np.log(3 << 20))))
        s = float(F32(1.0 + rng.uniform(0.0, 0.999)))
        cases.append((i, kind, n, int(rng.integers(0, 5)), s, bool(rng.integers(0, 2))))
    return cases


@pytest.mark.parametrize("case", _seeded_cases(), ids=lambda c: f"{c[0]}-{c[1]}-n{c[2]}")
def test_seeded_random_shapes(ctx, case):
    """Forty seeded draws of size, alignment, s, input kind (small normal
    values, zero runs, isolated spikes, unit-scale values) and accumulate:
    stream, M, residual and decoded output bit-exact against the oracle."""
    i, kind, n, offset, s, acc = case
    if kind == "normal":
        x = workloads.normal([760, i], n, 1e-3)
    elif kind == "runs":
        x = workloads.runs_tensor([760, i], n)
    elif kind == "wide":
        x = workloads.normal([760, i], n, 1.0)
    else:
        x = np.zeros(n, F32)
        js = np.random.default_rng([760, i]).integers(0, n, max(1, n // 5000))
        x[js] = workloads.normal([763, i], js.size, 1.0)
    r = workloads.normal([761, i], n, 1e-4) if i % 3 else np.zeros(n, F32)
    out0 = workloads.normal([762, i], n, 1e-3) if acc else None
    check_encode_decode(ctx, x, r, s, out0=out0, accumulate=acc, offset=offset,
                        tag=f"case {i} {kind} n={n} offset={offset} s={s}")
