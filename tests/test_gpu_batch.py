"""GPU parity of the batched entry points (tlc_compress_batch,
tlc_decompress_batch, tlc_decompress_sum) against the CPU oracle applied
tensor by tensor / stream by stream.  Bar: bit-exact."""
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
def bctx():
    from paper_1802_07389_amd import tlc
    c = tlc.Context(max_n=16 * workloads.C5_N, max_tensors=400)
    yield c
    c.close()


def batch_encode(ctx, xs, rs, ss, offsets=None):
    """Run tlc_compress_batch; return (status, per-tensor status, [(bytes,
    scale, residual)])."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    offsets = offsets or [0] * len(xs)
    xd = [g.to_dev(x, o) for x, o in zip(xs, offsets)]
    rd = [g.to_dev(r, o) for r, o in zip(rs, offsets)]
    outs = [torch.full((max(tlc.tlc_max_compressed_bytes(x.size), 1),), 0xAB,
                       dtype=torch.uint8, device="cuda") for x in xs]
    ptr = lambda t, n: t.data_ptr() if n else None
    st, lens, scales, stat = tlc.tlc_compress_batch(
        ctx.handle, [ptr(t, x.size) for t, x in zip(xd, xs)],
        [ptr(t, x.size) for t, x in zip(rd, xs)], [x.size for x in xs], ss,
        [o.data_ptr() for o in outs], [o.numel() for o in outs])
    torch.cuda.synchronize()
    res = [(o[:ln].cpu().numpy(), sc, r.cpu().numpy(), o.cpu().numpy())
           for o, ln, sc, r in zip(outs, lens, scales, rd)]
    return st, stat, res


def check_against_oracle(xs, rs, ss, res, tag):
    g = G()
    for t, (x, r, s) in enumerate(zip(xs, rs, ss)):
        r_ref = r.copy()
        st, C_ref, M_ref = oracle.compress(x, r_ref, s)
        C, M, r_gpu, _ = res[t]
        assert st == 0, (tag, t)
        assert M == M_ref, (tag, t, M, M_ref)
        assert np.array_equal(C, C_ref), (tag, t, C.size, C_ref.size)
        assert np.array_equal(g.bits(r_gpu), g.bits(r_ref)), (tag, t)


def test_batch_mixed_sizes_and_alignment(bctx):
    sizes = [0, 1, 5, 7, 13, 4096 * 5, 4096 * 5 + 3, 100003, 0, 5 * 14 * 4096 + 9, 262144]
    offs = [0, 0, 1, 0, 3, 0, 2, 0, 0, 1, 0]
    xs, rs, ss = [], [], []
    for t, n in enumerate(sizes):
        x = workloads.runs_tensor([700, t], n) if t % 2 else workloads.normal([701, t], n, 1.0)
        xs.append(x)
        rs.append(workloads.normal([702, t], n, 1e-4))
        ss.append([1.0, 1.5, 1.75, 1.9][t % 4])
    st, stat, res = batch_encode(bctx, xs, rs, ss, offs)
    assert st == 0 and all(v == 0 for v in stat)
    check_against_oracle(xs, rs, ss, res, "mixed")


def test_batch_nonfinite_tensor_is_refused_alone(bctx):
    from paper_1802_07389_amd import tlc
    g = G()
    sizes = [1000, 5000, 20481, 7]
    xs = [workloads.normal([710, t], n, 1.0) for t, n in enumerate(sizes)]
    rs = [workloads.normal([711, t], n, 1e-3) for t, n in enumerate(sizes)]
    xs[2][123] = np.nan
    ss = [1.0] * 4
    st, stat, res = batch_encode(bctx, xs, rs, ss)
    assert st == tlc.TLC_E_NONFINITE
    assert stat == [0, 0, tlc.TLC_E_NONFINITE, 0]
    C, M, r_gpu, raw = res[2]
    assert C.size == 0
    assert np.array_equal(g.bits(r_gpu), g.bits(rs[2]))  # residual untouched
    assert bool((raw == 0xAB).all())  # bytes untouched
    keep = [0, 1, 3]
    check_against_oracle([xs[i] for i in keep], [rs[i] for i in keep], [ss[i] for i in keep],
                         [res[i] for i in keep], "nonfinite-others")


def test_batch_fills_the_context(bctx):
    """A batch of exactly max_tensors tensors: the per-tensor results come
    back with the control block in one copy, up to the last slot of the
    context's readback block; then a smaller batch on the same context,
    whose results must not be stale ones from the first."""
    from paper_1802_07389_amd import tlc
    T = 40
    ctx = tlc.Context(max_n=T * 30000, max_tensors=T)
    try:
        sizes = [int(v) for v in np.random.default_rng(720).integers(1, 30000, size=T)]
        sizes[5] = 0
        xs = [workloads.normal([721, t], n, 1.0) for t, n in enumerate(sizes)]
        rs = [workloads.normal([722, t], n, 1e-3) for t, n in enumerate(sizes)]
        xs[T - 1][0] = np.inf  # the last slot reports its own error
        ss = [[1.0, 1.25, 1.5, 1.99][t % 4] for t in range(T)]
        st, stat, res = batch_encode(ctx, xs, rs, ss)
        assert st == tlc.TLC_E_NONFINITE
        assert stat == [0] * (T - 1) + [tlc.TLC_E_NONFINITE]
        assert res[T - 1][0].size == 0
        keep = [t for t in range(T - 1) if sizes[t]]
        check_against_oracle([xs[i] for i in keep], [rs[i] for i in keep], [ss[i] for i in keep],
                             [res[i] for i in keep], "full")
        k = 7
        xs2 = [workloads.normal([723, t], n, 1.0) for t, n in enumerate(sizes[:k])]
        rs2 = [np.zeros(n, F32) for n in sizes[:k]]
        st, stat, res = batch_encode(ctx, xs2, rs2, ss[:k])
        assert st == 0 and stat == [0] * k
        check_against_oracle(xs2, rs2, ss[:k], res, "smaller after full")
    finally:
        ctx.close()


def test_batch_argument_errors(bctx):
    import torch
    from paper_1802_07389_amd import tlc
    x = torch.zeros(100, device="cuda")
    r = torch.zeros(100, device="cuda")
    o = torch.zeros(100, dtype=torch.uint8, device="cuda")
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [x.data_ptr()], [r.data_ptr()], [100], [1.0],
                                    [o.data_ptr()], [19])
    assert st == tlc.TLC_E_CAPACITY
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [x.data_ptr()], [r.data_ptr()], [100], [2.0],
                                    [o.data_ptr()], [20])
    assert st == tlc.TLC_E_INVALID
    k = bctx.max_tensors + 1
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [x.data_ptr()] * k, [r.data_ptr()] * k,
                                    [0] * k, [1.0] * k, [o.data_ptr()] * k, [20] * k)
    assert st == tlc.TLC_E_INVALID
    assert tlc.tlc_sync(bctx.handle) == tlc.TLC_OK


def test_batch_c2_ten_steps_and_batch_decode(bctx):
    """C2 through the batched calls: 335 tensors, 10 steps, residuals carried;
    every step's streams decoded in one batch (odd steps accumulate).  Every
    tensor's stream, scale, residual and decoded output is compared with the
    oracle after every step."""
    import torch
    g = G()
    sizes = workloads.c2_sizes()
    rs_gpu = [torch.zeros(n, device="cuda") for n in sizes]
    rs_ref = [np.zeros(n, F32) for n in sizes]
    outs = [torch.full((n,), -0.0, device="cuda") for n in sizes]
    outs_ref = [np.full(n, -0.0, F32) for n in sizes]
    for step in range(workloads.C2_STEPS):
        xs = [workloads.c2_gradient(step, t, n) for t, n in enumerate(sizes)]
        xd = [torch.from_numpy(x).cuda() for x in xs]
        pays = bctx.compress_batch(xd, rs_gpu, workloads.C2_S)
        acc = step % 2 == 1
        for t, x in enumerate(xs):
            st, C_ref, M_ref = oracle.compress(x, rs_ref[t], workloads.C2_S)
            C, M = pays[t]
            assert st == 0 and M == M_ref, (step, t)
            assert np.array_equal(C.cpu().numpy(), C_ref), (step, t)
            st, outs_ref[t] = oracle.decompress(C_ref, M_ref, sizes[t], outs_ref[t],
                                                accumulate=acc)
            assert st == 0, (step, t)
        bctx.decompress_batch([p[0] for p in pays], [p[1] for p in pays], outs, accumulate=acc)
        bctx.sync()
        r_all = g.bits(torch.cat(rs_gpu).cpu().numpy())
        o_all = g.bits(torch.cat(outs).cpu().numpy())
        assert np.array_equal(r_all, g.bits(np.concatenate(rs_ref))), step
        assert np.array_equal(o_all, g.bits(np.concatenate(outs_ref))), step
        g.log(f"batched C2 step {step} ok: all 335 residuals and outputs")


def test_batch_overlapping_buffers_are_refused(bctx):
    """A residual or byte buffer shared between two tensors of one batch, or
    an output shared between two streams (or overlapping a stream's bytes),
    is an argument error: nothing runs.  One stream decoded into several
    outputs (read-only bytes shared) stays allowed."""
    import torch
    from paper_1802_07389_amd import tlc
    n = 5000
    m = tlc.tlc_max_compressed_bytes(n)
    x = torch.from_numpy(workloads.normal([990, 0], 2 * n, 1e-3)).cuda()
    r = torch.zeros(2 * n, device="cuda")
    b = torch.zeros(2 * m, dtype=torch.uint8, device="cuda")
    xp, rp, bp = x.data_ptr(), r.data_ptr(), b.data_ptr()
    r_before = r.clone()
    # the second tensor's residual starts inside the first one's
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [xp, xp + 4 * n], [rp, rp + 4 * (n - 1)],
                                    [n, n], [1.5, 1.5], [bp, bp + m], [m, m])
    assert st == tlc.TLC_E_INVALID
    # both tensors write the same bytes
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [xp, xp + 4 * n], [rp, rp + 4 * n],
                                    [n, n], [1.5, 1.5], [bp, bp], [m, m])
    assert st == tlc.TLC_E_INVALID
    # a residual over another tensor's input
    x2 = torch.from_numpy(workloads.normal([990, 1], n, 1e-3)).cuda()
    st, *_ = tlc.tlc_compress_batch(bctx.handle, [xp, x2.data_ptr()], [rp, xp + 8],
                                    [n, n], [1.5, 1.5], [bp, bp + m], [m, m])
    assert st == tlc.TLC_E_INVALID
    assert torch.equal(r, r_before)
    # disjoint buffers: accepted, and the same input read by both tensors is fine
    st, lens, scales, stat = tlc.tlc_compress_batch(
        bctx.handle, [xp, xp], [rp, rp + 4 * n], [n, n], [1.5, 1.5], [bp, bp + m], [m, m])
    assert st == tlc.TLC_OK and lens[0] == lens[1] and scales[0] == scales[1]
    o = torch.zeros(2 * n, device="cuda")
    op = o.data_ptr()
    # overlapping outputs
    st = tlc.tlc_decompress_batch(bctx.handle, [bp, bp], lens, scales, [n, n],
                                  [op, op + 4 * (n - 3)], 0)
    assert st == tlc.TLC_E_INVALID
    # an output over the other stream's bytes
    bb = torch.zeros(4 * n + m, dtype=torch.uint8, device="cuda")
    bb[:lens[0]].copy_(b[:lens[0]])
    st = tlc.tlc_decompress_batch(bctx.handle, [bb.data_ptr(), bp], lens, scales, [n, n],
                                  [op, bb.data_ptr() + 4], 0)
    assert st == tlc.TLC_E_INVALID
    assert tlc.tlc_sync(bctx.handle) == tlc.TLC_OK
    # one stream into two disjoint outputs: accepted, both decode the same values
    st = tlc.tlc_decompress_batch(bctx.handle, [bp, bp], [lens[0]] * 2, [scales[0]] * 2,
                                  [n, n], [op, op + 4 * n], 0)
    assert st == tlc.TLC_OK and tlc.tlc_sync(bctx.handle) == tlc.TLC_OK
    assert torch.equal(o[:n], o[n:])


def test_batch_overlap_check_after_repeated_calls(bctx):
    """The same buffers passed again skip the overlap sort (the previous
    call's ranges passed); a batch that differs is checked in full, a
    refused one is not remembered, and the good batch then passes again."""
    import torch
    from paper_1802_07389_amd import tlc
    n = 7000
    m = tlc.tlc_max_compressed_bytes(n)
    x = torch.from_numpy(workloads.normal([991, 0], 2 * n, 1e-3)).cuda()
    r = torch.zeros(2 * n, device="cuda")
    b = torch.zeros(2 * m, dtype=torch.uint8, device="cuda")
    o = torch.zeros(2 * n, device="cuda")
    xp, rp, bp, op = x.data_ptr(), r.data_ptr(), b.data_ptr(), o.data_ptr()
    good = ([xp, xp + 4 * n], [rp, rp + 4 * n], [n, n], [1.5, 1.5], [bp, bp + m], [m, m])
    bad = ([xp, xp + 4 * n], [rp, rp + 4 * (n - 1)], [n, n], [1.5, 1.5], [bp, bp + m], [m, m])
    for args in (good, good, bad, bad, good):
        r_before = r.clone()
        st, lens, scales, stat = tlc.tlc_compress_batch(bctx.handle, *args)
        if args is bad:
            assert st == tlc.TLC_E_INVALID and torch.equal(r, r_before)
        else:
            assert st == tlc.TLC_OK
    for outs, ok in (([op, op + 4 * n], True), ([op, op + 4 * n], True),
                     ([op, op + 4 * (n - 1)], False), ([op, op + 4 * (n - 1)], False),
                     ([op, op + 4 * n], True)):
        st = tlc.tlc_decompress_batch(bctx.handle, [bp, bp + m], lens, scales, [n, n], outs, 0)
        assert st == (tlc.TLC_OK if ok else tlc.TLC_E_INVALID)
        assert tlc.tlc_sync(bctx.handle) == tlc.TLC_OK


def test_batch_decode_corrupt_writes_nothing(bctx):
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    sizes = [5000, 20481, 300]
    xs = [workloads.runs_tensor([720, t], n) for t, n in enumerate(sizes)]
    pays = []
    for x in xs:
        st, C, M = oracle.compress(x, np.zeros(x.size, F32), 1.5)
        pays.append((C, M))
    bad = pays[1][0].copy()
    bad[len(bad) // 2] = 7 if bad[len(bad) // 2] >= 243 else 255
    streams = [pays[0][0], bad, pays[2][0]]
    outs0 = [workloads.normal([721, t], n) for t, n in enumerate(sizes)]
    outs = [torch.from_numpy(o.copy()).cuda() for o in outs0]
    cd = [torch.from_numpy(c).cuda() for c in streams]
    bctx.decompress_batch(cd, [p[1] for p in pays], outs, accumulate=True)
    assert tlc.tlc_sync(bctx.handle) == tlc.TLC_E_CORRUPT
    for o, o0 in zip(outs, outs0):
        assert np.array_equal(g.bits(o.cpu().numpy()), g.bits(o0))


@pytest.mark.parametrize("n,count,offset", [(1, 3, 0), (7, 2, 0), (4096 * 5 + 13, 3, 0),
                                            (4096 * 5 * 3, 5, 1), (100003, 4, 0),
                                            (262144, 2, 2)])
def test_decompress_sum_small(bctx, n, count, offset):
    """Streams summed in order equal sequential decode-accumulate, bit for bit."""
    g = G()
    import torch
    pays = []
    for p in range(count):
        x = workloads.runs_tensor([730, n, p], n) if p % 2 else workloads.normal([731, n, p], n)
        st, C, M = oracle.compress(x, np.zeros(n, F32), [1.0, 1.75, 1.5][p % 3])
        pays.append((C, M))
    out0 = workloads.normal([732, n], n, 1e-3)
    for acc in (False, True):
        ref = out0.copy()
        for p, (C, M) in enumerate(pays):
            st, ref = oracle.decompress(C, M, n, ref, accumulate=(acc or p > 0))
        od = g.to_dev(out0, offset)
        bctx.decompress_sum([torch.from_numpy(C).cuda() for C, _ in pays],
                            [M for _, M in pays], od, accumulate=acc)
        bctx.sync()
        assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(ref)), (n, count, acc)


@pytest.mark.parametrize("count", [64, 65, 131])
def test_decompress_sum_many_streams_odd_offsets(bctx, count):
    """More streams than one block stages at once, each stream starting at
    an odd byte offset of one shared buffer (slices at every alignment);
    summed in order, bit for bit against sequential decode-accumulate."""
    import torch
    g = G()
    n = 4096 * 5 * 2 + 11
    pays = []
    for p in range(count):
        x = workloads.runs_tensor([733, p], n) if p % 3 else workloads.normal([734, p], n)
        st, C, M = oracle.compress(x, np.zeros(n, F32), [1.0, 1.75, 1.5][p % 3])
        pays.append((C, M))
    buf = torch.zeros(sum(C.size + 3 for C, _ in pays) + 16, dtype=torch.uint8, device="cuda")
    views, at = [], 1
    for p, (C, _) in enumerate(pays):
        at += p % 4  # offsets of every residue mod 4
        buf[at:at + C.size] = torch.from_numpy(C).cuda()
        views.append(buf[at:at + C.size])
        at += C.size
    out0 = workloads.normal([735, count], n, 1e-3)
    ref = out0.copy()
    for C, M in pays:
        st, ref = oracle.decompress(C, M, n, ref, accumulate=True)
    od = torch.from_numpy(out0.copy()).cuda()
    bctx.decompress_sum(views, [M for _, M in pays], od, accumulate=True)
    bctx.sync()
    assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(ref)), count


def test_decompress_sum_corrupt_leaves_out(bctx):
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    n = 5 * 4096 * 2 + 3
    pays = []
    for p in range(3):
        x = workloads.runs_tensor([740, p], n)
        st, C, M = oracle.compress(x, np.zeros(n, F32), 1.5)
        pays.append((C, M))
    bad = pays[2][0][:-1]
    out0 = workloads.normal([741], n)
    od = torch.from_numpy(out0.copy()).cuda()
    bctx.decompress_sum([torch.from_numpy(c).cuda() for c in (pays[0][0], pays[1][0], bad)],
                        [M for _, M in pays], od, accumulate=True)
    assert tlc.tlc_sync(bctx.handle) == tlc.TLC_E_CORRUPT
    assert np.array_equal(g.bits(od.cpu().numpy()), g.bits(out0))


@pytest.mark.timeout(900)
def test_c5_aggregation_fused(bctx):
    """C5 with the fused aggregation: 16 payloads of 25.6M values summed in one
    pass; then the aggregate is re-encoded."""
    import torch
    g = G()
    n = workloads.C5_N
    payloads = []
    sum_ref = np.zeros(n, F32)
    for p in range(workloads.C5_PAYLOADS):
        x = workloads.c5_tensor(p)
        st, C, M = oracle.compress(x, np.zeros(n, F32), workloads.C5_S)
        assert st == 0
        st, sum_ref = oracle.decompress(C, M, n, sum_ref, accumulate=True)
        payloads.append((torch.from_numpy(C).cuda(), M))
    sumd = torch.zeros(n, device="cuda")
    bctx.decompress_sum([c for c, _ in payloads], [M for _, M in payloads], sumd,
                        accumulate=True)
    bctx.sync()
    assert np.array_equal(g.bits(sumd.cpu().numpy()), g.bits(sum_ref))
    g.log("C5 fused aggregation ok")


def test_shared_pull_one_payload_many_receivers(bctx):
    """Section 3 (shared compression of a pull): the server encodes one
    model delta once and every worker decodes the same payload into its own
    model replica.  One batched call with the stream repeated gives every
    replica exactly the oracle's decode-accumulate."""
    import torch
    g = G()
    n = 4096 * 5 * 3 + 7
    delta = workloads.runs_tensor([730], n)
    st, C, M = oracle.compress(delta, np.zeros(n, F32), 1.5)
    assert st == 0
    Cd = torch.from_numpy(C).cuda()
    replicas0 = [workloads.normal([731, w], n) for w in range(6)]
    outs = [torch.from_numpy(r.copy()).cuda() for r in replicas0]
    bctx.decompress_batch([Cd] * len(outs), [M] * len(outs), outs, accumulate=True)
    bctx.sync()
    for w, (o, r0) in enumerate(zip(outs, replicas0)):
        st, ref = oracle.decompress(C, M, n, r0.copy(), accumulate=True)
        assert st == 0 and np.array_equal(g.bits(o.cpu().numpy()), g.bits(ref)), w


@pytest.mark.parametrize("big", [False, True])
@pytest.mark.parametrize("corrupt", [False, True])
def test_batch_decode_short_and_long_streams(bctx, big, corrupt):
    """A batch of short streams (one or two 8 KiB scan tiles each), and one
    that also holds a stream of several scan tiles: both give the oracle's
    decode-accumulate bit for bit, and a corrupt stream in either (here the
    last, the long one in the second batch) leaves every output untouched.
    The kernel timers show one scan launch and one expansion launch."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()
    sizes = [300, 20481, 4096 * 5 + 3, 7] + ([1 << 20] if big else [])
    xs = [workloads.normal([740, t], n, 1.0) if n == 1 << 20 else
          workloads.runs_tensor([740, t], n) for t, n in enumerate(sizes)]
    pays = []
    for x in xs:
        st, C, M = oracle.compress(x, np.zeros(x.size, F32), 1.0)
        assert st == 0
        pays.append((C, M))
    longest = max(C.size for C, _ in pays)
    assert (longest > 2 * 8192) == big, longest
    streams = [C for C, _ in pays]
    if corrupt:
        bad = streams[-1].copy()
        bad[len(bad) // 2] = 7 if bad[len(bad) // 2] >= 243 else 255
        streams[-1] = bad
    outs0 = [workloads.normal([741, t], n) for t, n in enumerate(sizes)]
    outs = [torch.from_numpy(o.copy()).cuda() for o in outs0]
    bctx.profile(True, kernels=[tlc.TLC_KERNEL_ZRE_INDEX_BATCH,
                                tlc.TLC_KERNEL_EXPAND_DEQUANT_BATCH])
    bctx.profile_reset()
    bctx.decompress_batch([torch.from_numpy(C).cuda() for C in streams],
                          [M for _, M in pays], outs, accumulate=True)
    st = tlc.tlc_sync(bctx.handle)
    scans = bctx.profile_get(tlc.TLC_KERNEL_ZRE_INDEX_BATCH)[1]
    expands = bctx.profile_get(tlc.TLC_KERNEL_EXPAND_DEQUANT_BATCH)[1]
    bctx.profile(False)
    assert (scans, expands) == (1, 1)
    if corrupt:
        assert st == tlc.TLC_E_CORRUPT
        for o, o0 in zip(outs, outs0):
            assert np.array_equal(g.bits(o.cpu().numpy()), g.bits(o0))
        return
    assert st == tlc.TLC_OK
    for t, (o, o0) in enumerate(zip(outs, outs0)):
        st, ref = oracle.decompress(pays[t][0], pays[t][1], sizes[t], o0.copy(), True)
        assert st == 0 and np.array_equal(g.bits(o.cpu().numpy()), g.bits(ref)), t


def test_batch_calls_alternating_buffer_sets(bctx):
    """Batched encodes on one context that alternate between two sets of
    buffers, and repeat one, all match the oracle (the residuals carried
    from call to call): nothing of one call's descriptors leaks into the
    next."""
    import torch
    from paper_1802_07389_amd import tlc
    g = G()

    def make(sizes, seed):
        xs = [torch.empty(n, dtype=torch.float32, device="cuda") for n in sizes]
        rs = [torch.zeros(n, dtype=torch.float32, device="cuda") for n in sizes]
        outs = [torch.empty(tlc.tlc_max_compressed_bytes(n), dtype=torch.uint8, device="cuda")
                for n in sizes]
        return dict(sizes=sizes, xs=xs, rs=rs, outs=outs, r_ref=[np.zeros(n, F32) for n in sizes],
                    seed=seed)

    def run(b, step):
        xh = [workloads.normal([760, b["seed"], step, t], n, 1.0)
              for t, n in enumerate(b["sizes"])]
        for x, xd in zip(xh, b["xs"]):
            xd.copy_(torch.from_numpy(x))
        ss = [1.75] * len(xh)
        st, lens, scales, stat = tlc.tlc_compress_batch(
            bctx.handle, [t.data_ptr() for t in b["xs"]], [t.data_ptr() for t in b["rs"]],
            b["sizes"], ss, [o.data_ptr() for o in b["outs"]], [o.numel() for o in b["outs"]])
        torch.cuda.synchronize()
        assert st == 0 and all(v == 0 for v in stat), (b["seed"], step)
        for t, x in enumerate(xh):
            st_ref, C_ref, M_ref = oracle.compress(x, b["r_ref"][t], 1.75)
            assert st_ref == 0 and scales[t] == M_ref, (b["seed"], step, t)
            assert np.array_equal(b["outs"][t][:lens[t]].cpu().numpy(), C_ref), (b["seed"], step, t)
            assert np.array_equal(g.bits(b["rs"][t].cpu().numpy()), g.bits(b["r_ref"][t])), \
                (b["seed"], step, t)

    A = make([2 * 20480 + 7, 1000, 5], 1)
    B = make([333, 20480 + 1], 2)
    for step, b in enumerate([A, A, B, A, B, B, A]):
        run(b, step)
