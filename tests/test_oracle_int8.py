"""Pins of the oracle's 8-bit integer comparator (the "8-bit int" design
of Section 5.1: 255 codes -127..127, -128 unused).

The step is D = fl(M / 127), the code rint(fl(acc / D)) clamped to
[-127, 127], the value fl(q * D).  Each pin checks the oracle against a
closed form, a library routine it reduces to, or an invariant that holds
for every input -- not against a retyped copy of its own formula.
"""
import numpy as np
import pytest

import oracle
from paper_1802_07389_amd import workloads

F32 = np.float32
TINY = F32(2.0 ** -149)  # smallest subnormal


def codes(b):
    return np.asarray(b, np.uint8).view(np.int8).astype(np.int64)


def test_unit_step_is_round_half_even():
    """M = 127 gives D = 1 exactly, so the code is rint(acc) (ties to even,
    numpy's rint) and the residual acc - q is exact."""
    acc = (np.arange(-127 * 4, 127 * 4 + 1) / 4.0).astype(F32)  # quarters, ties included
    st, C, M = oracle.compress_int8(acc, None, 1.0)
    assert st == 0 and M == 127.0 and oracle.int8_step(M) == 1.0
    assert np.array_equal(codes(C), np.rint(acc).astype(np.int64))
    for v, q in [(0.5, 0), (1.5, 2), (2.5, 2), (-0.5, 0), (-1.5, -2), (126.5, 126), (-126.5, -126)]:
        assert codes(C)[np.flatnonzero(acc == F32(v))[0]] == q, v
    r = np.zeros_like(acc)
    st, C2, _ = oracle.compress_int8(acc, r, 1.0)
    assert np.array_equal(C2, C)
    assert np.array_equal(r.astype(np.float64), acc.astype(np.float64) - np.rint(acc))


@pytest.mark.parametrize("s", [1.0, 1.5, 1.99])
def test_code_range_and_extremes(s):
    x = workloads.normal([960, int(s * 100)], 100003, 1e-3)
    st, C, M = oracle.compress_int8(x, None, s)
    q = codes(C)
    assert st == 0 and C.size == x.size
    assert q.min() >= -127 and q.max() <= 127 and not (C == 0x80).any()
    i = int(np.argmax(np.abs(x)))
    if s == 1.0:  # the largest magnitude maps to the outermost code
        assert abs(q[i]) == 127 and np.sign(q[i]) == np.sign(x[i])
    else:  # it maps to about 127 / s
        assert abs(abs(q[i]) - 127.0 / s) <= 0.5 + 1e-6


@pytest.mark.parametrize("s", [1.0, 1.75])
def test_error_bound_and_monotone(s):
    """|acc - q D| <= D (1/2 + 127 * 2^-24) (one rounding of acc / D, then
    rint), and q is non-decreasing in acc."""
    x = np.sort(workloads.normal([961], 50000, 1.0))
    st, C, M = oracle.compress_int8(x, None, s)
    D = float(oracle.int8_step(M))
    q = codes(C)
    err = np.abs(x.astype(np.float64) - q * D)
    assert err.max() <= D * (0.5 + 127 * 2.0 ** -24)
    assert (np.diff(q) >= 0).all()


def test_subnormal_step_clamps_and_zero_step():
    # M = 190 * 2^-149: D = fl(190/127 * 2^-149) = 2^-149, M / D = 190 -> clamp
    x = np.array([190, -190, 3, 0], F32) * TINY
    r = np.zeros(4, F32)
    st, C, M = oracle.compress_int8(x, r, 1.0)
    assert st == 0 and M == F32(190) * TINY and oracle.int8_step(M) == TINY
    assert codes(C).tolist() == [127, -127, 3, 0]
    assert r.tolist() == (np.array([63, -63, 0, 0], F32) * TINY).tolist()
    # M = 63 * 2^-149: D rounds to 0, everything quantizes to 0
    x = np.array([63, -5, 1], F32) * TINY
    r = np.zeros(3, F32)
    st, C, M = oracle.compress_int8(x, r, 1.0)
    assert st == 0 and oracle.int8_step(M) == 0.0
    assert codes(C).tolist() == [0, 0, 0] and np.array_equal(r, x)


def test_zero_empty_and_nonfinite():
    st, C, M = oracle.compress_int8(np.zeros(1000, F32), None, 1.0)
    assert st == 0 and M == 0.0 and C.size == 1000 and not C.any()
    st, C, M = oracle.compress_int8(np.zeros(0, F32), None, 1.0)
    assert st == 0 and C.size == 0 and M == 0.0
    x = workloads.normal([962], 100)
    x[7] = np.inf
    r = workloads.normal([963], 100, 1e-3)
    r0 = r.copy()
    st, C, M = oracle.compress_int8(x, r, 1.0)
    assert st == oracle.E_NONFINITE and C.size == 0 and np.array_equal(r, r0)
    st, C, M = oracle.compress_int8(x, r, 1.0, in_place=True)  # step 1 done in the buffer
    assert st == oracle.E_NONFINITE and C.size == 0
    assert np.array_equal(r.view(np.uint32), (x + r0).view(np.uint32))
    st, *_ = oracle.compress_int8(np.ones(4, F32), None, 2.0)
    assert st == oracle.E_INVALID


def test_decode_closed_form():
    """Every byte at M = 127 (D = 1) decodes to its int8 value; accumulate
    adds it densely, so code 0 turns -0.0 into +0.0."""
    C = np.arange(256, dtype=np.uint8)
    st, out = oracle.decompress_int8(C, 127.0, 256)
    assert st == 0 and np.array_equal(out, C.view(np.int8).astype(F32))
    st, out = oracle.decompress_int8(C, 127.0, 256, np.full(256, -0.0, F32), accumulate=True)
    assert st == 0 and np.array_equal(out, C.view(np.int8).astype(F32))
    assert not np.signbit(out[0])
    # M = 254: D = 2 exactly
    st, out = oracle.decompress_int8(C, 254.0, 256, np.ones(256, F32), accumulate=True)
    assert np.array_equal(out, 2 * C.view(np.int8).astype(F32) + 1)


def test_decode_rejects_length_and_scale():
    out0 = workloads.normal([964], 10)
    out = out0.copy()
    st, out = oracle.decompress_int8(np.zeros(9, np.uint8), 1.0, 10, out)
    assert st == oracle.E_CORRUPT and np.array_equal(out, out0)
    st, _ = oracle.decompress_int8(np.zeros(10, np.uint8), -1.0, 10)
    assert st == oracle.E_INVALID
    st, _ = oracle.decompress_int8(np.zeros(10, np.uint8), float("nan"), 10)
    assert st == oracle.E_INVALID


def test_error_feedback_telescopes():
    """With error feedback, sum_t x_t = sum_t q_t D_t + r_T up to the fp32
    rounding of each step's adds (float64 check)."""
    n = 20000
    r = np.zeros(n, F32)
    sx = np.zeros(n)
    sd = np.zeros(n)
    for t in range(8):
        x = workloads.normal([965, t], n, 1e-3)
        st, C, M = oracle.compress_int8(x, r, 1.0)
        assert st == 0
        sx += x
        sd += codes(C) * float(oracle.int8_step(M))
    assert np.abs(sx - sd - r).max() <= 8 * 2 ** -24 * np.abs(sx).max() * 4 + 1e-12
    assert np.abs(r).max() <= 0.5 * 2e-3 / 127 * 5  # residual stays about half a step


def test_signed_zero_residual():
    """A value whose sum is -0.0 takes code 0, and its residual is
    -0.0 - 0 * D: the integer code 0 times D > 0 is +0, and -0.0 - (+0.0)
    is -0.0 in round-to-nearest, so the residual keeps the sign bit
    (0x80000000).  A sum of +0.0 keeps +0.0."""
    x = np.array([1.0, -0.0, -0.0, 0.5, 0.0], F32)
    r = np.array([0.0, -0.0, 0.0, 0.0, -0.0], F32)  # sums: 1, -0, +0, 0.5, +0
    st, C, M = oracle.compress_int8(x, r, 1.0)
    assert st == 0 and M == 1.0
    assert list(codes(C)) == [127, 0, 0, 64, 0]
    assert list(r.view(np.uint32)[1:3]) == [0x80000000, 0]
    assert r.view(np.uint32)[4] == 0
