"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  None of these needs a GPU, and none
compares the oracle only with itself: the expected values come from the
paper (tests/golden/paper_values.json), from hand derivations
(tests/golden/worked_examples.json), from closed forms, invariants, brute
force, or from the independently written numpy reference in defref.py.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import defref
import oracle
from paper_1802_07389_amd import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")
PAPER = json.load(open(os.path.join(GOLD, "paper_values.json")))
WORKED = json.load(open(os.path.join(GOLD, "worked_examples.json")))
F32 = np.float32


def pv(key):
    return PAPER[key]["value"]


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


# ------------------------------------------------------------------ Section 3.2
def test_qe_bijection_over_all_243_trit_groups():
    """Section 3.2: 3^5 = 243 codes, weights 81/27/9/3/1, decode inverts."""
    codes = set()
    for trits in itertools.product((0, 1, 2), repeat=5):
        q = np.array(trits, dtype=np.int8) - 1
        Q = oracle.quartic_encode(q)
        assert Q.size == 1
        expect = sum(w * t for w, t in zip(pv("qe_weights"), trits))
        assert int(Q[0]) == expect
        codes.add(int(Q[0]))
        assert np.array_equal(oracle.quartic_decode(Q, 5), q)
    assert len(codes) == pv("qe_distinct_codes")
    assert codes == set(range(pv("qe_max_byte") + 1))


def test_qe_zero_group_is_121_and_max_is_242():
    """Section 3.3: five zeros -> 121; Section 3.3: bytes never exceed 242."""
    assert oracle.quartic_encode(np.zeros(5, np.int8))[0] == pv("zero_group_byte")
    assert oracle.quartic_encode(np.ones(5, np.int8))[0] == pv("qe_max_byte")
    assert oracle.quartic_encode(-np.ones(5, np.int8))[0] == 0


def test_qe_partition_layout_single_element():
    """Section 3.2 steps 4-6 (contiguous partitions, p0 most significant).

    Setting element i of an otherwise zero tensor to +1 (or -1) changes only
    byte i mod m, by +-3^(4 - i // m).  A transposed (interleaved) layout or
    reversed digit weights fails this.
    """
    for n in (5, 9, 37, 50, 64):
        m = oracle.quartic_len(n)
        base = oracle.quartic_encode(np.zeros(n, np.int8)).astype(int)
        for i in range(n):
            for sign in (1, -1):
                q = np.zeros(n, np.int8)
                q[i] = sign
                d = oracle.quartic_encode(q).astype(int) - base
                expect = np.zeros(m, int)
                expect[i % m] = sign * 3 ** (4 - i // m)
                assert np.array_equal(d, expect), (n, i, sign)


def test_qe_pad_trits_are_zero():
    """Section 3.2 step 4 pads after the +1: pad trits are 0 (q = -1)."""
    for n in range(1, 41):
        m = oracle.quartic_len(n)
        pad = 5 * m - n
        Q = oracle.quartic_encode(np.zeros(n, np.int8))
        # pad positions are the last `pad` entries of p4 (the units digit)
        expect = np.full(m, 121, dtype=np.uint8)
        # p3 and p4 digits that fall past n are 0 instead of 1
        for flat in range(n, 5 * m):
            k, j = divmod(flat, m)
            expect[j] -= 3 ** (4 - k)
        assert np.array_equal(Q, expect), n
        assert pad == 5 * m - n


def test_qe_matches_numpy_reference_and_roundtrips_tiny():
    """Sizes 0..40 against defref (5 x m row view of the padded trits)."""
    rng = np.random.default_rng(7)
    for n in range(0, 41):
        for _ in range(5):
            q = rng.integers(-1, 2, size=n).astype(np.int8)
            Q = oracle.quartic_encode(q)
            assert np.array_equal(Q, defref.quartic(q))
            assert np.array_equal(oracle.quartic_decode(Q, n), q)
            assert Q.max(initial=0) <= 242


def test_qe_density_matches_paper():
    """Section 3.2: 1.6 bits per value, 0.95% above log2 3; 2-bit is ~26% above."""
    assert 8 / pv("qe_digits_per_byte") == pytest.approx(pv("qe_bits_per_value"))
    over = (pv("qe_bits_per_value") / math.log2(3) - 1) * 100
    assert over == pytest.approx(pv("qe_overhead_vs_log2_3_percent"), abs=0.005)
    assert (2 / math.log2(3) - 1) * 100 == pytest.approx(
        pv("two_bit_overhead_percent"), abs=0.5)


# ------------------------------------------------------------------ Section 3.3
def _zre_len_formula(seq):
    return sum(1 for b in seq if b != 121) + sum(
        -(-L // 14) for L in defref.runs(seq))


def test_zre_exhaustive_small_strings():
    """Section 3.3 on every string over {121, 7} of length <= 15."""
    for L in range(0, 16):
        for tup in itertools.product((121, 7), repeat=L):
            Q = np.array(tup, dtype=np.uint8)
            C = oracle.zre_encode(Q)
            assert C.size == _zre_len_formula(tup)
            assert np.array_equal(C, defref.zre(Q))
            st, back = oracle.zre_decode(C, L)
            assert st == oracle.OK and np.array_equal(back, Q)


def test_zre_codes_and_canonical_form():
    """Section 3.3: k in [2, 14] -> 243 + (k - 2); codes 243..255 only."""
    first, last = pv("zre_code_first"), pv("zre_code_last")
    kmin, kmax = pv("zre_run_min"), pv("zre_run_max")
    assert last - first == kmax - kmin
    for k in range(1, 60):
        C = oracle.zre_encode(np.full(k, 121, np.uint8))
        full, rem = divmod(k, kmax)
        expect = [last] * full
        if rem == 1:
            expect.append(121)
        elif rem >= kmin:
            expect.append(first + rem - kmin)
        assert C.tolist() == expect, k
        # within a run every code but the last is the full-chunk code
        assert all(b == last for b in C.tolist()[:-1])
    # runs embedded between data bytes
    for k in range(kmin, kmax + 1):
        Q = np.array([5] + [121] * k + [200], np.uint8)
        assert oracle.zre_encode(Q).tolist() == [5, first + k - kmin, 200]


def test_zre_random_long_streams_roundtrip():
    rng = np.random.default_rng(11)
    for trial in range(30):
        m = int(rng.integers(1, 5000))
        p121 = rng.choice([0.0, 0.5, 0.9, 0.99, 1.0])
        Q = np.where(rng.random(m) < p121, 121,
                     rng.integers(0, 243, size=m)).astype(np.uint8)
        C = oracle.zre_encode(Q)
        assert C.size == _zre_len_formula(Q.tolist())
        assert np.array_equal(C, defref.zre(Q))
        st, back = oracle.zre_decode(C, m)
        assert st == oracle.OK and np.array_equal(back, Q)


def test_zre_decode_rejects_wrong_length():
    """A stream that expands to more or fewer than m bytes is corrupt."""
    Q = np.array([7, 121, 121, 121, 9], np.uint8)
    C = oracle.zre_encode(Q)
    assert oracle.zre_decode(C, 5)[0] == oracle.OK
    assert oracle.zre_decode(C[:-1], 5)[0] == oracle.E_CORRUPT
    assert oracle.zre_decode(np.append(C, 7).astype(np.uint8), 5)[0] == oracle.E_CORRUPT
    assert oracle.zre_decode(C, 6)[0] == oracle.E_CORRUPT
    assert oracle.zre_decode(np.array([255], np.uint8), 13)[0] == oracle.E_CORRUPT


def test_all_zero_tensor_reaches_280x():
    """Section 3.3: an all-zero fp32 tensor compresses 280x (4 B * 5 * 14)."""
    target = pv("all_zero_fp32_ratio")
    for k in (1, 3, 100, 2000):
        n = 70 * k
        st, C, M = oracle.compress(np.zeros(n, F32), np.zeros(n, F32), 1.0)
        assert st == oracle.OK and M == 0.0
        assert C.size == k
        assert 4 * n / C.size == target


def test_no_zre_ratio_is_20x():
    """Table 2 'No ZRE': quartic bytes alone give 32 / 1.6 = 20x."""
    n = 5 * 1000
    q = np.random.default_rng(3).integers(-1, 2, n).astype(np.int8)
    assert 4 * n / oracle.quartic_encode(q).size == pv("no_zre_ratio")


# ------------------------------------------------------------------ worked examples
@pytest.mark.parametrize("case", [c for c in WORKED["cases"] if "x" in c],
                         ids=lambda c: c["name"])
def test_worked_example(case):
    x = np.array(case["x"], F32)
    r = np.array(case["r"], F32)
    st, C, M = oracle.compress(x, r, case["s"])
    assert st == oracle.OK
    assert M == case["scale"]
    assert C.tolist() == case["bytes"]
    assert np.array_equal(bits(r), bits(np.array(case["residual"], F32)))
    acc = oracle.accumulate(np.array(case["x"], F32), np.array(case["r"], F32))
    q, _ = oracle.quantize(acc, M)
    assert q.tolist() == case["q"]
    assert oracle.quartic_encode(q).tolist() == case["Q"]
    st, out = oracle.decompress(C, M, x.size)
    assert st == oracle.OK
    assert np.array_equal(bits(out), bits(np.array(case["decoded"], F32)))


def test_worked_two_step_error_feedback():
    case = next(c for c in WORKED["cases"] if c["name"] == "two_step_error_feedback")
    r = np.zeros(5, F32)
    for stp in case["steps"]:
        st, C, M = oracle.compress(np.array(stp["x"], F32), r, stp["s"])
        assert st == oracle.OK and M == stp["scale"]
        assert C.tolist() == stp["bytes"]
        assert r.tolist() == stp["residual"]


def test_worked_all_zero_runs():
    for n, expect in WORKED["all_zero_runs"].items():
        if n.startswith("_"):
            continue
        n = int(n)
        st, C, M = oracle.compress(np.zeros(n, F32), np.zeros(n, F32), 1.0)
        assert st == oracle.OK and C.tolist() == expect, n


def test_worked_all_zero_2p20():
    g = WORKED["all_zero_2p20"]
    n = g["n"]
    st, C, M = oracle.compress(np.zeros(n, F32), np.zeros(n, F32), 1.0)
    assert st == oracle.OK and C.size == g["len"]
    assert C[-4:].tolist() == g["tail_bytes"]
    assert set(C[:-4].tolist()) <= {255, 243 + (209712 % 14) - 2}


# ------------------------------------------------------------------ Section 3.1
def test_quantized_alphabet_and_error_bound():
    """Section 3.1: q in {-1,0,1}; |acc - M q| <= M/2 (plus the rounding of
    acc/M to 0.5, i.e. M * 2^-25); M/2 < max|acc| for s < 2."""
    for seed, s in [(1, 1.0), (2, 1.3), (3, 1.75), (4, 1.999)]:
        x = workloads.normal([seed], 20000, 1.0)
        acc = x.copy()
        st, M = oracle.absmax_scale(acc, s)
        q, r = oracle.quantize(acc, M)
        assert set(np.unique(q).tolist()) <= set(pv("quantized_alphabet"))
        err = np.abs(acc.astype(np.float64) - M * q.astype(np.float64))
        assert err.max() <= M * (0.5 + 2.0 ** -25)
        assert M / 2 < np.abs(acc).max()
        # the residual is acc - M q computed exactly (Sterbenz for q != 0)
        assert np.array_equal(r.astype(np.float64),
                              acc.astype(np.float64) - M * q.astype(np.float64))


def test_s1_preserves_max_magnitude():
    """Section 3.1: s = 1 keeps the largest magnitude through quantization."""
    for seed in range(5):
        x = workloads.normal([100, seed], 5000, 3e-2)
        i = int(np.argmax(np.abs(x)))
        st, C, M = oracle.compress(x, np.zeros_like(x), 1.0)
        st, out = oracle.decompress(C, M, x.size)
        assert out[i] == x[i]
        assert np.abs(out).max() == np.abs(x).max()


def test_max_element_never_zeroed_for_s_below_2():
    """Section 3.1: M/2 < max|T_in| whenever s < 2."""
    for s in (1.0, 1.5, 1.9, float(np.nextafter(F32(2.0), F32(0.0)))):
        x = workloads.normal([200], 3000, 1.0)
        acc = x.copy()
        st, M = oracle.absmax_scale(acc, s)
        q, _ = oracle.quantize(acc, M)
        i = int(np.argmax(np.abs(acc)))
        assert q[i] == np.sign(acc[i])


def test_larger_s_is_sparser():
    """Section 3.1: a larger s produces at least as many zeros."""
    x = workloads.normal([300], 50000, 1.0)
    zeros = []
    for s in np.linspace(1.0, 1.99, 23):
        st, M = oracle.absmax_scale(x, float(s))
        q, _ = oracle.quantize(x, M)
        zeros.append(int((q == 0).sum()))
    assert all(a <= b for a, b in zip(zeros, zeros[1:]))
    assert zeros[-1] > zeros[0]


def test_round_half_to_even_ties():
    """Eq. 2 uses round(); ties at +-0.5 go to 0 (half to even)."""
    acc = np.array([1.0, 0.5, -0.5, 0.5000001, -0.5000001], F32)
    st, M = oracle.absmax_scale(acc, 1.0)
    q, _ = oracle.quantize(acc, M)
    assert q.tolist() == [1, 0, 0, 1, -1]


def test_zero_tensor_scale_zero_residual_keeps_signed_zero():
    """M = 0: every q is 0 and the residual equals the sum, -0.0 included."""
    x = np.array([0.0, -0.0, 0.0, -0.0, 0.0, -0.0, 0.0], F32)
    r = np.zeros(7, F32)
    st, C, M = oracle.compress(x, r, 1.0)
    assert st == oracle.OK and M == 0.0
    assert np.array_equal(bits(r), bits(x + np.zeros(7, F32)))


def test_subnormal_inputs_and_scale():
    """No flush to zero: a subnormal tensor quantizes like a scaled normal one."""
    tiny = F32(2.0 ** -140)
    x = np.array([3, 1, -2, 0, 1.5], F32) * tiny
    st, C, M = oracle.compress(x, np.zeros(5, F32), 1.0)
    assert st == oracle.OK and M == 3 * tiny and M < np.finfo(F32).tiny
    acc = x.copy()
    q, _ = oracle.quantize(acc, M)
    # 1/3 -> 0, -2/3 -> -1, 1.5/3 = 0.5 -> 0
    assert q.tolist() == [1, 0, -1, 0, 0]


def test_nonfinite_is_rejected_and_leaves_state():
    """NaN/Inf, or max*s overflowing: no quantization exists, so the buffer
    and the bytes are left alone (reading A4); the in-place variant has
    done step 1 (Section 3.1, Fig. 3) in the buffer already, so it keeps
    x + r there."""
    for bad in (np.inf, -np.inf, np.nan):
        for enc in (oracle.compress, oracle.compress_nozre):
            x = workloads.normal([400], 100, 1.0)
            x[37] = bad
            r = workloads.normal([401], 100, 1.0)
            r0 = r.copy()
            st, C, M = enc(x, r, 1.0)
            assert st == oracle.E_NONFINITE and C.size == 0
            assert np.array_equal(bits(r), bits(r0))
            r = r0.copy()
            st, C, M = enc(x, r, 1.0, in_place=True)
            assert st == oracle.E_NONFINITE and C.size == 0
            assert np.array_equal(bits(r), bits(x + r0))
    # overflow of max * s: every sum is finite
    x = np.array([3.0e38, 1.0], F32)
    r = np.array([-0.0, 0.5], F32)
    assert oracle.compress(x, r, 1.5)[0] == oracle.E_NONFINITE
    assert np.array_equal(bits(r), bits(np.array([-0.0, 0.5], F32)))
    assert oracle.compress(x, r, 1.5, in_place=True)[0] == oracle.E_NONFINITE
    assert np.array_equal(bits(r), bits(np.array([3.0e38, 1.5], F32)))
    # argument errors leave the buffer alone in both forms
    r = np.ones(2, F32)
    for ip in (False, True):
        assert oracle.compress(x, r, 2.0, in_place=ip)[0] == oracle.E_INVALID
        assert oracle.compress(x, r, 1.0, cap=0, in_place=ip)[0] == oracle.E_CAPACITY
    assert r.tolist() == [1.0, 1.0]


def test_in_place_variant_matches_on_finite_input():
    x = workloads.normal([402], 5003, 1.0)
    r0 = workloads.normal([403], 5003, 1e-2)
    r1, r2 = r0.copy(), r0.copy()
    a = oracle.compress(x, r1, 1.5)
    b = oracle.compress(x, r2, 1.5, in_place=True)
    assert a[0] == b[0] == 0 and a[2] == b[2] and np.array_equal(a[1], b[1])
    assert np.array_equal(bits(r1), bits(r2))


def test_invalid_s_rejected():
    x = np.ones(10, F32)
    for s in (0.999, 2.0, 2.5, -1.0, float("nan")):
        assert oracle.compress(x, np.zeros(10, F32), s)[0] == oracle.E_INVALID
    assert oracle.compress(x, np.zeros(10, F32), 1.0, cap=1)[0] == oracle.E_CAPACITY


def test_empty_tensor():
    st, C, M = oracle.compress(np.zeros(0, F32), np.zeros(0, F32), 1.0)
    assert st == oracle.OK and C.size == 0 and M == 0.0
    assert oracle.decompress(C, 0.0, 0)[0] == oracle.OK


# ------------------------------------------------------------------ Eq. 3
def test_dequantize_and_signed_zero_accumulate():
    """Eq. 3 applied densely (reading A13): every element is written, so
    -0.0 + M*0 gives +0.0."""
    q = np.array([1, 0, -1, 0], np.int8)
    out = np.array([-0.0, -0.0, 2.0, 5.0], F32)
    oracle.dequantize(q, F32(0.25), out, accumulate=True)
    assert np.array_equal(bits(out), bits(np.array([0.25, 0.0, 1.75, 5.0], F32)))
    out = oracle.dequantize(q, F32(0.25))
    assert np.array_equal(bits(out), bits(np.array([0.25, 0.0, -0.25, 0.0], F32)))


def test_zero_update_accumulates_densely():
    """The encoding of an all-zero change accumulated into an aggregate adds
    +0.0 to every element: -0.0 becomes +0.0, every other finite value and
    the infinities keep their bits, NaNs stay NaN."""
    n = 1003
    special = np.array([0x80000000, 0x7F800000, 0xFF800000, 0x7FC00001, 0x00000001,
                        0x80000001], np.uint32)
    out0 = workloads.normal([502], n, 1.0)
    out0.view(np.uint32)[::7][:special.size] = special
    st, C, M = oracle.compress(np.zeros(n, F32), np.zeros(n, F32), 1.0)
    assert st == oracle.OK and M == 0.0
    expect = out0.copy()
    expect[(expect == 0) & np.signbit(expect)] = 0.0
    for scale in (0.0, 1.0):  # any scale: q = 0 everywhere
        st, out = oracle.decompress(C, scale, n, out0.copy(), accumulate=True)
        assert st == oracle.OK
        nan = np.isnan(expect)
        assert np.array_equal(np.isnan(out), nan)
        assert np.array_equal(bits(out[~nan]), bits(expect[~nan]))
        assert not (np.signbit(out) & (out == 0)).any()


def test_decompress_corrupt_leaves_out_unchanged():
    x = workloads.normal([500], 1000, 1.0)
    st, C, M = oracle.compress(x, np.zeros_like(x), 1.0)
    out = workloads.normal([501], 1000, 1.0)
    out0 = out.copy()
    for bad in (C[:-1], np.append(C, 3).astype(np.uint8)):
        st, _ = oracle.decompress(bad, M, 1000, out, accumulate=True)
        assert st == oracle.E_CORRUPT
        assert np.array_equal(bits(out), bits(out0))
    assert oracle.decompress(C, float("nan"), 1000, out)[0] == oracle.E_INVALID
    assert oracle.decompress(C, -1.0, 1000, out)[0] == oracle.E_INVALID


# ------------------------------------------------------------------ second implementation
@pytest.mark.parametrize("kind", ["c1", "runs", "c2_tensor"])
def test_oracle_matches_numpy_reference(kind):
    """Bit-equal against defref (numpy float32 division, np.rint, groupby)."""
    if kind == "c1":
        x, s = workloads.c1_tensor(), 1.0
        r = np.zeros_like(x)
    elif kind == "runs":
        x, s = workloads.runs_tensor([600], 300001), 1.5
        r = workloads.normal([601], 300001, 1e-4)
    else:
        x, s = workloads.c2_gradient(0, 100, 36864), 1.75
        r = workloads.normal([602], 36864, 1e-3)
    r_ref = r.copy()
    C_ref, M_ref, res_ref = defref.compress(x, r_ref, s)
    st, C, M = oracle.compress(x, r, s)
    assert st == oracle.OK
    assert bits(np.array([M]))[0] == bits(np.array([M_ref]))[0]
    assert np.array_equal(C, C_ref)
    assert np.array_equal(bits(r), bits(res_ref))
    out0 = workloads.normal([603], x.size, 1e-3)
    st, out = oracle.decompress(C, M, x.size, out0.copy(), accumulate=True)
    assert np.array_equal(bits(out), bits(defref.decompress(C_ref, M_ref, x.size, out0)))


# ------------------------------------------------------------------ error feedback
def test_error_feedback_telescopes():
    """Section 3.1, Fig. 3: what was not sent stays in the buffer.

    Over T steps, sum_t x_t = sum_t M_t q_t + r_T up to the fp32 rounding of
    the accumulation step alone (the residual update is exact).
    """
    n, T, s = 4096, 10, 1.75
    r = np.zeros(n, F32)
    sent = np.zeros(n, np.float64)
    total = np.zeros(n, np.float64)
    slack = np.zeros(n, np.float64)
    for t in range(T):
        x = workloads.normal([700, t], n, 1e-2)
        acc = oracle.accumulate(x, r)
        slack += np.abs(acc.astype(np.float64)) * 2.0 ** -24
        st, C, M = oracle.compress(x, r, s)
        st, dq = oracle.decompress(C, M, n)
        sent += dq.astype(np.float64)
        total += x.astype(np.float64)
    gap = np.abs(total - (sent + r.astype(np.float64)))
    assert np.all(gap <= slack + 1e-30)
