"""CPU-only checks of the HIP library's host side and of the facts its
kernels rely on (no GPU needed, no compute call into the library)."""
import os
import re
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
F32 = np.float32


def header_functions():
    text = open(os.path.join(ROOT, "include", "tlc.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(tlc_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    from paper_1802_07389_amd import build, tlc
    assert os.path.exists(build.LIB)
    declared = header_functions()
    assert len(declared) >= 16
    out = subprocess.run(["nm", "-D", "--defined-only", build.LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(tlc_\w+)$", out, flags=re.M))
    assert set(declared) <= exported, set(declared) - exported
    assert set(tlc.EXPORTS) == set(declared)
    for name in declared:
        getattr(tlc.lib, name)


@pytest.mark.parametrize("std", ["c99", "c11"])
def test_header_is_plain_c(tmp_path, std):
    """include/tlc.h is a C ABI: it compiles as strict C with every warning,
    and a C caller can name every entry point."""
    src = tmp_path / "use.c"
    calls = "\n".join(f"  (void){name};" for name in header_functions())
    src.write_text('#include "tlc.h"\nint main(void) {\n' + calls + "\n  return TLC_OK;\n}\n")
    subprocess.run(["gcc", f"-std={std}", "-pedantic", "-Wall", "-Wextra", "-Werror", "-c",
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(tmp_path / "use.o")],
                   check=True)


def test_binding_constants_match_header():
    """Every TLC_* integer #define of the C header has the same value in the
    Python binding."""
    from paper_1802_07389_amd import tlc
    text = open(os.path.join(ROOT, "include", "tlc.h")).read()
    defs = dict(re.findall(r"^#define\s+(TLC_\w+)\s+\(?(-?\d+)[uU]?L*L*\)?", text, flags=re.M))
    defs.update(re.findall(r"^#define\s+(TLC_MAX_N)\s+\(\(size_t\)(\d+)u\)", text, flags=re.M))
    assert len(defs) >= 25 and "TLC_MAX_N" in defs
    for name, val in defs.items():
        assert getattr(tlc, name) == int(val), name


def test_host_only_entry_points():
    from paper_1802_07389_amd import tlc
    for n in list(range(0, 50)) + [2 ** 20, 2 ** 28, 25_600_000, 4294967295]:
        assert tlc.tlc_max_compressed_bytes(n) == -(-n // 5)
    names = [tlc.tlc_kernel_name(k) for k in range(tlc.TLC_KERNEL_COUNT)]
    assert names == ["tlc_accum_absmax_kernel", "tlc_quant_encode_kernel", "tlc_zre_index_kernel",
                     "tlc_expand_dequant_kernel", "tlc_accum_absmax_batch_kernel",
                     "tlc_quant_encode_batch_kernel", "tlc_zre_index_batch_kernel",
                     "tlc_expand_dequant_batch_kernel", "tlc_expand_sum_kernel",
                     "tlc_quant_pack_kernel", "tlc_int8_quant_kernel",
                     "tlc_int8_dequant_kernel", "tlc_zre_chunk_kernel", "tlc_zre_compact_kernel",
                     "tlc_quant_encode_chained_kernel", "tlc_absmax_check_kernel",
                     "tlc_absmax_check_batch_kernel", "tlc_accum_quantize_kernel"]
    assert tlc.tlc_kernel_name(99) is None
    # every name is a __global__ function of the library's sources
    csrc = os.path.join(ROOT, "paper_1802_07389_amd", "csrc")
    src = "".join(open(os.path.join(csrc, f)).read() for f in os.listdir(csrc)
                  if f.endswith(".hip"))
    for name in filter(None, names):
        assert re.search(r"__global__[^;{]*\b" + name + r"\s*\(", src, flags=re.S), name


def test_ctx_create_fails_cleanly_without_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    from paper_1802_07389_amd import tlc
    with pytest.raises(tlc.TLCError) as e:
        tlc.tlc_ctx_create(1000, None)
    assert e.value.code == tlc.TLC_E_DEVICE
    with pytest.raises(tlc.TLCError) as e:
        tlc.tlc_ctx_create(0, None)
    assert e.value.code == tlc.TLC_E_INVALID


@pytest.fixture(scope="module")
def zsim(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("zsim") / "zre_tiling_sim")
    subprocess.run(["g++", "-std=c++17", "-O2", "-Wall", "-Werror", "-o", exe,
                    os.path.join(ROOT, "tests", "host", "zre_tiling_sim.cpp")], check=True)
    return exe


@pytest.mark.parametrize("tile,per", [(4096, 16), (64, 16), (16, 4), (14, 7), (5, 1), (28, 14)])
def test_zre_tiling_matches_oracle(zsim, tile, per):
    """The kernel's run-phase summaries, cut at arbitrary tile and thread
    boundaries, reproduce the sequential zero-run encoding exactly."""
    rng = np.random.default_rng(tile * 100 + per)
    for trial in range(60):
        m = int(rng.integers(0, 9000))
        p = rng.choice([0.0, 0.3, 0.9, 0.97, 0.999, 1.0])
        Q = np.where(rng.random(m) < p, 121, rng.integers(0, 243, m)).astype(np.uint8)
        r = subprocess.run([zsim, str(tile), str(per)], input=Q.tobytes(),
                           capture_output=True, check=True)
        assert np.array_equal(np.frombuffer(r.stdout, np.uint8), oracle.zre_encode(Q)), trial


@pytest.fixture(scope="module")
def zdef(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("zdef") / "zre_deferred_sim")
    subprocess.run(["g++", "-std=c++17", "-O2", "-Wall", "-Werror", "-o", exe,
                    os.path.join(ROOT, "tests", "host", "zre_deferred_sim.cpp")], check=True)
    return exe


@pytest.mark.parametrize("tile,per", [(4096, 16), (64, 16), (16, 4), (14, 7), (5, 1), (28, 14),
                                      (30, 2)])
def test_zre_three_pass_matches_oracle(zdef, tile, per):
    """The single-tensor encoder's three passes (each tile encoded from its
    first non-121 byte into its own slot, a scan of tile summaries, then the
    leading runs' codes written with the incoming phase) reproduce the
    sequential zero-run encoding exactly."""
    rng = np.random.default_rng(tile * 1000 + per)
    for trial in range(60):
        m = int(rng.integers(0, 9000))
        p = rng.choice([0.0, 0.3, 0.9, 0.97, 0.999, 1.0])
        Q = np.where(rng.random(m) < p, 121, rng.integers(0, 243, m)).astype(np.uint8)
        r = subprocess.run([zdef, str(tile), str(per)], input=Q.tobytes(),
                           capture_output=True, check=True)
        assert np.array_equal(np.frombuffer(r.stdout, np.uint8), oracle.zre_encode(Q)), trial


def quant_threshold(M):
    """Smallest float32 u with u > M * (0.5 + 2^-25) (exact in float64)."""
    T = np.float64(M) * (0.5 + 2.0 ** -25)
    f = np.float32(T)
    if np.float64(f) <= T:
        f = np.nextafter(f, np.float32(np.inf))
    return f


@pytest.mark.parametrize("M", [1.0, 1.5, 0.7071067, 3.0e-3, 1.9e30, 2.0 ** -126,
                               3 * 2.0 ** -140, 2.0 ** -149])
def test_quantization_threshold_lemma(M):
    """The kernels decide q = rint(fl(acc/M)) by comparing acc with U.

    Exhaustive over every float32 in [M/4, M] (both signs) plus zero: IEEE
    division followed by round-half-even agrees with (acc >= U) - (acc <= -U).
    Below M/4 both give 0.
    """
    M = F32(M)
    U = quant_threshold(M)
    assert M / 4 < U <= M
    lo = np.float32(M / 4).view(np.uint32)
    hi = M.view(np.uint32)
    for start in range(int(lo), int(hi) + 1, 1 << 22):
        stop = min(int(hi) + 1, start + (1 << 22))
        acc = np.arange(start, stop, dtype=np.uint32).view(F32)
        for a in (acc, -acc):
            q_div = np.rint(a / M).astype(np.int8)
            q_thr = (a >= U).astype(np.int8) - (a <= -U).astype(np.int8)
            assert np.array_equal(q_div, q_thr), (M, start)
    assert np.rint(F32(0) / M) == 0


def test_quantization_threshold_matches_oracle():
    """The same decision through the C oracle on values hugging U."""
    for M in [F32(1.0), F32(2.5e-3), F32(3 * 2.0 ** -140)]:
        U = quant_threshold(M)
        vals = [U]
        for _ in range(3):
            vals.append(np.nextafter(vals[-1], F32(0)))
        acc = np.array([M] + vals + [-v for v in vals], F32)
        st, Mo = oracle.absmax_scale(acc, 1.0)
        q, _ = oracle.quantize(acc, Mo)
        assert Mo == M
        expect = [1] + [1, 0, 0, 0] + [-1, 0, 0, 0]
        assert q.tolist() == expect


def test_byte_tricks_of_the_zero_run_kernels():
    """The word-level shortcuts the zero-run kernels take, exhaustively.

    * The index scan counts a stream byte's expansion beyond one quartic
      byte as (|b - 242| + b - 242) / 2, from two sums of absolute byte
      differences: it must equal expanded length - 1 (codes 243..255 stand
      for runs of 2..14 bytes of 121, every other byte for itself).
    * The first encode pass marks quartic byte i as non-121 from its five
      trits (q + 1): a byte is 121 exactly when all five trits are 1.
    * The spread byte mask gathers the four bytes' flags with one multiply
      (constant with bits 0, 6, 12, 18), whose partial products must not
      overlap.
    """
    b = np.arange(256, dtype=np.int64)
    expanded = np.where(b < 243, 1, b - 241)
    assert np.array_equal((np.abs(b - 242) + b - 242) // 2, expanded - 1)
    # five trits per byte, weights 81, 27, 9, 3, 1: only 11111 (base 3) is 121
    t = np.array(np.meshgrid(*[np.arange(3)] * 5, indexing="ij")).reshape(5, -1)
    byte = (t * np.array([81, 27, 9, 3, 1])[:, None]).sum(0)
    assert np.array_equal(byte == 121, (t == 1).all(0))
    # flags at bits 0, 8, 16, 24 times 0x41041: every partial product on its
    # own bit, and the four flags land on bits 18, 20, 22, 24
    bits = sorted(8 * f + k for f in range(4) for k in (0, 6, 12, 18) if 8 * f + k < 32)
    assert len(bits) == len(set(bits))
    for flags in range(16):
        y = sum(((flags >> f) & 1) << (8 * f) for f in range(4))
        spread = ((y * 0x00041041) & 0xFFFFFFFF) >> 18 & 0x55
        assert spread == sum(((flags >> f) & 1) << (2 * f) for f in range(4))
