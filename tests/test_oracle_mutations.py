"""The oracle's pins catch plausible mistakes.  Each case plants one
mistake in a copy of oracle/tlc_ref.c (a dropped term, a wrong sign,
weight, rounding, layout, bound or check), builds it, and runs the pin
file that covers that part against it (TLC_REF_LIBRARY) in a child
process: at least one pin must fail.  A control build of the unchanged
source passes every pin file."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
PINS = "tests/test_oracle_pins.py"
INT8 = "tests/test_oracle_int8.py"
MODES = "tests/test_oracle_modes.py"

# (name, pin file, text in tlc_ref.c, replacement)
MUTATIONS = [
    ("round half away from zero", PINS, "q[i] = (int8_t)rintf(v);", "q[i] = (int8_t)roundf(v);"),
    ("residual sign", PINS, "resid[i] = acc[i] - M * (float)q[i];",
     "resid[i] = acc[i] + M * (float)q[i];"),
    ("no error feedback", PINS, "acc[i] = x[i] + r[i];", "acc[i] = x[i];"),
    ("scale without s", PINS, "float M = A * s;", "float M = A;"),
    ("trit weights swapped", PINS, "p0[j] * 81u + p1[j] * 27u", "p0[j] * 27u + p1[j] * 81u"),
    ("padding with trit 1", PINS, "memset(u, 0, 5 * m);", "memset(u, 1, 5 * m);"),
    ("groups of five consecutive values", PINS,
     "u[k * m + j] = (uint8_t)((Q[j] / pow3[k]) % 3u);",
     "u[j * 5 + k] = (uint8_t)((Q[j] / pow3[k]) % 3u);"),
    ("runs cut at 13", PINS, "size_t k = L < REF_RUN_MAX ? L : REF_RUN_MAX;",
     "size_t k = L < 13u ? L : 13u;"),
    ("run code off by one", PINS, "(uint8_t)(REF_RUN_BASE + (k - REF_RUN_MIN))",
     "(uint8_t)(REF_RUN_BASE + (k - REF_RUN_MIN) + 1u)"),
    ("lone 121 coded as a run", PINS, "out[o++] = (k == 1) ? (uint8_t)REF_ZERO_GROUP",
     "out[o++] = (k == 0) ? (uint8_t)REF_ZERO_GROUP"),
    ("decode drops accumulate", PINS, "out[i] = accumulate ? out[i] + t : t;", "out[i] = t;"),
    ("decode skips zero terms", PINS, "    float t = M * (float)q[i];\n",
     "    if (q[i] == 0) continue;\n    float t = M * (float)q[i];\n"),
    ("no expanded-length check", PINS, "return pos == m ? TLC_REF_OK : TLC_REF_E_CORRUPT;",
     "return TLC_REF_OK;"),
    ("NaN not refused", PINS, "if (!isfinite(acc[i])) return TLC_REF_E_NONFINITE;",
     "if (0) return TLC_REF_E_NONFINITE;"),
    ("Philox multiplier", MODES, "ref_mulhilo(0xD2511F53u, c0,", "ref_mulhilo(0xD2511F55u, c0,"),
    ("Philox key schedule", MODES, "k0 += 0x9E3779B9u;", "k0 += 0x9E3779B8u;"),
    ("stochastic: wrong random word", MODES, "(double)(w[i % 4] >> 8)",
     "(double)(w[(i + 1) % 4] >> 8)"),
    ("no-ZRE: residual not kept", MODES,
     "  tlc_ref_quartic_encode(q, n, bytes); /* the quartic bytes are the payload */\n"
     "  memcpy(r, resid, n * sizeof(float));",
     "  tlc_ref_quartic_encode(q, n, bytes); /* the quartic bytes are the payload */"),
    ("8-bit: step M/128", INT8, "return M / 127.0f;", "return M / 128.0f;"),
    ("8-bit: round half away", INT8, "v = rintf(acc[i] / D);", "v = roundf(acc[i] / D);"),
    ("8-bit: truncate", INT8, "v = rintf(acc[i] / D);", "v = truncf(acc[i] / D);"),
    ("8-bit: no clamp", INT8, "      if (v > 127.0f) v = 127.0f;\n", ""),
    ("8-bit: clamp at -128", INT8, "if (v < -127.0f) v = -127.0f;",
     "if (v < -128.0f) v = -128.0f;"),
    ("8-bit: residual sign", INT8, "resid[i] = acc[i] - (float)q[i] * D;",
     "resid[i] = acc[i] + (float)q[i] * D;"),
    ("8-bit: residual from the float code", INT8, "resid[i] = acc[i] - (float)q[i] * D;",
     "resid[i] = acc[i] - v * D;"),
    ("8-bit: no error feedback", INT8, "tlc_ref_accumulate(x, r, n, acc); /* error feedback on */",
     "memcpy(acc, x, n * sizeof(float));"),
    ("8-bit: unsigned decode", INT8, "const float v = (float)(int8_t)bytes[i] * D;",
     "const float v = (float)bytes[i] * D;"),
    ("8-bit: decode drops accumulate", INT8, "out[i] = accumulate ? out[i] + v : v;",
     "out[i] = v;"),
    ("8-bit: no length check", INT8, "  if (len != n) return TLC_REF_E_CORRUPT;\n", ""),
]


def build(tmp, name, src):
    c = os.path.join(tmp, name + ".c")
    so = os.path.join(tmp, name + ".so")
    with open(c, "w") as f:
        f.write(src)
    subprocess.run(["gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC",
                    "-shared", "-w", "-I", ORACLE, "-o", so, c, "-lm"], check=True)
    return so


def run_pins(so, pinfile):
    env = dict(os.environ, TLC_REF_LIBRARY=so)
    p = subprocess.run([sys.executable, "-m", "pytest", pinfile, "-x", "-q", "-p",
                        "no:cacheprovider", "-m", "not gpu"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=300)
    return p.returncode, p.stdout[-600:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    original = open(os.path.join(ORACLE, "tlc_ref.c")).read()
    jobs = []
    for i, (name, pinfile, old, new) in enumerate(MUTATIONS):
        assert original.count(old) == 1, f"{name}: the text to change is not unique"
        jobs.append((name, pinfile, build(str(tmp_path), f"m{i}", original.replace(old, new))))
    control = build(str(tmp_path), "control", original)
    with ThreadPoolExecutor(max_workers=4) as ex:
        ctl = [ex.submit(run_pins, control, f) for f in (PINS, INT8, MODES)]
        res = [(name, f, ex.submit(run_pins, so, f)) for name, f, so in jobs]
        for fut in ctl:
            rc, out = fut.result()
            assert rc == 0, "the unchanged oracle must pass its pins:\n" + out
        survived = [(name, f, fut.result()[1]) for name, f, fut in res if fut.result()[0] == 0]
    assert not survived, "mistakes no pin caught: " + "; ".join(f"{n} ({f})" for n, f, _ in survived)
