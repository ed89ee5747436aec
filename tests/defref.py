"""Second, independently written reference of the 3LC path in numpy.

Used only to cross-check the C oracle on small and medium inputs.  It is
written from the paper's definitions with whole-array numpy operations and
itertools, so it shares neither structure nor code with ``oracle/tlc_ref.c``:

* Section 3.1: acc = x + r; M = max|acc| * s; q = round-half-even(acc / M);
  residual = acc - M q (numpy float32 arithmetic is IEEE binary32).
* Section 3.2: the trits t = q + 1 are zero-padded to 5m values, viewed as a
  5 x m array whose rows are the partitions p0..p4, and combined with
  weights 81, 27, 9, 3, 1.
* Section 3.3: runs of 121 are found with itertools.groupby and replaced by
  ceil(L/14) codes (full chunks of 14 first, remainder last).
"""
import itertools

import numpy as np

F32 = np.float32
WEIGHTS = np.array([81, 27, 9, 3, 1], dtype=np.int64)


def quantize(x, r, s):
    acc = (x.astype(F32) + r.astype(F32)).astype(F32)
    A = np.max(np.abs(acc)) if acc.size else F32(0)
    M = F32(F32(A) * F32(s))
    if M == 0:
        q = np.zeros(acc.size, dtype=np.int8)
    else:
        q = np.rint(acc / M).astype(np.int8)
    resid = (acc - M * q.astype(F32)).astype(F32)
    return acc, M, q, resid


def quartic(q):
    n = q.size
    m = -(-n // 5)
    t = np.zeros(5 * m, dtype=np.int64)
    t[:n] = q.astype(np.int64) + 1
    return (WEIGHTS @ t.reshape(5, m)).astype(np.uint8)


def unquartic(Q, n):
    m = Q.size
    digits = (Q.astype(np.int64)[None, :] // WEIGHTS[:, None]) % 3
    return (digits.reshape(5 * m)[:n] - 1).astype(np.int8)


def zre(Q):
    out = []
    for byte, grp in itertools.groupby(Q.tolist()):
        L = sum(1 for _ in grp)
        if byte != 121:
            out.extend([byte] * L)
            continue
        full, rem = divmod(L, 14)
        out.extend([255] * full)
        if rem == 1:
            out.append(121)
        elif rem >= 2:
            out.append(243 + rem - 2)
    return np.array(out, dtype=np.uint8)


def unzre(C):
    out = []
    for b in C.tolist():
        if b >= 243:
            out.extend([121] * (b - 241))
        else:
            out.append(b)
    return np.array(out, dtype=np.uint8)


def compress(x, r, s):
    """Return (bytes, M, new residual)."""
    _, M, q, resid = quantize(x, r, s)
    return zre(quartic(q)), M, resid


def decompress(C, M, n, out=None):
    q = unquartic(unzre(C), n)
    t = (F32(M) * q.astype(F32)).astype(F32)
    return t if out is None else (out + t).astype(F32)


def runs(seq):
    """Lengths of maximal runs of 121 in a byte sequence."""
    return [sum(1 for _ in g) for b, g in itertools.groupby(seq) if b == 121]
