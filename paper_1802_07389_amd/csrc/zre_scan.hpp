// zre_scan.hpp -- associative summary of a byte segment for parallel
// zero-run encoding (Section 3.3).
//
// Zero-run encoding cuts every run of L bytes equal to 121 into
// floor(L/14) full chunks (code 255) and a remainder chunk (code
// 243 + rho - 2 for rho >= 2, or 121 for rho == 1).  Where a chunk's code
// lands depends on how far into its run a byte is, and runs may cross any
// tile boundary, so a per-tile emit count cannot be computed without the
// prefix.  This header instead summarises a segment by
//
//   all : the segment is entirely 121 (or empty)
//   ld  : (length of the leading 121 run) mod 14     (== rem when all)
//   tr  : (length of the trailing 121 run) mod 14    (== rem when all)
//   cnt : output bytes the segment is certain to produce on its own:
//         floor(lead/14) + non-121 bytes + ceil(L/14) for every run closed
//         on both sides inside the segment + floor(trail/14);
//         for an all-121 segment of length len, floor(len/14)
//
// and combines two adjacent segments with an associative operator, so tile
// prefixes can be found with a decoupled look-back.  Emission convention
// used by the kernels: a full chunk's 255 is written at its 14th byte; the
// remainder code of a run is written just before the non-121 byte that
// closes it, or at the very end of the stream.
//
// Packed form (64 bits): cnt in bits 0..31, all in bit 32, ld in bits
// 33..36, tr in bits 37..40.
#pragma once

#include <stdint.h>

#ifndef TLC_HD
#if defined(__HIPCC__)
#define TLC_HD __host__ __device__ __forceinline__
#else
#define TLC_HD inline
#endif
#endif

namespace tlc {

constexpr uint32_t kZeroGroup = 121u;  // five zero values (Section 3.3)
constexpr uint32_t kRunBase = 243u;    // code of a run of two
constexpr uint32_t kRunMax = 14u;      // longest run one code covers
constexpr uint32_t kFullChunk = 255u;  // code of a run of fourteen

struct RunSum {
  uint64_t v;
};

TLC_HD uint32_t rs_cnt(RunSum a) { return (uint32_t)a.v; }
TLC_HD uint32_t rs_all(RunSum a) { return (uint32_t)(a.v >> 32) & 1u; }
TLC_HD uint32_t rs_ld(RunSum a) { return (uint32_t)(a.v >> 33) & 15u; }
TLC_HD uint32_t rs_tr(RunSum a) { return (uint32_t)(a.v >> 37) & 15u; }

TLC_HD RunSum rs_make(uint32_t all, uint32_t ld, uint32_t tr, uint32_t cnt) {
  RunSum r;
  r.v = (uint64_t)cnt | ((uint64_t)all << 32) | ((uint64_t)ld << 33) |
        ((uint64_t)tr << 37);
  return r;
}

// Empty segment: the identity of rs_combine.
TLC_HD RunSum rs_identity() { return rs_make(1u, 0u, 0u, 0u); }

// Summary of one byte.
TLC_HD RunSum rs_byte(uint32_t b) {
  return b == kZeroGroup ? rs_make(1u, 1u, 1u, 0u) : rs_make(0u, 0u, 0u, 1u);
}

// Run lengths are kept mod 14, so the sum s of two of them is at most 26:
// s / 14 is (s >= 14), s mod 14 is s or s - 14, and ceil(s / 14) is
// (s > 0) + (s > 14).
TLC_HD uint32_t rs_div14(uint32_t s) { return s >= kRunMax ? 1u : 0u; }
TLC_HD uint32_t rs_mod14(uint32_t s) { return s >= kRunMax ? s - kRunMax : s; }
TLC_HD uint32_t rs_ceil14(uint32_t s) { return (s != 0u ? 1u : 0u) + (s > kRunMax ? 1u : 0u); }

// Summary of segment a followed by segment b.
TLC_HD RunSum rs_combine(RunSum a, RunSum b) {
  uint32_t aall = rs_all(a), ball = rs_all(b);
  uint32_t cnt = rs_cnt(a) + rs_cnt(b);
  if (aall & ball) {
    uint32_t s = rs_ld(a) + rs_ld(b);
    return rs_make(1u, rs_mod14(s), rs_mod14(s), cnt + rs_div14(s));
  }
  if (aall) {  // the run at the end of a continues into b's leading run
    uint32_t s = rs_ld(a) + rs_ld(b);
    return rs_make(0u, rs_mod14(s), rs_tr(b), cnt + rs_div14(s));
  }
  if (ball) {  // b extends a's trailing run
    uint32_t s = rs_tr(a) + rs_ld(b);
    return rs_make(0u, rs_ld(a), rs_mod14(s), cnt + rs_div14(s));
  }
  // a's trailing run and b's leading run join into one run closed on both
  // sides: its remainder costs one more code if non-empty.
  uint32_t s = rs_tr(a) + rs_ld(b);
  return rs_make(0u, rs_ld(a), rs_tr(b), cnt + rs_ceil14(s));
}

// Bytes already written by everything before a point whose prefix (from
// the start of the stream) has summary p.  The leading run of the stream
// is closed by the stream start, so its remainder code has been written
// once a non-121 byte follows it.
TLC_HD uint32_t rs_emitted(RunSum p) {
  return rs_cnt(p) + ((!rs_all(p) && rs_ld(p) != 0u) ? 1u : 0u);
}

// Length of the open 121 run (mod 14) at the end of a prefix.
TLC_HD uint32_t rs_phase(RunSum p) { return rs_tr(p); }

// Total encoded length of a whole stream with summary t.
TLC_HD uint32_t rs_total(RunSum t) {
  return rs_emitted(t) + (rs_tr(t) != 0u ? 1u : 0u);
}

// Code of a run remainder of rho in [1, 14] bytes.
TLC_HD uint32_t rs_code(uint32_t rho) {
  return rho == 1u ? kZeroGroup : kRunBase + rho - 2u;
}

}  // namespace tlc

namespace tlc {

// Encode one quartic byte x arriving while the open 121 run has phi (mod
// 14) bytes; hands output bytes to put(byte) and returns the new phase.
template <class Put>
TLC_HD uint32_t rs_step(uint32_t x, uint32_t phi, Put&& put) {
  if (x == kZeroGroup) {
    if (++phi == kRunMax) {
      put(kFullChunk);
      phi = 0u;
    }
  } else {
    if (phi != 0u) put(rs_code(phi));
    phi = 0u;
    put(x);
  }
  return phi;
}

// Closed forms for a segment of len bytes that are all 121 (the common
// case: most groups of five values quantize to zero).  Its summary is
// (all, len mod 14, len mod 14, len / 14); encoding it after phase phi
// writes one 255 for every 14th byte of the grown run.
TLC_HD RunSum rs_zero_run(uint32_t len) {
  return rs_make(1u, len % kRunMax, len % kRunMax, len / kRunMax);
}

template <class Put>
TLC_HD uint32_t rs_zero_walk(uint32_t len, uint32_t phi, Put&& put) {
  const uint32_t t = phi + len;
  for (uint32_t e = 0; e < t / kRunMax; ++e) put(kFullChunk);
  return t % kRunMax;
}

// Closed forms for a short segment of len <= 16 bytes given by the mask nz
// of its non-121 bytes (bit i: byte i; no bits at or above len).  A run
// between two non-121 bytes is then at most 14 bytes long and costs
// exactly one code, so the summary needs only the leading and trailing run
// lengths, the count of non-121 bytes and the count of gaps between them
// (maximal runs of set bits, less one).  rs_mask_walk encodes the segment
// after phase phi, visiting only the non-121 bytes (byte(i) returns byte
// i), and returns the new phase.
TLC_HD RunSum rs_mask_summary(uint32_t nz, uint32_t len) {
  if (nz == 0u) return rs_zero_run(len);
  const uint32_t lead = (uint32_t)__builtin_ctz(nz);
  const uint32_t trail = len - 1u - (31u - (uint32_t)__builtin_clz(nz));
  const uint32_t runs = (uint32_t)__builtin_popcount(nz & ~(nz << 1));
  const uint32_t cnt =
      lead / kRunMax + (uint32_t)__builtin_popcount(nz) + (runs - 1u) + trail / kRunMax;
  return rs_make(0u, lead % kRunMax, trail % kRunMax, cnt);
}

template <class Byte, class Put>
TLC_HD uint32_t rs_mask_walk(uint32_t nz, uint32_t len, uint32_t phi, Byte&& byte, Put&& put) {
  uint32_t pos = 0u;
  while (nz) {
    const uint32_t p = (uint32_t)__builtin_ctz(nz);
    nz &= nz - 1u;
    phi = rs_zero_walk(p - pos, phi, put);
    if (phi != 0u) put(rs_code(phi));
    phi = 0u;
    put(byte(p));
    pos = p + 1u;
  }
  return rs_zero_walk(len - pos, phi, put);
}

// A segment that starts at a non-121 byte (phase 0) in terms of the gaps
// between its non-121 bytes: a gap of g bytes of 121 costs floor(g/14)
// codes 255 and, if g mod 14 != 0, one remainder code; each non-121 byte
// costs itself.  For the non-121 bytes of one thread (mask nz, bit
// kStep * i for position lo + i; kStep 2 is the spread form that 2-bit
// trits give directly) after the segment's previous non-121 byte at prev
// (prev < 0: none; the thread's first byte then opens the segment),
// rs_gaps_len counts the bytes they emit with their gaps and rs_gaps_emit
// emits them, handing each gap's k codes 255 to fill(k) and every other
// byte to put (a caller whose output already holds 255 everywhere only
// advances its offset in fill); the trailing run after the segment's last
// non-121 byte emits its floor(g/14) codes 255 separately.
TLC_HD uint32_t rs_gap_len(uint32_t g) { return g / kRunMax + (g % kRunMax != 0u ? 1u : 0u); }

// With nz covering at most 16 bytes, a gap between two of the thread's own
// bytes is at most 14 bytes and costs exactly one code if non-empty:
// besides the gap from prev, the count is one per non-121 byte plus one per
// maximal run of marked bytes after the first.
template <uint32_t kStep = 1>
TLC_HD uint32_t rs_gaps_len(uint32_t nz, uint32_t lo, int prev) {
  static_assert(kStep == 1 || kStep == 2, "one or two mask bits per byte");
  if (nz == 0u) return 0u;
  const uint32_t first = lo + (uint32_t)__builtin_ctz(nz) / kStep;
  const uint32_t runs = (uint32_t)__builtin_popcount(nz & ~(nz << kStep));
  return (prev >= 0 ? rs_gap_len(first - (uint32_t)prev - 1u) : 0u) +
         (uint32_t)__builtin_popcount(nz) + runs - 1u;
}

template <uint32_t kStep = 1, class Byte, class Put, class Fill>
TLC_HD void rs_gaps_emit(uint32_t nz, uint32_t lo, int prev, Byte&& byte, Put&& put,
                         Fill&& fill) {
  while (nz) {
    const uint32_t i = (uint32_t)__builtin_ctz(nz) / kStep;
    const uint32_t p = lo + i;
    nz &= nz - 1u;
    if (prev >= 0) {
      const uint32_t g = p - (uint32_t)prev - 1u;
      fill(g / kRunMax);
      if (g % kRunMax != 0u) put(rs_code(g % kRunMax));
    }
    put(byte(i));
    prev = (int)p;
  }
}

// rs_step over `count` bytes.  The caller writes the final remainder code
// (rs_code) if the stream ends with a non-zero phase.
template <class Put>
TLC_HD uint32_t rs_walk(const uint8_t* b, uint32_t count, uint32_t phi,
                        Put&& put) {
  for (uint32_t i = 0; i < count; ++i) phi = rs_step(b[i], phi, put);
  return phi;
}

}  // namespace tlc
