/*
 * tlc_ref.c -- plain, slow, single-threaded CPU oracle for the 3LC
 * compression path.  TEST INFRASTRUCTURE ONLY (see tlc_ref.h): only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Written from the paper's description, step by step, in its order and
 * notation.  No blocking, fusion or reordering: every stage materialises
 * its full output array before the next stage starts, so a reader can
 * check each function against Sections 3.1-3.3 by eye.
 *
 * Build: gcc -std=c11 -O2 -fno-fast-math -ffp-contract=off -shared -fPIC
 * (x86-64 SSE: fp32 divide is correctly rounded, no flush-to-zero, and
 * rintf uses the default round-to-nearest-even mode).
 */
#include "tlc_ref.h"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* Section 3.3: the byte that quartic encoding produces for five zero
 * values, and the first run code. */
#define REF_ZERO_GROUP 121u
#define REF_RUN_BASE 243u
#define REF_RUN_MIN 2u
#define REF_RUN_MAX 14u

static void* ref_alloc(size_t bytes) {
  void* p = malloc(bytes ? bytes : 1);
  if (!p) {
    fprintf(stderr, "tlc_ref: out of host memory (%zu bytes)\n", bytes);
    abort();
  }
  return p;
}

size_t tlc_ref_quartic_len(size_t n) { return (n + 4) / 5; }

/* Section 3.1, step 1: accumulate the input tensor into the local buffer. */
void tlc_ref_accumulate(const float* x, const float* r, size_t n, float* acc) {
  for (size_t i = 0; i < n; ++i) acc[i] = x[i] + r[i];
}

/* Section 3.1, Eq. 1: M = max(|T_in|) * s with 1 <= s < 2. */
int tlc_ref_absmax_scale(const float* acc, size_t n, float s, float* scale) {
  if (!(s >= 1.0f && s < 2.0f)) return TLC_REF_E_INVALID;
  float A = 0.0f;
  for (size_t i = 0; i < n; ++i) {
    if (!isfinite(acc[i])) return TLC_REF_E_NONFINITE;
    float a = fabsf(acc[i]);
    if (a > A) A = a;
  }
  float M = A * s;
  if (!isfinite(M)) return TLC_REF_E_NONFINITE;
  *scale = M;
  return TLC_REF_OK;
}

/* Section 3.1, Eq. 2 (T_quantized = round(T_in / M), round half to even)
 * and steps a/b (dequantize locally, keep the remaining error). */
void tlc_ref_quantize(const float* acc, size_t n, float M, int8_t* q,
                      float* resid) {
  for (size_t i = 0; i < n; ++i) {
    float v = (M == 0.0f) ? 0.0f : acc[i] / M;
    q[i] = (int8_t)rintf(v);
  }
  if (resid) {
    for (size_t i = 0; i < n; ++i) resid[i] = acc[i] - M * (float)q[i];
  }
}

/* Section 3.1, Eq. 3: T_out = M * T_quantized (optionally added to out). */
void tlc_ref_dequantize(const int8_t* q, size_t n, float M, float* out,
                        int accumulate) {
  for (size_t i = 0; i < n; ++i) {
    float t = M * (float)q[i];
    out[i] = accumulate ? out[i] + t : t; /* dense, every element */
  }
}

/* Section 3.2 encoding steps 1-6. */
void tlc_ref_quartic_encode(const int8_t* q, size_t n, uint8_t* Q) {
  size_t m = tlc_ref_quartic_len(n);
  /* steps 1-3: add 1, cast to u8, flatten (already flat) */
  /* step 4: pad with zeros to a multiple of 5 */
  uint8_t* u = (uint8_t*)ref_alloc(5 * m);
  memset(u, 0, 5 * m);
  for (size_t i = 0; i < n; ++i) u[i] = (uint8_t)(q[i] + 1);
  /* step 5: five partitions p0..p4, each of length m */
  const uint8_t* p0 = u;
  const uint8_t* p1 = u + m;
  const uint8_t* p2 = u + 2 * m;
  const uint8_t* p3 = u + 3 * m;
  const uint8_t* p4 = u + 4 * m;
  /* step 6: a = p0*81 + p1*27 + p2*9 + p3*3 + p4 */
  for (size_t j = 0; j < m; ++j)
    Q[j] = (uint8_t)(p0[j] * 81u + p1[j] * 27u + p2[j] * 9u + p3[j] * 3u +
                     p4[j]);
  free(u);
}

/* Section 3.2 decoding steps 1-4. */
void tlc_ref_quartic_decode(const uint8_t* Q, size_t n, int8_t* q) {
  size_t m = tlc_ref_quartic_len(n);
  static const unsigned pow3[5] = {81u, 27u, 9u, 3u, 1u};
  uint8_t* u = (uint8_t*)ref_alloc(5 * m);
  /* step 1: base-3 digits p_k = (a / 3^(4-k)) mod 3;
   * step 2: concatenate p0..p4 */
  for (size_t k = 0; k < 5; ++k)
    for (size_t j = 0; j < m; ++j)
      u[k * m + j] = (uint8_t)((Q[j] / pow3[k]) % 3u);
  /* step 3: unpad; step 4: subtract 1 */
  for (size_t i = 0; i < n; ++i) q[i] = (int8_t)((int)u[i] - 1);
  free(u);
}

/* Section 3.3: replace each run of k copies of 121 (2 <= k <= 14) by the
 * byte 243 + (k - 2).  Longer runs are cut into chunks of 14 from the left;
 * a chunk of one stays 121. */
size_t tlc_ref_zre_encode(const uint8_t* Q, size_t m, uint8_t* out) {
  size_t o = 0, j = 0;
  while (j < m) {
    if (Q[j] != REF_ZERO_GROUP) {
      out[o++] = Q[j++];
      continue;
    }
    size_t L = 0;
    while (j + L < m && Q[j + L] == REF_ZERO_GROUP) ++L;
    j += L;
    while (L > 0) {
      size_t k = L < REF_RUN_MAX ? L : REF_RUN_MAX;
      out[o++] = (k == 1) ? (uint8_t)REF_ZERO_GROUP
                          : (uint8_t)(REF_RUN_BASE + (k - REF_RUN_MIN));
      L -= k;
    }
  }
  return o;
}

/* Inverse of Section 3.3: a byte below 243 is a quartic byte; a byte
 * b >= 243 stands for (b - 243 + 2) copies of 121. */
int tlc_ref_zre_decode(const uint8_t* C, size_t c, uint8_t* Q, size_t m) {
  size_t pos = 0;
  for (size_t i = 0; i < c; ++i) {
    unsigned b = C[i];
    if (b < REF_RUN_BASE) {
      if (pos >= m) return TLC_REF_E_CORRUPT;
      Q[pos++] = (uint8_t)b;
    } else {
      size_t k = (size_t)(b - REF_RUN_BASE) + REF_RUN_MIN;
      if (pos + k > m) return TLC_REF_E_CORRUPT;
      for (size_t t = 0; t < k; ++t) Q[pos++] = (uint8_t)REF_ZERO_GROUP;
    }
  }
  return pos == m ? TLC_REF_OK : TLC_REF_E_CORRUPT;
}

static int ref_compress(const float* x, float* r, size_t n, float s, uint8_t* bytes,
                        size_t cap, size_t* len, float* scale, int in_place) {
  if (len) *len = 0;
  if (!len || !scale) return TLC_REF_E_INVALID;
  if (!(s >= 1.0f && s < 2.0f)) return TLC_REF_E_INVALID;
  if (n == 0) {
    *scale = 0.0f;
    return TLC_REF_OK;
  }
  if (!x || !r || !bytes) return TLC_REF_E_INVALID;
  size_t m = tlc_ref_quartic_len(n);
  if (cap < m) return TLC_REF_E_CAPACITY;

  float* acc = (float*)ref_alloc(n * sizeof(float));
  tlc_ref_accumulate(x, r, n, acc); /* step 1 */
  float M = 0.0f;
  int st = tlc_ref_absmax_scale(acc, n, s, &M); /* Eq. 1 */
  if (st != TLC_REF_OK) {
    if (in_place) memcpy(r, acc, n * sizeof(float)); /* step 1 already done in the buffer */
    free(acc);
    return st;
  }
  int8_t* q = (int8_t*)ref_alloc(n);
  float* resid = (float*)ref_alloc(n * sizeof(float));
  tlc_ref_quantize(acc, n, M, q, resid); /* Eq. 2, steps a and b */
  uint8_t* Q = (uint8_t*)ref_alloc(m);
  tlc_ref_quartic_encode(q, n, Q); /* Section 3.2 */
  uint8_t* C = (uint8_t*)ref_alloc(m);
  size_t c = tlc_ref_zre_encode(Q, m, C); /* Section 3.3 */

  memcpy(r, resid, n * sizeof(float));
  memcpy(bytes, C, c);
  *len = c;
  *scale = M;
  free(C);
  free(Q);
  free(resid);
  free(q);
  free(acc);
  return TLC_REF_OK;
}

int tlc_ref_compress(const float* x, float* r, size_t n, float s,
                     uint8_t* bytes, size_t cap, size_t* len, float* scale) {
  return ref_compress(x, r, n, s, bytes, cap, len, scale, 0);
}

int tlc_ref_compress_in_place(const float* x, float* r, size_t n, float s,
                              uint8_t* bytes, size_t cap, size_t* len, float* scale) {
  return ref_compress(x, r, n, s, bytes, cap, len, scale, 1);
}

int tlc_ref_decompress(const uint8_t* bytes, size_t len, float scale,
                       size_t n, float* out, int accumulate) {
  if (!isfinite(scale) || scale < 0.0f) return TLC_REF_E_INVALID;
  if (n == 0) return len == 0 ? TLC_REF_OK : TLC_REF_E_CORRUPT;
  if (!out || (len > 0 && !bytes)) return TLC_REF_E_INVALID;
  size_t m = tlc_ref_quartic_len(n);
  uint8_t* Q = (uint8_t*)ref_alloc(m);
  int st = tlc_ref_zre_decode(bytes, len, Q, m);
  if (st != TLC_REF_OK) {
    free(Q);
    return st;
  }
  int8_t* q = (int8_t*)ref_alloc(n);
  tlc_ref_quartic_decode(Q, n, q);
  tlc_ref_dequantize(q, n, scale, out, accumulate);
  free(q);
  free(Q);
  return TLC_REF_OK;
}

/* ---- comparison modes -------------------------------------------------- */

static void ref_mulhilo(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
  uint64_t p = (uint64_t)a * (uint64_t)b;
  *hi = (uint32_t)(p >> 32);
  *lo = (uint32_t)p;
}

void tlc_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { /* key schedule: bump the key between rounds */
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint32_t hi0, lo0, hi1, lo1;
    ref_mulhilo(0xD2511F53u, c0, &hi0, &lo0);
    ref_mulhilo(0xCD9E8D57u, c2, &hi1, &lo1);
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

int tlc_ref_compress_nozre(const float* x, float* r, size_t n, float s, uint8_t* bytes,
                           size_t cap, size_t* len, float* scale, int in_place) {
  if (len) *len = 0;
  if (!len || !scale) return TLC_REF_E_INVALID;
  if (!(s >= 1.0f && s < 2.0f)) return TLC_REF_E_INVALID;
  if (n == 0) {
    *scale = 0.0f;
    return TLC_REF_OK;
  }
  if (!x || !r || !bytes) return TLC_REF_E_INVALID;
  size_t m = tlc_ref_quartic_len(n);
  if (cap < m) return TLC_REF_E_CAPACITY;
  float* acc = (float*)ref_alloc(n * sizeof(float));
  tlc_ref_accumulate(x, r, n, acc);
  float M = 0.0f;
  int st = tlc_ref_absmax_scale(acc, n, s, &M);
  if (st != TLC_REF_OK) {
    if (in_place) memcpy(r, acc, n * sizeof(float)); /* step 1 already done in the buffer */
    free(acc);
    return st;
  }
  int8_t* q = (int8_t*)ref_alloc(n);
  float* resid = (float*)ref_alloc(n * sizeof(float));
  tlc_ref_quantize(acc, n, M, q, resid);
  tlc_ref_quartic_encode(q, n, bytes); /* the quartic bytes are the payload */
  memcpy(r, resid, n * sizeof(float));
  *len = m;
  *scale = M;
  free(resid);
  free(q);
  free(acc);
  return TLC_REF_OK;
}

int tlc_ref_compress_stochastic(const float* x, size_t n, float s, uint64_t seed,
                                uint64_t step, uint8_t* bytes, size_t cap, size_t* len,
                                float* scale) {
  if (len) *len = 0;
  if (!len || !scale) return TLC_REF_E_INVALID;
  if (!(s >= 1.0f && s < 2.0f)) return TLC_REF_E_INVALID;
  if (n == 0) {
    *scale = 0.0f;
    return TLC_REF_OK;
  }
  if (!x || !bytes) return TLC_REF_E_INVALID;
  size_t m = tlc_ref_quartic_len(n);
  if (cap < m) return TLC_REF_E_CAPACITY;
  float M = 0.0f;
  int st = tlc_ref_absmax_scale(x, n, s, &M); /* no error accumulation */
  if (st != TLC_REF_OK) return st;
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  int8_t* q = (int8_t*)ref_alloc(n);
  for (size_t i = 0; i < n; ++i) {
    const uint64_t blk = i / 4;
    const uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)step,
                             (uint32_t)(step >> 32)};
    uint32_t w[4];
    tlc_ref_philox4x32_10(ctr, key, w);
    const double u = (double)(w[i % 4] >> 8) / 16777216.0; /* uniform on [0, 1), 24 bits */
    const double a = fabs((double)x[i]);
    /* keep with probability |x|/M: u < |x|/M, i.e. u*M < |x| (exact in double) */
    const int keep = (M > 0.0f) && (u * (double)M < a);
    q[i] = keep ? (x[i] > 0.0f ? 1 : -1) : 0;
  }
  tlc_ref_quartic_encode(q, n, bytes);
  *len = m;
  *scale = M;
  free(q);
  return TLC_REF_OK;
}

/* ---- 8-bit integer comparator (Section 5.1, "8-bit int") ----------------
 * The paper fixes the code set (255 levels, -127..127, -128 unused) and
 * nothing else.  Reading: M as in Eq. 1, one step D = fl(M / 127) per
 * tensor, q = rint(fl(acc / D)) (round half to even) clamped to
 * [-127, 127], dequantized value fl(q * D).  The clamp only acts when D is
 * subnormal (its rounding can leave M / D above 127.5); D == 0 (M below
 * 127 * 2^-150) quantizes everything to 0. */
float tlc_ref_int8_step(float M) { return M / 127.0f; }

void tlc_ref_int8_quantize(const float* acc, size_t n, float M, int8_t* q, float* resid) {
  const float D = tlc_ref_int8_step(M);
  for (size_t i = 0; i < n; ++i) {
    float v = 0.0f;
    if (D > 0.0f) {
      v = rintf(acc[i] / D);
      if (v > 127.0f) v = 127.0f;
      if (v < -127.0f) v = -127.0f;
    }
    q[i] = (int8_t)v;
    if (resid) resid[i] = acc[i] - (float)q[i] * D;
  }
}

int tlc_ref_compress_int8(const float* x, float* r, size_t n, float s, uint8_t* bytes,
                          size_t cap, size_t* len, float* scale, int in_place) {
  if (len) *len = 0;
  if (!len || !scale) return TLC_REF_E_INVALID;
  if (!(s >= 1.0f && s < 2.0f)) return TLC_REF_E_INVALID;
  if (n == 0) {
    *scale = 0.0f;
    return TLC_REF_OK;
  }
  if (!x || !bytes) return TLC_REF_E_INVALID;
  if (cap < n) return TLC_REF_E_CAPACITY;
  float* acc = (float*)ref_alloc(n * sizeof(float));
  if (r)
    tlc_ref_accumulate(x, r, n, acc); /* error feedback on */
  else
    memcpy(acc, x, n * sizeof(float));
  float M = 0.0f;
  int st = tlc_ref_absmax_scale(acc, n, s, &M);
  if (st != TLC_REF_OK) {
    if (r && in_place) memcpy(r, acc, n * sizeof(float)); /* step 1 already done */
    free(acc);
    return st;
  }
  int8_t* q = (int8_t*)ref_alloc(n);
  float* resid = r ? (float*)ref_alloc(n * sizeof(float)) : NULL;
  tlc_ref_int8_quantize(acc, n, M, q, resid);
  for (size_t i = 0; i < n; ++i) bytes[i] = (uint8_t)q[i]; /* two's complement */
  if (r) memcpy(r, resid, n * sizeof(float));
  *len = n;
  *scale = M;
  free(resid);
  free(q);
  free(acc);
  return TLC_REF_OK;
}

int tlc_ref_decompress_int8(const uint8_t* bytes, size_t len, float scale, size_t n,
                            float* out, int accumulate) {
  if (!(scale >= 0.0f) || !isfinite(scale)) return TLC_REF_E_INVALID;
  if (n == 0) return len == 0 ? TLC_REF_OK : TLC_REF_E_CORRUPT;
  if (!bytes || !out) return TLC_REF_E_INVALID;
  if (len != n) return TLC_REF_E_CORRUPT;
  const float D = tlc_ref_int8_step(scale);
  for (size_t i = 0; i < n; ++i) {
    const float v = (float)(int8_t)bytes[i] * D;
    out[i] = accumulate ? out[i] + v : v; /* dense, every element */
  }
  return TLC_REF_OK;
}
