/*
 * tlc_ref.h -- plain, slow, single-threaded CPU oracle for the 3LC
 * compression path (3-value quantization with sparsity multiplication,
 * quartic encoding, zero-run encoding; paper Sections 3.1-3.3).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include,
 * link or call this file; only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark use it.  It shares no code, header,
 * table or constant with the HIP library.
 *
 * All pointers are HOST pointers.  Status codes use the same numeric
 * values as the product ABI (they are part of the contract), but are
 * defined here independently.
 *
 * Every function follows the paper's step order with fp32 arithmetic:
 *   acc = x + r                       (Section 3.1, error accumulation step 1)
 *   M   = max|acc| * s                (Section 3.1, Eq. 1)
 *   q   = round(acc / M)              (Section 3.1, Eq. 2; round half to even)
 *   r   = acc - M*q                   (Section 3.1, steps a and b)
 *   Q   = quartic encoding of q+1     (Section 3.2)
 *   C   = zero-run encoding of Q      (Section 3.3)
 * and the reverse for decoding, with out = M*q (Eq. 3) or out += M*q.
 */
#ifndef TLC_REF_H
#define TLC_REF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TLC_REF_OK            0
#define TLC_REF_E_INVALID    (-1)
#define TLC_REF_E_CAPACITY   (-2)
#define TLC_REF_E_NONFINITE  (-3)
#define TLC_REF_E_CORRUPT    (-4)

/* Number of quartic bytes for n values: ceil(n/5) (Section 3.2, padding
 * step).  Also the largest possible zero-run encoded length. */
size_t tlc_ref_quartic_len(size_t n);

/* Step 1 of error accumulation: acc[i] = x[i] + r[i] in fp32. */
void tlc_ref_accumulate(const float* x, const float* r, size_t n, float* acc);

/* Eq. 1: *scale = max_i |acc[i]| * s, in fp32.  Returns
 * TLC_REF_E_INVALID if s is outside [1, 2) or NaN, TLC_REF_E_NONFINITE if
 * any acc[i] is NaN or infinite or the product overflows.  n = 0 gives 0. */
int tlc_ref_absmax_scale(const float* acc, size_t n, float s, float* scale);

/* Eq. 2 and steps a/b: q[i] = rint(acc[i] / M) (0 when M == 0) and
 * resid[i] = acc[i] - M*q[i].  resid may be NULL. */
void tlc_ref_quantize(const float* acc, size_t n, float M, int8_t* q,
                      float* resid);

/* Eq. 3: out[i] = M*q[i], or out[i] = out[i] + M*q[i] when accumulate,
 * densely for every i (so -0.0 + M*0 gives +0.0). */
void tlc_ref_dequantize(const int8_t* q, size_t n, float M, float* out,
                        int accumulate);

/* Section 3.2 encoding: Q has ceil(n/5) bytes.  q values must be in
 * {-1, 0, 1}. */
void tlc_ref_quartic_encode(const int8_t* q, size_t n, uint8_t* Q);

/* Section 3.2 decoding: recovers q[0..n) from Q[0..ceil(n/5)). */
void tlc_ref_quartic_decode(const uint8_t* Q, size_t n, int8_t* q);

/* Section 3.3 encoding of Q[0..m) into out (capacity >= m).  Returns the
 * encoded length. */
size_t tlc_ref_zre_encode(const uint8_t* Q, size_t m, uint8_t* out);

/* Inverse of Section 3.3: expands C[0..c) into Q[0..m).  Returns
 * TLC_REF_E_CORRUPT if the expansion is not exactly m bytes long. */
int tlc_ref_zre_decode(const uint8_t* C, size_t c, uint8_t* Q, size_t m);

/* Whole encoder.  x is read only, r is the error-accumulation buffer
 * (in/out), bytes receives *len bytes (cap must be >= ceil(n/5)), *scale
 * receives M.  On any error r and bytes are left unchanged and *len = 0
 * (NaN/Inf: no meaningful quantization exists). */
int tlc_ref_compress(const float* x, float* r, size_t n, float s,
                     uint8_t* bytes, size_t cap, size_t* len, float* scale);

/* As tlc_ref_compress, except that step 1 (Section 3.1, Fig. 3) is taken as
 * accumulating x into the buffer itself before Eq. 1 is known: on
 * TLC_REF_E_NONFINITE r holds acc = x + r (argument errors still leave it
 * unchanged).  Every other result is identical. */
int tlc_ref_compress_in_place(const float* x, float* r, size_t n, float s,
                              uint8_t* bytes, size_t cap, size_t* len, float* scale);

/* Whole decoder.  On any error out is left unchanged. */
int tlc_ref_decompress(const uint8_t* bytes, size_t len, float scale,
                       size_t n, float* out, int accumulate);

/* ---- comparison modes -------------------------------------------------- */

/* Philox4x32-10 counter-based generator (Salmon, Moraes, Dror and Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC 2011): ten rounds of
 * two 32x32->64 multiplications with multipliers 0xD2511F53, 0xCD9E8D57 and
 * a Weyl key schedule 0x9E3779B9, 0xBB67AE85. */
void tlc_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Quantization + quartic encoding without zero-run encoding (Table 2, row
 * "No ZRE"): bytes receives the ceil(n/5) quartic bytes, error feedback as in
 * tlc_ref_compress (in_place != 0: as in tlc_ref_compress_in_place). */
int tlc_ref_compress_nozre(const float* x, float* r, size_t n, float s, uint8_t* bytes,
                           size_t cap, size_t* len, float* scale, int in_place);

/* Stochastic 3-value quantization + quartic encoding, no error feedback
 * (the "Stoch 3-value + QE" comparator of Section 5.1, described in Section
 * 3.1): M = max|x| * s; element i keeps sign(x_i) with probability |x_i|/M,
 * decided by u_i < |x_i|/M with u_i = (w >> 8) * 2^-24, w the 32-bit Philox
 * word (i mod 4) of counter (i/4 low, i/4 high, step low, step high) and key
 * (seed low, seed high).  bytes receives ceil(n/5) quartic bytes. */
int tlc_ref_compress_stochastic(const float* x, size_t n, float s, uint64_t seed,
                                uint64_t step, uint8_t* bytes, size_t cap, size_t* len,
                                float* scale);

/* 8-bit integer quantization (the "8-bit int" comparator of Section 5.1):
 * 255 codes -127..127.  Step D = fl(M / 127) with M = fl(max|acc| * s);
 * q_i = rint(fl(acc_i / D)) clamped to [-127, 127] (q = 0 when D == 0);
 * residual fl(acc_i - fl(q_i * D)).  tlc_ref_int8_quantize writes resid
 * only when it is not NULL. */
float tlc_ref_int8_step(float M);
void tlc_ref_int8_quantize(const float* acc, size_t n, float M, int8_t* q, float* resid);

/* Encoder: acc = x + r when r != NULL (error feedback, r updated), else acc
 * = x.  bytes receives the n codes as two's-complement int8 (cap >= n).
 * Errors as for tlc_ref_compress (in_place != 0: on TLC_REF_E_NONFINITE a
 * non-NULL r holds acc). */
int tlc_ref_compress_int8(const float* x, float* r, size_t n, float s, uint8_t* bytes,
                          size_t cap, size_t* len, float* scale, int in_place);

/* Decoder: out_i = fl(q_i * D) or fl(out_i + fl(q_i * D)), densely, D =
 * fl(scale / 127), every int8 code accepted; len != n is
 * TLC_REF_E_CORRUPT with out unchanged. */
int tlc_ref_decompress_int8(const uint8_t* bytes, size_t len, float scale, size_t n,
                            float* out, int accumulate);

#ifdef __cplusplus
}
#endif

#endif /* TLC_REF_H */
