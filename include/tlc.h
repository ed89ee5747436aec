/*
 * tlc.h -- C ABI of the MI355X (gfx950) 3LC compression library.
 *
 * 3LC compresses one fp32 state-change tensor (a gradient push or a model
 * delta pull) per call, as described in the paper "3LC: Lightweight and
 * Effective Traffic Compression for Distributed Machine Learning":
 *
 *   encode (Section 3.1, Fig. 3; Sections 3.2 and 3.3)
 *     acc = tensor + residual                        error accumulation
 *     M   = max|acc| * s,  1 <= s < 2                Eq. 1
 *     q   = round(acc / M) in {-1, 0, 1}             Eq. 2 (half to even)
 *     residual = acc - M*q                           steps a and b
 *     Q   = quartic encoding of q + 1                Section 3.2
 *     C   = zero-run encoding of Q                   Section 3.3
 *   decode
 *     Q = zero-run expansion of C; q = quartic decoding of Q;
 *     out = M*q (Eq. 3)  or  out += M*q (aggregation at a server).
 *
 * The payload of one call is the byte string C plus the fp32 scalar M.
 *
 * Layout conventions (bit-exact contract):
 *   - m = ceil(n/5) quartic bytes.  The n values are padded with trit 0 to
 *     5m and split into five CONTIGUOUS partitions p_k = [k*m, (k+1)*m);
 *     byte j = 81*t(j) + 27*t(m+j) + 9*t(2m+j) + 3*t(3m+j) + t(4m+j).
 *   - A run of L bytes equal to 121 becomes floor(L/14) bytes 255, then
 *     243 + (L mod 14) - 2 if L mod 14 >= 2, or 121 if L mod 14 == 1.
 *   - Division is IEEE fp32 and rounding is half-to-even, so results are
 *     bit-identical to a sequential fp32 implementation.
 *
 * Memory: every tensor / byte pointer passed to tlc_compress and
 * tlc_decompress is DEVICE memory owned by the caller (for example a torch
 * tensor's data_ptr()).  The context owns its device workspace and a small
 * pinned host buffer; nothing is allocated per call.
 *
 * Streams: a context is bound to one HIP stream (passed as void*; NULL is
 * the default stream).  All work of a context is ordered on that stream.  A
 * context must not be used by two host threads at once.
 *
 * Errors: functions return TLC_OK (0) or a negative TLC_E_* code; no C++
 * exception crosses this boundary.  tlc_last_error_string() describes the
 * most recent failure of the calling thread.
 */
#ifndef TLC_H
#define TLC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TLC_OK 0
#define TLC_E_INVALID (-1)   /* bad argument: NULL pointer, s not in [1,2), n > max_n, scale not finite */
#define TLC_E_CAPACITY (-2)  /* bytes_cap < tlc_max_compressed_bytes(n) */
#define TLC_E_NONFINITE (-3) /* NaN/Inf in tensor+residual, or max*s overflows */
#define TLC_E_CORRUPT (-4)   /* compressed stream does not expand to ceil(n/5) bytes */
#define TLC_E_DEVICE (-5)    /* HIP runtime error, or the context is unusable */

/* Largest number of values one call accepts, summed over a batch (the
 * quartic byte counts must fit the 30-bit counters of the zero-run scans). */
#define TLC_MAX_N ((size_t)4294967295u)

/* Largest number of tensors (or streams) one batched call accepts. */
#define TLC_MAX_TENSORS 65536

typedef struct tlc_ctx tlc_ctx;

/* Upper bound of the compressed length for n values: ceil(n/5).  Zero-run
 * encoding (Section 3.3) never lengthens the quartic byte string. */
size_t tlc_max_compressed_bytes(size_t n);

/* Create a context for tensors of up to max_n values (1 <= max_n <=
 * TLC_MAX_N) whose work is issued on `hip_stream` (a hipStream_t, or NULL).
 * Allocates one device workspace of about 0.81 * max_n bytes (218 MB for
 * max_n = 2^28): partial maxima, look-back status words, the decoder's
 * start index, and for the single-tensor encoder per-tile slots, records
 * and residual lists and two bytes per four values (bounds or trits of the
 * max pass).  No later call allocates device memory.  On success
 * *ctx receives the context; on failure *ctx is NULL.  Same as
 * tlc_ctx_create_batch(ctx, max_n, 1, hip_stream). */
int tlc_ctx_create(tlc_ctx** ctx, size_t max_n, void* hip_stream);

/* Create a context for batched calls: at most max_tensors tensors (or
 * streams) per call, 1 <= max_tensors <= TLC_MAX_TENSORS, and at most max_n
 * values per call summed over the batch (for tlc_decompress_sum: count * n).
 * Each tensor of a batch is still compressed on its own, with its own scale
 * and error buffer (Section 3: one compression context per tensor); the
 * batch only shares launches and the host synchronisation. */
int tlc_ctx_create_batch(tlc_ctx** ctx, size_t max_n, size_t max_tensors,
                         void* hip_stream);

/* Wait for the context's outstanding work and free it.  NULL is a no-op. */
int tlc_ctx_destroy(tlc_ctx* ctx);

/* Encode one tensor (Sections 3.1-3.3).
 *   tensor    device fp32[n], read only (the new state change).
 *   residual  device fp32[n], in/out: the error-accumulation buffer
 *             (Section 3.1, Fig. 3); on success it holds acc - M*q with
 *             acc = tensor + residual.  Must not overlap tensor.
 *   n         value count, 0 <= n <= max_n of the context.
 *   s         sparsity multiplier, 1 <= s < 2.
 *   bytes     device uint8[bytes_cap] receiving the zero-run encoded stream.
 *   bytes_cap must be >= tlc_max_compressed_bytes(n).
 *   bytes_len host out: stream length (0 on error).
 *   scale     host out: M (0 when n == 0).
 * Synchronous: returns after the stream length is known, which the encode
 * hands to the host a little before its last kernels end: the stream bytes
 * and the residual are complete in the order of the context's stream (work
 * issued there afterwards sees them; the host or another stream waits for
 * that stream, e.g. with tlc_sync, before reading them).  On
 * TLC_E_NONFINITE the residual and the bytes are left unchanged (with
 * TLC_OPT_IN_PLACE_FEEDBACK the residual holds acc instead). */
int tlc_compress(tlc_ctx* ctx, const float* tensor, float* residual, size_t n,
                 float s, uint8_t* bytes, size_t bytes_cap, size_t* bytes_len,
                 float* scale);

/* Decode one stream (inverse of Section 3.3, Section 3.2 decoding, Eq. 3).
 *   bytes       device uint8[bytes_len] from tlc_compress.
 *   scale       M from tlc_compress: finite and >= 0.
 *   n           value count of the encoded tensor, <= max_n.
 *   out         device fp32[n]: out = M*q (accumulate == 0) or
 *               out = out + M*q (accumulate != 0), for every element
 *               (-0.0 + M*0 gives +0.0; a value whose sum has the bits it
 *               already holds is not stored again).  Must not overlap
 *               bytes (TLC_E_INVALID).
 * Asynchronous on the context's stream; returns only errors detectable on
 * the host.  If the stream does not expand to exactly ceil(n/5) bytes, out
 * is left unchanged and the next tlc_sync() returns TLC_E_CORRUPT. */
int tlc_decompress(tlc_ctx* ctx, const uint8_t* bytes, size_t bytes_len,
                   float scale, size_t n, float* out, int accumulate);

/* ---- comparison encodings (decoded by tlc_decompress like any stream) --- */

#define TLC_MODE_3LC 0        /* Sections 3.1-3.3: same as tlc_compress */
#define TLC_MODE_NO_ZRE 1     /* 3-value quantization with error feedback and
                                 quartic encoding, no zero-run encoding
                                 (Table 2, row "No ZRE"): ceil(n/5) bytes */
#define TLC_MODE_STOCHASTIC 2 /* stochastic 3-value quantization + quartic
                                 encoding, no error feedback (the "Stoch
                                 3-value + QE" design of Section 5.1, TernGrad
                                 without clipping; Section 3.1) */
#define TLC_MODE_INT8 3       /* 8-bit integer quantization, codes -127..127
                                 (the "8-bit int" design of Section 5.1): n
                                 bytes, decoded by tlc_decompress_ex */

/* Encode with a comparison mode.  TLC_MODE_3LC forwards to tlc_compress
 * (seed and step unused).  TLC_MODE_NO_ZRE: as tlc_compress but the payload
 * is the ceil(n/5) quartic bytes.  TLC_MODE_STOCHASTIC: M = max|tensor| * s;
 * value i becomes sign(tensor[i]) with probability |tensor[i]|/M, else 0,
 * decided by u < |tensor[i]|/M with u = (w >> 8) * 2^-24 and w word (i mod
 * 4) of Philox4x32-10 (Salmon et al., SC 2011) at counter (i/4 low, i/4
 * high, step low, step high) and key (seed low, seed high); residual is not
 * used (may be NULL).  Both return *bytes_len = ceil(n/5); the bytes are
 * 0..242, so tlc_decompress decodes them unchanged.
 * TLC_MODE_INT8: acc = tensor + residual (error feedback, residual
 * rewritten) or, with residual == NULL, acc = tensor; M = max|acc| * s
 * (Eq. 1), step D = fl(M / 127); byte i is the two's-complement int8 code
 * rint(fl(acc_i / D)) clamped to [-127, 127] (0 when D == 0) and the
 * residual becomes fl(acc_i - fl(code * D)).  bytes_cap >= n; *bytes_len =
 * n.  Synchronous; on TLC_E_NONFINITE the residual and bytes are unchanged
 * (with TLC_OPT_IN_PLACE_FEEDBACK a non-NULL residual holds acc), as for
 * tlc_compress; the same holds for TLC_MODE_NO_ZRE. */
int tlc_compress_ex(tlc_ctx* ctx, int mode, const float* tensor, float* residual, size_t n,
                    float s, uint64_t seed, uint64_t step, uint8_t* bytes, size_t bytes_cap,
                    size_t* bytes_len, float* scale);

/* Decode a stream of any mode.  TLC_MODE_3LC, TLC_MODE_NO_ZRE and
 * TLC_MODE_STOCHASTIC forward to tlc_decompress.  TLC_MODE_INT8: bytes is
 * device uint8[n] of int8 codes (every code accepted), out = fl(code * D)
 * or out + fl(code * D) with D = fl(scale / 127); bytes_len != n returns
 * TLC_E_CORRUPT at once with out unchanged.  Asynchronous on the context's
 * stream. */
int tlc_decompress_ex(tlc_ctx* ctx, int mode, const uint8_t* bytes, size_t bytes_len,
                      float scale, size_t n, float* out, int accumulate);

/* Encode `count` tensors in one pass (two launches, one synchronisation):
 * for every t, exactly tlc_compress(ctx, tensors[t], residuals[t], ns[t],
 * s[t], bytes[t], caps[t], &bytes_len[t], &scales[t]).  All arrays are host
 * arrays of `count` entries; the pointers in them are device pointers, and
 * buffers of different tensors must not overlap.  Argument errors reject the
 * whole call before any work.  status[t] receives TLC_OK or
 * TLC_E_NONFINITE (that tensor's residual and bytes unchanged, or its
 * residual holding acc with TLC_OPT_IN_PLACE_FEEDBACK; bytes_len[t] = 0);
 * the call returns TLC_E_NONFINITE if any tensor was refused. */
int tlc_compress_batch(tlc_ctx* ctx, size_t count, const float* const* tensors,
                       float* const* residuals, const size_t* ns, const float* s,
                       uint8_t* const* bytes, const size_t* caps, size_t* bytes_len,
                       float* scales, int* status);

/* Decode `count` streams into `count` outputs in two launches: for every t,
 * tlc_decompress(ctx, bytes[t], bytes_len[t], scales[t], ns[t], outs[t],
 * accumulate).  Host arrays of device pointers; outputs must not overlap.
 * Asynchronous; if any stream is corrupt no output is written and the next
 * tlc_sync() returns TLC_E_CORRUPT. */
int tlc_decompress_batch(tlc_ctx* ctx, size_t count, const uint8_t* const* bytes,
                         const size_t* bytes_len, const float* scales, const size_t* ns,
                         float* const* outs, int accumulate);

/* Server-side aggregation (Section 2, Fig. 1; Section 3, Fig. 2): decode
 * `count` streams of the same n-value tensor and add them into one fp32
 * output in stream order, element by element:
 *   out = (((accumulate ? out : 0) + v_0) + v_1) + ... + v_{count-1}
 * (with accumulate == 0 the first term is v_0 itself), bit-identical to
 * tlc_decompress(stream 0, accumulate) followed by tlc_decompress(stream
 * t, accumulate = 1) for t = 1 .. count-1, but reading and writing out only
 * once.  Asynchronous; if any stream is corrupt out is left unchanged and
 * the next tlc_sync() returns TLC_E_CORRUPT.  count * n must not exceed the
 * context's max_n. */
int tlc_decompress_sum(tlc_ctx* ctx, size_t count, const uint8_t* const* bytes,
                       const size_t* bytes_len, const float* scales, size_t n, float* out,
                       int accumulate);

/* ---- encoding without a context (no allocation) ------------------------ */

/* Result of tlc_compress_noalloc, written to device memory by the call's
 * last kernel: status is TLC_OK, TLC_E_NONFINITE (residual and bytes left
 * unchanged, as for tlc_compress) or TLC_E_DEVICE (a look-back wait gave
 * up; the residual may then already hold its new values and no stream was
 * written); bytes_len and scale are those tlc_compress returns (0 unless
 * status is TLC_OK). */
typedef struct tlc_result {
  int32_t status;
  uint32_t bytes_len;
  float scale;
  uint32_t reserved; /* 0 */
} tlc_result;

/* Largest n tlc_compress_noalloc accepts: 2^23 values (at most 410 encoder
 * tiles, whose scratch is 8 KiB of device memory). */
#define TLC_NOALLOC_MAX_N ((size_t)8388608u)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * tlc_compress without a context.  Same encoding, bit for bit, with the
 * default error policy (the check pass leaves residual and bytes unchanged
 * on NaN/Inf), for n <= TLC_NOALLOC_MAX_N (larger n: TLC_E_INVALID, nothing
 * runs).
 *   tensor, residual, n, s, bytes, bytes_cap   as for tlc_compress.
 *   result      device pointer to one tlc_result (16 bytes), written last.
 *   hip_stream  a hipStream_t of the calling thread's current device (or
 *               NULL, the default stream); every pointer belongs to that
 *               device.
 * Asynchronous: returns after queueing its kernels (argument errors are
 * returned at once, and nothing runs); read *result after the stream has
 * reached it.  No device or pinned memory is allocated, and no library
 * routine that allocates is called: the scratch (a control block, partial
 * maxima, look-back status words) is a static device array of 8 KiB per
 * device, located once per device on the first call there.  Every call on
 * a device shares that array and clears it first, so calls that may
 * overlap on one device (other streams, other host threads) race and must
 * be ordered by the caller. */
int tlc_compress_noalloc(const float* tensor, float* residual, size_t n, float s,
                         uint8_t* bytes, size_t bytes_cap, tlc_result* result,
                         void* hip_stream);

/* ---- options ------------------------------------------------------------ */

/* TLC_OPT_IN_PLACE_FEEDBACK: take step 1 of error accumulation (Section
 * 3.1, Fig. 3: the tensor is added into the buffer) as done in the
 * residual itself before Eq. 1 is known.  The encoders then read tensor and
 * residual once instead of twice (12 instead of 20 bytes per value for the
 * 3-value modes); every result is the same, except that after
 * TLC_E_NONFINITE the residual holds tensor + residual instead of being
 * left unchanged.  For callers that check their tensors for NaN/Inf
 * themselves, or reset the residual after such an error. */
#define TLC_OPT_IN_PLACE_FEEDBACK 1u

/* Set the context's options (a combination of TLC_OPT_*; 0, the default,
 * is the behaviour documented above).  Takes effect from the next call. */
int tlc_ctx_set_options(tlc_ctx* ctx, uint32_t options);

/* Wait for all work of the context and return (then clear) the sticky
 * status of asynchronous decodes: TLC_OK or TLC_E_CORRUPT. */
int tlc_sync(tlc_ctx* ctx);

/* Look-back epochs.  Every launch of a chained or batched encode and every
 * decode tags the status words of its scan with the next value of a
 * per-context counter (encode 1 .. TLC_ENC_EPOCH_MAX, decode 1 ..
 * TLC_DEC_EPOCH_MAX), so the words need no clearing between launches;
 * when a counter wraps, its status words are cleared first (and for the
 * decode counter the range starts, the verdict and the mark that flags a
 * corrupt stream's launch). */
#define TLC_ENC_EPOCH_MAX 8388607  /* 2^23 - 1 */
#define TLC_DEC_EPOCH_MAX 67108863 /* 2^26 - 1 */

/* For tests of the wrap: wait for the context's work, clear the
 * epoch-tagged words of both scans (status words, the decoder's range
 * starts and its verdict: no word of an earlier launch can then carry a
 * future epoch) and set the counters to the last epochs used, enc_epoch
 * <= TLC_ENC_EPOCH_MAX and dec_epoch <= TLC_DEC_EPOCH_MAX (else
 * TLC_E_INVALID).  The corrupt-stream mark is left as it is: only the wrap
 * clears it. */
int tlc_ctx_set_epochs(tlc_ctx* ctx, uint32_t enc_epoch, uint32_t dec_epoch);

/* Text of the calling thread's most recent error (never NULL). */
const char* tlc_last_error_string(void);

/* ---- per-kernel timing (HIP events on the context's stream) ----------- */

#define TLC_KERNEL_ABSMAX 0         /* step 1 into the residual, partial max (Eq. 1) */
#define TLC_KERNEL_QUANT_ENCODE 1   /* Eq. 1-2, residual, quartic pack, each tile's own
                                       zero-run encoding */
#define TLC_KERNEL_ZRE_INDEX 2      /* zero-run scan: where each output range starts
                                       (a small stream's scan runs in the next kernel) */
#define TLC_KERNEL_EXPAND_DEQUANT 3 /* zero-run expansion, quartic unpack, Eq. 3 (for a
                                       small stream, with the scan in its first blocks) */
#define TLC_KERNEL_ABSMAX_BATCH 4
#define TLC_KERNEL_QUANT_ENCODE_BATCH 5
#define TLC_KERNEL_ZRE_INDEX_BATCH 6
#define TLC_KERNEL_EXPAND_DEQUANT_BATCH 7
#define TLC_KERNEL_EXPAND_SUM 8     /* multi-stream expansion + summed dequantization */
#define TLC_KERNEL_QUANT_PACK 9     /* comparison modes: quantize + quartic pack */
#define TLC_KERNEL_INT8_QUANT 10    /* 8-bit comparator: codes and residual */
#define TLC_KERNEL_INT8_DEQUANT 11  /* 8-bit comparator: decode */
#define TLC_KERNEL_ZRE_CHUNKS 12    /* zero-run encoding: summaries of tile chunks */
#define TLC_KERNEL_ZRE_COMPACT 13   /* zero-run encoding: tiles compacted into the stream */
#define TLC_KERNEL_QUANT_ENCODE_CHAINED 14 /* a small tensor's encode in one chained pass */
#define TLC_KERNEL_ABSMAX_CHECK 15  /* partial max of |tensor + residual|, nothing written */
#define TLC_KERNEL_ABSMAX_CHECK_BATCH 16
#define TLC_KERNEL_ACCUM_QUANTIZE 17 /* after the check pass: step 1, Eq. 2 and the residual
                                        for every value, 2-bit trits (large tensors) */
#define TLC_KERNEL_COUNT 18

/* Enable (on != 0) or disable recording of a start/stop event pair around
 * every kernel launch of the context (of the kernels selected by
 * tlc_profile_mask; all of them by default). */
int tlc_profile_enable(tlc_ctx* ctx, int on);

/* Select which kernels are timed while profiling is enabled: bit k of mask
 * selects kernel id k (TLC_KERNEL_*).  Each timed launch adds an event pair
 * to the stream, whose ordering costs some microseconds of device time, so
 * a caller measuring throughput may time only the kernel it needs. */
int tlc_profile_mask(tlc_ctx* ctx, uint32_t mask);

/* Synchronize, then report the summed device time (ms) and the number of
 * timed launches of kernel `kernel` since the last reset. */
int tlc_profile_get(tlc_ctx* ctx, int kernel, double* total_ms,
                    uint64_t* launches);

/* Zero the accumulated timings. */
int tlc_profile_reset(tlc_ctx* ctx);

/* Name of a kernel id (the __global__ function's name), or NULL. */
const char* tlc_kernel_name(int kernel);

#ifdef __cplusplus
}
#endif

#endif /* TLC_H */
