// device_common.hpp -- device helpers shared by the encode and decode
// kernels of the 3LC path.
#pragma once

#include <float.h>

#include "lookback.hpp"
#include "tlc_internal.h"
#include "wave_scan.hpp"
#include "zre_scan.hpp"

namespace tlc {

constexpr int kWaves = kThreads / 64;

// Unsigned min/max with both operands of one type.  HIP's mixed-type
// min/max (what min<T>(a, b) selects when b has another type, an int
// constant for instance) converts to double and calls fmin: several f64
// instructions, and values from 2^53 on would round.
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }

// A store into the pinned host readback (HostMirror) at system scope, so
// that it is in host memory when the kernel completes; p null: nothing.
__device__ __forceinline__ void host_put(uint32_t* p, uint32_t v) {
  if (p) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ void host_put_result(EncResult* h, uint32_t err, float scale) {
  if (h) {
    host_put(&h->err, err);
    host_put(reinterpret_cast<uint32_t*>(&h->scale), __float_as_uint(scale));
  }
}

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ uint32_t abs_bits(float v) {
  return __float_as_uint(v) & 0x7fffffffu;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  return wave_last(wave_incl_scan(v, 0u, OpMax()));
}

// Block-wide max over a block of kW waves; every thread gets the result.
// Uses lds[kW] and one barrier; callers that reuse lds must barrier again
// first.
template <int kW = kWaves>
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* lds) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) lds[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = lds[0];
#pragma unroll
  for (int w = 1; w < kW; ++w) r = max(r, lds[w]);
  return r;
}

// Block-wide exclusive prefix of u32 values over a block of kW waves:
// returns (exclusive prefix of this thread, block total).  Uses lds[kW] and
// one barrier.
struct ScanU32 {
  uint32_t excl, total;
};
template <int kW = kWaves>
__device__ __forceinline__ ScanU32 block_scan_u32(uint32_t v, uint32_t* lds) {
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v, 0u, OpAdd());
  if (lane == 63) lds[wid] = incl;
  __syncthreads();
  ScanU32 r;
  r.excl = incl - v;
  r.total = 0;
#pragma unroll
  for (int w = 0; w < kW; ++w) {
    if ((uint32_t)w < wid) r.excl += lds[w];
    r.total += lds[w];
  }
  return r;
}

// Exclusive max-scan over a block of kW waves (0 for thread 0) and the
// block's max (all threads; ends with a barrier-protected read of lds).
template <int kW = kWaves>
__device__ __forceinline__ ScanU32 block_scan_max_u32(uint32_t v, uint32_t* lds) {
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v, 0u, OpMax());
  const uint32_t excl = wave_prev_lane(incl, 0u);
  if (lane == 63) lds[wid] = incl;
  __syncthreads();
  ScanU32 r;
  r.excl = excl;
  r.total = 0u;
#pragma unroll
  for (int w = 0; w < kW; ++w) {
    if ((uint32_t)w < wid) r.excl = max(r.excl, lds[w]);
    r.total = max(r.total, lds[w]);
  }
  return r;
}

// How a kernel reaches the five partitions of a tile: one float4 per
// partition slice (m % 4 == 0, 16-byte aligned tensors), aligned float4
// cells off the slice grid (aligned tensors, m % 4 != 0), or one quartic
// byte per lane with scalar accesses (unaligned tensors).
constexpr int kPathVec = 0;
constexpr int kPathShift = 1;
constexpr int kPathByte = 2;

// Streaming float4 accesses (16-byte aligned addresses) with the
// nontemporal hint, for tensors read or written once per kernel and far
// larger than the caches.  Measured on gfx950: the max reduction reads
// 25 % faster with it, the 8-bit kernels (contiguous read/write streams,
// both sides hinted) 10-15 % faster, and the decoder's partition-by-
// partition sweep gains too (its hinted stores leave no dirty lines for the
// next encode).  The 3LC encoder hints only its loads of the tensor, which
// nothing reads again (a C4 round trip 1.5 % faster); hinting its residual
// loads or stores slowed it or the decode that follows.  The hint changes
// neither values nor visibility: the next kernel on the stream sees the
// stores.
typedef float tlc_f4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld_stream(const float* p) {
  const tlc_f4 v = __builtin_nontemporal_load(reinterpret_cast<const tlc_f4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st_stream(float* p, float4 v) {
  tlc_f4 w;
  w.x = v.x;
  w.y = v.y;
  w.z = v.z;
  w.w = v.w;
  __builtin_nontemporal_store(w, reinterpret_cast<tlc_f4*>(p));
}

// Place value of partition k's trit in a quartic byte (p0 most significant).
__device__ __forceinline__ uint32_t trit_weight(int k) {
  return k == 0 ? 81u : (k == 1 ? 27u : (k == 2 ? 9u : (k == 3 ? 3u : 1u)));
}

// ---------------------------------------------------------------- Eq. 1-2
struct Scale {
  float M;       // max|acc| * s
  float U;       // smallest fp32 u with rint(u / M) == 1
  uint32_t bad;  // NaN/Inf input or overflowing product
};

// rint(fl(a / M)) for |a| <= M is 1 exactly when fl(a / M) > 0.5, i.e. (the
// tie at 0.5 + 2^-25 rounds down to the even 0.5) when a > M * (0.5 +
// 2^-25).  That product has at most 49 significant bits, so it is exact in
// double; U is the smallest float above it.  The test a >= U therefore
// gives the same q as an IEEE divide followed by round-half-even, and by
// symmetry a <= -U gives q = -1.  M = 0 makes U the smallest subnormal, so
// q = 0 for the (all-zero) tensor.
__device__ __forceinline__ float quant_threshold(float M) {
  const double h = 0.5000000298023223876953125;  // 0.5 + 2^-25
  const double T = (double)M * h;
  float f = __double2float_rn(T);
  if ((double)f <= T) f = __uint_as_float(__float_as_uint(f) + 1u);
  return f;
}

// M and U from the partial maxima of one tensor (all kT threads of the
// block).
template <int kT = kThreads>
__device__ __forceinline__ Scale finish_scale(const uint32_t* __restrict__ partials,
                                              uint32_t np, float s, uint32_t* lds) {
  static_assert(kT % 64 == 0, "whole waves");
  uint32_t v = 0;
  for (uint32_t i = threadIdx.x; i < np; i += kT) v = max(v, partials[i]);
  const uint32_t A = block_max<kT / 64>(v, lds);
  Scale sc;
  sc.M = 0.0f;
  sc.U = 0.0f;
  sc.bad = 1u;
  if (A >= 0x7f800000u) return sc;
  const float M = __uint_as_float(A) * s;
  if (!(M <= FLT_MAX)) return sc;
  sc.M = M;
  sc.U = quant_threshold(M);
  sc.bad = 0u;
  return sc;
}

// q = round(acc / M) in {-1, 0, 1} (returned as the trit q + 1) and the
// residual acc - M*q.  M*q is exact, so acc - M, acc + M and acc are the
// bit patterns of acc - M*q for q = 1, -1, 0 (acc - (+0) == acc, -0 kept).
__device__ __forceinline__ uint32_t quantize_one(float acc, float M, float U,
                                                 float& res) {
  const bool pos = acc >= U;
  const bool neg = acc <= -U;
  res = pos ? acc - M : (neg ? acc + M : acc);
  return pos ? 2u : (neg ? 0u : 1u);
}

// Quartic byte j < m: quantizes the five accumulated values r[j + k*m]
// (contiguous partitions, p0 most significant; elements past n are the zero
// padding of Section 3.2, step 4) and returns the byte.  A value with q = 0
// keeps acc as its residual, which the buffer already holds, so only q != 0
// writes back.  kX (after the check pass has given M): the buffer still
// holds the previous residual, acc = x + r is formed here (step 1 of
// Section 3.1) and every value's residual is stored.
template <bool kX = false>
__device__ __forceinline__ uint32_t quantize_byte(const float* __restrict__ x,
                                                  float* __restrict__ r, uint64_t n,
                                                  uint64_t m, uint64_t j, float M, float U) {
  uint32_t code = 0u;
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    const uint64_t e = k * m + j;
    uint32_t t = 0u;
    if (e < n) {
      float o;
      t = quantize_one(kX ? x[e] + r[e] : r[e], M, U, o);
      if (kX || t != 1u) r[e] = o;
    }
    code = code * 3u + t;
  }
  return code;
}

// Quartic bytes j .. j+3 (j % 4 == 0) with m % 4 == 0 and r 16-byte
// aligned (and x, with kX): every partition slice is one float4.
// group4_full says whether all twenty values exist (only the last groups
// reach into the padding of p4); load_group4 fetches the five slices (the
// sums x + r with kX) and quantize_group4_loaded quantizes them, stores
// back a slice if one of its values has q != 0 (every slice with kX), and
// returns the four bytes packed little-endian.  Split so a caller can keep
// the loads of several groups in flight at once.
__device__ __forceinline__ bool group4_full(uint64_t n, uint64_t m, uint64_t j) {
  return 4 * m + j + 4 <= n;
}

template <bool kX = false>
__device__ __forceinline__ void load_group4(const float* __restrict__ x,
                                            const float* __restrict__ r, uint64_t m,
                                            uint64_t j, float4 (&a)[5]) {
#pragma unroll
  for (int k = 0; k < 5; ++k) a[k] = *reinterpret_cast<const float4*>(r + k * m + j);
  if (kX) {
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      const float4 b = *reinterpret_cast<const float4*>(x + k * m + j);
      a[k] = make_float4(b.x + a[k].x, b.y + a[k].y, b.z + a[k].z, b.w + a[k].w);
    }
  }
}

template <bool kX = false>
__device__ __forceinline__ uint32_t quantize_group4_loaded(float* __restrict__ r, uint64_t m,
                                                           uint64_t j, const float4 (&a)[5],
                                                           float M, float U) {
  uint32_t code[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    float4 o;
    const uint32_t t0 = quantize_one(a[k].x, M, U, o.x);
    const uint32_t t1 = quantize_one(a[k].y, M, U, o.y);
    const uint32_t t2 = quantize_one(a[k].z, M, U, o.z);
    const uint32_t t3 = quantize_one(a[k].w, M, U, o.w);
    code[0] = code[0] * 3u + t0;
    code[1] = code[1] * 3u + t1;
    code[2] = code[2] * 3u + t2;
    code[3] = code[3] * 3u + t3;
    if (kX || ((t0 ^ 1u) | (t1 ^ 1u) | (t2 ^ 1u) | (t3 ^ 1u)))
      *reinterpret_cast<float4*>(r + k * m + j) = o;
  }
  return code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
}

// The group by single bytes (any group, including those in the padding).
template <bool kX = false>
__device__ __forceinline__ uint32_t quantize_group4_bytes(const float* __restrict__ x,
                                                          float* __restrict__ r, uint64_t n,
                                                          uint64_t m, uint64_t j, float M,
                                                          float U) {
  uint32_t w = 0u;
#pragma unroll
  for (int c = 0; c < 4; ++c) w |= quantize_byte<kX>(x, r, n, m, j + c, M, U) << (8 * c);
  return w;
}

template <bool kX = false>
__device__ __forceinline__ uint32_t quantize_group4(const float* __restrict__ x,
                                                    float* __restrict__ r, uint64_t n,
                                                    uint64_t m, uint64_t j, float M,
                                                    float U) {
  if (!group4_full(n, m, j)) return quantize_group4_bytes<kX>(x, r, n, m, j, M, U);
  float4 a[5];
  load_group4<kX>(x, r, m, j, a);
  return quantize_group4_loaded<kX>(r, m, j, a, M, U);
}

// ---------------------------------------------------------------- stochastic mode
// Philox4x32-10 (Salmon et al., SC 2011): ten rounds, each multiplying two
// counter words by 0xD2511F53 and 0xCD9E8D57 (high halves XORed with the
// other two words and the key), the key advancing by 0x9E3779B9 /
// 0xBB67AE85 between rounds.
struct Philox4 {
  uint32_t v[4];
};
__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  Philox4 r;
  r.v[0] = c0;
  r.v[1] = c1;
  r.v[2] = c2;
  r.v[3] = c3;
  return r;
}

// Random words for elements 4b .. 4b+3 of a tensor: counter (b, step),
// key = seed.
__device__ __forceinline__ Philox4 element_words(uint64_t b, uint64_t step, uint64_t seed) {
  return philox4x32_10((uint32_t)b, (uint32_t)(b >> 32), (uint32_t)step,
                       (uint32_t)(step >> 32), (uint32_t)seed, (uint32_t)(seed >> 32));
}

// Stochastic 3-value quantization of one value: sign(x) kept with
// probability |x|/M, i.e. when u*M < |x| for u = (w >> 8) * 2^-24; the
// product of a 24-bit integer and an fp32 is exact in double, so the
// decision is exact.  Returns the trit q + 1.
__device__ __forceinline__ uint32_t stochastic_trit(float x, float M, uint32_t w) {
  const double u = (double)(w >> 8) * (1.0 / 16777216.0);
  const bool keep = (M > 0.0f) && (u * (double)M < fabs((double)x));
  return keep ? (x > 0.0f ? 2u : 0u) : 1u;
}

// ---------------------------------------------------------------- Section 3.3
using EncSW = StatusWord<39>;  // RunSum with a 30-bit count
using DecSW = StatusWord<36>;  // expanded byte count

__device__ __forceinline__ uint64_t rs_to_payload(RunSum a) {
  return (a.v & 0x3fffffffull) | ((a.v >> 32) << 30);
}
__device__ __forceinline__ RunSum rs_from_payload(uint64_t p) {
  RunSum r;
  r.v = (p & 0x3fffffffull) | ((p >> 30) << 32);
  return r;
}

struct EncOp {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    return rs_to_payload(rs_combine(rs_from_payload(a), rs_from_payload(b)));
  }
};
struct SumOp {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};

__device__ __forceinline__ void unpack16(uint4 v, uint8_t* b) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    b[i] = (uint8_t)(v.x >> (8 * i));
    b[4 + i] = (uint8_t)(v.y >> (8 * i));
    b[8 + i] = (uint8_t)(v.z >> (8 * i));
    b[12 + i] = (uint8_t)(v.w >> (8 * i));
  }
}

// Wave scans of segment summaries (zre_scan.hpp), in lane order.
struct OpRun {
  __device__ __forceinline__ uint64_t operator()(uint64_t a, uint64_t b) const {
    RunSum x, y;
    x.v = a;
    y.v = b;
    return rs_combine(x, y).v;
  }
};
__device__ __forceinline__ RunSum wave_incl_scan_rs(RunSum v) {
  RunSum r;
  r.v = wave_incl_scan(v.v, rs_identity().v, OpRun());
  return r;
}
__device__ __forceinline__ RunSum wave_prev_lane_rs(RunSum v) {
  RunSum r;
  r.v = wave_prev_lane(v.v, rs_identity().v);
  return r;
}

// Number of quartic bytes a stream byte stands for: data bytes (< 243) one,
// run codes 243 + (k - 2) k copies of 121.
__device__ __forceinline__ uint32_t expanded_len(uint32_t b) {
  return b < kRunBase ? 1u : b - (kRunBase - 2u);
}

// What the four stream bytes of w expand to beyond one quartic byte each:
// byte b adds max(b - 242, 0) (expanded_len less one), which is
// (|b - 242| + b - 242) / 2, and two sums of absolute byte differences
// (v_sad_u8) give that for the four bytes at once.  A zero byte adds 0.
__device__ __forceinline__ uint32_t run_extra4(uint32_t w) {
  constexpr uint32_t kPivot = kRunBase - 1u;  // 242 in every byte below
  const uint32_t s =
      __builtin_amdgcn_sad_u8(w, kPivot * 0x01010101u, __builtin_amdgcn_sad_u8(w, 0u, 0u));
  return (s - 4u * kPivot) >> 1;
}

// ---------------------------------------------------------------- Eq. 3
// The dequantized value M*q for trit t = q + 1 is -M, M*0 or M (M*(-1) is
// the exact negation; M*0 is +0, or -0 for a scale of -0.0, which the
// decoder accepts as >= 0).
__device__ __forceinline__ float trit_value(uint32_t t, float M) {
  return t == 0u ? -M : (t == 1u ? M * 0.0f : M);
}

// Eq. 3 accumulated densely into out (every value: out + M*q, so -0.0 + 0
// gives +0.0).  acc_trit4 returns whether any of the four sums has other
// bits than its input: a store of identical bits can be skipped without
// changing any result, and with few values q != 0 most stores are.
__device__ __forceinline__ float acc_trit(float out, uint32_t t, float M) {
  return out + trit_value(t, M);
}

__device__ __forceinline__ bool acc_trit4(float4& o, const uint32_t (&d)[4], float M) {
  const float4 r = make_float4(o.x + trit_value(d[0], M), o.y + trit_value(d[1], M),
                               o.z + trit_value(d[2], M), o.w + trit_value(d[3], M));
  const bool changed = ((__float_as_uint(r.x) ^ __float_as_uint(o.x)) |
                        (__float_as_uint(r.y) ^ __float_as_uint(o.y)) |
                        (__float_as_uint(r.z) ^ __float_as_uint(o.z)) |
                        (__float_as_uint(r.w) ^ __float_as_uint(o.w))) != 0u;
  o = r;
  return changed;
}

// out[e] += M*q, stored only if the bits change.
__device__ __forceinline__ void acc_trit_at(float* __restrict__ out, uint64_t e, uint32_t t,
                                            float M) {
  const float o = out[e];
  const float r = o + trit_value(t, M);
  if (__float_as_uint(r) != __float_as_uint(o)) out[e] = r;
}

// Mask of the non-121 bytes among the 16 quartic bytes q[lo .. lo + cnt)
// (cnt <= 16; q + lo 16-byte aligned) that one thread holds: bit i for
// byte lo + i.
// Four bits: byte i of w differs from 121.  x = w ^ 0x79797979 has a zero
// byte exactly where w holds 121; bit 7 of ((x & 0x7f..) + 0x7f..) | x is
// set in every other byte (no carry leaves a byte); the multiply gathers
// the four bit-7 flags, shifted to bits 0, 8, 16, 24, into bits 21..24
// (the partial products occupy distinct bits, so nothing carries).
__device__ __forceinline__ uint32_t nonzero_byte_mask4(uint32_t w) {
  const uint32_t x = w ^ 0x79797979u;
  const uint32_t y = (x | ((x & 0x7f7f7f7fu) + 0x7f7f7f7fu)) & 0x80808080u;
  return ((y >> 7) * 0x00204081u) >> 21 & 0xfu;
}

__device__ __forceinline__ uint32_t nonzero_mask16(const uint4& w, uint32_t cnt) {
  static_assert(kZeroGroup == 0x79u, "the mask compares against bytes of 121");
  const uint32_t nz = nonzero_byte_mask4(w.x) | (nonzero_byte_mask4(w.y) << 4) |
                      (nonzero_byte_mask4(w.z) << 8) | (nonzero_byte_mask4(w.w) << 12);
  return cnt >= 16u ? nz : nz & ((1u << cnt) - 1u);
}

// The same mask in spread form, bit 2i for byte lo + i (rs_gaps_len<2>):
// the multiply places the four bit-7 flags, shifted to bits 0, 8, 16, 24,
// at bits 18, 20, 22, 24 (again no two partial products share a bit).
__device__ __forceinline__ uint32_t nonzero_byte_mask4_spread(uint32_t w) {
  const uint32_t x = w ^ 0x79797979u;
  const uint32_t y = (x | ((x & 0x7f7f7f7fu) + 0x7f7f7f7fu)) & 0x80808080u;
  return ((y >> 7) * 0x00041041u) >> 18 & 0x55u;
}

__device__ __forceinline__ uint32_t nonzero_mask16_spread(const uint4& w, uint32_t cnt) {
  const uint32_t nz = nonzero_byte_mask4_spread(w.x) | (nonzero_byte_mask4_spread(w.y) << 8) |
                      (nonzero_byte_mask4_spread(w.z) << 16) |
                      (nonzero_byte_mask4_spread(w.w) << 24);
  return cnt >= 16u ? nz : nz & ((1u << (2u * cnt)) - 1u);
}

// The spread mask of the 16 quartic bytes that five trit words pack (word
// k holds partition k's trits, trit i in bits 2i and 2i + 1, as q + 1):
// byte i is 121 exactly when all five of its trits are 1 (Section 3.2: 121
// is 11111 in base 3), i.e. when bits 2i, 2i + 1 read 01 in every word.
__device__ __forceinline__ uint32_t nonzero_mask_trits(const uint32_t (&d)[5]) {
  constexpr uint32_t kOnes = 0x55555555u;  // trit 1 in every field
  const uint32_t z = (d[0] ^ kOnes) | (d[1] ^ kOnes) | (d[2] ^ kOnes) | (d[3] ^ kOnes) |
                     (d[4] ^ kOnes);
  return (z | (z >> 1)) & kOnes;
}

__device__ __forceinline__ uint32_t nonzero_group_mask(const uint8_t* q, uint32_t lo,
                                                       uint32_t cnt) {
  return nonzero_mask16(*reinterpret_cast<const uint4*>(q + lo), cnt);
}

// Byte i (< 16) of four little-endian words, by selects on the values (an
// indexed array would be placed in LDS or scratch memory).
__device__ __forceinline__ uint32_t byte_of16(uint32_t x, uint32_t y, uint32_t z, uint32_t w,
                                              uint32_t i) {
  const uint32_t lo = (i & 4u) ? y : x, hi = (i & 4u) ? w : z;
  return ((i & 8u) ? hi : lo) >> (8u * (i & 3u)) & 255u;
}

// Base-3 digits of a quartic byte, most significant first (weights 81, 27,
// 9, 3, 1): Section 3.2, decoding step 1.
__device__ __forceinline__ void digits5(uint32_t byte, uint32_t (&t)[5]) {
  t[0] = byte / 81u;
  byte -= t[0] * 81u;
  t[1] = byte / 27u;
  byte -= t[1] * 27u;
  t[2] = byte / 9u;
  byte -= t[2] * 9u;
  t[3] = byte / 3u;
  t[4] = byte - t[3] * 3u;
}

// Index of the last descriptor whose `first` field is <= key (descriptors
// sorted by `first`, descs[0].first == 0).
template <class D, class F>
__device__ __forceinline__ uint32_t find_desc(const D* __restrict__ descs, uint32_t count,
                                              uint32_t key, F first) {
  uint32_t lo = 0, hi = count;  // invariant: first(descs[lo]) <= key
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (first(descs[mid]) <= key)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

}  // namespace tlc
