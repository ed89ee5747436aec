// tlc_kernels.hip -- gfx950 kernels of the 3LC encode/decode path.
//
//   tlc_absmax_kernel          partial maxima of |tensor + residual|   (Eq. 1)
//   tlc_quant_encode_kernel    M, 3-value quantization, residual write-back,
//                              quartic pack and zero-run encoding in one
//                              pass              (Eq. 1-2, Sections 3.2-3.3)
//   tlc_zre_index_kernel       zero-run scan: where each 4096-byte range of
//                              quartic bytes starts in the stream
//   tlc_expand_dequant_kernel  zero-run expansion into LDS, quartic unpack,
//                              Eq. 3, optional accumulate
//
// All of it is HBM streaming or byte scanning; nothing is a dense
// contraction, so there is no MFMA here.  fp32 arithmetic is exactly the
// paper's sequence (add, scale, divide+round, subtract, multiply, add); see
// quantize_one for how the divide is decided without dividing.
#include <float.h>

#include "lookback.hpp"
#include "tlc_internal.h"
#include "zre_scan.hpp"

namespace tlc {

constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint32_t abs_bits(float v) {
  return __float_as_uint(v) & 0x7fffffffu;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, d, 64));
  return v;
}

// Block-wide max; every thread gets the result.
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* lds) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) lds[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = lds[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r = max(r, lds[w]);
  return r;
}

// ---------------------------------------------------------------- Eq. 1
// max |x + r| is taken on the bit patterns with the sign cleared: for
// non-negative IEEE values integer order equals numeric order, so the u32
// max is exact and independent of reduction order, and any NaN/Inf makes
// the result >= 0x7f800000.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void tlc_absmax_kernel(
    const float* __restrict__ x, const float* __restrict__ r, uint64_t n,
    uint32_t* __restrict__ partials) {
  __shared__ uint32_t lds[kWaves];
  uint32_t mx = 0;
  const uint64_t tid = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads;
  if (kVec) {
    const float4* __restrict__ x4 = reinterpret_cast<const float4*>(x);
    const float4* __restrict__ r4 = reinterpret_cast<const float4*>(r);
    const uint64_t nv = n >> 2;
    uint64_t i = tid;
    for (; i + 3 * stride < nv; i += 4 * stride) {
      float4 a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = x4[i + u * stride];
#pragma unroll
      for (int u = 0; u < 4; ++u) b[u] = r4[i + u * stride];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        mx = max(mx, abs_bits(a[u].x + b[u].x));
        mx = max(mx, abs_bits(a[u].y + b[u].y));
        mx = max(mx, abs_bits(a[u].z + b[u].z));
        mx = max(mx, abs_bits(a[u].w + b[u].w));
      }
    }
    for (; i < nv; i += stride) {
      float4 a = x4[i], b = r4[i];
      mx = max(mx, abs_bits(a.x + b.x));
      mx = max(mx, abs_bits(a.y + b.y));
      mx = max(mx, abs_bits(a.z + b.z));
      mx = max(mx, abs_bits(a.w + b.w));
    }
    for (uint64_t e = (nv << 2) + tid; e < n; e += stride)
      mx = max(mx, abs_bits(x[e] + r[e]));
  } else {
    for (uint64_t e = tid; e < n; e += stride) mx = max(mx, abs_bits(x[e] + r[e]));
  }
  mx = block_max(mx, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = mx;
}

// ---------------------------------------------------------------- Eq. 2
struct Scale {
  float M;      // max|acc| * s
  float U;      // smallest fp32 u with rint(u / M) == 1
  uint32_t bad; // NaN/Inf input or overflowing product
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

__device__ __forceinline__ Scale finish_scale(const uint32_t* __restrict__ partials,
                                              uint32_t np, float s, uint32_t* lds) {
  uint32_t v = 0;
  for (uint32_t i = threadIdx.x; i < np; i += kThreads) v = max(v, partials[i]);
  const uint32_t A = block_max(v, lds);
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

__device__ __forceinline__ RunSum shfl_up_rs(RunSum v, int d) {
  RunSum o;
  o.v = __shfl_up(v.v, d, 64);
  return o;
}

// Quartic byte j < m: quantizes the five elements j + k*m (contiguous
// partitions, p0 most significant; elements past n are the zero padding of
// Section 3.2, step 4), writes their residuals and returns the byte.
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
      t = quantize_one(x[e] + r[e], M, U, o);
      r[e] = o;
    }
    code = code * 3u + t;
  }
  return code;
}

// Quartic bytes j .. j+3 (j % 4 == 0) with m % 4 == 0 and 16-byte aligned x
// and r, so every partition slice is one float4; returns the four bytes
// packed little-endian.
__device__ __forceinline__ uint32_t quantize_group4(const float* __restrict__ x,
                                                    float* __restrict__ r, uint64_t n,
                                                    uint64_t m, uint64_t j, float M,
                                                    float U) {
  if (4 * m + j + 4 > n) {  // the group that reaches into the padding of p4
    uint32_t w = 0u;
#pragma unroll
    for (int c = 0; c < 4; ++c) w |= quantize_byte(x, r, n, m, j + c, M, U) << (8 * c);
    return w;
  }
  uint32_t code[4] = {0u, 0u, 0u, 0u};
  float4 a[5], b[5];
#pragma unroll
  for (int k = 0; k < 5; ++k) a[k] = *reinterpret_cast<const float4*>(x + k * m + j);
#pragma unroll
  for (int k = 0; k < 5; ++k) b[k] = *reinterpret_cast<const float4*>(r + k * m + j);
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    float4 o;
    code[0] = code[0] * 3u + quantize_one(a[k].x + b[k].x, M, U, o.x);
    code[1] = code[1] * 3u + quantize_one(a[k].y + b[k].y, M, U, o.y);
    code[2] = code[2] * 3u + quantize_one(a[k].z + b[k].z, M, U, o.z);
    code[3] = code[3] * 3u + quantize_one(a[k].w + b[k].w, M, U, o.w);
    *reinterpret_cast<float4*>(r + k * m + j) = o;
  }
  return code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
}

// One tile = kEncTile quartic bytes (5 * kEncTile values).  Phase 1: the
// block quantizes its values (threads take groups of 4 bytes, or single
// bytes when the partitions are not 16-byte aligned, interleaved so every
// load and store instruction is coalesced) and keeps the quartic bytes in
// LDS.  Phase 2: each thread takes kEncTile/256 consecutive bytes,
// summarises them as a RunSum, the block scans the summaries, the tile gets
// its prefix by decoupled look-back, and every thread zero-run encodes its
// bytes from its own prefix into LDS; the block then copies the tile's
// output into the stream.  The quartic bytes never go to HBM.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void tlc_quant_encode_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n, uint32_t m, float s,
    const uint32_t* __restrict__ partials, uint32_t np, uint8_t* __restrict__ out,
    uint64_t* __restrict__ status, uint32_t ticket_base, uint32_t epoch,
    Ctrl* __restrict__ ctrl) {
  constexpr int kBytes = kEncTile / kThreads;  // zero-run bytes per thread
  static_assert(kBytes % 16 == 0, "threads read whole uint4s of quartic bytes");
  __shared__ uint32_t s_max[kWaves];
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_fault;
  __shared__ RunSum s_wave[kWaves];
  __shared__ RunSum s_excl;
  __shared__ __align__(16) uint8_t s_q[kEncTile];
  __shared__ __align__(16) uint8_t s_out[kEncTile + 16];

  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->enc_ticket) - ticket_base;
  const Scale sc = finish_scale(partials, np, s, s_max);  // includes a barrier
  const uint32_t tile = s_tile;
  if (tile == 0 && threadIdx.x == 0) {
    ctrl->enc_err = sc.bad;
    ctrl->enc_scale = sc.M;
  }
  if (sc.bad) return;  // NaN/Inf or overflow: residual and stream untouched

  // ---- phase 1: Eq. 1-2, residual write-back, quartic pack
  const uint64_t q0 = (uint64_t)tile * kEncTile;
  const uint32_t tile_bytes = (uint32_t)min<uint64_t>(kEncTile, (uint64_t)m - q0);
  if (kVec) {  // 4 bytes per thread: float4 loads and stores
    for (uint32_t g = threadIdx.x; g * 4u < tile_bytes; g += kThreads)
      *reinterpret_cast<uint32_t*>(s_q + g * 4u) =
          quantize_group4(x, r, n, m, q0 + g * 4u, sc.M, sc.U);
  } else {  // 1 byte per thread: dword accesses, still contiguous per wave
    for (uint32_t lj = threadIdx.x; lj < tile_bytes; lj += kThreads)
      s_q[lj] = (uint8_t)quantize_byte(x, r, n, m, q0 + lj, sc.M, sc.U);
  }
  __syncthreads();

  // ---- phase 2: Section 3.3
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint32_t lo = threadIdx.x * kBytes;
  const uint32_t cnt = lo < tile_bytes ? min<uint32_t>(kBytes, tile_bytes - lo) : 0u;
  uint8_t b[kBytes];
#pragma unroll
  for (int h = 0; h < kBytes / 16; ++h)
    unpack16(*reinterpret_cast<const uint4*>(s_q + lo + 16 * h), b + 16 * h);
  RunSum sum = rs_identity();
#pragma unroll
  for (int i = 0; i < kBytes; ++i)
    if ((uint32_t)i < cnt) sum = rs_combine(sum, rs_byte(b[i]));

  RunSum incl = sum;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    RunSum o = shfl_up_rs(incl, d);
    if (lane >= (uint32_t)d) incl = rs_combine(o, incl);
  }
  RunSum excl_lane = shfl_up_rs(incl, 1);
  if (lane == 0) excl_lane = rs_identity();
  if (lane == 63) s_wave[wid] = incl;
  __syncthreads();
  RunSum wpre = rs_identity();
  RunSum agg = rs_identity();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if ((uint32_t)w < wid) wpre = rs_combine(wpre, s_wave[w]);
    agg = rs_combine(agg, s_wave[w]);
  }

  if (wid == 0) {
    bool fault = false;
    uint64_t ex = rs_to_payload(rs_identity());
    if (tile == 0) {
      if (lane == 0)
        status_publish(&status[0], EncSW::pack(rs_to_payload(agg), kFlagPrefix, epoch));
    } else {
      ex = lookback_wave<EncSW>(status, tile, rs_to_payload(agg), ex, epoch, EncOp(),
                                &fault);
    }
    if (lane == 0) {
      s_excl = rs_from_payload(ex);
      s_fault = fault ? 1u : 0u;
      if (fault)
        __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (s_fault) return;

  const RunSum tex = s_excl;
  const RunSum P = rs_combine(rs_combine(tex, wpre), excl_lane);
  const uint32_t tile_begin = rs_emitted(tex);
  uint32_t o = rs_emitted(P) - tile_begin;
  uint32_t phi = rs_phase(P);
  auto put = [&](uint32_t c) {
    if (o < sizeof(s_out)) s_out[o] = (uint8_t)c;
    ++o;
  };
#pragma unroll
  for (int i = 0; i < kBytes; ++i)
    if ((uint32_t)i < cnt) phi = rs_step(b[i], phi, put);
  if (cnt && q0 + lo + cnt == m && phi) put(rs_code(phi));  // stream ends in a run

  const bool last_tile = q0 + kEncTile >= m;
  const RunSum tincl = rs_combine(tex, agg);
  const uint32_t tile_end = last_tile ? rs_total(tincl) : rs_emitted(tincl);
  __syncthreads();
  // a tile emits at most kEncTile + 1 bytes; the clamps only keep a logic
  // error from writing outside the caller's m-byte buffer
  const uint32_t count =
      tile_end >= tile_begin ? min<uint32_t>(tile_end - tile_begin, kEncTile + 1) : 0u;
  for (uint32_t i = threadIdx.x; i < count; i += kThreads)
    if (tile_begin + i < m) out[tile_begin + i] = s_out[i];
  if (last_tile && threadIdx.x == 0) ctrl->enc_len = tile_end;
}

// ---------------------------------------------------------------- expansion
__device__ __forceinline__ uint32_t expanded_len(uint32_t b) {
  return b < kRunBase ? 1u : b - (kRunBase - 2u);
}

// One tile = 256 threads x 32 stream bytes.  Expansion lengths are scanned
// in the block and across tiles (decoupled look-back), which places every
// stream byte's expansion in the quartic byte string.  Nothing is expanded
// here: the byte whose expansion contains position k * kDecRange records
// (its index, how far into its expansion that position lies) in start[k],
// so each block of the expanding kernel can find its part of the stream
// with one load.  The last tile flags the launch's epoch as corrupt when
// the expansion total is not exactly m.
__global__ __launch_bounds__(kThreads) void tlc_zre_index_kernel(
    const uint8_t* __restrict__ C, uint32_t c, uint32_t m, uint64_t* __restrict__ start,
    uint64_t* __restrict__ status, uint32_t ticket_base, uint32_t epoch,
    Ctrl* __restrict__ ctrl) {
  constexpr int kBytes = kZreBytesPerThread;
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_fault;
  __shared__ uint32_t s_wave[kWaves];
  __shared__ uint64_t s_excl;

  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->dec_ticket) - ticket_base;
  __syncthreads();
  const uint32_t tile = s_tile;
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint64_t j0 = (uint64_t)tile * kZreTile + threadIdx.x * kBytes;
  const uint32_t cnt = j0 < c ? (uint32_t)min<uint64_t>(kBytes, c - j0) : 0u;

  uint8_t b[kBytes];
  if (cnt == (uint32_t)kBytes && ((reinterpret_cast<uintptr_t>(C + j0) & 15u) == 0u)) {
#pragma unroll
    for (int h = 0; h < kBytes / 16; ++h)
      unpack16(*reinterpret_cast<const uint4*>(C + j0 + 16 * h), b + 16 * h);
  } else {
#pragma unroll
    for (int i = 0; i < kBytes; ++i) b[i] = (uint32_t)i < cnt ? C[j0 + i] : (uint8_t)0;
  }
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kBytes; ++i)
    if ((uint32_t)i < cnt) sum += expanded_len(b[i]);

  uint32_t incl = sum;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t o = __shfl_up(incl, d, 64);
    if (lane >= (uint32_t)d) incl += o;
  }
  if (lane == 63) s_wave[wid] = incl;
  __syncthreads();
  uint32_t wpre = 0, agg = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if ((uint32_t)w < wid) wpre += s_wave[w];
    agg += s_wave[w];
  }

  if (wid == 0) {
    bool fault = false;
    uint64_t ex = 0;
    if (tile == 0) {
      if (lane == 0) status_publish(&status[0], DecSW::pack(agg, kFlagPrefix, epoch));
    } else {
      ex = lookback_wave<DecSW>(status, tile, agg, 0, epoch, SumOp(), &fault);
    }
    if (lane == 0) {
      s_excl = ex;
      s_fault = fault ? 1u : 0u;
      if (fault)
        __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const bool last_tile = (uint64_t)(tile + 1) * kZreTile >= c;
      if (last_tile && (fault || ex + agg != m)) {
        __hip_atomic_store(&ctrl->dec_bad_epoch, epoch, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&ctrl->dec_corrupt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  __syncthreads();
  if (s_fault) return;

  uint64_t o = s_excl + wpre + incl - sum;  // where this thread's first byte expands
#pragma unroll
  for (int i = 0; i < kBytes; ++i) {
    if ((uint32_t)i < cnt) {
      const uint32_t len = expanded_len(b[i]);
      const uint64_t k = (o + kDecRange - 1) / kDecRange;  // first range start >= o
      const uint64_t at = k * kDecRange;
      if (at < o + len && at < m) start[k] = ((j0 + i) << 8) | (at - o);
      o += len;
    }
  }
}

// ---------------------------------------------------------------- Eq. 3
// The dequantized value M*q for trit t = q + 1 is -M, +0 or M (M*(-1) is
// the exact negation and M*0 is +0 for finite M >= 0).
__device__ __forceinline__ float trit_value(uint32_t t, float M) {
  return t == 0u ? -M : (t == 1u ? 0.0f : M);
}

__device__ __forceinline__ void digits5(uint32_t byte, uint32_t (&t)[5]) {
  // base-3 digits, most significant first (weights 81, 27, 9, 3, 1)
  t[0] = byte / 81u;
  byte -= t[0] * 81u;
  t[1] = byte / 27u;
  byte -= t[1] * 27u;
  t[2] = byte / 9u;
  byte -= t[2] * 9u;
  t[3] = byte / 3u;
  t[4] = byte - t[3] * 3u;
}

// Writes bytes of 121 at lds[lo..hi).
__device__ __forceinline__ void fill_zero_groups(uint8_t* lds, uint32_t lo, uint32_t hi) {
  while (lo < hi && (lo & 3u)) lds[lo++] = (uint8_t)kZeroGroup;
  for (; lo + 4 <= hi; lo += 4) *reinterpret_cast<uint32_t*>(lds + lo) = 0x79797979u;
  while (lo < hi) lds[lo++] = (uint8_t)kZeroGroup;
}

// One block = quartic bytes [k*kDecRange, (k+1)*kDecRange).  Phase 1
// expands the stream bytes that cover the range (found through start[k])
// into LDS: the bytes are spread over the threads, a block scan of their
// expansion lengths gives each one its position, and each thread writes
// its expansions.  Phase 2 unpacks the base-3 digits of every quartic byte
// (Section 3.2 decoding), dequantizes (Eq. 3) and stores or accumulates
// into the five partitions of out, with float4 accesses when m % 4 == 0
// and out is 16-byte aligned.
template <bool kVec, bool kAcc>
__global__ __launch_bounds__(kThreads) void tlc_expand_dequant_kernel(
    const uint8_t* __restrict__ C, uint32_t c, const uint64_t* __restrict__ start,
    uint64_t n, uint64_t m, float M, float* __restrict__ out, uint32_t epoch,
    const Ctrl* __restrict__ ctrl) {
  constexpr int kBytes = kDecRange / kThreads;  // stream bytes per thread (at most)
  __shared__ uint32_t s_wave[kWaves];
  __shared__ __align__(16) uint8_t s_q[kDecRange];
  if (ctrl->dec_bad_epoch == epoch) return;  // corrupt stream: out untouched

  // ---- phase 1: zero-run expansion of this range into LDS
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint64_t q0 = (uint64_t)blockIdx.x * kDecRange;
  const uint32_t qn = (uint32_t)min<uint64_t>(kDecRange, m - q0);
  const uint64_t s0 = start[blockIdx.x];
  const uint32_t i0 = (uint32_t)(s0 >> 8);
  const uint32_t skip = (uint32_t)(s0 & 255u);
  uint32_t i1 = c;  // one past the last stream byte that reaches into the range
  if (q0 + kDecRange < m) {
    const uint64_t s1 = start[blockIdx.x + 1];
    i1 = (uint32_t)(s1 >> 8) + ((s1 & 255u) ? 1u : 0u);
  }
  i1 = min(i1, c);
  const uint32_t count = i1 > i0 ? min<uint32_t>(i1 - i0, kDecRange) : 0u;
  const uint32_t lo = threadIdx.x * kBytes;
  const uint32_t cnt = lo < count ? min<uint32_t>(kBytes, count - lo) : 0u;
  uint8_t b[kBytes];
#pragma unroll
  for (int i = 0; i < kBytes; ++i) b[i] = (uint32_t)i < cnt ? C[i0 + lo + i] : (uint8_t)0;
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kBytes; ++i)
    if ((uint32_t)i < cnt) sum += expanded_len(b[i]);
  uint32_t incl = sum;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t o = __shfl_up(incl, d, 64);
    if (lane >= (uint32_t)d) incl += o;
  }
  if (lane == 63) s_wave[wid] = incl;
  __syncthreads();
  uint32_t wpre = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w)
    if ((uint32_t)w < wid) wpre += s_wave[w];
  int pos = (int)(wpre + incl - sum) - (int)skip;  // range-relative start of b[0]
#pragma unroll
  for (int i = 0; i < kBytes; ++i) {
    if ((uint32_t)i < cnt) {
      const uint32_t x = b[i];
      const int len = (int)expanded_len(x);
      const uint32_t a = (uint32_t)max(pos, 0);
      const uint32_t e = (uint32_t)min(pos + len, (int)qn);
      if (a < e) {
        if (x < kRunBase)
          s_q[a] = (uint8_t)x;
        else
          fill_zero_groups(s_q, a, e);
      }
      pos += len;
    }
  }
  __syncthreads();

  // ---- phase 2: Section 3.2 decoding and Eq. 3
  if (kVec) {
#pragma unroll
    for (int g = 0; g < kDecRange / (4 * kThreads); ++g) {
      const uint32_t jl = 4u * (threadIdx.x + kThreads * g);
      if (jl >= qn) break;
      const uint64_t j = q0 + jl;
      const uint32_t w = *reinterpret_cast<const uint32_t*>(s_q + jl);
      uint32_t t[4][5];
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) digits5((w >> (8 * cc)) & 0xffu, t[cc]);
      if (4 * m + j + 4 <= n) {
        float4 o[5];
        if (kAcc) {
#pragma unroll
          for (int k = 0; k < 5; ++k) o[k] = *reinterpret_cast<const float4*>(out + k * m + j);
        }
#pragma unroll
        for (int k = 0; k < 5; ++k) {
          if (kAcc) {
            o[k].x = o[k].x + trit_value(t[0][k], M);
            o[k].y = o[k].y + trit_value(t[1][k], M);
            o[k].z = o[k].z + trit_value(t[2][k], M);
            o[k].w = o[k].w + trit_value(t[3][k], M);
          } else {
            o[k].x = trit_value(t[0][k], M);
            o[k].y = trit_value(t[1][k], M);
            o[k].z = trit_value(t[2][k], M);
            o[k].w = trit_value(t[3][k], M);
          }
          *reinterpret_cast<float4*>(out + k * m + j) = o[k];
        }
      } else {  // the group whose p4 slice reaches into the padding
#pragma unroll
        for (int k = 0; k < 5; ++k) {
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const uint64_t e = k * m + j + cc;
            if (e < n) {
              const float v = trit_value(t[cc][k], M);
              out[e] = kAcc ? out[e] + v : v;
            }
          }
        }
      }
    }
  } else {
    for (uint32_t jl = threadIdx.x; jl < qn; jl += kThreads) {
      const uint64_t j = q0 + jl;
      uint32_t t[5];
      digits5(s_q[jl], t);
#pragma unroll
      for (int k = 0; k < 5; ++k) {
        const uint64_t e = k * m + j;
        if (e < n) {
          const float v = trit_value(t[k], M);
          out[e] = kAcc ? out[e] + v : v;
        }
      }
    }
  }
}

static inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0u;
}

static inline uint32_t blocks_for(uint64_t items, uint64_t per_block,
                                             uint32_t cap) {
  uint64_t b = (items + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (uint32_t)b;
}

hipError_t launch_absmax(const float* x, const float* r, uint64_t n,
                         uint32_t* partials, uint32_t* nblocks, hipStream_t st) {
  const bool vec = aligned16(x) && aligned16(r);
  const uint64_t items = vec ? (n >> 2) : n;
  const uint32_t blocks = blocks_for(items, (uint64_t)kThreads * 4, kAbsmaxMaxBlocks);
  *nblocks = blocks;
  if (vec)
    tlc_absmax_kernel<true><<<blocks, kThreads, 0, st>>>(x, r, n, partials);
  else
    tlc_absmax_kernel<false><<<blocks, kThreads, 0, st>>>(x, r, n, partials);
  return hipGetLastError();
}

hipError_t launch_quant_encode(const float* x, float* r, uint64_t n, uint32_t m, float s,
                              const uint32_t* partials, uint32_t npartials, uint8_t* out,
                              uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                              uint32_t epoch, Ctrl* ctrl, hipStream_t st) {
  const bool vec = (m % 4 == 0) && aligned16(x) && aligned16(r);
  if (vec)
    tlc_quant_encode_kernel<true><<<ntiles, kThreads, 0, st>>>(
        x, r, n, m, s, partials, npartials, out, status, ticket_base, epoch, ctrl);
  else
    tlc_quant_encode_kernel<false><<<ntiles, kThreads, 0, st>>>(
        x, r, n, m, s, partials, npartials, out, status, ticket_base, epoch, ctrl);
  return hipGetLastError();
}

hipError_t launch_zre_index(const uint8_t* C, uint32_t c, uint32_t m, uint64_t* start,
                           uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                           uint32_t epoch, Ctrl* ctrl, hipStream_t st) {
  tlc_zre_index_kernel<<<ntiles, kThreads, 0, st>>>(C, c, m, start, status, ticket_base, epoch,
                                                    ctrl);
  return hipGetLastError();
}

hipError_t launch_expand_dequant(const uint8_t* C, uint32_t c, const uint64_t* start,
                                 uint64_t n, uint64_t m, float scale, float* out,
                                 int accumulate, uint32_t epoch, const Ctrl* ctrl,
                                 hipStream_t st) {
  const bool vec = (m % 4 == 0) && aligned16(out);
  const uint32_t blocks = (uint32_t)((m + kDecRange - 1) / kDecRange);
#define TLC_LAUNCH(V, A)                                                                     \
  tlc_expand_dequant_kernel<V, A><<<blocks, kThreads, 0, st>>>(C, c, start, n, m, scale, out, \
                                                               epoch, ctrl)
  if (vec) {
    if (accumulate) TLC_LAUNCH(true, true); else TLC_LAUNCH(true, false);
  } else {
    if (accumulate) TLC_LAUNCH(false, true); else TLC_LAUNCH(false, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

}  // namespace tlc
