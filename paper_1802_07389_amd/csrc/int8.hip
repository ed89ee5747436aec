// int8.hip -- gfx950 kernels of the 8-bit integer comparator (the "8-bit
// int" design of Section 5.1): 255 codes -127..127 at one step D = M / 127
// per tensor, M from Eq. 1.
//
//   tlc_int8_quant_kernel    code = rint(acc / D) clamped to [-127, 127]
//                            (0 when D == 0), residual acc - code * D,
//                            one int8 byte per value; acc is the buffer
//                            that tlc_accum_absmax_kernel has accumulated
//                            (error feedback) or the tensor itself
//   tlc_int8_dequant_kernel  out = code * D, or out + code * D
//
// Both are elementwise streams: a block covers kI8Rows rows of 1024 values;
// in a row lane t owns values 4t .. 4t + 3 (one float4 per tensor and one
// 32-bit word of codes), so every load and store instruction of a wave is
// one contiguous span.  Divides, products and sums use the _rn intrinsics,
// so each is one IEEE operation rounded to nearest even, as in the
// definition.
#include "device_common.hpp"

namespace tlc {

constexpr int kI8Rows = 16;                    // rows per block
constexpr uint32_t kI8Row = kThreads * 4u;     // values per row
constexpr int kI8Batch = 4;                    // rows whose loads are in flight together

__device__ __forceinline__ float int8_step(float M) { return __fdiv_rn(M, 127.0f); }

// Code of one accumulated value, as a float holding an integer in
// [-127, 127].
__device__ __forceinline__ float int8_code(float acc, float D) {
  if (!(D > 0.0f)) return 0.0f;
  const float v = rintf(__fdiv_rn(acc, D));
  return fminf(fmaxf(v, -127.0f), 127.0f);
}

__device__ __forceinline__ uint32_t int8_byte(float code) {
  return (uint32_t)(int32_t)code & 0xffu;
}

// Value of one byte: fl(code * D) (code 0 gives +0).
__device__ __forceinline__ float int8_value(uint32_t byte, float D) {
  return __fmul_rn((float)(int32_t)(int8_t)(uint8_t)byte, D);
}

// out + fl(code * D), densely (code 0 adds +0).
__device__ __forceinline__ float int8_acc(float out, uint32_t byte, float D) {
  return __fadd_rn(out, int8_value(byte, D));
}

// One value: code byte and (kResid) residual acc - fl(code * D).  The
// product is taken from the integer code: rint leaves -0.0 for acc = -0.0,
// whose product -0 would turn the residual -0.0 - (-0) into +0.0, while
// the integer 0 gives +0 and keeps acc = -0.0 as its residual.
template <bool kResid>
__device__ __forceinline__ uint32_t int8_one(float acc, float D, float& res) {
  const float code = int8_code(acc, D);
  if (kResid) res = __fsub_rn(acc, __fmul_rn((float)(int32_t)code, D));
  return int8_byte(code);
}

// kVec: the values read (r or x) 16-byte aligned, out 4-byte aligned.
// kResid: error feedback, acc = r (already x + r) and r is rewritten, x is
// unused; otherwise acc = x and r is unused.
template <bool kVec, bool kResid>
__global__ __launch_bounds__(kThreads) void tlc_int8_quant_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n, float s,
    const uint32_t* __restrict__ partials, uint32_t np, uint8_t* __restrict__ out,
    Ctrl* __restrict__ ctrl) {
  __shared__ uint32_t red[kWaves];
  const Scale sc = finish_scale(partials, np, s, red);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctrl->enc.err = sc.bad;
    ctrl->enc.scale = sc.M;
    ctrl->enc.len = sc.bad ? 0u : (uint32_t)n;
  }
  if (sc.bad) return;  // NaN/Inf or overflow: no bytes, the buffer keeps acc
  const float D = int8_step(sc.M);
  const uint64_t base = (uint64_t)blockIdx.x * kI8Row * kI8Rows;
  const float* __restrict__ src = kResid ? r : x;
  if (kVec) {
#pragma unroll 1
    for (int h = 0; h < kI8Rows; h += kI8Batch) {
      float4 a[kI8Batch];
      bool full[kI8Batch];
#pragma unroll
      for (int i = 0; i < kI8Batch; ++i) {
        const uint64_t e = base + (uint64_t)(h + i) * kI8Row + 4u * threadIdx.x;
        full[i] = e + 4u <= n;
        if (full[i]) a[i] = ld_stream(src + e);
      }
#pragma unroll
      for (int i = 0; i < kI8Batch; ++i) {
        const uint64_t e = base + (uint64_t)(h + i) * kI8Row + 4u * threadIdx.x;
        if (full[i]) {
          float4 o;
          const uint32_t w = int8_one<kResid>(a[i].x, D, o.x) |
                             int8_one<kResid>(a[i].y, D, o.y) << 8 |
                             int8_one<kResid>(a[i].z, D, o.z) << 16 |
                             int8_one<kResid>(a[i].w, D, o.w) << 24;
          if (kResid) st_stream(r + e, o);
          *reinterpret_cast<uint32_t*>(out + e) = w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if (e + c < n) {
              float o = 0.0f;
              out[e + c] = (uint8_t)int8_one<kResid>(src[e + c], D, o);
              if (kResid) r[e + c] = o;
            }
          }
        }
      }
    }
  } else {
    for (uint32_t k = threadIdx.x; k < kI8Row * kI8Rows; k += kThreads) {
      const uint64_t e = base + k;
      if (e >= n) break;
      float o = 0.0f;
      out[e] = (uint8_t)int8_one<kResid>(src[e], D, o);
      if (kResid) r[e] = o;
    }
  }
}

// kVec: C 4-byte aligned, out 16-byte aligned.
template <bool kVec, bool kAcc>
__global__ __launch_bounds__(kThreads) void tlc_int8_dequant_kernel(
    const uint8_t* __restrict__ C, uint64_t n, float M, float* __restrict__ out) {
  const float D = int8_step(M);
  const uint64_t base = (uint64_t)blockIdx.x * kI8Row * kI8Rows;
  if (kVec) {
#pragma unroll 1
    for (int h = 0; h < kI8Rows; h += kI8Batch) {
      uint32_t w[kI8Batch];
      float4 o[kI8Batch];
      bool full[kI8Batch];
#pragma unroll
      for (int i = 0; i < kI8Batch; ++i) {
        const uint64_t e = base + (uint64_t)(h + i) * kI8Row + 4u * threadIdx.x;
        full[i] = e + 4u <= n;
        if (full[i]) {
          w[i] = *reinterpret_cast<const uint32_t*>(C + e);
          if (kAcc) o[i] = ld_stream(out + e);
        }
      }
#pragma unroll
      for (int i = 0; i < kI8Batch; ++i) {
        const uint64_t e = base + (uint64_t)(h + i) * kI8Row + 4u * threadIdx.x;
        if (full[i]) {
          float4 res;
          if (kAcc) {
            res = make_float4(int8_acc(o[i].x, w[i], D), int8_acc(o[i].y, w[i] >> 8, D),
                              int8_acc(o[i].z, w[i] >> 16, D), int8_acc(o[i].w, w[i] >> 24, D));
          } else {
            res = make_float4(int8_value(w[i], D), int8_value(w[i] >> 8, D),
                              int8_value(w[i] >> 16, D), int8_value(w[i] >> 24, D));
          }
          st_stream(out + e, res);
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if (e + c < n)
              out[e + c] = kAcc ? int8_acc(out[e + c], C[e + c], D) : int8_value(C[e + c], D);
          }
        }
      }
    }
  } else {
    for (uint32_t k = threadIdx.x; k < kI8Row * kI8Rows; k += kThreads) {
      const uint64_t e = base + k;
      if (e >= n) break;
      out[e] = kAcc ? int8_acc(out[e], C[e], D) : int8_value(C[e], D);
    }
  }
}

// ---------------------------------------------------------------- launchers
namespace {
inline bool aligned(const void* p, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(p) & (a - 1u)) == 0u;
}
inline uint32_t int8_blocks(uint64_t n) {
  const uint64_t per = (uint64_t)kI8Row * kI8Rows;
  return (uint32_t)((n + per - 1) / per);
}
}  // namespace

hipError_t launch_int8_quant(const float* x, float* r, uint64_t n, float s,
                             const uint32_t* partials, uint32_t npartials, uint8_t* out,
                             Ctrl* ctrl, hipStream_t st) {
  const uint32_t blocks = int8_blocks(n);
  const bool vec = aligned(r ? r : x, 16) && aligned(out, 4);
  if (r) x = nullptr;  // the buffer already holds x + r
#define TLC_LAUNCH(V, R)                                                                 \
  launch_k(tlc_int8_quant_kernel<V, R>, blocks, kThreads, st, x, r, n, s, partials, npartials, \
                                                           out, ctrl)
  if (r) {
    if (vec) TLC_LAUNCH(true, true); else TLC_LAUNCH(false, true);
  } else {
    if (vec) TLC_LAUNCH(true, false); else TLC_LAUNCH(false, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

hipError_t launch_int8_dequant(const uint8_t* C, uint64_t n, float M, float* out,
                               int accumulate, hipStream_t st) {
  const uint32_t blocks = int8_blocks(n);
  const bool vec = aligned(C, 4) && aligned(out, 16);
#define TLC_LAUNCH(V, A) launch_k(tlc_int8_dequant_kernel<V, A>, blocks, kThreads, st, C, n, M, out)
  if (accumulate) {
    if (vec) TLC_LAUNCH(true, true); else TLC_LAUNCH(false, true);
  } else {
    if (vec) TLC_LAUNCH(true, false); else TLC_LAUNCH(false, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

}  // namespace tlc
