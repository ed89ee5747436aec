// wave_scan.hpp -- scans across the 64 lanes of a wavefront on the lane
// moves of gfx950's data-parallel primitives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tlc {

// Lane moves of the data-parallel primitives (DPP) of GFX9 parts, which
// stay in the vector ALU instead of a round trip through the LDS crossbar
// (ds_bpermute): row_shr:k hands lane i - k of the same 16-lane row to lane
// i, row_bcast:15 the last lane of each row to the whole next row,
// row_bcast:31 lane 31 to rows 2 and 3, wave_shr:1 lane i - 1 to lane i.
// A lane whose source lies outside its row (or the wave), or whose row is
// not in the row mask, gets `old` instead.  Every lane of the wave must be
// active.
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppWaveShr1 = 0x138;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_mov(uint64_t old, uint64_t v) {
  return (uint64_t)dpp_mov<kCtrl, kRowMask>((uint32_t)old, (uint32_t)v) |
         ((uint64_t)dpp_mov<kCtrl, kRowMask>((uint32_t)(old >> 32), (uint32_t)(v >> 32)) << 32);
}

// Inclusive scan in lane order under an associative op with identity e,
// op(a, b) being segment a followed by segment b: doubling shifts inside
// each row, then the rows' totals carried to the rows after them.
template <class T, class Op>
__device__ __forceinline__ T wave_incl_scan(T x, T e, Op op) {
  x = op(dpp_mov<kDppRowShr1, 0xf>(e, x), x);
  x = op(dpp_mov<kDppRowShr2, 0xf>(e, x), x);
  x = op(dpp_mov<kDppRowShr4, 0xf>(e, x), x);
  x = op(dpp_mov<kDppRowShr8, 0xf>(e, x), x);
  x = op(dpp_mov<kDppRowBcast15, 0xa>(e, x), x);
  x = op(dpp_mov<kDppRowBcast31, 0xc>(e, x), x);
  return x;
}

// Lane i - 1's value (e in lane 0): an inclusive scan made exclusive.
template <class T>
__device__ __forceinline__ T wave_prev_lane(T x, T e) {
  return dpp_mov<kDppWaveShr1, 0xf>(e, x);
}

// Lane 63's value, the same in every lane.
__device__ __forceinline__ uint32_t wave_last(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

struct OpAdd {
  __device__ __forceinline__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; }
};
struct OpMax {
  __device__ __forceinline__ uint32_t operator()(uint32_t a, uint32_t b) const {
    return a > b ? a : b;
  }
};

}  // namespace tlc
