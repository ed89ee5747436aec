// lookback.hpp -- status words for single-pass decoupled look-back scans on
// a multi-XCD gfx950.
//
// Each tile owns one 64-bit status word holding
//   payload (low bits) | flag << kFlagShift | epoch << kEpochShift
// with flag 1 = the tile's own aggregate, 2 = inclusive prefix, 3 = a
// predecessor gave up (look-back fault; successors give up too).  The epoch
// is a per-launch tag, so words left by earlier launches never match and
// the array needs no clearing between launches; the host clears it when
// the epoch counter wraps.
//
// The L2 caches of the eight XCDs are not coherent with each other, so
// status words are only touched with agent-scope atomics.  Tiles are taken
// in order from an atomic ticket, so a tile only ever waits for tiles that
// already run, and every wait is bounded (kSpinLimit) so each wave exits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tlc {

constexpr uint32_t kFlagAgg = 1u;
constexpr uint32_t kFlagPrefix = 2u;
constexpr uint32_t kFlagFault = 3u;
constexpr uint32_t kSpinLimit = 1u << 22;

template <int PayloadBits>
struct StatusWord {
  static constexpr int kFlagShift = PayloadBits;
  static constexpr int kEpochShift = PayloadBits + 2;
  static constexpr int kEpochBits = 64 - kEpochShift;
  static constexpr uint64_t kPayloadMask = (uint64_t(1) << PayloadBits) - 1u;
  static constexpr uint32_t kEpochMask = (uint32_t)((uint64_t(1) << kEpochBits) - 1u);

  __device__ static uint64_t pack(uint64_t payload, uint32_t flag, uint32_t epoch) {
    return (payload & kPayloadMask) | ((uint64_t)flag << kFlagShift) |
           ((uint64_t)epoch << kEpochShift);
  }
  __device__ static uint64_t payload(uint64_t w) { return w & kPayloadMask; }
  __device__ static uint32_t flag(uint64_t w) { return (uint32_t)(w >> kFlagShift) & 3u; }
  __device__ static uint32_t epoch(uint64_t w) { return (uint32_t)(w >> kEpochShift); }
};

__device__ __forceinline__ void status_publish(uint64_t* p, uint64_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t status_read(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_ACQUIRE,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t take_ticket(uint32_t* counter) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

// Single-thread look-back for tile `tile` (> 0) over an associative
// operator op(earlier, later).  Publishes the aggregate, folds predecessor
// words until an inclusive prefix is found, publishes the tile's inclusive
// prefix and returns the exclusive prefix.  On a bounded-wait timeout or a
// predecessor fault it publishes a fault word and sets *fault.
template <class SW, class Op>
__device__ uint64_t lookback_exclusive(uint64_t* status, uint32_t tile,
                                       uint64_t agg, uint64_t identity,
                                       uint32_t epoch, Op op, bool* fault) {
  status_publish(&status[tile], SW::pack(agg, kFlagAgg, epoch));
  uint64_t run = identity;
  uint32_t i = tile - 1u;
  uint32_t spins = 0;
  for (;;) {
    uint64_t w = status_read(&status[i]);
    uint32_t f = SW::flag(w);
    if (SW::epoch(w) != epoch || f == 0u) {
      if (++spins > kSpinLimit) {
        *fault = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    if (f == kFlagFault) {
      *fault = true;
      break;
    }
    run = op(SW::payload(w), run);
    if (f == kFlagPrefix) break;
    --i;  // an aggregate word never belongs to tile 0, so i stays >= 0
  }
  if (*fault) {
    status_publish(&status[tile], SW::pack(0, kFlagFault, epoch));
    return identity;
  }
  status_publish(&status[tile], SW::pack(op(run, agg), kFlagPrefix, epoch));
  return run;
}

}  // namespace tlc
