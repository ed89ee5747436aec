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

#include "wave_scan.hpp"

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

// The payload lives inside the status word, so no other memory has to be
// made visible with it: relaxed agent-scope atomics are enough and avoid the
// L2 write-back / invalidate that release / acquire imply on gfx950.
//
// Built with TLC_DELAY_INJECT (the stress build of the look-back scans
// only, never the product library), every publish first sleeps for a
// pseudo-random 0 to 7 times 127 * 64 clocks (up to about 25 us), a
// function of the word's address and contents: tiles then publish in a
// scrambled order and their successors see every mix of missing,
// aggregate and prefix words.
__device__ __forceinline__ void status_publish(uint64_t* p, uint64_t w) {
#ifdef TLC_DELAY_INJECT
  uint64_t h = (reinterpret_cast<uintptr_t>(p) ^ (w * 0x9E3779B97F4A7C15ull)) + 0x632BE59BD9B4E019ull;
  h = (h ^ (h >> 31)) * 0xD6E8FEB86659FD93ull;
  for (uint32_t d = (uint32_t)(h >> 61); d > 0u; --d) __builtin_amdgcn_s_sleep(127);
#endif
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t status_read(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t take_ticket(uint32_t* counter) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

// Wave-parallel look-back for tile `tile` (> floor), run by all 64 lanes of
// one wave, over an associative operator op(earlier, later).  Tiles
// [floor, tile) belong to the same scan (a batch keeps several scans in one
// status array); tile `floor` always publishes its inclusive prefix.  Lane l
// polls the word of tile (base - l), so one poll covers 64 predecessors (a
// higher lane holds an earlier tile).  The words from the nearest inclusive
// prefix up to tile - 1 are folded in order by a DPP scan of the lanes under
// op with its arguments swapped, which leaves the fold in lane 63.
// Publishes the tile's aggregate first and its inclusive prefix last;
// returns the exclusive prefix in every lane.  A bounded wait or a
// predecessor fault publishes a fault word and sets *fault.
template <class Op>
struct OpLaterFirst {
  Op op;
  __device__ __forceinline__ uint64_t operator()(uint64_t later, uint64_t earlier) const {
    return op(earlier, later);
  }
};

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  return (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane) |
         ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane) << 32);
}

template <class SW, class Op>
__device__ uint64_t lookback_wave(uint64_t* status, uint32_t floor, uint32_t tile,
                                  uint64_t agg, uint64_t identity, uint32_t epoch, Op op,
                                  bool* fault) {
  const uint32_t lane = threadIdx.x & 63u;
  if (lane == 0) status_publish(&status[tile], SW::pack(agg, kFlagAgg, epoch));
  uint64_t run = identity;
  int64_t base = (int64_t)tile - 1;
  uint32_t spins = 0;
  bool failed = false;
  for (;;) {
    const int64_t idx = base - (int64_t)lane;
    uint64_t val = identity;
    bool ready = true, is_prefix = true, is_fault = false;
    if (idx >= (int64_t)floor) {  // lanes before the scan's first tile act as an (ignored) prefix
      const uint64_t w = status_read(&status[idx]);
      const uint32_t f = SW::flag(w);
      ready = SW::epoch(w) == epoch && f != 0u;
      is_prefix = ready && f == kFlagPrefix;
      is_fault = ready && f == kFlagFault;
      val = SW::payload(w);
    }
    const uint64_t pmask = __ballot(is_prefix);
    const uint32_t p = pmask ? (uint32_t)(__ffsll((unsigned long long)pmask) - 1) : 64u;
    const bool need = lane <= p;  // the nearest prefix and the tiles after it
    if (__ballot(is_fault && need)) {
      failed = true;
      break;
    }
    if (__ballot(!ready && need)) {
      if (++spins > kSpinLimit) {
        failed = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    const uint64_t fold = wave_incl_scan(need ? val : identity, identity, OpLaterFirst<Op>{op});
    run = op(readlane64(fold, 63), run);
    if (p < 64u) break;
    base -= 64;
  }
  *fault = failed;
  if (lane == 0) {
    status_publish(&status[tile], failed ? SW::pack(0, kFlagFault, epoch)
                                         : SW::pack(op(run, agg), kFlagPrefix, epoch));
  }
  return failed ? identity : run;
}

}  // namespace tlc
