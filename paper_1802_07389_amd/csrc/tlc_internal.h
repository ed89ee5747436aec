// tlc_internal.h -- definitions shared by the kernels and the host side of
// the library (not part of the public ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tlc.h"

namespace tlc {

constexpr int kThreads = 256;             // every kernel: 4 wave64 per block
constexpr int kZreBytesPerThread = 64;    // zero-run index scan: four uint4 per thread
constexpr int kZreTile = kThreads * kZreBytesPerThread;  // 16384 stream bytes per tile
// the batched scans, over many streams that mostly fit one tile, and the
// index role of the single-launch decode take half as many bytes per
// thread (shorter per-thread loops on short streams; the fused decode
// kernel then stays within the expanding blocks' 64 registers)
constexpr int kZreBatchBytesPerThread = 32;
constexpr int kZreBatchTile = kThreads * kZreBatchBytesPerThread;  // 8192
constexpr int kEncTile = 4096;            // quartic bytes per encoder tile
constexpr int kDecRange = 4096;           // quartic bytes per expand/dequantize block
constexpr uint32_t kAbsmaxMaxBlocks = 256;  // partial maxima per encode (one block per CU)
// Tensors of at least this many encoder tiles take the three-pass encoder
// (no waits between tiles); smaller ones the single chained pass.
constexpr uint32_t kThreePassMinTiles = 512;

// Per-tensor encode result (device), written by the encoder's tiles.
struct EncResult {
  uint32_t err;    // 1: NaN/Inf in tensor + residual, or max*s overflow
  uint32_t len;    // zero-run stream length
  float scale;     // M
  uint32_t reserved;
};

// Device control block (one per context, in the workspace).  The first 32
// bytes are copied to pinned host memory by tlc_sync and after the encodes
// whose kernels do not write their result there themselves (HostMirror).
struct Ctrl {
  EncResult enc;           // single-tensor encode result
  uint32_t fault;          // sticky: a look-back wait timed out
  uint32_t dec_corrupt;    // sticky: a decoded stream had the wrong length
  uint32_t dec_bad_epoch;  // epoch of the last decode launch with a bad stream
  uint32_t enc_ticket;     // tile tickets of the encoder
  uint32_t dec_ticket;     // tile tickets of the zero-run index scan
  uint32_t dec_verdict;    // epoch << 1 | bad of the last single-stream decode's stream
  uint32_t chunk_done;     // blocks of the tile-chunk pass done (0 between calls)
  uint32_t pad[53];
};
static_assert(sizeof(Ctrl) == 256, "Ctrl is one 256-byte slot");

struct HostReadback {
  EncResult enc;
  uint32_t fault;
  uint32_t dec_corrupt;
  uint32_t pad[2];
};

// Device pointers into the pinned host readback that the encoders (and the
// decoders, for the fault and bad-stream flags) also write a call's result to,
// so that the host needs no copy before it reads it; null: not mirrored.
// res: the result (one per tensor of a batch); fault: the look-back fault
// flag; corrupt: the decoder's sticky bad-stream flag.
struct HostMirror {
  EncResult* res = nullptr;
  uint32_t* fault = nullptr;
  uint32_t* corrupt = nullptr;
};

// One tensor of a batched encode (device copy of the host's description).
struct EncDesc {
  const float* x;
  float* r;
  uint8_t* out;
  uint64_t n;
  uint32_t m;
  float s;
  uint32_t tile0;  // first encoder tile (global tile numbering of the launch)
  uint32_t blk0;   // first absmax block / partial maximum of this tensor
  uint32_t nblk;   // absmax blocks of this tensor
  uint32_t vec;    // bit 0: m % 4 == 0 and r 16-byte aligned; bit 1: r aligned;
                   // bit 2: x and r aligned (float4 accumulation)
  uint32_t pad[2];
};
static_assert(sizeof(EncDesc) == 64, "EncDesc is 64 bytes");

// Per-tile record of the single-tensor encoder's first pass: the zero-run
// summary of the whole tile (RunSum bits), the length of its leading run of
// 121 bytes, how many bytes it wrote into its slot (its encoding from the
// first non-121 byte on), and how many residuals it left in its fix list.
struct TileRec {
  uint64_t agg;
  uint16_t lead;  // <= kEncTile
  uint16_t len;   // <= kEncTile
  uint32_t nfix;  // <= kFixCap
};
static_assert(sizeof(TileRec) == 16, "TileRec is 16 bytes");

// Residuals with q != 0 that a first-pass tile of the float4 path leaves to
// the compaction pass, as (k * kEncTile + position in the tile, value
// bits): a few scattered stores cost far less in a pass of their own than
// mixed into the first pass's read stream.  Further ones are stored at once.
constexpr uint32_t kFixCap = 256;
static_assert(sizeof(TileRec) == 16, "TileRec is 16 bytes");

// One stream of a batched decode or of a decode-sum.
struct DecDesc {
  const uint8_t* C;
  float* out;      // batched decode: this stream's output (decode-sum: unused)
  uint64_t n;
  uint32_t c;
  uint32_t m;
  float scale;
  uint32_t tile0;   // first index-scan tile (global numbering of the launch)
  uint32_t range0;  // first start-index entry / expand block of this stream
  uint32_t vec;     // 1: m % 4 == 0 and out 16-byte aligned; 2: only out aligned
  uint32_t pad[4];
};
static_assert(sizeof(DecDesc) == 64, "DecDesc is 64 bytes");

// Kernel launches of the library.  While tlc_profile_* times a launcher
// (timed_launch), g_launch_events holds its event pair: the first kernel
// the launcher dispatches takes the start event and every kernel the stop
// event (the last one's stands), recorded by the dispatches themselves
// (hipExtLaunchKernelGGL), so timing adds no marker packets between
// kernels.  Untimed launches are plain launches.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

template <class... Formals, class... Args>
inline void launch_k(void (*kernel)(Formals...), dim3 grid, dim3 block, hipStream_t st,
                     Args... args) {
  LaunchEvents& ev = g_launch_events;
  if (ev.start || ev.stop) {
    hipEvent_t a = ev.start;
    ev.start = nullptr;
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, a, ev.stop, 0, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
  }
}

// Launchers (encode.hip, decode.hip, int8.hip).  All return the hipError_t of the
// launch.
// The check pass: partial maxima of |x + r|, nothing written.
hipError_t launch_absmax_check(const float* x, const float* r, uint64_t n, uint32_t* partials,
                               uint32_t* nblocks, hipStream_t st);
// summ (may be NULL): per float4 of r, the top half of its largest |acc|;
// only written on the float4 path (x and r 16-byte aligned).  guard (may
// be NULL): the check pass's guard_np partial maxima; if they give a bad
// scale (with s), nothing is written and the partials mark the tensor bad.
// trit: after the check pass (guard) on the float4 path, the pass quantizes
// every value (final residuals in r, 2-bit trits in summ, one byte per
// float4) and launch_quant_encode(trit) only packs the trits.
hipError_t launch_accum_absmax(const float* x, float* r, uint64_t n,
                               uint32_t* partials, uint32_t* nblocks, uint16_t* summ,
                               const uint32_t* guard, uint32_t guard_np, float s, bool trit,
                               hipStream_t st);
hipError_t launch_quant_encode(float* r, uint64_t n, uint32_t m, float s,
                               const uint32_t* partials, uint32_t npartials, uint8_t* slots,
                               TileRec* recs, uint2* fix, const uint16_t* summ, bool trit,
                               Ctrl* ctrl, HostMirror hm, hipStream_t st);
// x != NULL: the tiles form acc = x + r themselves from the check pass's
// partials (r still holds the previous residual); x == NULL: r holds acc.
hipError_t launch_quant_encode_chained(const float* x, float* r, uint64_t n, uint32_t m,
                                       float s, const uint32_t* partials, uint32_t npartials,
                                       uint8_t* out, uint64_t* status, uint32_t ntiles,
                                       uint32_t ticket_base, uint32_t epoch, Ctrl* ctrl,
                                       HostMirror hm, hipStream_t st);
hipError_t launch_zre_chunks(const TileRec* recs, uint32_t ntiles, uint64_t* local_pre,
                             uint64_t* chunk_agg, Ctrl* ctrl, hipStream_t st);
hipError_t launch_zre_compact(const TileRec* recs, const uint64_t* chunk_pre,
                              const uint64_t* local_pre, const uint8_t* slots, uint32_t m,
                              uint8_t* out, const uint2* fix, float* r, uint64_t n, Ctrl* ctrl,
                              HostMirror hm, hipStream_t st);
hipError_t launch_quant_pack(const float* x, float* r, uint64_t n, uint32_t m, float s,
                             int stochastic, uint64_t seed, uint64_t step,
                             const uint32_t* partials, uint32_t npartials, uint8_t* out,
                             Ctrl* ctrl, hipStream_t st);
hipError_t launch_int8_quant(const float* x, float* r, uint64_t n, float s,
                             const uint32_t* partials, uint32_t npartials, uint8_t* out,
                             Ctrl* ctrl, hipStream_t st);
hipError_t launch_int8_dequant(const uint8_t* C, uint64_t n, float M, float* out,
                               int accumulate, hipStream_t st);
hipError_t launch_absmax_check_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_blocks, uint32_t* partials, hipStream_t st);
hipError_t launch_accum_absmax_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_blocks, uint32_t* partials,
                                     const uint32_t* guard, hipStream_t st);
// fused: as x != NULL for the chained encoder (partials: the check pass's).
hipError_t launch_quant_encode_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_tiles, const uint32_t* partials,
                                     bool fused, EncResult* results, uint64_t* status,
                                     uint32_t ticket_base, uint32_t epoch, Ctrl* ctrl,
                                     HostMirror hm, hipStream_t st);
// One stream's decode.  Small decodes (at most kFusedMaxBlocks blocks in
// all, so every block is resident at once) run in one launch: the first
// blocks scan the stream (kZreBatchTile bytes each), the others expand.
// Larger ones run the scan (kZreTile bytes per block), then the expansion:
// thousands of expanding blocks waiting inside one launch for a scan of
// hundreds of tiles slowed it down more than the launch boundary costs.
constexpr uint32_t kFusedMaxBlocks = 256;
inline uint32_t decode_ranges(uint64_t m) { return (uint32_t)((m + kDecRange - 1) / kDecRange); }
inline bool decode_fused(uint64_t c, uint64_t m) {
  return (c + kZreBatchTile - 1) / kZreBatchTile + decode_ranges(m) <= kFusedMaxBlocks;
}
// The scan's tiles; the tickets a decode takes (the host advances the
// decoder's ticket base by decode_tickets(c, m)).
inline uint32_t decode_index_tiles(uint64_t c, uint64_t m) {
  const uint64_t tile = decode_fused(c, m) ? kZreBatchTile : kZreTile;
  return (uint32_t)((c + tile - 1) / tile);
}
inline uint32_t decode_tickets(uint64_t c, uint64_t m) {
  return decode_index_tiles(c, m) + (decode_fused(c, m) ? decode_ranges(m) : 0u);
}
// The scan of one stream (not decode_fused), then its expansion; or, when
// decode_fused, both in the expansion's launch (ticket_base then counts
// the scan's tiles too).
hipError_t launch_zre_index(const uint8_t* C, uint32_t c, uint32_t m, uint64_t* start,
                            uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                            uint32_t epoch, Ctrl* ctrl, HostMirror hm, hipStream_t st);
hipError_t launch_expand_dequant(const uint8_t* C, uint32_t c, uint64_t* start,
                                 uint64_t* status, uint32_t ticket_base, uint64_t n, uint64_t m,
                                 float scale, float* out, int accumulate, uint32_t epoch,
                                 Ctrl* ctrl, HostMirror hm, hipStream_t st);
hipError_t launch_zre_index_batch(const DecDesc* descs, uint32_t count, uint32_t total_tiles,
                                  uint64_t* start, uint64_t* status, uint32_t ticket_base,
                                  uint32_t epoch, Ctrl* ctrl, HostMirror hm, hipStream_t st);
hipError_t launch_expand_dequant_batch(const DecDesc* descs, uint32_t count,
                                       uint32_t total_ranges, const uint64_t* start,
                                       int accumulate, uint32_t epoch, const Ctrl* ctrl,
                                       hipStream_t st);
hipError_t launch_expand_sum(const DecDesc* descs, uint32_t count, const uint64_t* start,
                             uint64_t n, uint64_t m, float* out, int vec, int accumulate,
                             uint32_t epoch, const Ctrl* ctrl, hipStream_t st);

// Epoch widths of the two look-back status layouts.
constexpr uint32_t kEncEpochMax = (1u << 23) - 1u;
constexpr uint32_t kDecEpochMax = (1u << 26) - 1u;
static_assert(kEncEpochMax == TLC_ENC_EPOCH_MAX && kDecEpochMax == TLC_DEC_EPOCH_MAX,
              "the header states the epoch maxima");

// Sets the calling thread's error text (tlc_last_error_string) and returns
// code.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

}  // namespace tlc
