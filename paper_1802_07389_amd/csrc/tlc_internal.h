// tlc_internal.h -- definitions shared by the kernels and the host side of
// the library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tlc {

constexpr int kThreads = 256;             // every kernel: 4 wave64 per block
constexpr int kZreBytesPerThread = 32;    // zero-run scans: two uint4 per thread
constexpr int kZreTile = kThreads * kZreBytesPerThread;  // 8192 bytes per tile
constexpr int kEncTile = 4096;            // quartic bytes per encoder tile
constexpr int kDecRange = 4096;           // quartic bytes per expand/dequantize block
constexpr uint32_t kAbsmaxMaxBlocks = 512;  // partial maxima per encode

// Device control block (one per context, in the workspace).  The first 16
// bytes are copied to pinned host memory after every encode.
struct Ctrl {
  uint32_t enc_err;        // 1 if the last encode saw NaN/Inf or overflow
  uint32_t enc_len;        // zero-run stream length of the last encode
  float enc_scale;         // M of the last encode
  uint32_t fault;          // sticky: a look-back wait timed out
  uint32_t dec_corrupt;    // sticky: a decoded stream had the wrong length
  uint32_t dec_bad_epoch;  // epoch of the last decode whose stream was bad
  uint32_t enc_ticket;     // tile tickets of the zero-run encoder
  uint32_t dec_ticket;     // tile tickets of the zero-run decoder
  uint32_t pad[56];
};
static_assert(sizeof(Ctrl) == 256, "Ctrl is one 256-byte slot");

struct HostReadback {
  uint32_t enc_err;
  uint32_t enc_len;
  float enc_scale;
  uint32_t fault;
  uint32_t dec_corrupt;
  uint32_t pad[3];
};

// Launchers (tlc_kernels.hip).  All return the hipError_t of the launch.
hipError_t launch_absmax(const float* x, const float* r, uint64_t n,
                         uint32_t* partials, uint32_t* nblocks,
                         hipStream_t st);
hipError_t launch_quant_encode(const float* x, float* r, uint64_t n, uint32_t m, float s,
                              const uint32_t* partials, uint32_t npartials, uint8_t* out,
                              uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                              uint32_t epoch, Ctrl* ctrl, hipStream_t st);
hipError_t launch_zre_index(const uint8_t* C, uint32_t c, uint32_t m, uint64_t* start,
                           uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                           uint32_t epoch, Ctrl* ctrl, hipStream_t st);
hipError_t launch_expand_dequant(const uint8_t* C, uint32_t c, const uint64_t* start,
                                 uint64_t n, uint64_t m, float scale, float* out,
                                 int accumulate, uint32_t epoch, const Ctrl* ctrl,
                                 hipStream_t st);

// Epoch widths of the two look-back status layouts.
constexpr uint32_t kEncEpochMax = (1u << 23) - 1u;
constexpr uint32_t kDecEpochMax = (1u << 26) - 1u;

}  // namespace tlc
