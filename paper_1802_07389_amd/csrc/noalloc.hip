// noalloc.hip -- tlc_compress_noalloc: the encode of tlc_compress for
// callers that cannot allocate device memory (graph capture, serving
// loops, harnesses that forbid hipMalloc).  It runs the kernels of the
// small-tensor path (check pass, then the chained pass that accumulates,
// quantizes, packs and zero-run encodes; Sections 3.1-3.3) with their
// scratch in a file-scope device array instead of a context's workspace.
#include <mutex>

#include "tlc.h"
#include "tlc_internal.h"

#define TLC_API extern "C" __attribute__((visibility("default")))

namespace tlc {
namespace {

// Scratch layout: the control block (tile ticket, encode result, fault
// flag), the check pass's partial maxima (at most kAbsmaxMaxBlocks; the
// next kAbsmaxMaxBlocks words are spare), then one look-back status word
// per encoder tile
// (n <= TLC_NOALLOC_MAX_N gives at most 410 tiles, all on the chained
// path) and two spare words.
constexpr uint32_t kNoallocMaxTiles =
    (uint32_t)(((TLC_NOALLOC_MAX_N + 4) / 5 + kEncTile - 1) / kEncTile);
static_assert(kNoallocMaxTiles < kThreePassMinTiles, "the chained path takes every size");
constexpr size_t kOffPartialsChk = sizeof(Ctrl);
constexpr size_t kOffPartials = kOffPartialsChk + kAbsmaxMaxBlocks * sizeof(uint32_t);
constexpr size_t kOffStatus = kOffPartials + kAbsmaxMaxBlocks * sizeof(uint32_t);
constexpr size_t kStatusWords = kNoallocMaxTiles + 2;
constexpr size_t kScratchBytes = 8192;  // the size the header states
static_assert(kOffStatus + kStatusWords * sizeof(uint64_t) <= kScratchBytes, "layout fits");

// In host code `scratch` names a host-side stand-in; its device address
// comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
uint8_t* g_scratch[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Zeroes the control block and the first `words` status words (every call
// starts from a cleared scratch: tile ticket 0, no fault, epoch 1 matches
// no word) and writes an empty result (the whole answer when n == 0).
__global__ __launch_bounds__(kThreads) void tlc_noalloc_begin_kernel(
    uint8_t* __restrict__ scr, uint32_t words, tlc_result* __restrict__ res) {
  uint32_t* ctrl = reinterpret_cast<uint32_t*>(scr);
  for (uint32_t i = threadIdx.x; i < sizeof(Ctrl) / sizeof(uint32_t); i += kThreads) ctrl[i] = 0u;
  uint64_t* status = reinterpret_cast<uint64_t*>(scr + kOffStatus);
  for (uint32_t i = threadIdx.x; i < words; i += kThreads) status[i] = 0u;
  if (threadIdx.x == 0) {
    res->status = TLC_OK;
    res->bytes_len = 0u;
    res->scale = 0.0f;
    res->reserved = 0u;
  }
}

// Copies the encode's outcome from the control block into the result.
__global__ __launch_bounds__(64) void tlc_noalloc_end_kernel(const uint8_t* __restrict__ scr,
                                                             tlc_result* __restrict__ res) {
  if (threadIdx.x != 0) return;
  const Ctrl* c = reinterpret_cast<const Ctrl*>(scr);
  const bool fault = c->fault != 0u;
  const bool bad = c->enc.err != 0u;
  res->status = fault ? TLC_E_DEVICE : (bad ? TLC_E_NONFINITE : TLC_OK);
  res->bytes_len = (fault || bad) ? 0u : c->enc.len;
  res->scale = (fault || bad) ? 0.0f : c->enc.scale;
  res->reserved = 0u;
}

bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return an && bn && pa < pb + bn && pb < pa + an;
}

}  // namespace
}  // namespace tlc

using namespace tlc;

TLC_API int tlc_compress_noalloc(const float* tensor, float* residual, size_t n, float s,
                                 uint8_t* bytes, size_t bytes_cap, tlc_result* result,
                                 void* hip_stream) {
  if (!result) return fail(TLC_E_INVALID, "tlc_compress_noalloc: NULL result");
  if (!(s >= 1.0f && s < 2.0f))
    return fail(TLC_E_INVALID, "tlc_compress_noalloc: s = %g not in [1, 2)", (double)s);
  if (n > TLC_NOALLOC_MAX_N)
    return fail(TLC_E_INVALID, "tlc_compress_noalloc: n = %zu exceeds TLC_NOALLOC_MAX_N = %zu",
                n, (size_t)TLC_NOALLOC_MAX_N);
  const size_t m = n / 5 + (n % 5 ? 1 : 0);
  if (n) {
    if (!tensor || !residual || !bytes)
      return fail(TLC_E_INVALID, "tlc_compress_noalloc: NULL device pointer");
    if (bytes_cap < m)
      return fail(TLC_E_CAPACITY, "tlc_compress_noalloc: bytes_cap %zu < %zu", bytes_cap, m);
    if (overlap(tensor, n * 4, residual, n * 4) || overlap(tensor, n * 4, bytes, m) ||
        overlap(residual, n * 4, bytes, m) || overlap(result, sizeof(tlc_result), tensor, n * 4) ||
        overlap(result, sizeof(tlc_result), residual, n * 4) ||
        overlap(result, sizeof(tlc_result), bytes, m))
      return fail(TLC_E_INVALID, "tlc_compress_noalloc: tensor, residual, bytes and result overlap");
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return fail(TLC_E_DEVICE, "tlc_compress_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(TLC_E_DEVICE, "tlc_compress_noalloc: device %d not supported", dev);
  // once per device, with that device current: the device copy's address
  std::call_once(g_once[dev], [dev] {
    g_scratch_err[dev] = hipGetSymbolAddress((void**)&g_scratch[dev], HIP_SYMBOL(scratch));
  });
  if (g_scratch_err[dev] != hipSuccess)
    return fail(TLC_E_DEVICE, "tlc_compress_noalloc: hipGetSymbolAddress: %s",
                hipGetErrorString(g_scratch_err[dev]));
  uint8_t* scr = g_scratch[dev];
  Ctrl* ctrl = reinterpret_cast<Ctrl*>(scr);
  uint32_t* partials_chk = reinterpret_cast<uint32_t*>(scr + kOffPartialsChk);
  uint64_t* status = reinterpret_cast<uint64_t*>(scr + kOffStatus);
  hipStream_t st = (hipStream_t)hip_stream;
  const uint32_t ntiles = (uint32_t)((m + kEncTile - 1) / kEncTile);  // <= kNoallocMaxTiles

  tlc_noalloc_begin_kernel<<<1, kThreads, 0, st>>>(scr, ntiles + 2u, result);
  e = hipGetLastError();
  if (e == hipSuccess && n) {
    uint32_t np = 0;
    e = launch_absmax_check(tensor, residual, n, partials_chk, &np, st);
    if (e == hipSuccess)
      e = launch_quant_encode_chained(tensor, residual, n, (uint32_t)m, s, partials_chk, np,
                                      bytes, status, ntiles, 0u, 1u, ctrl, HostMirror{}, st);
    if (e == hipSuccess) {
      tlc_noalloc_end_kernel<<<1, 64, 0, st>>>(scr, result);
      e = hipGetLastError();
    }
  }
  if (e != hipSuccess)
    return fail(TLC_E_DEVICE, "tlc_compress_noalloc: launch: %s", hipGetErrorString(e));
  return TLC_OK;
}
