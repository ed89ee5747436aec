// tlc_api.hip -- host side of the C ABI declared in include/tlc.h: argument
// checks, the per-context device workspace, kernel launches on the
// context's stream, status readback and optional per-kernel event timing.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <vector>

#include "tlc.h"
#include "tlc_internal.h"

#define TLC_API extern "C" __attribute__((visibility("default")))

using namespace tlc;

namespace {

thread_local char g_err[512] = "no error";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(TLC_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

size_t quartic_len(size_t n) { return n / 5 + (n % 5 ? 1 : 0); }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return an && bn && pa < pb + bn && pb < pa + an;
}

const char* const kKernelNames[TLC_KERNEL_COUNT] = {
    "tlc_absmax_kernel", "tlc_quant_encode_kernel", "tlc_zre_index_kernel",
    "tlc_expand_dequant_kernel"};

struct PendingTiming {
  int kernel;
  hipEvent_t start, stop;
};

}  // namespace

struct tlc_ctx {
  hipStream_t stream = nullptr;
  int device = 0;
  size_t max_n = 0;
  size_t max_m = 0;
  // device workspace (one allocation)
  void* ws = nullptr;
  Ctrl* ctrl = nullptr;
  uint32_t* partials = nullptr;
  uint64_t* enc_status = nullptr;
  uint64_t* dec_status = nullptr;
  uint64_t* start = nullptr;  // per kDecRange quartic bytes: (stream index, skip)
  size_t enc_status_words = 0;
  size_t dec_status_words = 0;
  // pinned host readback
  HostReadback* rb = nullptr;
  // look-back bookkeeping
  uint32_t enc_ticket_base = 0, dec_ticket_base = 0;
  uint32_t enc_epoch = 0, dec_epoch = 0;
  bool broken = false;
  // profiling
  bool profiling = false;
  std::vector<hipEvent_t> free_events;
  std::vector<PendingTiming> pending;
  double total_ms[TLC_KERNEL_COUNT] = {};
  uint64_t launches[TLC_KERNEL_COUNT] = {};
};

namespace {

int ensure_device(tlc_ctx* c) {
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (cur != c->device) {
    e = hipSetDevice(c->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
  }
  return TLC_OK;
}

hipEvent_t take_event(tlc_ctx* c) {
  if (!c->free_events.empty()) {
    hipEvent_t ev = c->free_events.back();
    c->free_events.pop_back();
    return ev;
  }
  hipEvent_t ev = nullptr;
  if (hipEventCreate(&ev) != hipSuccess) return nullptr;
  return ev;
}

// Resolve recorded event pairs; call only after the stream is idle.
void collect_timings(tlc_ctx* c) {
  for (const PendingTiming& p : c->pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
      c->total_ms[p.kernel] += ms;
      c->launches[p.kernel] += 1;
    }
    c->free_events.push_back(p.start);
    c->free_events.push_back(p.stop);
  }
  c->pending.clear();
}

// Launch helper: brackets the launch with events when profiling is on.
template <class F>
int timed_launch(tlc_ctx* c, int kernel, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  if (c->profiling) {
    a = take_event(c);
    b = take_event(c);
    if (a && b && hipEventRecord(a, c->stream) != hipSuccess) {
      c->free_events.push_back(a);
      c->free_events.push_back(b);
      a = b = nullptr;
    }
  }
  hipError_t e = launch();
  if (e != hipSuccess) {
    c->broken = true;  // ticket counters may no longer match their bases
    if (a) c->free_events.push_back(a);
    if (b) c->free_events.push_back(b);
    return hip_fail(e, kKernelNames[kernel]);
  }
  if (a && b) {
    if (hipEventRecord(b, c->stream) == hipSuccess) {
      c->pending.push_back(PendingTiming{kernel, a, b});
    } else {
      c->free_events.push_back(a);
      c->free_events.push_back(b);
    }
  }
  return TLC_OK;
}

// Next look-back epoch (never 0, the value of cleared status words).  When
// the counter wraps, the caller clears the status array first.
uint32_t next_epoch(uint32_t* epoch, uint32_t max_epoch, bool* need_clear) {
  *need_clear = *epoch >= max_epoch;
  if (*need_clear) *epoch = 0;
  return ++*epoch;
}

int sync_and_read(tlc_ctx* c) {
  hipError_t e = hipMemcpyAsync(c->rb, c->ctrl, sizeof(HostReadback),
                                hipMemcpyDeviceToHost, c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(readback)");
  e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  collect_timings(c);
  return TLC_OK;
}

}  // namespace

TLC_API size_t tlc_max_compressed_bytes(size_t n) { return quartic_len(n); }

TLC_API const char* tlc_last_error_string(void) { return g_err; }

TLC_API const char* tlc_kernel_name(int kernel) {
  return (kernel >= 0 && kernel < TLC_KERNEL_COUNT) ? kKernelNames[kernel] : nullptr;
}

TLC_API int tlc_ctx_create(tlc_ctx** out, size_t max_n, void* hip_stream) {
  if (!out) return fail(TLC_E_INVALID, "tlc_ctx_create: ctx pointer is NULL");
  *out = nullptr;
  if (max_n == 0 || max_n > TLC_MAX_N)
    return fail(TLC_E_INVALID, "tlc_ctx_create: max_n %zu not in [1, %zu]", max_n,
                (size_t)TLC_MAX_N);
  tlc_ctx* c = new (std::nothrow) tlc_ctx();
  if (!c) return fail(TLC_E_DEVICE, "tlc_ctx_create: out of host memory");
  c->stream = (hipStream_t)hip_stream;
  c->max_n = max_n;
  c->max_m = quartic_len(max_n);
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "hipGetDevice");
  }
  // layout: ctrl | partials | enc status | dec status | start index
  c->enc_status_words = (c->max_m + kEncTile - 1) / kEncTile + 1;
  c->dec_status_words = (c->max_m + kZreTile - 1) / kZreTile + 1;
  const size_t off_partials = sizeof(Ctrl);
  const size_t off_enc = round_up(off_partials + kAbsmaxMaxBlocks * sizeof(uint32_t), 256);
  const size_t off_dec = round_up(off_enc + c->enc_status_words * sizeof(uint64_t), 256);
  const size_t off_start = round_up(off_dec + c->dec_status_words * sizeof(uint64_t), 256);
  const size_t start_words = (c->max_m + kDecRange - 1) / kDecRange + 1;
  const size_t total = off_start + start_words * sizeof(uint64_t);
  e = hipMalloc(&c->ws, total);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "hipMalloc(workspace)");
  }
  uint8_t* base = (uint8_t*)c->ws;
  c->ctrl = (Ctrl*)base;
  c->partials = (uint32_t*)(base + off_partials);
  c->enc_status = (uint64_t*)(base + off_enc);
  c->dec_status = (uint64_t*)(base + off_dec);
  c->start = (uint64_t*)(base + off_start);
  e = hipMemset(c->ws, 0, total);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess)
    e = hipHostMalloc((void**)&c->rb, sizeof(HostReadback), hipHostMallocDefault);
  if (e != hipSuccess) {
    (void)hipFree(c->ws);
    delete c;
    return hip_fail(e, "tlc_ctx_create: workspace init");
  }
  memset(c->rb, 0, sizeof(HostReadback));
  *out = c;
  return TLC_OK;
}

TLC_API int tlc_ctx_destroy(tlc_ctx* c) {
  if (!c) return TLC_OK;
  ensure_device(c);
  (void)hipStreamSynchronize(c->stream);
  collect_timings(c);
  for (hipEvent_t ev : c->free_events) (void)hipEventDestroy(ev);
  if (c->rb) (void)hipHostFree(c->rb);
  if (c->ws) (void)hipFree(c->ws);
  delete c;
  return TLC_OK;
}

TLC_API int tlc_compress(tlc_ctx* c, const float* tensor, float* residual, size_t n,
                         float s, uint8_t* bytes, size_t bytes_cap, size_t* bytes_len,
                         float* scale) {
  if (bytes_len) *bytes_len = 0;
  if (!c || !bytes_len || !scale) return fail(TLC_E_INVALID, "tlc_compress: NULL argument");
  if (c->broken) return fail(TLC_E_DEVICE, "tlc_compress: context unusable after a device error");
  if (!(s >= 1.0f && s < 2.0f))
    return fail(TLC_E_INVALID, "tlc_compress: s = %g not in [1, 2)", (double)s);
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_compress: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  if (n == 0) {
    *scale = 0.0f;
    return TLC_OK;
  }
  if (!tensor || !residual || !bytes)
    return fail(TLC_E_INVALID, "tlc_compress: NULL device pointer");
  const size_t m = quartic_len(n);
  if (bytes_cap < m)
    return fail(TLC_E_CAPACITY, "tlc_compress: bytes_cap %zu < %zu", bytes_cap, m);
  if (overlap(tensor, n * 4, residual, n * 4) || overlap(tensor, n * 4, bytes, m) ||
      overlap(residual, n * 4, bytes, m))
    return fail(TLC_E_INVALID, "tlc_compress: tensor, residual and bytes overlap");
  int st = ensure_device(c);
  if (st) return st;

  uint32_t np = 0;
  st = timed_launch(c, TLC_KERNEL_ABSMAX, [&] {
    return launch_absmax(tensor, residual, n, c->partials, &np, c->stream);
  });
  if (st) return st;
  bool clear = false;
  const uint32_t epoch = next_epoch(&c->enc_epoch, kEncEpochMax, &clear);
  if (clear) {
    hipError_t e = hipMemsetAsync(c->enc_status, 0, c->enc_status_words * 8, c->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync(status)");
  }
  const uint32_t ntiles = (uint32_t)((m + kEncTile - 1) / kEncTile);
  st = timed_launch(c, TLC_KERNEL_QUANT_ENCODE, [&] {
    return launch_quant_encode(tensor, residual, n, (uint32_t)m, s, c->partials, np, bytes,
                               c->enc_status, ntiles, c->enc_ticket_base, epoch, c->ctrl,
                               c->stream);
  });
  if (st) return st;
  c->enc_ticket_base += ntiles;
  st = sync_and_read(c);
  if (st) return st;
  if (c->rb->fault) {
    c->broken = true;
    return fail(TLC_E_DEVICE, "tlc_compress: look-back wait timed out");
  }
  if (c->rb->enc_err)
    return fail(TLC_E_NONFINITE, "tlc_compress: NaN/Inf in tensor+residual or max*s overflow");
  *bytes_len = c->rb->enc_len;
  *scale = c->rb->enc_scale;
  return TLC_OK;
}

TLC_API int tlc_decompress(tlc_ctx* c, const uint8_t* bytes, size_t bytes_len, float scale,
                           size_t n, float* out, int accumulate) {
  if (!c) return fail(TLC_E_INVALID, "tlc_decompress: NULL context");
  if (c->broken) return fail(TLC_E_DEVICE, "tlc_decompress: context unusable after a device error");
  if (!isfinite(scale) || scale < 0.0f)
    return fail(TLC_E_INVALID, "tlc_decompress: scale %g is not finite and >= 0", (double)scale);
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_decompress: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  if (n == 0) {
    if (bytes_len != 0) return fail(TLC_E_CORRUPT, "tlc_decompress: bytes for an empty tensor");
    return TLC_OK;
  }
  if (!out || (bytes_len && !bytes)) return fail(TLC_E_INVALID, "tlc_decompress: NULL device pointer");
  const size_t m = quartic_len(n);
  if (bytes_len == 0 || bytes_len > m)
    return fail(TLC_E_CORRUPT, "tlc_decompress: stream length %zu impossible for n = %zu",
                bytes_len, n);
  int st = ensure_device(c);
  if (st) return st;
  bool clear = false;
  const uint32_t epoch = next_epoch(&c->dec_epoch, kDecEpochMax, &clear);
  if (clear) {
    hipError_t e = hipMemsetAsync(c->dec_status, 0, c->dec_status_words * 8, c->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync(status)");
  }
  const uint32_t ntiles = (uint32_t)((bytes_len + kZreTile - 1) / kZreTile);
  st = timed_launch(c, TLC_KERNEL_ZRE_INDEX, [&] {
    return launch_zre_index(bytes, (uint32_t)bytes_len, (uint32_t)m, c->start, c->dec_status,
                            ntiles, c->dec_ticket_base, epoch, c->ctrl, c->stream);
  });
  if (st) return st;
  c->dec_ticket_base += ntiles;
  st = timed_launch(c, TLC_KERNEL_EXPAND_DEQUANT, [&] {
    return launch_expand_dequant(bytes, (uint32_t)bytes_len, c->start, n, m, scale, out,
                                 accumulate, epoch, c->ctrl, c->stream);
  });
  return st;
}

TLC_API int tlc_sync(tlc_ctx* c) {
  if (!c) return fail(TLC_E_INVALID, "tlc_sync: NULL context");
  int st = ensure_device(c);
  if (st) return st;
  st = sync_and_read(c);
  if (st) return st;
  if (c->rb->fault) {
    c->broken = true;
    return fail(TLC_E_DEVICE, "look-back wait timed out");
  }
  if (c->rb->dec_corrupt) {
    hipError_t e = hipMemsetAsync(&c->ctrl->dec_corrupt, 0, sizeof(uint32_t), c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "tlc_sync: clearing status");
    return fail(TLC_E_CORRUPT, "a decoded stream did not expand to ceil(n/5) bytes");
  }
  return TLC_OK;
}

TLC_API int tlc_profile_enable(tlc_ctx* c, int on) {
  if (!c) return fail(TLC_E_INVALID, "tlc_profile_enable: NULL context");
  c->profiling = on != 0;
  return TLC_OK;
}

TLC_API int tlc_profile_get(tlc_ctx* c, int kernel, double* total_ms, uint64_t* launches) {
  if (!c || !total_ms || !launches || kernel < 0 || kernel >= TLC_KERNEL_COUNT)
    return fail(TLC_E_INVALID, "tlc_profile_get: bad argument");
  int st = ensure_device(c);
  if (st) return st;
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  collect_timings(c);
  *total_ms = c->total_ms[kernel];
  *launches = c->launches[kernel];
  return TLC_OK;
}

TLC_API int tlc_profile_reset(tlc_ctx* c) {
  if (!c) return fail(TLC_E_INVALID, "tlc_profile_reset: NULL context");
  int st = ensure_device(c);
  if (st) return st;
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  collect_timings(c);
  for (int k = 0; k < TLC_KERNEL_COUNT; ++k) {
    c->total_ms[k] = 0.0;
    c->launches[k] = 0;
  }
  return TLC_OK;
}
