// tlc_api.hip -- host side of the C ABI declared in include/tlc.h: argument
// checks, the per-context device workspace, kernel launches on the
// context's stream, status readback and optional per-kernel event timing.
#include <math.h>
#include <stddef.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "tlc.h"
#include "tlc_internal.h"

#define TLC_API extern "C" __attribute__((visibility("default")))

using namespace tlc;

namespace {
thread_local char g_err[512] = "no error";
}  // namespace

thread_local LaunchEvents tlc::g_launch_events;

int tlc::fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(TLC_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

size_t quartic_len(size_t n) { return n / 5 + (n % 5 ? 1 : 0); }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

size_t ceil_div(size_t a, size_t b) { return (a + b - 1) / b; }

bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return an && bn && pa < pb + bn && pb < pa + an;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0u; }

const char* const kKernelNames[TLC_KERNEL_COUNT] = {
    "tlc_accum_absmax_kernel",       "tlc_quant_encode_kernel",
    "tlc_zre_index_kernel",          "tlc_expand_dequant_kernel",
    "tlc_accum_absmax_batch_kernel", "tlc_quant_encode_batch_kernel",
    "tlc_zre_index_batch_kernel",    "tlc_expand_dequant_batch_kernel",
    "tlc_expand_sum_kernel",         "tlc_quant_pack_kernel",
    "tlc_int8_quant_kernel",         "tlc_int8_dequant_kernel",
    "tlc_zre_chunk_kernel",          "tlc_zre_compact_kernel",
    "tlc_quant_encode_chained_kernel", "tlc_absmax_check_kernel",
    "tlc_absmax_check_batch_kernel", "tlc_accum_quantize_kernel"};

// A device address range of one call's arguments; `written` ranges must
// not overlap any other range of the call.
struct Span {
  uintptr_t lo, hi;
  bool written;
};

// Sorts the spans by start address and reports whether a written span
// overlaps another span (read-only spans may overlap each other: one stream
// decoded into several outputs, one tensor read twice).  In start order a
// span overlaps an earlier one exactly when it starts below that one's end,
// so it suffices to keep the largest end of all earlier spans and of the
// earlier written ones.  std::sort works in place: nothing is allocated.
bool spans_conflict(std::vector<Span>& v) {
  std::sort(v.begin(), v.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
  uintptr_t end_all = 0, end_written = 0;
  for (const Span& sp : v) {
    if (sp.lo < (sp.written ? end_all : end_written)) return true;
    end_all = std::max(end_all, sp.hi);
    if (sp.written) end_written = std::max(end_written, sp.hi);
  }
  return false;
}

// spans_conflict for a call whose spans may repeat the previous call's
// (`last`: the spans of the last call that passed, in call order).  A
// training loop passes the same buffers every step: the list then equals
// `last`, which was checked already, and the sort is skipped.  `last`
// has the capacity of `v`, so nothing is allocated.
bool spans_conflict_cached(std::vector<Span>& v, std::vector<Span>& last) {
  if (v.size() == last.size() &&
      std::equal(v.begin(), v.end(), last.begin(), [](const Span& a, const Span& b) {
        return a.lo == b.lo && a.hi == b.hi && a.written == b.written;
      }))
    return false;
  last = v;
  if (!spans_conflict(v)) return false;
  last.clear();
  return true;
}

void add_span(std::vector<Span>& v, const void* p, size_t bytes, bool written) {
  if (bytes) v.push_back(Span{(uintptr_t)p, (uintptr_t)p + bytes, written});
}

struct PendingTiming {
  int kernel;
  hipEvent_t start, stop;
};

constexpr int kStagingSlots = 4;

}  // namespace

struct tlc_ctx {
  hipStream_t stream = nullptr;
  int device = 0;
  size_t max_n = 0;        // values per call (summed over a batch)
  size_t max_tensors = 0;  // tensors or streams per call
  // device workspace (one allocation)
  void* ws = nullptr;
  Ctrl* ctrl = nullptr;
  uint32_t* partials = nullptr;
  uint32_t* partials_chk = nullptr;  // the check pass's partial maxima
  size_t partials_cap = 0;
  uint64_t* enc_status = nullptr;
  size_t enc_status_words = 0;
  uint64_t* dec_status = nullptr;
  size_t dec_status_words = 0;
  uint64_t* start = nullptr;  // per kDecRange quartic bytes: (stream index, skip)
  size_t start_words = 0;
  EncDesc* enc_descs = nullptr;
  DecDesc* dec_descs = nullptr;
  EncResult* enc_results = nullptr;
  // single-tensor encoder: per-tile slots and records, chunk summaries
  uint8_t* slots = nullptr;
  TileRec* recs = nullptr;
  uint64_t* chunk_agg = nullptr;  // chunk summaries, scanned in place into chunk prefixes
  uint64_t* local_pre = nullptr;  // every tile's prefix within its chunk
  uint2* fix = nullptr;           // per tile kFixCap deferred residuals
  uint16_t* summ = nullptr;       // per float4 of the buffer: top half of max |acc|
  // pinned host memory: status readback, batch results, descriptor staging
  HostReadback* rb = nullptr;
  EncResult* host_results = nullptr;
  HostReadback* rb_dev = nullptr;  // the same pinned memory, as the device addresses it
  uint8_t* staging = nullptr;  // kStagingSlots slots of max_tensors * 64 bytes
  hipEvent_t staging_done[kStagingSlots] = {};
  bool staging_used[kStagingSlots] = {};
  int staging_next = 0;
  // look-back bookkeeping
  uint32_t enc_ticket_base = 0, dec_ticket_base = 0;
  uint32_t enc_epoch = 0, dec_epoch = 0;
  bool broken = false;
  uint32_t options = 0;  // TLC_OPT_*
  // profiling
  bool profiling = false;
  uint32_t profile_mask = 0xffffffffu;  // bit k: time kernel id k
  // host-side descriptor tables of the batched calls (capacity max_tensors,
  // reserved at creation, so the calls do not allocate)
  std::vector<EncDesc> enc_host;
  std::vector<DecDesc> dec_host;
  std::vector<size_t> which;
  std::vector<Span> spans;  // address ranges of a batched call (3 per tensor)
  std::vector<Span> enc_spans_ok, dec_spans_ok;  // the last batched calls that passed
  std::vector<hipEvent_t> free_events;
  std::vector<PendingTiming> pending;
  double total_ms[TLC_KERNEL_COUNT] = {};
  uint64_t launches[TLC_KERNEL_COUNT] = {};
};

namespace {

// Makes the context's device current for one entry point and restores the
// caller's device when the entry point returns.
class DeviceScope {
 public:
  explicit DeviceScope(int dev) {
    err_ = hipGetDevice(&prev_);
    if (err_ == hipSuccess && prev_ != dev) {
      err_ = hipSetDevice(dev);
      switched_ = err_ == hipSuccess;
    }
  }
  ~DeviceScope() {
    if (switched_) (void)hipSetDevice(prev_);
  }
  DeviceScope(const DeviceScope&) = delete;
  DeviceScope& operator=(const DeviceScope&) = delete;
  int status() const { return err_ == hipSuccess ? TLC_OK : hip_fail(err_, "hipSetDevice"); }

 private:
  int prev_ = -1;
  bool switched_ = false;
  hipError_t err_ = hipSuccess;
};

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
// Adds the finished timed launches to the totals; a pair whose kernels are
// still running (an encode returns once its result has arrived) stays
// pending for the next call.
void collect_timings(tlc_ctx* c) {
  size_t keep = 0;
  for (const PendingTiming& p : c->pending) {
    float ms = 0.0f;
    const hipError_t e = hipEventElapsedTime(&ms, p.start, p.stop);
    if (e == hipErrorNotReady) {
      c->pending[keep++] = p;
      continue;
    }
    if (e == hipSuccess) {
      c->total_ms[p.kernel] += ms;
      c->launches[p.kernel] += 1;
    }
    c->free_events.push_back(p.start);
    c->free_events.push_back(p.stop);
  }
  c->pending.resize(keep);
}

// Launch helper: brackets the launch with events when profiling is on.
// The launcher's kernels record the event pair themselves (launch_k): the
// first one's start and the last one's end.
template <class F>
int timed_launch(tlc_ctx* c, int kernel, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  if (c->profiling && ((c->profile_mask >> kernel) & 1u)) {
    a = take_event(c);
    b = take_event(c);
    if (!a || !b) {
      if (a) c->free_events.push_back(a);
      if (b) c->free_events.push_back(b);
      a = b = nullptr;
    }
  }
  g_launch_events = LaunchEvents{a, b};
  hipError_t e = launch();
  const bool started = g_launch_events.start == nullptr;  // a kernel took the start event
  g_launch_events = LaunchEvents{};
  if (e != hipSuccess) {
    c->broken = true;  // ticket counters may no longer match their bases
    if (a) c->free_events.push_back(a);
    if (b) c->free_events.push_back(b);
    return hip_fail(e, kKernelNames[kernel]);
  }
  if (a && b) {
    if (started) {
      c->pending.push_back(PendingTiming{kernel, a, b});
    } else {  // the launcher dispatched no kernel
      c->free_events.push_back(a);
      c->free_events.push_back(b);
    }
  }
  return TLC_OK;
}

// Next look-back epoch (never 0, the value of cleared status words); when
// the counter wraps the status array is cleared on the stream first.
// Next launch epoch (1 .. max_epoch).  When the counter wraps, the status
// words are cleared, and so is `stale` (a device word that may hold an
// epoch number of the old cycle: the decoder's bad-stream mark), so that no
// old value can match a new launch.
int next_epoch(tlc_ctx* c, uint32_t* epoch, uint32_t max_epoch, uint64_t* status,
               size_t words, uint32_t* stale, uint32_t* out) {
  if (*epoch >= max_epoch) {
    *epoch = 0;
    hipError_t e = hipMemsetAsync(status, 0, words * sizeof(uint64_t), c->stream);
    if (e == hipSuccess && stale) e = hipMemsetAsync(stale, 0, sizeof(uint32_t), c->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync(status)");
  }
  *out = ++*epoch;
  return TLC_OK;
}

// The decoder's epoch.  Its wrap also clears what carries a decode epoch
// besides the status words: the corrupt-stream mark, the single-stream
// verdict and the start entries.
int next_dec_epoch(tlc_ctx* c, uint32_t* out) {
  if (c->dec_epoch >= kDecEpochMax) {
    hipError_t e = hipMemsetAsync(&c->ctrl->dec_verdict, 0, sizeof(uint32_t), c->stream);
    if (e == hipSuccess)
      e = hipMemsetAsync(c->start, 0, c->start_words * sizeof(uint64_t), c->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync(decoder epoch wrap)");
  }
  return next_epoch(c, &c->dec_epoch, kDecEpochMax, c->dec_status, c->dec_status_words,
                    &c->ctrl->dec_bad_epoch, out);
}

// Copies `bytes` of host descriptors to `dst` on the stream through a
// pinned staging slot.  A slot is reused only after its previous copy has
// executed, so back-to-back asynchronous calls cannot overwrite a
// descriptor table that is still in flight.
int upload(tlc_ctx* c, void* dst, const void* src, size_t bytes) {
  const int slot = c->staging_next;
  c->staging_next = (slot + 1) % kStagingSlots;
  if (c->staging_used[slot]) {
    hipError_t e = hipEventSynchronize(c->staging_done[slot]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(staging)");
  }
  uint8_t* host = c->staging + (size_t)slot * c->max_tensors * 64;
  memcpy(host, src, bytes);
  hipError_t e = hipMemcpyAsync(dst, host, bytes, hipMemcpyHostToDevice, c->stream);
  if (e == hipSuccess) e = hipEventRecord(c->staging_done[slot], c->stream);
  if (e != hipSuccess) {
    c->broken = true;
    return hip_fail(e, "descriptor upload");
  }
  c->staging_used[slot] = true;
  return TLC_OK;
}

// Copies the control block's readback fields to the pinned block, then
// waits.
int sync_and_read(tlc_ctx* c) {
  hipError_t e =
      hipMemcpyAsync(c->rb, c->ctrl, sizeof(HostReadback), hipMemcpyDeviceToHost, c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(readback)");
  e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  collect_timings(c);
  return TLC_OK;
}

// Waits for the stream; for calls whose kernels wrote their result into the
// pinned readback themselves (HostMirror), no copy is needed first.
int sync_mirrored(tlc_ctx* c) {
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  collect_timings(c);
  return TLC_OK;
}

// Where an encode's kernels mirror the single-tensor result and the fault
// flag (the pinned readback, as the device addresses it).
HostMirror enc_mirror(tlc_ctx* c) {
  return HostMirror{&c->rb_dev->enc, &c->rb_dev->fault};
}
HostMirror fault_mirror(tlc_ctx* c) {
  return HostMirror{nullptr, &c->rb_dev->fault, &c->rb_dev->dec_corrupt};
}
// A batch: the per-tensor results follow the control block's slot in the
// readback (as host_results does on the host).
HostMirror batch_mirror(tlc_ctx* c) {
  return HostMirror{
      reinterpret_cast<EncResult*>(reinterpret_cast<uint8_t*>(c->rb_dev) + sizeof(Ctrl)),
      &c->rb_dev->fault};
}

// An encode whose kernels mirror their results (enc_mirror, batch_mirror):
// before its launches the host fills each result's err, len and scale words
// with kPending, which none of their values takes (err is 0 or 1, a length
// is below 2^31, a scale is finite), and then waits for the words to change
// rather than for the stream: a tensor's first tile writes err and the
// scale (and a zero length on error), its last tile, or the compaction's
// last, the length, a little before the kernels end.
constexpr uint32_t kPending = 0xffffffffu;

static_assert(offsetof(EncResult, err) == 0 && offsetof(EncResult, len) == 4 &&
                  offsetof(EncResult, scale) == 8 && sizeof(EncResult) == 16,
              "err, len and scale are the first three of a result's four words");

void arm_results(EncResult* r, uint32_t count) {
  volatile uint32_t* w = reinterpret_cast<volatile uint32_t*>(r);
  for (uint32_t i = 0; i < count; ++i) {
    w[4 * i] = kPending;
    w[4 * i + 1] = kPending;
    w[4 * i + 2] = kPending;
  }
}

bool result_pending(const EncResult* r) {
  const volatile uint32_t* w = reinterpret_cast<const volatile uint32_t*>(r);
  const uint32_t err = w[0];
  return err == kPending || w[2] == kPending || (err == 0u && w[1] == kPending);
}

// Polls the armed results; falls back to waiting for the stream once the
// stream has finished (or a look-back fault was flagged) without them.
int wait_results(tlc_ctx* c, const EncResult* r, uint32_t count) {
  const volatile uint32_t* fault = &c->rb->fault;
  uint32_t i = 0;  // results before i have arrived
  for (uint32_t spin = 1;; ++spin) {
    if (*fault) break;
    while (i < count && !result_pending(&r[i])) ++i;
    if (i == count) {
      __atomic_thread_fence(__ATOMIC_ACQUIRE);  // the results' plain reads come after
      collect_timings(c);
      return TLC_OK;
    }
    if ((spin & 255u) == 0u) {
      const hipError_t q = hipStreamQuery(c->stream);
      if (q == hipSuccess) break;
      if (q != hipErrorNotReady) return hip_fail(q, "hipStreamQuery");
    }
#if defined(__x86_64__) || defined(__i386__)
    __builtin_ia32_pause();  // a spin-wait hint to the core
#endif
  }
  int st = sync_mirrored(c);
  if (st) return st;
  if (!*fault)
    for (; i < count; ++i)
      if (result_pending(&r[i])) {
        c->broken = true;
        return fail(TLC_E_DEVICE, "the encode wrote no result for a tensor");
      }
  return TLC_OK;
}

// Waits for an encode and reports its result (the stream length and M);
// mirrored: the kernels wrote it into the readback (enc_mirror), which
// arm_result prepared.
int finish_compress(tlc_ctx* c, const char* fn, size_t* bytes_len, float* scale,
                    bool mirrored = false) {
  int st = mirrored ? wait_results(c, &c->rb->enc, 1) : sync_and_read(c);
  if (st) return st;
  if (c->rb->fault) {
    c->broken = true;
    return fail(TLC_E_DEVICE, "%s: look-back wait timed out", fn);
  }
  if (c->rb->enc.err)
    return fail(TLC_E_NONFINITE, "%s: NaN/Inf in tensor+residual or max*s overflow", fn);
  *bytes_len = c->rb->enc.len;
  *scale = c->rb->enc.scale;
  return TLC_OK;
}

int check_usable(tlc_ctx* c, const char* fn) {
  if (!c) return fail(TLC_E_INVALID, "%s: NULL context", fn);
  if (c->broken) return fail(TLC_E_DEVICE, "%s: context unusable after a device error", fn);
  return TLC_OK;
}

// Absmax blocks given to one tensor of a batch (proportional to its size,
// `items` float4 pairs or single values).
uint32_t batch_absmax_blocks(size_t items) {
  size_t b = ceil_div(items, (size_t)kThreads * 4);
  return (uint32_t)std::max<size_t>(1, std::min<size_t>(b, kAbsmaxMaxBlocks));
}

}  // namespace

TLC_API size_t tlc_max_compressed_bytes(size_t n) { return quartic_len(n); }

TLC_API const char* tlc_last_error_string(void) { return g_err; }

TLC_API const char* tlc_kernel_name(int kernel) {
  return (kernel >= 0 && kernel < TLC_KERNEL_COUNT) ? kKernelNames[kernel] : nullptr;
}

TLC_API int tlc_ctx_create_batch(tlc_ctx** out, size_t max_n, size_t max_tensors,
                                 void* hip_stream) {
  if (!out) return fail(TLC_E_INVALID, "tlc_ctx_create: ctx pointer is NULL");
  *out = nullptr;
  if (max_n == 0 || max_n > TLC_MAX_N)
    return fail(TLC_E_INVALID, "tlc_ctx_create: max_n %zu not in [1, %zu]", max_n,
                (size_t)TLC_MAX_N);
  if (max_tensors == 0 || max_tensors > TLC_MAX_TENSORS)
    return fail(TLC_E_INVALID, "tlc_ctx_create: max_tensors %zu not in [1, %d]", max_tensors,
                TLC_MAX_TENSORS);
  tlc_ctx* c = new (std::nothrow) tlc_ctx();
  if (!c) return fail(TLC_E_DEVICE, "tlc_ctx_create: out of host memory");
  c->stream = (hipStream_t)hip_stream;
  c->max_n = max_n;
  c->max_tensors = max_tensors;
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "hipGetDevice");
  }
  // Bounds over any call: the sum of m_t is at most max_n/5 + tensors, and a
  // tensor has at most m_t/tile + 1 tiles.
  const size_t mm = max_n / 5 + max_tensors;
  c->partials_cap =
      std::max<size_t>(kAbsmaxMaxBlocks, max_n / ((size_t)kThreads * 4) + max_tensors + 1);
  const size_t tiles1 = ceil_div(quartic_len(max_n), (size_t)kEncTile);  // one tensor
  c->enc_status_words = mm / kEncTile + max_tensors + 2;
  c->dec_status_words = mm / kZreBatchTile + max_tensors + 2;  // the smaller tile
  c->start_words = mm / kDecRange + max_tensors + 2;
  // layout: ctrl | enc results | partials | check partials | enc status | dec status |
  //         start | enc descs | dec descs | tile records | chunk summaries |
  //         tile prefixes in their chunks | fix lists | float4 summaries | slots
  // (the batch results follow the control block, so that one copy reads both)
  static_assert(sizeof(Ctrl) % alignof(EncResult) == 0, "results follow the control block");
  const size_t off_res = sizeof(Ctrl);
  size_t off = round_up(off_res + max_tensors * sizeof(EncResult), 256);
  const size_t off_partials = off;
  off = round_up(off + c->partials_cap * sizeof(uint32_t), 256);
  const size_t off_partials_chk = off;
  off = round_up(off + c->partials_cap * sizeof(uint32_t), 256);
  const size_t off_enc = off;
  off = round_up(off + c->enc_status_words * sizeof(uint64_t), 256);
  const size_t off_dec = off;
  off = round_up(off + c->dec_status_words * sizeof(uint64_t), 256);
  const size_t off_start = off;
  off = round_up(off + c->start_words * sizeof(uint64_t), 256);
  const size_t off_edesc = off;
  off = round_up(off + max_tensors * sizeof(EncDesc), 256);
  const size_t off_ddesc = off;
  off = round_up(off + max_tensors * sizeof(DecDesc), 256);
  const size_t off_recs = off;
  off = round_up(off + tiles1 * sizeof(TileRec), 256);
  const size_t off_chunks = off;
  off = round_up(off + (tiles1 / 64 + 1) * sizeof(uint64_t), 256);
  const size_t off_local = off;
  off = round_up(off + tiles1 * sizeof(uint64_t), 256);
  const size_t off_fix = off;
  off = round_up(off + tiles1 * (size_t)kFixCap * sizeof(uint2), 256);
  const size_t off_summ = off;
  off = round_up(off + (max_n / 4) * sizeof(uint16_t), 256);
  const size_t off_slots = off;
  const size_t total = round_up(off + tiles1 * (size_t)kEncTile, 256);
  e = hipMalloc(&c->ws, total);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "hipMalloc(workspace)");
  }
  uint8_t* base = (uint8_t*)c->ws;
  c->ctrl = (Ctrl*)base;
  c->partials = (uint32_t*)(base + off_partials);
  c->partials_chk = (uint32_t*)(base + off_partials_chk);
  c->enc_status = (uint64_t*)(base + off_enc);
  c->dec_status = (uint64_t*)(base + off_dec);
  c->start = (uint64_t*)(base + off_start);
  c->enc_descs = (EncDesc*)(base + off_edesc);
  c->dec_descs = (DecDesc*)(base + off_ddesc);
  c->enc_results = (EncResult*)(base + off_res);
  c->recs = (TileRec*)(base + off_recs);
  c->chunk_agg = (uint64_t*)(base + off_chunks);
  c->local_pre = (uint64_t*)(base + off_local);
  c->fix = (uint2*)(base + off_fix);
  c->summ = (uint16_t*)(base + off_summ);
  c->slots = base + off_slots;
  e = hipMemset(c->ws, 0, total);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  // pinned readback block, laid out as the workspace's head: the control
  // block's slot, then the batch results
  if (e == hipSuccess)
    e = hipHostMalloc((void**)&c->rb, sizeof(Ctrl) + max_tensors * sizeof(EncResult),
                      hipHostMallocDefault);
  if (e == hipSuccess)
    c->host_results =
        reinterpret_cast<EncResult*>(reinterpret_cast<uint8_t*>(c->rb) + sizeof(Ctrl));
  if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&c->rb_dev, c->rb, 0);
  if (e == hipSuccess)
    e = hipHostMalloc((void**)&c->staging, kStagingSlots * max_tensors * 64,
                      hipHostMallocDefault);
  for (int i = 0; i < kStagingSlots && e == hipSuccess; ++i)
    e = hipEventCreateWithFlags(&c->staging_done[i], hipEventDisableTiming);
  if (e != hipSuccess) {
    for (int i = 0; i < kStagingSlots; ++i)
      if (c->staging_done[i]) (void)hipEventDestroy(c->staging_done[i]);
    if (c->staging) (void)hipHostFree(c->staging);
    if (c->rb) (void)hipHostFree(c->rb);
    (void)hipFree(c->ws);
    delete c;
    return hip_fail(e, "tlc_ctx_create: workspace init");
  }
  memset(c->rb, 0, sizeof(HostReadback));
  try {
    c->enc_host.reserve(max_tensors);
    c->dec_host.reserve(max_tensors);
    c->which.reserve(max_tensors);
    c->spans.reserve(3 * max_tensors);
    c->enc_spans_ok.reserve(3 * max_tensors);
    c->dec_spans_ok.reserve(3 * max_tensors);
  } catch (...) {
    tlc_ctx_destroy(c);
    return fail(TLC_E_DEVICE, "tlc_ctx_create: out of host memory");
  }
  *out = c;
  return TLC_OK;
}

TLC_API int tlc_ctx_create(tlc_ctx** out, size_t max_n, void* hip_stream) {
  return tlc_ctx_create_batch(out, max_n, 1, hip_stream);
}

TLC_API int tlc_ctx_destroy(tlc_ctx* c) {
  if (!c) return TLC_OK;
  DeviceScope dev(c->device);
  (void)hipStreamSynchronize(c->stream);
  collect_timings(c);
  for (const PendingTiming& p : c->pending) {  // left only if the stream failed
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  for (hipEvent_t ev : c->free_events) (void)hipEventDestroy(ev);
  for (int i = 0; i < kStagingSlots; ++i)
    if (c->staging_done[i]) (void)hipEventDestroy(c->staging_done[i]);
  if (c->staging) (void)hipHostFree(c->staging);
  if (c->rb) (void)hipHostFree(c->rb);  // holds host_results too
  if (c->ws) (void)hipFree(c->ws);
  delete c;
  return TLC_OK;
}

// ---------------------------------------------------------------- encode
namespace {

// Step 1 and Eq. 1 for one tensor (r may be NULL: no error buffer).  With
// the default error policy a check pass first reduces max|x + r| without
// writing, and the writing pass leaves a tensor whose scale is bad
// untouched, so the buffer keeps its values on TLC_E_NONFINITE;
// TLC_OPT_IN_PLACE_FEEDBACK drops the check pass.
// With summ (the three-pass float4 path) after a check pass, the writing
// pass quantizes every value and leaves trits in summ (*trit set); in place
// it leaves acc and bounds.
int launch_max_passes(tlc_ctx* c, const float* x, float* r, size_t n, float s, uint16_t* summ,
                      uint32_t* np, bool* trit = nullptr) {
  if (trit) *trit = false;
  const uint32_t* guard = nullptr;
  uint32_t guard_np = 0;
  if (r && !(c->options & TLC_OPT_IN_PLACE_FEEDBACK)) {
    int st = timed_launch(c, TLC_KERNEL_ABSMAX_CHECK, [&] {
      return launch_absmax_check(x, r, n, c->partials_chk, &guard_np, c->stream);
    });
    if (st) return st;
    guard = c->partials_chk;
  }
  const bool quantize = summ != nullptr && guard != nullptr;
  if (trit) *trit = quantize;
  return timed_launch(c, quantize ? TLC_KERNEL_ACCUM_QUANTIZE : TLC_KERNEL_ABSMAX, [&] {
    return launch_accum_absmax(x, r, n, c->partials, np, summ, guard, guard_np, s, quantize,
                               c->stream);
  });
}

}  // namespace

TLC_API int tlc_ctx_set_options(tlc_ctx* c, uint32_t options) {
  if (!c) return fail(TLC_E_INVALID, "tlc_ctx_set_options: NULL context");
  if (options & ~TLC_OPT_IN_PLACE_FEEDBACK)
    return fail(TLC_E_INVALID, "tlc_ctx_set_options: unknown option bits 0x%x", options);
  c->options = options;
  return TLC_OK;
}

TLC_API int tlc_compress(tlc_ctx* c, const float* tensor, float* residual, size_t n,
                         float s, uint8_t* bytes, size_t bytes_cap, size_t* bytes_len,
                         float* scale) {
  if (bytes_len) *bytes_len = 0;
  int st = check_usable(c, "tlc_compress");
  if (st) return st;
  if (!bytes_len || !scale) return fail(TLC_E_INVALID, "tlc_compress: NULL argument");
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
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;

  arm_results(&c->rb->enc, 1);
  const uint32_t ntiles = (uint32_t)ceil_div(m, kEncTile);
  // The three passes' float4 path: after the check pass the max pass
  // quantizes every value and keeps 2-bit trits per value in summ; in place
  // it keeps a bound per float4 there, and the quantizer skips float4s of
  // the buffer whose bound is below U.
  // (The bounds take the float4 slices of the partitions, so m % 4 == 0;
  // the trits are kept per float4 of the buffer and serve any m.)
  const bool in_place = (c->options & TLC_OPT_IN_PLACE_FEEDBACK) != 0u;
  uint16_t* summ = (ntiles >= kThreePassMinTiles && aligned16(tensor) && aligned16(residual) &&
                    (m % 4 == 0 || !in_place))
                       ? c->summ
                       : nullptr;
  if (ntiles < kThreePassMinTiles) {  // small tensor: one chained pass
    // default policy: the check pass, then the chained tiles form acc = x + r
    // themselves; in place: step 1 into the buffer first, as for large tensors
    uint32_t np = 0;
    const uint32_t* partials = c->partials;
    if (in_place) {
      st = launch_max_passes(c, tensor, residual, n, s, nullptr, &np);
    } else {
      partials = c->partials_chk;
      st = timed_launch(c, TLC_KERNEL_ABSMAX_CHECK, [&] {
        return launch_absmax_check(tensor, residual, n, c->partials_chk, &np, c->stream);
      });
    }
    if (st) return st;
    uint32_t epoch = 0;
    st = next_epoch(c, &c->enc_epoch, kEncEpochMax, c->enc_status, c->enc_status_words, nullptr,
                    &epoch);
    if (st) return st;
    st = timed_launch(c, TLC_KERNEL_QUANT_ENCODE_CHAINED, [&] {
      return launch_quant_encode_chained(in_place ? nullptr : tensor, residual, n, (uint32_t)m,
                                         s, partials, np, bytes, c->enc_status, ntiles,
                                         c->enc_ticket_base, epoch, c->ctrl, enc_mirror(c),
                                         c->stream);
    });
    if (st) return st;
    c->enc_ticket_base += ntiles;
    return finish_compress(c, "tlc_compress", bytes_len, scale, true);
  }
  uint32_t np = 0;
  bool trit = false;
  st = launch_max_passes(c, tensor, residual, n, s, summ, &np, &trit);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_QUANT_ENCODE, [&] {
    return launch_quant_encode(residual, n, (uint32_t)m, s, c->partials, np, c->slots, c->recs,
                               c->fix, summ, trit, c->ctrl, enc_mirror(c), c->stream);
  });
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_ZRE_CHUNKS, [&] {
    return launch_zre_chunks(c->recs, ntiles, c->local_pre, c->chunk_agg, c->ctrl, c->stream);
  });
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_ZRE_COMPACT, [&] {
    return launch_zre_compact(c->recs, c->chunk_agg, c->local_pre, c->slots, (uint32_t)m, bytes,
                              c->fix, residual, n, c->ctrl, enc_mirror(c), c->stream);
  });
  if (st) return st;
  return finish_compress(c, "tlc_compress", bytes_len, scale, true);
}

namespace {

// TLC_MODE_INT8 of tlc_compress_ex (residual may be NULL: no error feedback).
int compress_int8(tlc_ctx* c, const float* tensor, float* residual, size_t n, float s,
                  uint8_t* bytes, size_t bytes_cap, size_t* bytes_len, float* scale) {
  if (!bytes_len || !scale) return fail(TLC_E_INVALID, "tlc_compress_ex: NULL argument");
  if (!(s >= 1.0f && s < 2.0f))
    return fail(TLC_E_INVALID, "tlc_compress_ex: s = %g not in [1, 2)", (double)s);
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_compress_ex: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  if (n == 0) {
    *scale = 0.0f;
    return TLC_OK;
  }
  if (!tensor || !bytes) return fail(TLC_E_INVALID, "tlc_compress_ex: NULL device pointer");
  if (bytes_cap < n)
    return fail(TLC_E_CAPACITY, "tlc_compress_ex: bytes_cap %zu < n = %zu", bytes_cap, n);
  if (overlap(tensor, n * 4, bytes, n) ||
      (residual && (overlap(tensor, n * 4, residual, n * 4) || overlap(residual, n * 4, bytes, n))))
    return fail(TLC_E_INVALID, "tlc_compress_ex: tensor, residual and bytes overlap");
  DeviceScope dev(c->device);
  int st = dev.status();
  if (st) return st;
  uint32_t np = 0;
  st = launch_max_passes(c, tensor, residual, n, s, nullptr, &np);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_INT8_QUANT, [&] {
    return launch_int8_quant(tensor, residual, n, s, c->partials, np, bytes, c->ctrl,
                             c->stream);
  });
  if (st) return st;
  st = sync_and_read(c);
  if (st) return st;
  if (c->rb->enc.err)
    return fail(TLC_E_NONFINITE, "tlc_compress_ex: NaN/Inf in the input or max*s overflow");
  *bytes_len = c->rb->enc.len;
  *scale = c->rb->enc.scale;
  return TLC_OK;
}

}  // namespace

TLC_API int tlc_compress_ex(tlc_ctx* c, int mode, const float* tensor, float* residual,
                            size_t n, float s, uint64_t seed, uint64_t step, uint8_t* bytes,
                            size_t bytes_cap, size_t* bytes_len, float* scale) {
  if (mode == TLC_MODE_3LC)
    return tlc_compress(c, tensor, residual, n, s, bytes, bytes_cap, bytes_len, scale);
  if (bytes_len) *bytes_len = 0;
  int st = check_usable(c, "tlc_compress_ex");
  if (st) return st;
  if (mode == TLC_MODE_INT8)
    return compress_int8(c, tensor, residual, n, s, bytes, bytes_cap, bytes_len, scale);
  if (mode != TLC_MODE_NO_ZRE && mode != TLC_MODE_STOCHASTIC)
    return fail(TLC_E_INVALID, "tlc_compress_ex: unknown mode %d", mode);
  const bool stoch = mode == TLC_MODE_STOCHASTIC;
  if (!bytes_len || !scale) return fail(TLC_E_INVALID, "tlc_compress_ex: NULL argument");
  if (!(s >= 1.0f && s < 2.0f))
    return fail(TLC_E_INVALID, "tlc_compress_ex: s = %g not in [1, 2)", (double)s);
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_compress_ex: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  if (n == 0) {
    *scale = 0.0f;
    return TLC_OK;
  }
  if (!tensor || !bytes || (!stoch && !residual))
    return fail(TLC_E_INVALID, "tlc_compress_ex: NULL device pointer");
  const size_t m = quartic_len(n);
  if (bytes_cap < m)
    return fail(TLC_E_CAPACITY, "tlc_compress_ex: bytes_cap %zu < %zu", bytes_cap, m);
  if (overlap(tensor, n * 4, bytes, m) ||
      (!stoch && (overlap(tensor, n * 4, residual, n * 4) || overlap(residual, n * 4, bytes, m))))
    return fail(TLC_E_INVALID, "tlc_compress_ex: tensor, residual and bytes overlap");
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  float* r = stoch ? nullptr : residual;  // the stochastic mode has no error feedback
  uint32_t np = 0;
  st = launch_max_passes(c, tensor, r, n, s, nullptr, &np);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_QUANT_PACK, [&] {
    return launch_quant_pack(tensor, r, n, (uint32_t)m, s, stoch ? 1 : 0, seed, step,
                             c->partials, np, bytes, c->ctrl, c->stream);
  });
  if (st) return st;
  st = sync_and_read(c);
  if (st) return st;
  if (c->rb->enc.err)
    return fail(TLC_E_NONFINITE, "tlc_compress_ex: NaN/Inf in the input or max*s overflow");
  *bytes_len = c->rb->enc.len;
  *scale = c->rb->enc.scale;
  return TLC_OK;
}

TLC_API int tlc_compress_batch(tlc_ctx* c, size_t count, const float* const* tensors,
                               float* const* residuals, const size_t* ns, const float* s,
                               uint8_t* const* bytes, const size_t* caps, size_t* bytes_len,
                               float* scales, int* status) {
  int st = check_usable(c, "tlc_compress_batch");
  if (st) return st;
  if (count == 0) return TLC_OK;
  if (!tensors || !residuals || !ns || !s || !bytes || !caps || !bytes_len || !scales ||
      !status)
    return fail(TLC_E_INVALID, "tlc_compress_batch: NULL argument");
  if (count > c->max_tensors)
    return fail(TLC_E_INVALID, "tlc_compress_batch: %zu tensors exceed the context's %zu",
                count, c->max_tensors);
  size_t total_n = 0;
  for (size_t t = 0; t < count; ++t) {
    bytes_len[t] = 0;
    scales[t] = 0.0f;
    status[t] = TLC_OK;
  }
  for (size_t t = 0; t < count; ++t) {
    if (!(s[t] >= 1.0f && s[t] < 2.0f))
      return fail(TLC_E_INVALID, "tlc_compress_batch: tensor %zu: s = %g not in [1, 2)", t,
                  (double)s[t]);
    if (ns[t] > c->max_n)
      return fail(TLC_E_INVALID, "tlc_compress_batch: tensor %zu: n = %zu too large", t, ns[t]);
    total_n += ns[t];
    if (ns[t] == 0) continue;
    const size_t m = quartic_len(ns[t]);
    if (!tensors[t] || !residuals[t] || !bytes[t])
      return fail(TLC_E_INVALID, "tlc_compress_batch: tensor %zu: NULL device pointer", t);
    if (caps[t] < m)
      return fail(TLC_E_CAPACITY, "tlc_compress_batch: tensor %zu: capacity %zu < %zu", t,
                  caps[t], m);
    if (overlap(tensors[t], ns[t] * 4, residuals[t], ns[t] * 4) ||
        overlap(tensors[t], ns[t] * 4, bytes[t], m) ||
        overlap(residuals[t], ns[t] * 4, bytes[t], m))
      return fail(TLC_E_INVALID, "tlc_compress_batch: tensor %zu: buffers overlap", t);
  }
  if (total_n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_compress_batch: %zu values exceed the context's max_n %zu",
                total_n, c->max_n);
  c->spans.clear();
  for (size_t t = 0; t < count; ++t) {
    if (ns[t] == 0) continue;
    add_span(c->spans, tensors[t], ns[t] * 4, false);
    add_span(c->spans, residuals[t], ns[t] * 4, true);
    add_span(c->spans, bytes[t], quartic_len(ns[t]), true);
  }
  if (spans_conflict_cached(c->spans, c->enc_spans_ok))
    return fail(TLC_E_INVALID,
                "tlc_compress_batch: a residual or byte buffer overlaps another tensor's buffer");
  std::vector<EncDesc>& d = c->enc_host;
  std::vector<size_t>& which = c->which;  // batch position of each launched tensor
  d.clear();
  which.clear();
  uint32_t blocks = 0, tiles = 0;
  for (size_t t = 0; t < count; ++t) {
    if (ns[t] == 0) continue;
    EncDesc e = {};
    e.x = tensors[t];
    e.r = residuals[t];
    e.out = bytes[t];
    e.n = ns[t];
    e.m = (uint32_t)quartic_len(ns[t]);
    e.s = s[t];
    e.tile0 = tiles;
    e.blk0 = blocks;
    const bool ral = aligned16(residuals[t]);
    const bool al = ral && aligned16(tensors[t]);
    e.nblk = batch_absmax_blocks(al ? ns[t] / 4 : ns[t]);
    e.vec = ((e.m % 4 == 0 && ral) ? 1u : 0u) | (ral ? 2u : 0u) | (al ? 4u : 0u);
    blocks += e.nblk;
    tiles += (uint32_t)ceil_div(e.m, kEncTile);
    d.push_back(e);
    which.push_back(t);
  }
  if (d.empty()) return TLC_OK;
  if (blocks > c->partials_cap || tiles > c->enc_status_words)
    return fail(TLC_E_INVALID, "tlc_compress_batch: batch exceeds the context's workspace");
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  const uint32_t cnt = (uint32_t)d.size();
  st = upload(c, c->enc_descs, d.data(), cnt * sizeof(EncDesc));
  if (st) return st;
  arm_results(c->host_results, cnt);
  // default policy: the check pass, then every tile forms acc = x + r itself
  // from its tensor (no writing max pass); in place: step 1 into the buffers
  // with the partial maxima of the sums, then the tiles quantize the buffers
  const bool check = !(c->options & TLC_OPT_IN_PLACE_FEEDBACK);
  if (check) {
    st = timed_launch(c, TLC_KERNEL_ABSMAX_CHECK_BATCH, [&] {
      return launch_absmax_check_batch(c->enc_descs, cnt, blocks, c->partials_chk, c->stream);
    });
  } else {
    st = timed_launch(c, TLC_KERNEL_ABSMAX_BATCH, [&] {
      return launch_accum_absmax_batch(c->enc_descs, cnt, blocks, c->partials, nullptr,
                                       c->stream);
    });
  }
  if (st) return st;
  uint32_t epoch = 0;
  st = next_epoch(c, &c->enc_epoch, kEncEpochMax, c->enc_status, c->enc_status_words, nullptr,
                  &epoch);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_QUANT_ENCODE_BATCH, [&] {
    return launch_quant_encode_batch(c->enc_descs, cnt, tiles,
                                     check ? c->partials_chk : c->partials, check,
                                     c->enc_results, c->enc_status, c->enc_ticket_base, epoch,
                                     c->ctrl, batch_mirror(c), c->stream);
  });
  if (st) return st;
  c->enc_ticket_base += tiles;
  st = wait_results(c, c->host_results, cnt);
  if (st) return st;
  if (c->rb->fault) {
    c->broken = true;
    return fail(TLC_E_DEVICE, "tlc_compress_batch: look-back wait timed out");
  }
  int worst = TLC_OK;
  for (uint32_t i = 0; i < cnt; ++i) {
    const size_t t = which[i];
    const EncResult& r = c->host_results[i];
    if (r.err) {
      status[t] = TLC_E_NONFINITE;
      worst = TLC_E_NONFINITE;
    } else {
      bytes_len[t] = r.len;
      scales[t] = r.scale;
    }
  }
  if (worst) fail(worst, "tlc_compress_batch: NaN/Inf or overflow in at least one tensor");
  return worst;
}

// ---------------------------------------------------------------- decode
namespace {

// Shared checks of one stream; *skip is set for an empty tensor.
int check_stream(const char* fn, size_t t, const uint8_t* bytes, size_t len, float scale,
                 size_t n, const float* out, bool* skip) {
  *skip = false;
  if (!isfinite(scale) || scale < 0.0f)
    return fail(TLC_E_INVALID, "%s: stream %zu: scale %g is not finite and >= 0", fn, t,
                (double)scale);
  if (n == 0) {
    if (len != 0) return fail(TLC_E_CORRUPT, "%s: stream %zu: bytes for an empty tensor", fn, t);
    *skip = true;
    return TLC_OK;
  }
  if (!out || (len && !bytes)) return fail(TLC_E_INVALID, "%s: stream %zu: NULL pointer", fn, t);
  if (len == 0 || len > quartic_len(n))
    return fail(TLC_E_CORRUPT, "%s: stream %zu: length %zu impossible for n = %zu", fn, t, len,
                n);
  if (overlap(bytes, len, out, n * 4))
    return fail(TLC_E_INVALID, "%s: stream %zu: bytes overlap the output", fn, t);
  return TLC_OK;
}

}  // namespace

TLC_API int tlc_decompress(tlc_ctx* c, const uint8_t* bytes, size_t bytes_len, float scale,
                           size_t n, float* out, int accumulate) {
  int st = check_usable(c, "tlc_decompress");
  if (st) return st;
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_decompress: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  bool skip = false;
  st = check_stream("tlc_decompress", 0, bytes, bytes_len, scale, n, out, &skip);
  if (st || skip) return st;
  const size_t m = quartic_len(n);
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  uint32_t epoch = 0;
  st = next_dec_epoch(c, &epoch);
  if (st) return st;
  if (!decode_fused(bytes_len, m)) {  // the scan in a launch of its own
    const uint32_t ntiles = decode_index_tiles(bytes_len, m);
    st = timed_launch(c, TLC_KERNEL_ZRE_INDEX, [&] {
      return launch_zre_index(bytes, (uint32_t)bytes_len, (uint32_t)m, c->start, c->dec_status,
                              ntiles, c->dec_ticket_base, epoch, c->ctrl, fault_mirror(c),
                              c->stream);
    });
    if (st) return st;
  }
  st = timed_launch(c, TLC_KERNEL_EXPAND_DEQUANT, [&] {
    return launch_expand_dequant(bytes, (uint32_t)bytes_len, c->start, c->dec_status,
                                 c->dec_ticket_base, n, m, scale, out, accumulate, epoch,
                                 c->ctrl, fault_mirror(c), c->stream);
  });
  if (st) return st;
  c->dec_ticket_base += decode_tickets(bytes_len, m);
  return TLC_OK;
}

TLC_API int tlc_decompress_ex(tlc_ctx* c, int mode, const uint8_t* bytes, size_t bytes_len,
                              float scale, size_t n, float* out, int accumulate) {
  if (mode == TLC_MODE_3LC || mode == TLC_MODE_NO_ZRE || mode == TLC_MODE_STOCHASTIC)
    return tlc_decompress(c, bytes, bytes_len, scale, n, out, accumulate);
  int st = check_usable(c, "tlc_decompress_ex");
  if (st) return st;
  if (mode != TLC_MODE_INT8)
    return fail(TLC_E_INVALID, "tlc_decompress_ex: unknown mode %d", mode);
  if (!isfinite(scale) || scale < 0.0f)
    return fail(TLC_E_INVALID, "tlc_decompress_ex: scale %g is not finite and >= 0",
                (double)scale);
  if (n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_decompress_ex: n = %zu exceeds the context's max_n %zu", n,
                c->max_n);
  if (bytes_len != n)
    return fail(TLC_E_CORRUPT, "tlc_decompress_ex: %zu bytes for n = %zu int8 codes",
                bytes_len, n);
  if (n == 0) return TLC_OK;
  if (!bytes || !out) return fail(TLC_E_INVALID, "tlc_decompress_ex: NULL pointer");
  if (overlap(bytes, n, out, n * 4))
    return fail(TLC_E_INVALID, "tlc_decompress_ex: bytes overlap the output");
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  return timed_launch(c, TLC_KERNEL_INT8_DEQUANT, [&] {
    return launch_int8_dequant(bytes, n, scale, out, accumulate, c->stream);
  });
}

TLC_API int tlc_decompress_batch(tlc_ctx* c, size_t count, const uint8_t* const* bytes,
                                 const size_t* bytes_len, const float* scales, const size_t* ns,
                                 float* const* outs, int accumulate) {
  int st = check_usable(c, "tlc_decompress_batch");
  if (st) return st;
  if (count == 0) return TLC_OK;
  if (!bytes || !bytes_len || !scales || !ns || !outs)
    return fail(TLC_E_INVALID, "tlc_decompress_batch: NULL argument");
  if (count > c->max_tensors)
    return fail(TLC_E_INVALID, "tlc_decompress_batch: %zu streams exceed the context's %zu",
                count, c->max_tensors);
  size_t total_n = 0;
  std::vector<DecDesc>& d = c->dec_host;
  d.clear();
  uint32_t tiles = 0, ranges = 0;
  for (size_t t = 0; t < count; ++t) {
    if (ns[t] > c->max_n)
      return fail(TLC_E_INVALID, "tlc_decompress_batch: stream %zu: n = %zu too large", t,
                  ns[t]);
    bool skip = false;
    st = check_stream("tlc_decompress_batch", t, bytes[t], bytes_len[t], scales[t], ns[t],
                      outs[t], &skip);
    if (st) return st;
    total_n += ns[t];
    if (skip) continue;
    DecDesc e = {};
    e.C = bytes[t];
    e.out = outs[t];
    e.n = ns[t];
    e.c = (uint32_t)bytes_len[t];
    e.m = (uint32_t)quartic_len(ns[t]);
    e.scale = scales[t];
    e.tile0 = tiles;
    e.range0 = ranges;
    e.vec = aligned16(outs[t]) ? (e.m % 4 == 0 ? 1u : 2u) : 0u;
    tiles += (uint32_t)ceil_div(e.c, kZreBatchTile);
    ranges += (uint32_t)ceil_div(e.m, kDecRange);
    d.push_back(e);
  }
  if (total_n > c->max_n)
    return fail(TLC_E_INVALID, "tlc_decompress_batch: %zu values exceed the context's max_n %zu",
                total_n, c->max_n);
  if (d.empty()) return TLC_OK;
  c->spans.clear();
  for (const DecDesc& e : d) {
    add_span(c->spans, e.C, e.c, false);
    add_span(c->spans, e.out, e.n * 4, true);
  }
  if (spans_conflict_cached(c->spans, c->dec_spans_ok))
    return fail(TLC_E_INVALID, "tlc_decompress_batch: an output overlaps another stream's "
                               "output or bytes");
  if (tiles > c->dec_status_words || ranges > c->start_words)
    return fail(TLC_E_INVALID, "tlc_decompress_batch: batch exceeds the context's workspace");
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  const uint32_t cnt = (uint32_t)d.size();
  st = upload(c, c->dec_descs, d.data(), cnt * sizeof(DecDesc));
  if (st) return st;
  uint32_t epoch = 0;
  st = next_dec_epoch(c, &epoch);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_ZRE_INDEX_BATCH, [&] {
    return launch_zre_index_batch(c->dec_descs, cnt, tiles, c->start, c->dec_status,
                                  c->dec_ticket_base, epoch, c->ctrl, fault_mirror(c),
                                  c->stream);
  });
  if (st) return st;
  c->dec_ticket_base += tiles;
  return timed_launch(c, TLC_KERNEL_EXPAND_DEQUANT_BATCH, [&] {
    return launch_expand_dequant_batch(c->dec_descs, cnt, ranges, c->start, accumulate, epoch,
                                       c->ctrl, c->stream);
  });
}

TLC_API int tlc_decompress_sum(tlc_ctx* c, size_t count, const uint8_t* const* bytes,
                               const size_t* bytes_len, const float* scales, size_t n,
                               float* out, int accumulate) {
  int st = check_usable(c, "tlc_decompress_sum");
  if (st) return st;
  if (count == 0) return fail(TLC_E_INVALID, "tlc_decompress_sum: no streams");
  if (!bytes || !bytes_len || !scales)
    return fail(TLC_E_INVALID, "tlc_decompress_sum: NULL argument");
  if (count > c->max_tensors)
    return fail(TLC_E_INVALID, "tlc_decompress_sum: %zu streams exceed the context's %zu",
                count, c->max_tensors);
  if (n > c->max_n / count)
    return fail(TLC_E_INVALID,
                "tlc_decompress_sum: %zu streams of %zu values exceed the context's max_n %zu",
                count, n, c->max_n);
  const size_t m = quartic_len(n);
  const uint32_t nranges = (uint32_t)ceil_div(m, kDecRange);
  std::vector<DecDesc>& d = c->dec_host;
  d.clear();
  uint32_t tiles = 0;
  for (size_t t = 0; t < count; ++t) {
    bool skip = false;
    st = check_stream("tlc_decompress_sum", t, bytes[t], bytes_len[t], scales[t], n, out, &skip);
    if (st) return st;
    if (skip) continue;  // n == 0: nothing to do for any stream
    DecDesc e = {};
    e.C = bytes[t];
    e.out = out;
    e.n = n;
    e.c = (uint32_t)bytes_len[t];
    e.m = (uint32_t)m;
    e.scale = scales[t];
    e.tile0 = tiles;
    e.range0 = (uint32_t)t * nranges;
    tiles += (uint32_t)ceil_div(e.c, kZreBatchTile);
    d.push_back(e);
  }
  if (d.empty()) return TLC_OK;
  if (tiles > c->dec_status_words || (size_t)count * nranges > c->start_words)
    return fail(TLC_E_INVALID, "tlc_decompress_sum: streams exceed the context's workspace");
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  const uint32_t cnt = (uint32_t)d.size();
  st = upload(c, c->dec_descs, d.data(), cnt * sizeof(DecDesc));
  if (st) return st;
  uint32_t epoch = 0;
  st = next_dec_epoch(c, &epoch);
  if (st) return st;
  st = timed_launch(c, TLC_KERNEL_ZRE_INDEX_BATCH, [&] {
    return launch_zre_index_batch(c->dec_descs, cnt, tiles, c->start, c->dec_status,
                                  c->dec_ticket_base, epoch, c->ctrl, fault_mirror(c),
                                  c->stream);
  });
  if (st) return st;
  c->dec_ticket_base += tiles;
  const int vec = (m % 4 == 0 && aligned16(out)) ? 1 : 0;
  return timed_launch(c, TLC_KERNEL_EXPAND_SUM, [&] {
    return launch_expand_sum(c->dec_descs, cnt, c->start, n, m, out, vec, accumulate, epoch,
                             c->ctrl, c->stream);
  });
}

TLC_API int tlc_sync(tlc_ctx* c) {
  if (!c) return fail(TLC_E_INVALID, "tlc_sync: NULL context");
  DeviceScope dev(c->device);
  int st = dev.status();
  if (st) return st;
  // every kernel that sets the fault or bad-stream flag also writes it
  // into the pinned readback
  st = sync_mirrored(c);
  if (st) return st;
  if (c->rb->fault) {
    c->broken = true;
    return fail(TLC_E_DEVICE, "look-back wait timed out");
  }
  if (c->rb->dec_corrupt) {
    hipError_t e = hipMemsetAsync(&c->ctrl->dec_corrupt, 0, sizeof(uint32_t), c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "tlc_sync: clearing status");
    c->rb->dec_corrupt = 0u;
    return fail(TLC_E_CORRUPT, "a decoded stream did not expand to ceil(n/5) bytes");
  }
  return TLC_OK;
}

TLC_API int tlc_ctx_set_epochs(tlc_ctx* c, uint32_t enc_epoch, uint32_t dec_epoch) {
  int st = check_usable(c, "tlc_ctx_set_epochs");
  if (st) return st;
  if (enc_epoch > kEncEpochMax || dec_epoch > kDecEpochMax)
    return fail(TLC_E_INVALID, "tlc_ctx_set_epochs: epochs %u, %u above %u, %u", enc_epoch,
                dec_epoch, kEncEpochMax, kDecEpochMax);
  DeviceScope dev(c->device);
  st = dev.status();
  if (st) return st;
  // every epoch-tagged word: status words, range starts and the
  // single-stream verdict (a word from an earlier use of an epoch must not
  // match)
  hipError_t e = hipMemsetAsync(c->enc_status, 0, c->enc_status_words * sizeof(uint64_t),
                                c->stream);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->dec_status, 0, c->dec_status_words * sizeof(uint64_t), c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->start, 0, c->start_words * sizeof(uint64_t), c->stream);
  if (e == hipSuccess)
    e = hipMemsetAsync(&c->ctrl->dec_verdict, 0, sizeof(uint32_t), c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "tlc_ctx_set_epochs");
  c->enc_epoch = enc_epoch;
  c->dec_epoch = dec_epoch;
  return TLC_OK;
}

// ---------------------------------------------------------------- profiling
TLC_API int tlc_profile_enable(tlc_ctx* c, int on) {
  if (!c) return fail(TLC_E_INVALID, "tlc_profile_enable: NULL context");
  c->profiling = on != 0;
  return TLC_OK;
}

TLC_API int tlc_profile_mask(tlc_ctx* c, uint32_t mask) {
  if (!c) return fail(TLC_E_INVALID, "tlc_profile_mask: NULL context");
  c->profile_mask = mask;
  return TLC_OK;
}

TLC_API int tlc_profile_get(tlc_ctx* c, int kernel, double* total_ms, uint64_t* launches) {
  if (!c || !total_ms || !launches || kernel < 0 || kernel >= TLC_KERNEL_COUNT)
    return fail(TLC_E_INVALID, "tlc_profile_get: bad argument");
  DeviceScope dev(c->device);
  int st = dev.status();
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
  DeviceScope dev(c->device);
  int st = dev.status();
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
