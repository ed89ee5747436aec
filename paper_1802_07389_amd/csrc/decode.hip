// decode.hip -- gfx950 decode kernels of the 3LC path.
//
//   tlc_zre_index_kernel / _batch_kernel
//       zero-run scan: where each kDecRange-byte range of quartic bytes
//       starts in the stream; checks the expanded length
//   tlc_expand_dequant_kernel / _batch_kernel
//       zero-run expansion into LDS, quartic unpack (Section 3.2), Eq. 3,
//       optional accumulate; a small stream's decode runs the scan in the
//       first blocks of the same launch
//   tlc_expand_sum_kernel
//       the same for P streams of one tensor, summed in stream order into
//       one output in a single pass over it (server-side aggregation)
//
// The quartic bytes are never stored in HBM: each block rebuilds its range
// of them in LDS from the stream.
#include "device_common.hpp"

namespace tlc {

// ---------------------------------------------------------------- index scan
// A start entry: (stream byte << 8 | how far into its expansion) with the
// launch's epoch above it, published with an agent-scope atomic store like
// a look-back status word, so that a reader in the same launch knows by the
// tag alone that the entry is this launch's.  The byte index is below 2^30
// (a stream is at most m < 2^30 bytes) and the offset below 14.
constexpr int kStartPayloadBits = 38;
constexpr uint64_t kStartPayloadMask = (uint64_t(1) << kStartPayloadBits) - 1u;
static_assert(kDecEpochMax < (1u << (64 - kStartPayloadBits)), "the epoch fits above the payload");

__device__ __forceinline__ uint64_t start_payload(uint64_t w) { return w & kStartPayloadMask; }
__device__ __forceinline__ uint32_t start_epoch(uint64_t w) {
  return (uint32_t)(w >> kStartPayloadBits);
}

// The last index tile's verdict on the stream, for the same launch's
// expanding blocks: epoch << 1 | 1 when the expansion total is not m (or a
// look-back gave up), epoch << 1 when it is.
__device__ __forceinline__ uint32_t verdict_word(uint32_t epoch, bool bad) {
  return (epoch << 1) | (bad ? 1u : 0u);
}

struct IdxShared {
  uint32_t red[kWaves];
  uint32_t fault;
  uint64_t excl;
};

// Tile `lt` (kThreads * kBytes stream bytes) of one stream: expansion lengths are
// scanned in the block and across tiles (decoupled look-back, status slot
// floor + lt), which places every stream byte's expansion in the quartic
// byte string.  The byte whose expansion contains position k * kDecRange
// records (its index, how far into its expansion that position lies) in
// start[k], so each expanding block finds its part of the stream with one
// load.  The stream's last tile flags the launch's epoch as corrupt when
// the expansion total is not exactly m.
template <int kBytes>
__device__ __forceinline__ void index_tile(const uint8_t* __restrict__ C, uint32_t c, uint32_t m,
                                           uint64_t* __restrict__ start,
                                           uint64_t* __restrict__ status, uint32_t floor,
                                           uint32_t lt, uint32_t epoch, Ctrl* __restrict__ ctrl,
                                           uint32_t* hfault, uint32_t* hcorrupt,
                                           IdxShared& sh) {
  constexpr uint32_t kTile = kThreads * kBytes;
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint64_t j0 = (uint64_t)lt * kTile + threadIdx.x * kBytes;
  const uint32_t cnt = j0 < c ? (uint32_t)umin64(kBytes, c - j0) : 0u;

  // the thread's bytes stay packed four to a word; byte i is bits 8*(i%4) of w[i/4]
  uint32_t w[kBytes / 4];
  if (cnt == (uint32_t)kBytes && ((reinterpret_cast<uintptr_t>(C + j0) & 15u) == 0u)) {
#pragma unroll
    for (int h = 0; h < kBytes / 16; ++h) {
      const uint4 v = *reinterpret_cast<const uint4*>(C + j0 + 16 * h);
      w[4 * h] = v.x;
      w[4 * h + 1] = v.y;
      w[4 * h + 2] = v.z;
      w[4 * h + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < kBytes / 4; ++q) {
      uint32_t x = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((uint32_t)(4 * q + i) < cnt) x |= (uint32_t)C[j0 + 4 * q + i] << (8 * i);
      w[q] = x;
    }
  }
  // one quartic byte per stream byte and the runs' extra bytes word by
  // word (the zero bytes past cnt add nothing)
  uint32_t wx[kBytes / 4];
  uint32_t sum = cnt;
#pragma unroll
  for (int q = 0; q < kBytes / 4; ++q) {
    wx[q] = run_extra4(w[q]);
    sum += wx[q];
  }
  const ScanU32 sc = block_scan_u32(sum, sh.red);
  const uint32_t agg = sc.total;

  if (wid == 0) {
    bool fault = false;
    uint64_t ex = 0;
    if (lt == 0) {
      if (lane == 0) status_publish(&status[floor], DecSW::pack(agg, kFlagPrefix, epoch));
    } else {
      ex = lookback_wave<DecSW>(status, floor, floor + lt, agg, 0, epoch, SumOp(), &fault);
    }
    if (lane == 0) {
      sh.excl = ex;
      sh.fault = fault ? 1u : 0u;
      if (fault) {
        __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        host_put(hfault, 1u);
      }
      const bool last_tile = (uint64_t)(lt + 1) * kTile >= c;
      const bool bad = fault || ex + agg != m;
      if (last_tile && bad) {
        __hip_atomic_store(&ctrl->dec_bad_epoch, epoch, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&ctrl->dec_corrupt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        host_put(hcorrupt, 1u);
      }
      if (last_tile)
        __hip_atomic_store(&ctrl->dec_verdict, verdict_word(epoch, bad), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (sh.fault) return;

  // The thread's bytes expand to at most 14 * kBytes < kDecRange quartic
  // bytes, so at most one range start falls among them: the first one at or
  // after the thread's first position o.
  static_assert(14 * kBytes < kDecRange, "one range start per thread at most");
  const uint64_t o = sh.excl + sc.excl;
  const uint64_t k = (o + kDecRange - 1) / kDecRange;
  const uint64_t at = k * kDecRange;
  if (at < m && at < o + sum) {
    const uint32_t d = (uint32_t)(at - o);  // the start's distance into the thread's expansion
    // The word whose expansion holds position d (the words' expansions tile
    // [0, sum), so exactly one has d - rel < its length), then the byte in
    // it.  Every word before it holds four of the thread's bytes; the zero
    // bytes past cnt come after the start's byte and are never reached.
    uint32_t rel = 0, hq = 0, hw = 0, hrel = 0;
#pragma unroll
    for (int q = 0; q < kBytes / 4; ++q) {
      const uint32_t wl = 4u + wx[q];
      const bool here = d - rel < wl;  // d < rel wraps to a large difference
      hq = here ? (uint32_t)q : hq;
      hw = here ? w[q] : hw;
      hrel = here ? rel : hrel;
      rel += wl;
    }
    uint32_t hit = 4u * hq, into = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t len = expanded_len((hw >> (8 * c)) & 255u);
      const bool here = d - hrel < len;
      hit = here ? 4u * hq + (uint32_t)c : hit;
      into = here ? d - hrel : into;
      hrel += len;
    }
    status_publish(&start[k], ((uint64_t)epoch << kStartPayloadBits) | ((j0 + hit) << 8) | into);
  }
}

__global__ __launch_bounds__(kThreads) void tlc_zre_index_kernel(
    const uint8_t* __restrict__ C, uint32_t c, uint32_t m, uint64_t* __restrict__ start,
    uint64_t* __restrict__ status, uint32_t ticket_base, uint32_t epoch,
    Ctrl* __restrict__ ctrl, HostMirror hm) {
  __shared__ IdxShared sh;
  __shared__ uint32_t s_tile;
  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->dec_ticket) - ticket_base;
  __syncthreads();
  index_tile<kZreBytesPerThread>(C, c, m, start, status, 0, s_tile, epoch, ctrl, hm.fault,
                                 hm.corrupt, sh);
}

__global__ __launch_bounds__(kThreads) void tlc_zre_index_batch_kernel(
    const DecDesc* __restrict__ descs, uint32_t count, uint64_t* __restrict__ start,
    uint64_t* __restrict__ status, uint32_t ticket_base, uint32_t epoch,
    Ctrl* __restrict__ ctrl, HostMirror hm) {
  __shared__ IdxShared sh;
  __shared__ uint32_t s_tile;
  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->dec_ticket) - ticket_base;
  __syncthreads();
  const uint32_t T = s_tile;
  const uint32_t t = find_desc(descs, count, T, [](const DecDesc& d) { return d.tile0; });
  const DecDesc d = descs[t];
  index_tile<kZreBatchBytesPerThread>(d.C, d.c, d.m, start + d.range0, status, d.tile0,
                                      T - d.tile0, epoch, ctrl, hm.fault, hm.corrupt, sh);
}

// ---------------------------------------------------------------- expansion
// The stream bytes that expand into range k of one stream: the first one,
// how far into its expansion the range starts, and how many (at most
// kDecRange: the range's qn quartic bytes come from at most qn stream bytes).
// s0, s1: the payloads of the start entries of ranges k and k + 1 (s1 is
// not read when range k is the stream's last).
struct Slice {
  uint32_t i0, skip, count;
};

__device__ __forceinline__ Slice slice_from(uint64_t s0, uint64_t s1, bool last, uint32_t c) {
  Slice r;
  r.i0 = (uint32_t)(s0 >> 8);
  r.skip = (uint32_t)(s0 & 255u);
  // one past the last stream byte that reaches into the range
  const uint32_t i1 = last ? c : umin32((uint32_t)(s1 >> 8) + ((s1 & 255u) ? 1u : 0u), c);
  r.count = i1 > r.i0 ? umin32(i1 - r.i0, kDecRange) : 0u;
  return r;
}

// The same from the start entries of a stream that an earlier launch wrote.
__device__ __forceinline__ Slice slice_of(const uint64_t* __restrict__ starts, uint32_t k,
                                          uint64_t m, uint32_t c) {
  const bool last = (uint64_t)(k + 1) * kDecRange >= m;
  return slice_from(start_payload(starts[k]), last ? 0u : start_payload(starts[k + 1]), last,
                    c);
}

constexpr int kSliceBytes = kDecRange / kThreads;  // stream bytes per thread (at most)

// Expands a slice into s_q, the range's quartic bytes [0, qn): the thread
// holds slice bytes lo .. lo + cnt - 1 (lo = threadIdx.x * kSliceBytes),
// byte(i) giving byte lo + i.  Every run code expands to bytes of 121, so
// the range is first filled with 121 (one 16-byte store per thread, before
// the scan's barrier) and only the data bytes other than 121 are written,
// each at the position a block scan of the expansion lengths gives it: the
// work no longer follows the length of the runs a thread holds.  The same
// scan counts those data bytes (packed as length + (count << 16): a slice
// expands to fewer than kDecRange + 28 bytes and holds at most kDecRange
// bytes, so no carry crosses), which is returned.  Ends with a barrier.
static_assert(kDecRange == 16 * kThreads, "the fill of s_q is one uint4 per thread");
template <class ByteAt>
__device__ __forceinline__ uint32_t expand_slice(ByteAt byte, uint32_t cnt, uint32_t skip,
                                                 uint32_t qn, uint8_t* s_q, uint32_t* red) {
  reinterpret_cast<uint4*>(s_q)[threadIdx.x] =
      make_uint4(0x79797979u, 0x79797979u, 0x79797979u, 0x79797979u);
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kSliceBytes; ++i) {
    if ((uint32_t)i < cnt) {
      const uint32_t x = byte(i);
      sum += expanded_len(x) + (x < kRunBase && x != kZeroGroup ? 1u << 16 : 0u);
    }
  }
  const ScanU32 sc = block_scan_u32(sum, red);
  int pos = (int)(sc.excl & 0xffffu) - (int)skip;  // range-relative start of byte 0
#pragma unroll
  for (int i = 0; i < kSliceBytes; ++i) {
    if ((uint32_t)i < cnt) {
      const uint32_t x = byte(i);
      if (x < kRunBase && x != kZeroGroup && pos >= 0 && pos < (int)qn) s_q[pos] = (uint8_t)x;
      pos += (int)expanded_len(x);
    }
  }
  __syncthreads();
  return sc.total >> 16;
}

// Expands quartic bytes [k*kDecRange, k*kDecRange + qn) of one stream into
// s_q (the stream bytes covering the range found through the start entries,
// spread over the threads); returns the slice's count of data bytes other
// than 121.  Ends with a barrier.
__device__ __forceinline__ uint32_t expand_range(const uint8_t* __restrict__ C, uint32_t c,
                                             const uint64_t* __restrict__ starts, uint32_t k,
                                             uint64_t m, uint32_t qn, uint8_t* s_q,
                                             uint32_t* red) {
  const Slice sl = slice_of(starts, k, m, c);
  const uint32_t lo = threadIdx.x * kSliceBytes;
  const uint32_t cnt = lo < sl.count ? umin32(kSliceBytes, sl.count - lo) : 0u;
  uint8_t b[kSliceBytes];
#pragma unroll
  for (int i = 0; i < kSliceBytes; ++i) b[i] = (uint32_t)i < cnt ? C[sl.i0 + lo + i] : (uint8_t)0;
  return expand_slice([&](int i) -> uint32_t { return b[i]; }, cnt, sl.skip, qn, s_q, red);
}

// ---------------------------------------------------------------- Eq. 3
// Partition K of quartic bytes s_q[0, qn) (global bytes q0 + jl) when out
// is 16-byte aligned: the partition starts a = (K*m + q0) mod 4 values past
// a float4 boundary (a = 0 when m % 4 == 0), and cell f of its aligned
// float4 grid takes digit K of bytes 4f - a .. 4f + 3 - a (two LDS words).
// Cells shared with a neighbouring range or partition, or reaching past n,
// are written value by value.  The block sweeps one partition at a time.
// kNT: the full cells use nontemporal loads and stores.  That pays when out
// is far larger than the 256 MB last-level cache: on gfx950 the hinted
// sweep then beat the plain one and five-partition float4 groups, and its
// stores leave no dirty lines for the next encode to write back.  Outputs
// that fit the cache decode faster with plain accesses.
constexpr int kSweepCells = (kDecRange + 6) / 4 / kThreads + 1;  // cells per lane, a <= 3

// Accumulating, a sweep stores only the float4s whose sums change bits,
// unless its range's stream slice has more than this many data bytes other
// than 121: then most float4s change, and storing every one keeps the
// writes a contiguous stream (scattered stores inside the read stream cost
// far more than their bytes).  Either way every value gets out + M*q.
constexpr uint32_t kDenseLiterals = kDecRange / 4;

// The kAcc loads of partition K's full cells (the cells the sweep below
// adds to), issued before the range's zero-run expansion so that their
// latency overlaps it.
template <int K, bool kNT>
__device__ __forceinline__ void sweep_preload(uint64_t q0, uint32_t qn, uint64_t n, uint64_t m,
                                              const float* __restrict__ out,
                                              float4 (&o)[kSweepCells]) {
  const uint64_t base = (uint64_t)K * m + q0;
  const uint32_t a = (uint32_t)(base & 3u);
  const uint64_t e0 = base - a;
  const uint32_t nf = (qn + a + 3u) >> 2;
#pragma unroll
  for (int i = 0; i < kSweepCells; ++i) {
    const uint32_t f = threadIdx.x + kThreads * i;
    if (f < nf && 4u * f >= a && 4u * f + 4u <= qn + a && e0 + 4ull * f + 4u <= n)
      o[i] = kNT ? ld_stream(out + e0 + 4ull * f)
                 : *reinterpret_cast<const float4*>(out + e0 + 4ull * f);
  }
}

template <int K, bool kAcc, bool kNT, bool kPre = false>
__device__ __forceinline__ void dequant_partition_shifted(const uint8_t* s_q, uint64_t q0,
                                                          uint32_t qn, uint64_t n, uint64_t m,
                                                          float M, float* __restrict__ out,
                                                          bool dense,
                                                          const float4* pre = nullptr) {
  constexpr uint32_t kPlace = K == 0 ? 81u : (K == 1 ? 27u : (K == 2 ? 9u : (K == 3 ? 3u : 1u)));
  constexpr int kCells = kSweepCells;
  const uint32_t* qw = reinterpret_cast<const uint32_t*>(s_q);
  const uint64_t base = (uint64_t)K * m + q0;
  const uint32_t a = (uint32_t)(base & 3u);
  const uint64_t e0 = base - a;
  const uint32_t nf = (qn + a + 3u) >> 2;
  float4 o[kCells];
  bool full[kCells];
#pragma unroll
  for (int i = 0; i < kCells; ++i) {
    const uint32_t f = threadIdx.x + kThreads * i;
    full[i] = f < nf && 4u * f >= a && 4u * f + 4u <= qn + a && e0 + 4ull * f + 4u <= n;
    if (kAcc && full[i]) {
      if (kPre)
        o[i] = pre[i];
      else
        o[i] = kNT ? ld_stream(out + e0 + 4ull * f)
                   : *reinterpret_cast<const float4*>(out + e0 + 4ull * f);
    }
  }
#pragma unroll
  for (int i = 0; i < kCells; ++i) {
    const uint32_t f = threadIdx.x + kThreads * i;
    if (f >= nf) break;
    const uint64_t e = e0 + 4ull * f;
    // bytes 4f - a .. 4f + 3 - a: the top a bytes of word f - 1, then word f
    const uint32_t lo = (a != 0u && f >= 1u) ? qw[f - 1] : 0u;
    const uint32_t hi = 4u * f < qn ? qw[f] : 0u;
    const uint32_t w4 = a ? (uint32_t)((((uint64_t)hi << 32) | lo) >> (8u * (4u - a))) : hi;
    uint32_t d[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) d[c] = (((w4 >> (8 * c)) & 0xffu) / kPlace) % 3u;
    if (full[i]) {
      bool store = true;
      if (kAcc) {
        store = acc_trit4(o[i], d, M) || dense;
      } else {
        o[i] = make_float4(trit_value(d[0], M), trit_value(d[1], M), trit_value(d[2], M),
                           trit_value(d[3], M));
      }
      if (store) {
        if (kNT)
          st_stream(out + e, o[i]);
        else
          *reinterpret_cast<float4*>(out + e) = o[i];
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t p = 4u * f + c;
        if (p >= a && p - a < qn && e + c < n) {
          if (kAcc)
            acc_trit_at(out, e + c, d[c], M);
          else
            out[e + c] = trit_value(d[c], M);
        }
      }
    }
  }
}

// Unpacks the base-3 digits of quartic bytes s_q[0, qn) (global bytes
// q0 + jl), dequantizes (Eq. 3) and stores or accumulates into the five
// partitions of out.  kPathShift: aligned float4 cells partition by
// partition (aligned out; the large outputs also take the nontemporal
// hint).  kPathVec: each lane takes 4 bytes and their five float4 slices
// at once (aligned out, m % 4 == 0; fewer dependent memory round trips per
// block, which is what outputs that fit the cache are bound by).
// kPathByte: one quartic byte per lane with scalar accesses.
template <int kPath, bool kAcc, bool kNT = false>
__device__ __forceinline__ void dequant_range(const uint8_t* s_q, uint64_t q0, uint32_t qn,
                                              uint64_t n, uint64_t m, float M,
                                              float* __restrict__ out, bool dense) {
  if (kPath == kPathShift) {
    dequant_partition_shifted<0, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<1, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<2, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<3, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<4, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
  } else if (kPath == kPathVec) {
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
          bool store = true;
          if (kAcc) {
            const uint32_t dk[4] = {t[0][k], t[1][k], t[2][k], t[3][k]};
            store = acc_trit4(o[k], dk, M) || dense;
          } else {
            o[k].x = trit_value(t[0][k], M);
            o[k].y = trit_value(t[1][k], M);
            o[k].z = trit_value(t[2][k], M);
            o[k].w = trit_value(t[3][k], M);
          }
          if (store) *reinterpret_cast<float4*>(out + k * m + j) = o[k];
        }
      } else {  // the group whose p4 slice reaches into the padding
#pragma unroll
        for (int k = 0; k < 5; ++k) {
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const uint64_t e = k * m + j + cc;
            if (e < n) {
              if (kAcc)
                acc_trit_at(out, e, t[cc][k], M);
              else
                out[e] = trit_value(t[cc][k], M);
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
          if (kAcc)
            acc_trit_at(out, e, t[k], M);
          else
            out[e] = trit_value(t[k], M);
        }
      }
    }
  }
}

// Lane 0 of an expanding block: waits for a start entry of this launch (its
// epoch tag) and returns its payload.  Gives up (kNoStart) when the
// launch's verdict says the stream is bad (its entries may never come) or
// the wait runs past kSpinLimit (then the fault flag is set).
constexpr uint64_t kNoStart = ~uint64_t(0);  // above any payload

// Up to a few thousand resident blocks wait at once, so they poll gently:
// a pause of 8 * 64 clocks between reads, and the verdict on every fourth.
__device__ uint64_t wait_start(const uint64_t* p, uint32_t epoch, Ctrl* ctrl, uint32_t* hfault) {
  for (uint32_t spins = 0;; ++spins) {
    const uint64_t v = status_read(p);
    if (start_epoch(v) == epoch) return start_payload(v);
    if ((spins & 3u) == 3u) {
      const uint32_t vd = __hip_atomic_load(&ctrl->dec_verdict, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
      if (vd == verdict_word(epoch, true)) return kNoStart;
    }
    if (spins > kSpinLimit) {
      __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      host_put(hfault, 1u);
      return kNoStart;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}

// Lane 0 of an expanding block: waits for the launch's verdict; true when
// the stream is good.
__device__ bool wait_verdict(uint32_t epoch, Ctrl* ctrl, uint32_t* hfault) {
  for (uint32_t spins = 0;; ++spins) {
    const uint32_t vd = __hip_atomic_load(&ctrl->dec_verdict, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
    if ((vd >> 1) == epoch) return (vd & 1u) == 0u;
    if (spins > kSpinLimit) {
      __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      host_put(hfault, 1u);
      return false;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}

// One stream's expansion: range k (quartic bytes [k*kDecRange,
// (k+1)*kDecRange)) per block.
// kFused = false: the scan ran in its own launch before; range k =
// blockIdx.x, the start entries are read as they are, and a corrupt stream
// (flagged by the scan) is left alone.
// kFused = true (small decodes, every block resident at once): blocks take
// tickets in order; the first `ntiles` run the scan (index_tile), every
// later one expands range k = ticket - ntiles.  An expanding block issues
// the output loads it can, waits for its start entries (tagged with the
// launch's epoch, written by scan tiles, which hold lower tickets and so
// already run), expands the range into LDS, and waits for the last scan
// tile's verdict before it stores anything: a corrupt stream leaves out
// untouched.  The scan's latency then overlaps the expanding blocks' work
// and no kernel boundary separates the two steps.
template <int kPath, bool kAcc, bool kNT, bool kFused>
__global__ __launch_bounds__(kThreads) void tlc_expand_dequant_kernel(
    const uint8_t* __restrict__ C, uint32_t c, uint64_t* __restrict__ start,
    uint64_t* __restrict__ status, uint32_t ntiles, uint32_t ticket_base, uint64_t n,
    uint64_t m, float M, float* __restrict__ out, uint32_t epoch, Ctrl* __restrict__ ctrl,
    HostMirror hm) {
  __shared__ IdxShared ish;
  __shared__ uint32_t red[kWaves];
  __shared__ __align__(16) uint8_t s_q[kDecRange];
  __shared__ uint32_t s_t, s_ok;
  __shared__ uint64_t s_se[2];
  uint32_t k;
  if constexpr (kFused) {
    if (threadIdx.x == 0) s_t = take_ticket(&ctrl->dec_ticket) - ticket_base;
    __syncthreads();
    const uint32_t T = s_t;
    if (T < ntiles) {
      index_tile<kZreBatchBytesPerThread>(C, c, (uint32_t)m, start, status, 0, T, epoch, ctrl,
                                          hm.fault, hm.corrupt, ish);
      return;
    }
    k = T - ntiles;
  } else {
    if (ctrl->dec_bad_epoch == epoch) return;  // corrupt stream: out untouched
    k = blockIdx.x;
  }
  const uint64_t q0 = (uint64_t)k * kDecRange;
  const uint32_t qn = (uint32_t)umin64(kDecRange, m - q0);
  const bool last = q0 + kDecRange >= m;
  constexpr bool kPre = kPath == kPathShift && kAcc && kNT;
  // large outputs: the first two partitions' loads go out before the
  // expansion (on gfx950 15 us of 410 on a 2^28-value decode; outputs that
  // fit the cache gained nothing)
  float4 p0[kPre ? kSweepCells : 1], p1[kPre ? kSweepCells : 1];
  if constexpr (kPre) {
    sweep_preload<0, kNT>(q0, qn, n, m, out, p0);
    sweep_preload<1, kNT>(q0, qn, n, m, out, p1);
  }
  Slice sl;
  if constexpr (kFused) {
    if (threadIdx.x == 0) {
      const uint64_t s0 = wait_start(&start[k], epoch, ctrl, hm.fault);
      const uint64_t s1 =
          last || s0 == kNoStart ? 0u : wait_start(&start[k + 1], epoch, ctrl, hm.fault);
      s_se[0] = s0;
      s_se[1] = s1;
      s_ok = s0 != kNoStart && s1 != kNoStart ? 1u : 0u;
    }
    __syncthreads();
    if (!s_ok) return;
    sl = slice_from(s_se[0], s_se[1], last, c);
  } else {
    sl = slice_of(start, k, m, c);
  }
  const uint32_t lo = threadIdx.x * kSliceBytes;
  const uint32_t cnt = lo < sl.count ? umin32(kSliceBytes, sl.count - lo) : 0u;
  uint8_t b[kSliceBytes];
#pragma unroll
  for (int i = 0; i < kSliceBytes; ++i) b[i] = (uint32_t)i < cnt ? C[sl.i0 + lo + i] : (uint8_t)0;
  const bool dense =
      expand_slice([&](int i) -> uint32_t { return b[i]; }, cnt, sl.skip, qn, s_q, red) >
      kDenseLiterals;
  if constexpr (kFused) {
    if (threadIdx.x == 0) s_ok = wait_verdict(epoch, ctrl, hm.fault) ? 1u : 0u;
    __syncthreads();
    if (!s_ok) return;  // a corrupt stream: out untouched
  }
  if constexpr (kPre) {
    dequant_partition_shifted<0, kAcc, kNT, true>(s_q, q0, qn, n, m, M, out, dense, p0);
    dequant_partition_shifted<1, kAcc, kNT, true>(s_q, q0, qn, n, m, M, out, dense, p1);
    dequant_partition_shifted<2, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<3, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
    dequant_partition_shifted<4, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
  } else {
    dequant_range<kPath, kAcc, kNT>(s_q, q0, qn, n, m, M, out, dense);
  }
}

template <bool kAcc>
__global__ __launch_bounds__(kThreads) void tlc_expand_dequant_batch_kernel(
    const DecDesc* __restrict__ descs, uint32_t count, const uint64_t* __restrict__ start,
    uint32_t epoch, const Ctrl* __restrict__ ctrl) {
  __shared__ uint32_t red[kWaves];
  __shared__ __align__(16) uint8_t s_q[kDecRange];
  if (ctrl->dec_bad_epoch == epoch) return;  // a corrupt stream: no output written
  const uint32_t t =
      find_desc(descs, count, blockIdx.x, [](const DecDesc& d) { return d.range0; });
  const DecDesc d = descs[t];
  const uint32_t k = blockIdx.x - d.range0;
  const uint64_t q0 = (uint64_t)k * kDecRange;
  const uint32_t qn = (uint32_t)umin64(kDecRange, (uint64_t)d.m - q0);
  const bool dense =
      expand_range(d.C, d.c, start + d.range0, k, d.m, qn, s_q, red) > kDenseLiterals;
  if (d.vec & 1u)
    dequant_range<kPathVec, kAcc>(s_q, q0, qn, d.n, d.m, d.scale, d.out, dense);
  else if (d.vec & 2u)
    dequant_range<kPathShift, kAcc>(s_q, q0, qn, d.n, d.m, d.scale, d.out, dense);
  else
    dequant_range<kPathByte, kAcc>(s_q, q0, qn, d.n, d.m, d.scale, d.out, dense);
}

// ---------------------------------------------------------------- aggregation
// Streams whose slices a block stages per pass of the summed decode: one
// wave reads their descriptors and start entries together.
constexpr int kSumChunk = 64;
// Stream bytes a wave expands per round (16 per lane).
constexpr uint32_t kWaveSliceBytes = 64u * 16u;

struct SumSlice {
  const uint8_t* C;  // the slice's first byte
  uint32_t count;
  uint32_t skip;
  float scale;
  uint32_t pad;
};

// Stream bytes lo .. lo + 15 of a slice (those below count) as words,
// byte i in bits 8 * (i % 4) of word i / 4 once aligned by sh.  Reads only
// the aligned dwords that hold them (none when lo >= count): each dword
// read holds at least one byte of the slice, so no read leaves the pages
// the stream lies in.  Bytes past the slice's end are unspecified and
// never used.
struct SliceWords {
  uint32_t w[5];
  uint32_t sh;  // byte offset of the first byte inside w[0]
};

__device__ __forceinline__ SliceWords load_slice_words(const SumSlice& s, uint32_t lo) {
  const uint32_t cnt = lo < s.count ? umin32(16u, s.count - lo) : 0u;
  const uintptr_t first = reinterpret_cast<uintptr_t>(s.C) + lo;
  const uint32_t* base = reinterpret_cast<const uint32_t*>(first & ~(uintptr_t)3);
  SliceWords r;
  r.sh = (uint32_t)(first & 3u);
#pragma unroll
  for (int j = 0; j < 5; ++j) r.w[j] = cnt && (uint32_t)(4 * j) < r.sh + cnt ? base[j] : 0u;
  return r;
}

__device__ __forceinline__ uint32_t slice_word_byte(const SliceWords& s, int i) {
  // byte i lies in w[(sh + i) / 4]; alignbyte selects it from a word pair
  const uint32_t q = (uint32_t)i >> 2;
  const uint32_t word = __builtin_amdgcn_alignbyte(s.w[q + 1], s.w[q], s.sh);
  return (word >> (8 * (i & 3))) & 255u;
}

// One wave expands a slice into s_q (the range's quartic bytes [0, qn)):
// it fills the range with 121, then each lane takes 16 stream bytes per
// round, a wave scan of their expansion lengths places them, and the data
// bytes other than 121 are written.  `pre` holds the lane's bytes of the
// first round.  No block barrier: the caller's barrier publishes s_q.
__device__ __forceinline__ void wave_expand(const SumSlice& sl, const SliceWords& pre,
                                            uint32_t qn, uint8_t* s_q) {
  const uint32_t lane = threadIdx.x & 63u;
#pragma unroll
  for (int i = 0; i < kDecRange / (16 * 64); ++i)
    reinterpret_cast<uint4*>(s_q)[lane + 64 * i] =
        make_uint4(0x79797979u, 0x79797979u, 0x79797979u, 0x79797979u);
  int base = -(int)sl.skip;  // range-relative start of the round's first byte
  for (uint32_t r0 = 0; r0 < sl.count; r0 += kWaveSliceBytes) {
    const uint32_t lo = r0 + 16u * lane;
    const SliceWords w = r0 == 0 ? pre : load_slice_words(sl, lo);
    const uint32_t cnt = lo < sl.count ? umin32(16u, sl.count - lo) : 0u;
    uint32_t len = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if ((uint32_t)i < cnt) len += expanded_len(slice_word_byte(w, i));
    const uint32_t incl = wave_incl_scan(len, 0u, OpAdd());
    int pos = base + (int)(incl - len);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if ((uint32_t)i < cnt) {
        const uint32_t x = slice_word_byte(w, i);
        if (x < kRunBase && x != kZeroGroup && pos >= 0 && pos < (int)qn) s_q[pos] = (uint8_t)x;
        pos += (int)expanded_len(x);
      }
    }
    base += (int)wave_last(incl);
  }
}

// Range k of `count` streams of the same n-value tensor, summed into out in
// stream order per element (out = ((out + v0) + v1) + ..., or starting
// from v0 without accumulate): the same fp32 additions, in the same order,
// as decoding the streams one after another, but out is read and written
// once.  Values stay in registers between streams.  The descriptors and
// start entries of up to kSumChunk streams are read in one round trip; the
// streams then go in groups of kWaves, one per wave, each expanded by its
// wave into its own LDS range, with one block barrier per group; the next
// group's bytes load while the current group is summed, and the groups'
// LDS ranges alternate between two sets.
template <bool kVec, bool kAcc>
__global__ __launch_bounds__(kThreads) void tlc_expand_sum_kernel(
    const DecDesc* __restrict__ descs, uint32_t count, const uint64_t* __restrict__ start,
    uint64_t n, uint64_t m, float* __restrict__ out, uint32_t epoch,
    const Ctrl* __restrict__ ctrl) {
  constexpr int kPer = kVec ? kDecRange / kThreads / 4 : kDecRange / kThreads;  // slots
  constexpr int kW = kVec ? 4 : 1;                                              // bytes/slot
  constexpr uint32_t kZeroWord = kVec ? 0x79797979u : kZeroGroup;  // a slot of zero groups
  __shared__ __align__(16) uint8_t s_q[2][kWaves][kDecRange];
  __shared__ SumSlice s_sl[kSumChunk];
  if (ctrl->dec_bad_epoch == epoch) return;  // a corrupt stream: out untouched
  const uint32_t k = blockIdx.x;
  const uint64_t q0 = (uint64_t)k * kDecRange;
  const uint32_t qn = (uint32_t)umin64(kDecRange, m - q0);
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;

  // slot g covers quartic bytes jl(g) .. jl(g) + kW - 1 and their 5 partitions
  float acc[kPer][5][kW];
  auto jl_of = [&](int g) -> uint32_t {
    return kVec ? 4u * (threadIdx.x + kThreads * g) : threadIdx.x + kThreads * g;
  };
  if (kAcc) {
#pragma unroll
    for (int g = 0; g < kPer; ++g) {
      const uint32_t jl = jl_of(g);
      if (jl >= qn) continue;
      const uint64_t j = q0 + jl;
#pragma unroll
      for (int kk = 0; kk < 5; ++kk) {
        if (kVec && 4 * m + j + 4 <= n) {
          const float4 v = *reinterpret_cast<const float4*>(out + kk * m + j);
          acc[g][kk][0] = v.x;
          acc[g][kk][kW > 1 ? 1 : 0] = v.y;
          acc[g][kk][kW > 2 ? 2 : 0] = v.z;
          acc[g][kk][kW > 3 ? 3 : 0] = v.w;
        } else {
#pragma unroll
          for (int cc = 0; cc < kW; ++cc) {
            const uint64_t e = kk * m + j + cc;
            acc[g][kk][cc] = e < n ? out[e] : 0.0f;
          }
        }
      }
    }
  }

  bool clean = false;  // no value is -0.0 and every NaN is quiet
  for (uint32_t p0 = 0; p0 < count; p0 += kSumChunk) {
    const uint32_t pc = umin32(kSumChunk, count - p0);
    if (threadIdx.x < pc) {
      const DecDesc d = descs[p0 + threadIdx.x];
      const Slice sl = slice_of(start + d.range0, k, m, d.c);
      s_sl[threadIdx.x] = SumSlice{d.C + sl.i0, sl.count, sl.skip, d.scale, 0u};
    }
    __syncthreads();
    SliceWords cur{};
    if (wid < pc) cur = load_slice_words(s_sl[wid], 16u * lane);
    for (uint32_t g0 = 0; g0 < pc; g0 += kWaves) {
      const uint32_t gn = umin32(kWaves, pc - g0);
      SliceWords nxt{};
      if (g0 + kWaves + wid < pc) nxt = load_slice_words(s_sl[g0 + kWaves + wid], 16u * lane);
      // Group g0 / kWaves fills set (g0 / kWaves) & 1.  A wave reaches that
      // fill only past the barrier of the previous group, which every
      // thread passes only after summing the group two back from the same
      // set, so the sets alternate without a barrier of their own.
      uint8_t(*set)[kDecRange] = s_q[(g0 / kWaves) & 1u];
      if (wid < gn) wave_expand(s_sl[g0 + wid], cur, qn, set[wid]);
      __syncthreads();
      for (uint32_t s = 0; s < gn; ++s) {
        const float scale = s_sl[g0 + s].scale;
        const bool first = !kAcc && p0 + g0 + s == 0;
        const bool dense = first || !clean;
        const uint8_t* sq = set[s];
#pragma unroll
        for (int g = 0; g < kPer; ++g) {
          const uint32_t jl = jl_of(g);
          if (jl >= qn) continue;
          const uint32_t w = kVec ? *reinterpret_cast<const uint32_t*>(sq + jl) : sq[jl];
          if (!dense && w == kZeroWord) continue;  // every term +-0: no value changes
#pragma unroll
          for (int cc = 0; cc < kW; ++cc) {
            uint32_t t[5];
            digits5((w >> (8 * cc)) & 0xffu, t);
#pragma unroll
            for (int kk = 0; kk < 5; ++kk)
              acc[g][kk][cc] = first ? trit_value(t[kk], scale)
                                     : acc_trit(acc[g][kk][cc], t[kk], scale);
          }
        }
        // After a dense pass with M > 0 every value was given one of -M,
        // +0, M, so none is -0.0 (a rounded-to-nearest sum that is zero is
        // +0) and every NaN is quiet; no later term of +-0 (a zero group,
        // with any M >= 0) then changes a value, and none makes a -0.0 again.
        if (dense && scale > 0.0f) clean = true;
      }
      cur = nxt;
    }
    __syncthreads();  // s_sl and the sets are rewritten for the next chunk
  }

#pragma unroll
  for (int g = 0; g < kPer; ++g) {
    const uint32_t jl = jl_of(g);
    if (jl >= qn) continue;
    const uint64_t j = q0 + jl;
#pragma unroll
    for (int kk = 0; kk < 5; ++kk) {
      if (kVec && 4 * m + j + 4 <= n) {
        *reinterpret_cast<float4*>(out + kk * m + j) =
            make_float4(acc[g][kk][0], acc[g][kk][kW > 1 ? 1 : 0], acc[g][kk][kW > 2 ? 2 : 0],
                        acc[g][kk][kW > 3 ? 3 : 0]);
      } else {
#pragma unroll
        for (int cc = 0; cc < kW; ++cc) {
          const uint64_t e = kk * m + j + cc;
          if (e < n) out[e] = acc[g][kk][cc];
        }
      }
    }
  }
}

// ---------------------------------------------------------------- launchers
// Outputs of at least this size decode with nontemporal hints (twice the
// 256 MB last-level cache of the part).
constexpr uint64_t kNtMinBytes = 512ull << 20;

static inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0u;
}

hipError_t launch_zre_index(const uint8_t* C, uint32_t c, uint32_t m, uint64_t* start,
                            uint64_t* status, uint32_t ntiles, uint32_t ticket_base,
                            uint32_t epoch, Ctrl* ctrl, HostMirror hm, hipStream_t st) {
  launch_k(tlc_zre_index_kernel, ntiles, kThreads, st, C, c, m, start, status, ticket_base,
           epoch, ctrl, hm);
  return hipGetLastError();
}

hipError_t launch_expand_dequant(const uint8_t* C, uint32_t c, uint64_t* start,
                                 uint64_t* status, uint32_t ticket_base, uint64_t n, uint64_t m,
                                 float scale, float* out, int accumulate, uint32_t epoch,
                                 Ctrl* ctrl, HostMirror hm, hipStream_t st) {
  const bool al = aligned16(out);
  const bool nt = al && n * sizeof(float) >= kNtMinBytes;
  const bool fused = decode_fused(c, m);
  const uint32_t ntiles = fused ? decode_index_tiles(c, m) : 0u;
  const uint32_t blocks = ntiles + decode_ranges(m);
#define TLC_LAUNCH(V, A, N, F)                                                              \
  launch_k(tlc_expand_dequant_kernel<V, A, N, F>, blocks, kThreads, st, C, c, start, status, \
           ntiles, ticket_base, n, m, scale, out, epoch, ctrl, hm)
#define TLC_LAUNCH2(V, A, N) \
  if (fused) TLC_LAUNCH(V, A, N, true); else TLC_LAUNCH(V, A, N, false)
  if (nt) {
    // outputs of 512 MiB or more have far more blocks than a fused launch takes
    if (accumulate) TLC_LAUNCH(kPathShift, true, true, false);
    else TLC_LAUNCH(kPathShift, false, true, false);
  } else if (al && m % 4 == 0) {
    if (accumulate) { TLC_LAUNCH2(kPathVec, true, false); } else { TLC_LAUNCH2(kPathVec, false, false); }
  } else if (al) {
    if (accumulate) { TLC_LAUNCH2(kPathShift, true, false); } else { TLC_LAUNCH2(kPathShift, false, false); }
  } else {
    if (accumulate) { TLC_LAUNCH2(kPathByte, true, false); } else { TLC_LAUNCH2(kPathByte, false, false); }
  }
#undef TLC_LAUNCH2
#undef TLC_LAUNCH
  return hipGetLastError();
}

hipError_t launch_zre_index_batch(const DecDesc* descs, uint32_t count, uint32_t total_tiles,
                                  uint64_t* start, uint64_t* status, uint32_t ticket_base,
                                  uint32_t epoch, Ctrl* ctrl, HostMirror hm, hipStream_t st) {
  launch_k(tlc_zre_index_batch_kernel, total_tiles, kThreads, st, descs, count, start, status,
           ticket_base, epoch, ctrl, hm);
  return hipGetLastError();
}

hipError_t launch_expand_dequant_batch(const DecDesc* descs, uint32_t count,
                                       uint32_t total_ranges, const uint64_t* start,
                                       int accumulate, uint32_t epoch, const Ctrl* ctrl,
                                       hipStream_t st) {
  if (accumulate)
    launch_k(tlc_expand_dequant_batch_kernel<true>, total_ranges, kThreads, st, descs, count,
                                                                             start, epoch, ctrl);
  else
    launch_k(tlc_expand_dequant_batch_kernel<false>, total_ranges, kThreads, st,
        descs, count, start, epoch, ctrl);
  return hipGetLastError();
}

hipError_t launch_expand_sum(const DecDesc* descs, uint32_t count, const uint64_t* start,
                             uint64_t n, uint64_t m, float* out, int vec, int accumulate,
                             uint32_t epoch, const Ctrl* ctrl, hipStream_t st) {
  const uint32_t blocks = (uint32_t)((m + kDecRange - 1) / kDecRange);
#define TLC_LAUNCH(V, A)                                                                 \
  launch_k(tlc_expand_sum_kernel<V, A>, blocks, kThreads, st, descs, count, start, n, m, out, \
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
