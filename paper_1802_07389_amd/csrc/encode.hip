// encode.hip -- gfx950 encode kernels of the 3LC path.
//
//   tlc_absmax_check_kernel / _batch_kernel
//       partial maxima of |tensor + buffer|, nothing written: lets the
//       default error policy refuse NaN/Inf before the buffer changes
//   tlc_accum_absmax_kernel / _batch_kernel
//       step 1 of error accumulation (the tensor is added into the buffer,
//       in place) and partial maxima of the sums               (Section 3.1,
//                                                               Fig. 3, Eq. 1)
//   tlc_accum_quantize_kernel
//       after the check pass, on large aligned tensors: acc = x + r,
//       3-value quantization, the residual stored in place and 2-bit
//       trits for the quartic pack                  (Section 3.1, Eq. 1-2)
//   tlc_quant_encode_kernel, tlc_zre_chunk(_scan)_kernel, tlc_zre_compact_kernel
//       one tensor: M, 3-value quantization of the buffer, residual
//       write-back where q != 0 (or the quartic pack from the writing
//       pass's trits), each tile's own zero-run encoding; then a scan of the
//       tile summaries and the compaction into one stream
//                                              (Eq. 1-2, Sections 3.2-3.3)
//   tlc_quant_encode_chained_kernel, tlc_quant_encode_batch_kernel
//       a small tensor, or many tensors, in one pass: tiles chained by
//       decoupled look-back
//
// The batch kernels run many tensors in one launch: every block maps its
// index (absmax) or its ticket (encoder) to a tensor through the sorted
// first-block / first-tile fields of the tensor descriptors, then runs the
// same max reduction and tile quantization as the single-tensor kernels.
// Everything is HBM streaming; nothing is a dense contraction, so there is
// no MFMA.
#include "device_common.hpp"

namespace tlc {

// ---------------------------------------------------------------- Eq. 1
// Step 1 and Eq. 1 in one read of the tensor: with kResid the buffer
// becomes acc = x + r (the quantizer then reads only the buffer and writes
// back just the values with q != 0, whose residual differs from acc);
// without, acc = x and nothing is written.  max |acc| is taken on the bit
// patterns with the sign cleared: for non-negative IEEE values integer
// order equals numeric order, so the u32 max is exact and independent of
// reduction order, and any NaN/Inf makes the result >= 0x7f800000.  Block
// `blk` of `nblk` strides over [0, n).  The float4 path marks its loads and
// stores nontemporal: nothing here is read again before the whole tensor
// has streamed through, and the hint measured faster for this kernel and
// for the quantizer that follows.
//
// kSum (float4 path with a buffer): also store, for float4 number i of the
// buffer, the top 16 bits of the bit pattern of its largest |acc|.  That
// half-word h bounds the four values from above (|acc| < (h + 1) * 2^16 as
// bit patterns), so the quantizer can skip every float4 whose h lies below
// the top half of its threshold U: all four have q = 0 and keep acc.
//
// kStore false (with kResid): the check pass of the default error policy,
// which only reduces max|x + r| and writes nothing.
template <bool kVec, bool kResid = true, bool kSum = false, bool kStore = kResid>
__device__ __forceinline__ uint32_t absmax_part(const float* __restrict__ x,
                                                float* __restrict__ r, uint64_t n,
                                                uint32_t blk, uint32_t nblk,
                                                uint16_t* __restrict__ summ = nullptr) {
  static_assert(!kSum || (kVec && kStore), "summaries come from the float4 buffer path");
  static_assert(!kStore || kResid, "only a buffer is stored");
  uint32_t mx = 0;
  const uint64_t tid = (uint64_t)blk * kThreads + threadIdx.x;
  const uint64_t stride = (uint64_t)nblk * kThreads;
  if (kVec) {
    const uint64_t nv = n >> 2;
    uint64_t i = tid;
    for (; i + 3 * stride < nv; i += 4 * stride) {
      float4 a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = ld_stream(x + 4 * (i + u * stride));
#pragma unroll
      for (int u = 0; u < 4; ++u)
        b[u] = kResid ? ld_stream(r + 4 * (i + u * stride)) : make_float4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 v = kResid ? make_float4(a[u].x + b[u].x, a[u].y + b[u].y,
                                              a[u].z + b[u].z, a[u].w + b[u].w)
                                : a[u];
        if (kStore) st_stream(r + 4 * (i + u * stride), v);
        const uint32_t m4 =
            max(max(abs_bits(v.x), abs_bits(v.y)), max(abs_bits(v.z), abs_bits(v.w)));
        if (kSum) summ[i + u * stride] = (uint16_t)(m4 >> 16);
        mx = max(mx, m4);
      }
    }
    for (; i < nv; i += stride) {
      const float4 a = ld_stream(x + 4 * i);
      float4 v = a;
      if (kResid) {
        const float4 b = ld_stream(r + 4 * i);
        v = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
        if (kStore) st_stream(r + 4 * i, v);
      }
      const uint32_t m4 =
          max(max(abs_bits(v.x), abs_bits(v.y)), max(abs_bits(v.z), abs_bits(v.w)));
      if (kSum) summ[i] = (uint16_t)(m4 >> 16);
      mx = max(mx, m4);
    }
    for (uint64_t e = (nv << 2) + tid; e < n; e += stride) {
      const float v = kResid ? x[e] + r[e] : x[e];
      if (kStore) r[e] = v;
      mx = max(mx, abs_bits(v));
    }
  } else {
    for (uint64_t e = tid; e < n; e += stride) {
      const float v = kResid ? x[e] + r[e] : x[e];
      if (kStore) r[e] = v;
      mx = max(mx, abs_bits(v));
    }
  }
  return mx;
}

// The writing pass of the default error policy on the float4 path, once the
// check pass has given M (Eq. 1): acc = x + r, q = round(acc / M) and the
// residual acc - M*q (Eq. 2, Fig. 3 steps a-b) for every value; the
// residual is stored in place and q + 1 kept as a 2-bit trit, one byte per
// float4 of the buffer (value 4i + c in bits 2c, 2c + 1), from which the
// quantizer packs the quartic bytes without reading the buffer again.  The
// last n % 4 values are taken by one thread, which writes their byte.
__device__ __forceinline__ void accum_quantize_part(const float* __restrict__ x,
                                                    float* __restrict__ r, uint64_t n,
                                                    uint32_t blk, uint32_t nblk, float M,
                                                    float U, uint8_t* __restrict__ trits) {
  const uint64_t tid = (uint64_t)blk * kThreads + threadIdx.x;
  const uint64_t stride = (uint64_t)nblk * kThreads;
  const uint64_t nv = n >> 2;
  auto put4 = [&](uint64_t i, const float4& a, const float4& b) {
    float4 o;
    const uint32_t t0 = quantize_one(a.x + b.x, M, U, o.x);
    const uint32_t t1 = quantize_one(a.y + b.y, M, U, o.y);
    const uint32_t t2 = quantize_one(a.z + b.z, M, U, o.z);
    const uint32_t t3 = quantize_one(a.w + b.w, M, U, o.w);
    st_stream(r + 4 * i, o);
    trits[i] = (uint8_t)(t0 | (t1 << 2) | (t2 << 4) | (t3 << 6));
  };
  uint64_t i = tid;
  for (; i + 3 * stride < nv; i += 4 * stride) {
    float4 a[4], b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = ld_stream(x + 4 * (i + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u) b[u] = ld_stream(r + 4 * (i + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u) put4(i + u * stride, a[u], b[u]);
  }
  for (; i < nv; i += stride) put4(i, ld_stream(x + 4 * i), ld_stream(r + 4 * i));
  if (tid == 0 && (n & 3u)) {
    uint32_t tb = 0u;
    for (uint64_t e = nv << 2; e < n; ++e) {
      float o;
      tb |= quantize_one(x[e] + r[e], M, U, o) << (2u * (uint32_t)(e & 3u));
      r[e] = o;
    }
    trits[nv] = (uint8_t)tb;
  }
}

// Partial maxima of |x + r| that write nothing: the check pass that lets
// the default error policy refuse NaN/Inf before the buffer is touched.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void tlc_absmax_check_kernel(
    const float* __restrict__ x, const float* __restrict__ r, uint64_t n,
    uint32_t* __restrict__ partials) {
  __shared__ uint32_t lds[kWaves];
  const uint32_t mx = block_max(
      absmax_part<kVec, true, false, false>(x, const_cast<float*>(r), n, blockIdx.x, gridDim.x),
      lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = mx;
}

// The guard of a writing pass: with the check pass's partial maxima (guard
// != nullptr), a tensor whose scale would be NaN/Inf or overflow is left
// untouched, and the pass posts a partial that makes every later kernel
// refuse it as well.  Returns true when the block must stop.  Ends with a
// barrier when it reads the guard.
__device__ __forceinline__ bool refused_by_guard(const uint32_t* __restrict__ guard,
                                                 uint32_t guard_np, float s, uint32_t* lds,
                                                 uint32_t* __restrict__ partial) {
  if (guard == nullptr) return false;
  const Scale g = finish_scale(guard, guard_np, s, lds);
  __syncthreads();  // lds is reused by the caller
  if (!g.bad) return false;
  if (threadIdx.x == 0) *partial = 0xffffffffu;
  return true;
}

template <bool kVec, bool kResid, bool kSum>
__global__ __launch_bounds__(kThreads) void tlc_accum_absmax_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n,
    uint32_t* __restrict__ partials, uint16_t* __restrict__ summ,
    const uint32_t* __restrict__ guard, uint32_t guard_np, float s) {
  __shared__ uint32_t lds[kWaves];
  if (refused_by_guard(guard, guard_np, s, lds, &partials[blockIdx.x])) return;
  const uint32_t mx =
      block_max(absmax_part<kVec, kResid, kSum>(x, r, n, blockIdx.x, gridDim.x, summ), lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = mx;
}

// The writing pass of the default error policy on the float4 path of large
// tensors (steps 1, a and b of Section 3.1 with Eq. 2): the check pass's
// partial maxima give M (Eq. 1), then every value's acc = x + r is
// quantized, its residual stored in place and q + 1 kept as a 2-bit trit
// (accum_quantize_part).  A scale that is NaN/Inf or overflows leaves the
// buffer untouched.  The block's partial is the check pass's own.
__global__ __launch_bounds__(kThreads) void tlc_accum_quantize_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n,
    uint32_t* __restrict__ partials, uint8_t* __restrict__ trits,
    const uint32_t* __restrict__ guard, uint32_t guard_np, float s) {
  __shared__ uint32_t lds[kWaves];
  const Scale g = finish_scale(guard, guard_np, s, lds);
  if (g.bad) {  // NaN/Inf or overflow: nothing written, later kernels refuse too
    if (threadIdx.x == 0) partials[blockIdx.x] = 0xffffffffu;
    return;
  }
  accum_quantize_part(x, r, n, blockIdx.x, gridDim.x, g.M, g.U, trits);
  if (threadIdx.x == 0) partials[blockIdx.x] = guard[blockIdx.x];
}

// One block of the batch's max passes.  kStore false: the check pass.
// guard (kStore): the check pass's partial maxima, same block numbering.
template <bool kStore>
__device__ __forceinline__ void accum_absmax_batch_block(const EncDesc* __restrict__ descs,
                                                         uint32_t count,
                                                         uint32_t* __restrict__ partials,
                                                         const uint32_t* __restrict__ guard,
                                                         uint32_t* lds) {
  const uint32_t t =
      find_desc(descs, count, blockIdx.x, [](const EncDesc& d) { return d.blk0; });
  const EncDesc& d = descs[t];
  const uint32_t blk = blockIdx.x - d.blk0;
  if (kStore && refused_by_guard(guard ? guard + d.blk0 : nullptr, d.nblk, d.s, lds,
                                 &partials[blockIdx.x]))
    return;
  const uint32_t mx = (d.vec & 4u)
                          ? absmax_part<true, true, false, kStore>(d.x, d.r, d.n, blk, d.nblk)
                          : absmax_part<false, true, false, kStore>(d.x, d.r, d.n, blk, d.nblk);
  const uint32_t bm = block_max(mx, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = bm;
}

__global__ __launch_bounds__(kThreads) void tlc_absmax_check_batch_kernel(
    const EncDesc* __restrict__ descs, uint32_t count, uint32_t* __restrict__ partials) {
  __shared__ uint32_t lds[kWaves];
  accum_absmax_batch_block<false>(descs, count, partials, nullptr, lds);
}

__global__ __launch_bounds__(kThreads) void tlc_accum_absmax_batch_kernel(
    const EncDesc* __restrict__ descs, uint32_t count, uint32_t* __restrict__ partials,
    const uint32_t* __restrict__ guard) {
  __shared__ uint32_t lds[kWaves];
  accum_absmax_batch_block<true>(descs, count, partials, guard, lds);
}

// ---------------------------------------------------------------- Eq. 2, 3.2
// Phase 1 of a tile (quartic bytes [q0, q0 + T), T <= kEncTile) when
// m % 4 != 0 but the buffer r is 16-byte aligned.  Partition k of the tile
// starts a = (k*m + q0) mod 4 values past a float4 boundary, so the block
// sweeps it in aligned float4 cells: cell f holds the values of tile bytes
// 4f - a .. 4f + 3 - a.  A cell shared with a neighbouring tile or
// partition, or reaching past n, is read and written value by value, so
// every value's residual has one writer (and only values with q != 0 are
// written).  Partition 0 (a = 0, as q0 is a
// multiple of 4) stores the bytes; partitions 1-4 add their weighted trits
// with LDS atomics on the two words a cell straddles: a byte's total stays
// below 243, so no carry crosses into the next byte.
template <bool kX = false>
__device__ __forceinline__ void quantize_tile_shifted(const float* __restrict__ x,
                                                      float* __restrict__ r, uint64_t n,
                                                      uint64_t m, uint64_t q0, uint32_t T,
                                                      float M, float U, uint32_t* qw) {
  constexpr int kCells = (kEncTile + 6) / 4 / kThreads + 1;  // cells per lane, a <= 3
#pragma unroll 1
  for (int k = 0; k < 5; ++k) {
    const uint64_t base = (uint64_t)k * m + q0;
    const uint32_t a = (uint32_t)(base & 3u);
    const uint64_t e0 = base - a;  // first value of cell 0
    const uint32_t nf = (T + a + 3u) >> 2;
    const uint32_t w = trit_weight(k);
    float4 ra[kCells];
    bool full[kCells];
#pragma unroll
    for (int i = 0; i < kCells; ++i) {
      const uint32_t f = threadIdx.x + kThreads * i;
      const uint64_t e = e0 + 4ull * f;
      full[i] = f < nf && 4u * f >= a && 4u * f + 4u <= T + a && e + 4u <= n;
      if (full[i]) {
        ra[i] = *reinterpret_cast<const float4*>(r + e);
        if (kX) {
          const float4 b = *reinterpret_cast<const float4*>(x + e);
          ra[i] = make_float4(b.x + ra[i].x, b.y + ra[i].y, b.z + ra[i].z, b.w + ra[i].w);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kCells; ++i) {
      const uint32_t f = threadIdx.x + kThreads * i;
      if (f >= nf) break;
      const uint64_t e = e0 + 4ull * f;
      uint32_t t[4] = {0u, 0u, 0u, 0u};  // padding and other tiles' values add nothing
      if (full[i]) {
        float4 o;
        t[0] = quantize_one(ra[i].x, M, U, o.x);
        t[1] = quantize_one(ra[i].y, M, U, o.y);
        t[2] = quantize_one(ra[i].z, M, U, o.z);
        t[3] = quantize_one(ra[i].w, M, U, o.w);
        if (kX || ((t[0] ^ 1u) | (t[1] ^ 1u) | (t[2] ^ 1u) | (t[3] ^ 1u)))
          *reinterpret_cast<float4*>(r + e) = o;
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t p = 4u * f + c;  // position in the partition's cell grid
          if (p >= a && p - a < T && e + c < n) {
            float o;
            t[c] = quantize_one(kX ? x[e + c] + r[e + c] : r[e + c], M, U, o);
            if (kX || t[c] != 1u) r[e + c] = o;
          }
        }
      }
      // byte 4f + c - a: word f - 1 for c < a, word f otherwise
      uint32_t lo = 0u, hi = 0u;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t v = t[c] * w;
        if ((uint32_t)c < a)
          lo |= v << (8u * (4u + c - a));
        else
          hi |= v << (8u * (c - a));
      }
      if (k == 0) {
        qw[f] = hi;  // a == 0: the cell is word f
      } else {
        if (lo) atomicAdd(&qw[f - 1], lo);  // lo != 0 only when f >= 1
        if (hi) atomicAdd(&qw[f], hi);
      }
    }
    if (k == 0) __syncthreads();  // partition 0 has stored every word
  }
}

// ---------------------------------------------------------------- Eq. 2, 3.2, 3.3
struct EncShared {
  uint32_t red[kWaves];
  uint32_t fault;
  uint32_t nfix;   // entries taken in the tile's fix list (may pass kFixCap)
  uint32_t nneed;  // float4 slices the tile has to load (summaries)
  uint32_t red2[kWaves];
  uint32_t lead;   // the tile's first non-121 byte (first pass)
  RunSum wave[kWaves];
  RunSum excl;
  __align__(16) uint8_t q[kEncTile];
  __align__(16) uint8_t out[kEncTile + 16];
};

static_assert(kEncTile / kThreads == 16, "one uint4 of quartic bytes per thread");
constexpr int kGroupsPerThread = kEncTile / 4 / kThreads;  // groups of 4 bytes per thread

// Phase 1 of a tile (Eq. 2, residual write-back, quartic pack): the block
// quantizes the 5 * tile_bytes accumulated values of quartic bytes
// [q0, q0 + tile_bytes), held in the buffer r, and leaves the bytes in q
// (LDS).  kPath: threads take groups of 4 bytes,
// aligned float4 cells of one partition at a time, or single bytes,
// interleaved so every load and store instruction is coalesced.  kDeep
// (float4 path): in a whole tile whose every group lies before n, all of a
// thread's groups are loaded, without branches between them, before the
// first is quantized: one memory round trip per tile instead of one per
// group, at the cost of registers, for grids small enough to stay resident
// (the chained and batched encoders).  Ends with a barrier.
template <int kPath, bool kX = false, bool kDeep = false>
__device__ __forceinline__ void quantize_tile(const float* __restrict__ x, float* __restrict__ r,
                                              uint64_t n, uint32_t m, const Scale& sc,
                                              uint64_t q0, uint32_t tile_bytes, uint8_t* q) {
  if (kPath == kPathVec && kDeep && tile_bytes == (uint32_t)kEncTile &&
      group4_full(n, m, q0 + kEncTile - 4u)) {
    float4 v[kGroupsPerThread][5];
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it)
      load_group4<kX>(x, r, m, q0 + (threadIdx.x + kThreads * it) * 4u, v[it]);
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it) {
      const uint32_t g = threadIdx.x + kThreads * it;
      *reinterpret_cast<uint32_t*>(q + g * 4u) =
          quantize_group4_loaded<kX>(r, m, q0 + g * 4u, v[it], sc.M, sc.U);
    }
  } else if (kPath == kPathVec) {  // 4 bytes per thread: float4 loads and stores
    // The thread's groups g = threadIdx.x + kThreads * it: the next group's
    // ten loads are issued before the current group is quantized, so a
    // tile takes about one memory round trip per thread instead of one per
    // group (the groups' values are disjoint).  A group reaching into the
    // padding of p4 takes the byte path.
    auto ok = [&](uint32_t g) {
      return g * 4u < tile_bytes && group4_full(n, m, q0 + g * 4u);
    };
    float4 cur[5];
    if (ok(threadIdx.x)) load_group4<kX>(x, r, m, q0 + threadIdx.x * 4u, cur);
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it) {
      const uint32_t g = threadIdx.x + kThreads * it;
      if (g * 4u >= tile_bytes) break;
      const uint64_t j = q0 + g * 4u;
      float4 nxt[5];
      const bool next = it + 1 < kGroupsPerThread && ok(g + kThreads);
      if (next) load_group4<kX>(x, r, m, j + 4u * kThreads, nxt);
      *reinterpret_cast<uint32_t*>(q + g * 4u) =
          ok(g) ? quantize_group4_loaded<kX>(r, m, j, cur, sc.M, sc.U)
                : quantize_group4_bytes<kX>(x, r, n, m, j, sc.M, sc.U);
      if (next) {
#pragma unroll
        for (int k = 0; k < 5; ++k) cur[k] = nxt[k];
      }
    }
  } else if (kPath == kPathShift) {  // aligned float4 cells off the slice grid
    quantize_tile_shifted<kX>(x, r, n, m, q0, tile_bytes, sc.M, sc.U,
                              reinterpret_cast<uint32_t*>(q));
  } else {  // 1 byte per thread: dword accesses, still contiguous per wave
    for (uint32_t lj = threadIdx.x; lj < tile_bytes; lj += kThreads)
      q[lj] = (uint8_t)quantize_byte<kX>(x, r, n, m, q0 + lj, sc.M, sc.U);
  }
  __syncthreads();
}

// Encodes tile `lt` (kEncTile quartic bytes) of one tensor of a batch whose
// scale is sc.  Phase 1: quantize_tile.  Phase 2: each thread takes
// kEncTile/256 consecutive bytes and summarises them as a RunSum; the block
// scans the summaries, the tile gets its prefix by decoupled look-back
// (status slot floor + lt; slot floor is the tensor's first tile), and
// every thread zero-run encodes its bytes from its own prefix into LDS; the
// block then copies the tile's output into the stream.  The last tile
// stores the stream length in res->len.
template <int kPath, bool kX>
__device__ __forceinline__ void encode_tile(const float* __restrict__ x, float* __restrict__ r,
                                            uint64_t n, uint32_t m, const Scale& sc,
                                            uint32_t lt, uint32_t floor,
                                            uint8_t* __restrict__ out,
                                            uint64_t* __restrict__ status, uint32_t epoch,
                                            Ctrl* __restrict__ ctrl, EncResult* res,
                                            EncResult* hres, uint32_t* hfault,
                                            EncShared& sh) {
  constexpr int kBytes = kEncTile / kThreads;  // zero-run bytes per thread
  static_assert(kBytes % 16 == 0, "threads read whole uint4s of quartic bytes");

  // ---- phase 1: Eq. 1-2, residual write-back, quartic pack
  const uint64_t q0 = (uint64_t)lt * kEncTile;
  const uint32_t tile_bytes = (uint32_t)umin64(kEncTile, (uint64_t)m - q0);
  quantize_tile<kPath, kX, true>(x, r, n, m, sc, q0, tile_bytes, sh.q);

  // ---- phase 2: Section 3.3
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint32_t lo = threadIdx.x * kBytes;
  const uint32_t cnt = lo < tile_bytes ? umin32(kBytes, tile_bytes - lo) : 0u;
  const uint32_t nz = cnt ? nonzero_group_mask(sh.q, lo, cnt) : 0u;
  const RunSum sum = rs_mask_summary(nz, cnt);

  const RunSum incl = wave_incl_scan_rs(sum);
  const RunSum excl_lane = wave_prev_lane_rs(incl);
  if (lane == 63) sh.wave[wid] = incl;
  __syncthreads();
  RunSum wpre = rs_identity();
  RunSum agg = rs_identity();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if ((uint32_t)w < wid) wpre = rs_combine(wpre, sh.wave[w]);
    agg = rs_combine(agg, sh.wave[w]);
  }

  if (wid == 0) {
    bool fault = false;
    uint64_t ex = rs_to_payload(rs_identity());
    if (lt == 0) {
      if (lane == 0)
        status_publish(&status[floor], EncSW::pack(rs_to_payload(agg), kFlagPrefix, epoch));
    } else {
      ex = lookback_wave<EncSW>(status, floor, floor + lt, rs_to_payload(agg), ex, epoch,
                                EncOp(), &fault);
    }
    if (lane == 0) {
      sh.excl = rs_from_payload(ex);
      sh.fault = fault ? 1u : 0u;
      if (fault) {
        __hip_atomic_store(&ctrl->fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        host_put(hfault, 1u);
      }
    }
  }
  __syncthreads();
  if (sh.fault) return;

  const RunSum tex = sh.excl;
  const RunSum P = rs_combine(rs_combine(tex, wpre), excl_lane);
  const uint32_t tile_begin = rs_emitted(tex);
  uint32_t o = rs_emitted(P) - tile_begin;
  uint32_t phi = rs_phase(P);
  auto put = [&](uint32_t c) {
    if (o < sizeof(sh.out)) sh.out[o] = (uint8_t)c;
    ++o;
  };
  phi = rs_mask_walk(nz, cnt, phi, [&](uint32_t i) { return (uint32_t)sh.q[lo + i]; }, put);
  if (cnt && q0 + lo + cnt == m && phi) put(rs_code(phi));  // stream ends in a run

  const bool last_tile = q0 + kEncTile >= m;
  const RunSum tincl = rs_combine(tex, agg);
  const uint32_t tile_end = last_tile ? rs_total(tincl) : rs_emitted(tincl);
  __syncthreads();
  // a tile emits at most kEncTile + 1 bytes; the clamps only keep a logic
  // error from writing outside the m-byte output buffer
  const uint32_t count =
      tile_end >= tile_begin ? umin32(tile_end - tile_begin, kEncTile + 1) : 0u;
  for (uint32_t i = threadIdx.x; i < count; i += kThreads)
    if (tile_begin + i < m) out[tile_begin + i] = sh.out[i];
  if (last_tile && threadIdx.x == 0) {
    res->len = tile_end;
    if (hres) host_put(&hres->len, tile_end);
  }
}

// ---------------------------------------------------------------- single tensor, three passes
// A single tensor is encoded without any wait between tiles:
//   pass A (tlc_quant_encode_kernel, one block per tile): quantize_tile, then
//     zero-run encode the tile from its first non-121 byte on into its own
//     slot.  That part does not depend on earlier tiles: the byte closes the
//     run before it, so the encoder is at phase 0 there.  Each tile records
//     its summary (RunSum), the length of its leading 121 run and the slot
//     length.
//   pass B (tlc_zre_chunk_kernel): every tile's prefix within its chunk of
//     64 tiles and the chunk summaries; the pass's last block scans the
//     chunk summaries.
//   pass C (tlc_zre_compact_kernel, one wave per tile): the tile's prefix
//     (its output offset and incoming run phase) from its chunk's prefix
//     and its own within the chunk, then the leading run's codes, which
//     need the incoming phase (one 255 per 14th byte of the grown run, then
//     its remainder code if the tile has a non-121 byte), and the slot; the
//     last tile adds the remainder of a run that ends the stream.

// Residual v of the tile's value `local` (k * kEncTile + position) when
// `has`: the wave takes consecutive entries of the tile's fix list (in LDS)
// with one LDS atomic; a value whose entry falls past kFixCap is stored at
// dst at once.
__device__ __forceinline__ void fix_put(bool has, uint32_t local, float v, float* dst,
                                        uint32_t* nfix, uint2* fix) {
  const uint64_t bal = __ballot(has);
  if (bal == 0u) return;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t leader = (uint32_t)__ffsll((unsigned long long)bal) - 1u;
  const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
      (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  uint32_t base = 0u;
  if (lane == leader) base = atomicAdd(nfix, (uint32_t)__popcll(bal));
  base = (uint32_t)__shfl((int)base, (int)leader, 64);
  if (has) {
    const uint32_t slot = base + rank;
    if (slot < kFixCap)
      fix[slot] = make_uint2(local, __float_as_uint(v));
    else
      *dst = v;
  }
}

// Slice k of group g (values j..j+3 of partition k, loaded as a) of a
// first-pass tile: the four trits, and the residuals of q != 0 put into the
// tile's fix list.
__device__ __forceinline__ void quantize_slice(const float4& a, uint32_t k, uint32_t g,
                                               float* e, const Scale& sc, uint32_t (&t)[4],
                                               uint32_t* nfix, uint2* s_fix) {
  float4 o;
  t[0] = quantize_one(a.x, sc.M, sc.U, o.x);
  t[1] = quantize_one(a.y, sc.M, sc.U, o.y);
  t[2] = quantize_one(a.z, sc.M, sc.U, o.z);
  t[3] = quantize_one(a.w, sc.M, sc.U, o.w);
  const uint32_t local = k * kEncTile + g * 4u;
  fix_put(t[0] != 1u, local, o.x, e, nfix, s_fix);
  fix_put(t[1] != 1u, local + 1u, o.y, e + 1, nfix, s_fix);
  fix_put(t[2] != 1u, local + 2u, o.z, e + 2, nfix, s_fix);
  fix_put(t[3] != 1u, local + 3u, o.w, e + 3, nfix, s_fix);
}

// A tile with at most this many float4 slices to load (of 5 * 1024) takes
// the sparse form below.
constexpr uint32_t kSparseSlices = 512;
// Slices a thread of a sparse tile loads together (more go one at a time).
constexpr int kSparseBatch = 4;

// The max pass's bounds of this thread's slices (group it = threadIdx.x +
// kThreads * it, partition k); 0 for groups that are missing or reach into
// the padding.  They do not depend on M, so the loads are issued before the
// block reduces it.
__device__ __forceinline__ void load_bounds(const uint16_t* __restrict__ summ, uint64_t n,
                                            uint32_t m, uint64_t q0, uint32_t tile_bytes,
                                            uint32_t (&h)[kGroupsPerThread][5]) {
#pragma unroll
  for (int it = 0; it < kGroupsPerThread; ++it) {
    const uint32_t g = threadIdx.x + kThreads * it;
    const uint64_t j = q0 + g * 4u;
    const bool full = g * 4u < tile_bytes && group4_full(n, m, j);
#pragma unroll
    for (int k = 0; k < 5; ++k) h[it][k] = full ? summ[(k * (uint64_t)m + j) >> 2] : 0u;
  }
}

// Phase 1 of a first-pass tile on the float4 path: quantize_tile<kPathVec>
// with the residuals of q != 0 put into the tile's fix list, which is built
// in LDS (s_fix) and then copied out whole, so HBM sees a few full lines
// per tile rather than one partial line per value.
//
// With the max pass's bounds (kSum; h from load_bounds) a slice is needed
// only if its bound reaches the top half of U; the others hold four values
// with q = 0, contribute trit 1 and are neither read nor written.  If the
// block needs few slices (typical: most groups of five values quantize to
// zero), every group starts from the all-zero byte 121 and its owner loads
// its first kSparseBatch needed slices together, moving each byte by
// (t - 1) * 3^(4-k); otherwise the groups are quantized in turn with their
// needed slices loaded together.  The groups that reach into the padding
// store theirs directly.  Ends with a barrier.
template <bool kSum>
__device__ __forceinline__ void quantize_tile_vec_deferred(
    float* __restrict__ r, uint64_t n, uint32_t m, const Scale& sc, uint64_t q0,
    uint32_t tile_bytes, uint8_t* q, uint2* s_fix, uint32_t* nfix, uint32_t* nneed,
    uint2* __restrict__ fix, const uint32_t (&h)[kGroupsPerThread][5]) {
  static_assert(kEncTile == 4096, "fix entries hold k * 4096 + position");
  static_assert(kGroupsPerThread * 5 <= 32, "a thread's slices fit one mask");
  uint32_t* qw = reinterpret_cast<uint32_t*>(q);
  uint32_t need = 0u;  // bit 5 * it + k: slice k of group it is loaded
  bool sparse = false;
  if (kSum) {
    const uint32_t hU = __float_as_uint(sc.U) >> 16;
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it)
#pragma unroll
      for (int k = 0; k < 5; ++k) need |= (h[it][k] >= hU ? 1u : 0u) << (5 * it + k);
    if (need) atomicAdd(nneed, (uint32_t)__popc(need));
    __syncthreads();
    sparse = *nneed <= kSparseSlices;
  }
  if (sparse) {
    int code[kGroupsPerThread][4];
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it)
#pragma unroll
      for (int c = 0; c < 4; ++c) code[it][c] = 121;  // five zero values per byte
    // the first kSparseBatch needed slices: loads issued together
    float4 a[kSparseBatch];
    uint32_t sel[kSparseBatch];
    uint32_t rest = need;
#pragma unroll
    for (int b = 0; b < kSparseBatch; ++b) {
      sel[b] = rest ? (uint32_t)__ffs(rest) - 1u : 32u;
      rest &= rest - 1u;
      if (sel[b] < 32u) {
        const uint32_t it = sel[b] / 5u, k = sel[b] % 5u;
        a[b] = *reinterpret_cast<const float4*>(r + (uint64_t)k * m + q0 +
                                                (threadIdx.x + kThreads * it) * 4u);
      }
    }
    auto apply = [&](uint32_t bit, const float4& v) {
      const uint32_t it = bit / 5u, k = bit % 5u;
      const uint32_t g = threadIdx.x + kThreads * it;
      float* e = r + (uint64_t)k * m + q0 + g * 4u;
      uint32_t t[4];
      quantize_slice(v, k, g, e, sc, t, nfix, s_fix);
      const int w = (int)trit_weight((int)k);
#pragma unroll
      for (int gi = 0; gi < kGroupsPerThread; ++gi)
        if ((uint32_t)gi == it) {
#pragma unroll
          for (int c = 0; c < 4; ++c) code[gi][c] += ((int)t[c] - 1) * w;
        }
    };
#pragma unroll
    for (int b = 0; b < kSparseBatch; ++b)
      if (sel[b] < 32u) apply(sel[b], a[b]);
    while (rest) {  // rare: more needed slices than one batch
      const uint32_t bit = (uint32_t)__ffs(rest) - 1u;
      rest &= rest - 1u;
      const uint32_t it = bit / 5u, k = bit % 5u;
      apply(bit, *reinterpret_cast<const float4*>(r + (uint64_t)k * m + q0 +
                                                  (threadIdx.x + kThreads * it) * 4u));
    }
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it) {
      const uint32_t g = threadIdx.x + kThreads * it;
      if (g * 4u >= tile_bytes) break;
      const uint64_t j = q0 + g * 4u;
      qw[g] = group4_full(n, m, j)
                  ? (uint32_t)code[it][0] | ((uint32_t)code[it][1] << 8) |
                        ((uint32_t)code[it][2] << 16) | ((uint32_t)code[it][3] << 24)
                  : quantize_group4_bytes(nullptr, r, n, m, j, sc.M, sc.U);
    }
  } else {
#pragma unroll
    for (int it = 0; it < kGroupsPerThread; ++it) {
      const uint32_t g = threadIdx.x + kThreads * it;
      if (g * 4u >= tile_bytes) break;
      const uint64_t j = q0 + g * 4u;
      if (!group4_full(n, m, j)) {
        qw[g] = quantize_group4_bytes(nullptr, r, n, m, j, sc.M, sc.U);
        continue;
      }
      float4 a[5];
      if (kSum) {
#pragma unroll
        for (int k = 0; k < 5; ++k)
          a[k] = (need >> (5 * it + k)) & 1u ? *reinterpret_cast<const float4*>(r + (uint64_t)k * m + j)
                                             : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {
        load_group4(nullptr, r, m, j, a);
      }
      uint32_t code[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int k = 0; k < 5; ++k) {
        uint32_t t[4];
        quantize_slice(a[k], (uint32_t)k, g, r + (uint64_t)k * m + j, sc, t, nfix, s_fix);
#pragma unroll
        for (int c = 0; c < 4; ++c) code[c] = code[c] * 3u + t[c];
      }
      qw[g] = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
    }
  }
  __syncthreads();
  const uint32_t nf = umin32(*nfix, kFixCap);
  for (uint32_t i = threadIdx.x; i < nf; i += kThreads) fix[i] = s_fix[i];
}

// Phase 1 of a first-pass tile when the max pass has quantized every value
// (kTrit).  load_trits fetches, for each of this thread's groups (quartic
// bytes j..j+3, g = threadIdx.x + kThreads * it, as in the float4 path) and
// each partition k, the trits of values e = k*m + j .. e + 3 as one byte:
// they start at bit 2*(e mod 4) of trit byte e/4 and run into the next one
// when e mod 4 != 0 (m % 4 != 0).  They do not depend on M, so the loads
// are issued before the block reduces it.  pack_trits then forms the
// quartic bytes (Section 3.2), with the values past n as the zero padding
// (trit 0), and ends with a barrier.
template <int kT = kThreads>
__device__ __forceinline__ void load_trits(const uint8_t* __restrict__ trits, uint64_t n,
                                           uint32_t m, uint64_t q0, uint32_t tile_bytes,
                                           uint32_t (&tb)[kEncTile / 4 / kT][5]) {
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    // group g's first value is e = base + 4g; q0 is a multiple of 4, so
    // e mod 4 = base mod 4 = a for the whole block, e / 4 = base / 4 + g,
    // and the values before n are those with 4g < n - base
    const uint64_t base = (uint64_t)k * m + q0;
    const uint32_t a = (uint32_t)(base & 3u);
    const uint8_t* tp = trits + (base >> 2);
    const uint64_t left = n > base ? n - base : 0u;  // values of the partition from base on
    const uint32_t lim = (uint32_t)umin64(left, tile_bytes);
    const uint32_t cap = (uint32_t)umin64(left + a, 2u * kEncTile);
#pragma unroll
    for (int it = 0; it < kEncTile / 4 / kT; ++it) {
      const uint32_t g = threadIdx.x + kT * it;
      uint32_t v = 0u;
      if (g * 4u < lim) {
        v = tp[g];
        if (a != 0u) {
          // trit byte e/4 + 1 holds values from e + 4 - a on: it exists when
          // 4g + 4 - a < left (4g + 4 <= tile_bytes + 3 < 2 * kEncTile)
          if (g * 4u + 4u < cap) v |= (uint32_t)tp[g + 1u] << 8;
          v = (v >> (2u * a)) & 0xffu;
        }
      }
      tb[it][k] = v;
    }
  }
}

// The trits of this thread's own 16 values in each partition of a tile
// (values k*m + q0 + 16*tid + [0, 16), so that the thread packs the 16
// quartic bytes it encodes): 32 consecutive bits of the trit array from bit
// 2*(k*m + q0) + 32*tid on, taken from the aligned word at or before them
// and the next one (alignbit; the bit offset within the word is the same
// for the whole partition, so any m works).  The trits fill the first n/4
// bytes of a 256-byte aligned region of max_n/2 bytes, so that next word
// lies inside it too.
__device__ __forceinline__ void load_trit_words(const uint8_t* __restrict__ trits, uint32_t m,
                                                uint64_t q0, uint32_t (&d)[5]) {
  const uint32_t* tw = reinterpret_cast<const uint32_t*>(trits);
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    const uint64_t e0 = (uint64_t)k * m + q0;  // the partition's first value in the tile
    const uint32_t sh = 2u * (uint32_t)(e0 & 15u);
    const uint32_t* wp = tw + (e0 >> 4) + threadIdx.x;
    const uint32_t lo = wp[0];
    d[k] = sh ? __builtin_amdgcn_alignbit(wp[1], lo, sh) : lo;
  }
}

__device__ __forceinline__ uint32_t spread_trits(uint32_t tb) {
  // the four 2-bit trits of one byte into the low bits of four bytes
  tb = (tb | (tb << 12)) & 0x000f000fu;
  return (tb | (tb << 6)) & 0x03030303u;
}

// Tables of spread trits times the partition's weight (Section 3.2: 81, 27,
// 9, 3, 1): lut[k][b] holds, in byte lane c, 3^(4-k) times trit c of trit
// byte b.  The sum of one entry per partition is the four quartic bytes of
// a group (each at most 242, so no carry crosses a lane): five LDS reads
// and four adds instead of five spreads and four multiply-adds.  Written
// before a barrier of the caller.
template <int kT = kThreads>
__device__ __forceinline__ void init_trit_luts(uint32_t (*lut)[256]) {
  static_assert(256 % kT == 0, "whole rounds of table entries");
#pragma unroll
  for (uint32_t b = threadIdx.x; b < 256u; b += kT) {
    const uint32_t sp = spread_trits(b);
    lut[0][b] = 81u * sp;
    lut[1][b] = 27u * sp;
    lut[2][b] = 9u * sp;
    lut[3][b] = 3u * sp;
    lut[4][b] = sp;
  }
}

// This thread's 16 quartic bytes from its trit words (load_trit_words):
// byte g of each word holds the trits of its values 4g..4g+3.
__device__ __forceinline__ uint4 pack_trit_words(const uint32_t (&d)[5],
                                                 const uint32_t (*lut)[256]) {
  uint32_t o[4];
#pragma unroll
  for (int g = 0; g < 4; ++g)
    o[g] = lut[0][(d[0] >> (8 * g)) & 255u] + lut[1][(d[1] >> (8 * g)) & 255u] +
           lut[2][(d[2] >> (8 * g)) & 255u] + lut[3][(d[3] >> (8 * g)) & 255u] +
           lut[4][(d[4] >> (8 * g)) & 255u];
  return make_uint4(o[0], o[1], o[2], o[3]);
}

template <int kT = kThreads>
__device__ __forceinline__ void pack_trits(const uint32_t (&tb)[kEncTile / 4 / kT][5], uint64_t n,
                                           uint32_t m, uint64_t q0, uint32_t tile_bytes,
                                           const uint32_t (*lut)[256], uint8_t* q) {
  uint32_t* qw = reinterpret_cast<uint32_t*>(q);
#pragma unroll
  for (int it = 0; it < kEncTile / 4 / kT; ++it) {
    const uint32_t g = threadIdx.x + kT * it;
    if (g * 4u >= tile_bytes) break;
    const uint64_t j = q0 + g * 4u;
    if (4ull * m + j + 4u <= n) {
      // all 20 values exist: the four bytes at once
      qw[g] = lut[0][tb[it][0]] + lut[1][tb[it][1]] + lut[2][tb[it][2]] + lut[3][tb[it][3]] +
              lut[4][tb[it][4]];
      continue;
    }
    uint32_t code[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      const uint64_t e = (uint64_t)k * m + j;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        code[c] = code[c] * 3u + (e + c < n ? (tb[it][k] >> (2 * c)) & 3u : 0u);
    }
    qw[g] = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
  }
  __syncthreads();
}

// kTrit (kPathVec only): the buffer already holds the residuals and `summ`
// the trits of every value (the max pass after the check pass); phase 1
// only packs them, and the tile's residual list stays empty.
template <int kPath, bool kTrit = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(5)))
void tlc_quant_encode_kernel(
    float* __restrict__ r, uint64_t n, uint32_t m, float s,
    const uint32_t* __restrict__ partials, uint32_t np, uint8_t* __restrict__ slots,
    TileRec* __restrict__ recs, uint2* __restrict__ fix, const uint16_t* __restrict__ summ,
    Ctrl* __restrict__ ctrl, HostMirror hm) {
  constexpr int kBytes = kEncTile / kThreads;  // zero-run bytes per thread
  static_assert(kBytes % 16 == 0, "threads read whole uint4s of quartic bytes");
  static_assert(!kTrit || kPath == kPathVec, "trits are kept on the float4 path");
  __shared__ EncShared sh;
  __shared__ uint2 s_fix[(kPath == kPathVec && !kTrit) ? kFixCap : 1];
  __shared__ uint32_t s_lut[kTrit ? 5 : 1][256];
  __shared__ uint32_t s_scale[kWaves];  // M's reduction: the scans below reuse sh.red
  if (threadIdx.x == 0) {
    sh.nfix = 0u;
    sh.nneed = 0u;
  }
  const uint32_t t = blockIdx.x;
  const uint64_t q0 = (uint64_t)t * kEncTile;
  const uint32_t tile_bytes = (uint32_t)umin64(kEncTile, (uint64_t)m - q0);
  // an interior tile (whole, every value before n): each thread packs its
  // own 16 quartic bytes in registers; other tiles pack through sh.q
  const bool own = kTrit && tile_bytes == (uint32_t)kEncTile && 4ull * m + q0 + kEncTile <= n;
  uint32_t h[kGroupsPerThread][5];  // bounds, or with kTrit the trits
  if (kTrit) {
    const uint8_t* trits = reinterpret_cast<const uint8_t*>(summ);
    if (own)
      load_trit_words(trits, m, q0, h[0]);
    else
      load_trits(trits, n, m, q0, tile_bytes, h);
    init_trit_luts(s_lut);
  } else if (kPath == kPathVec && summ) {
    load_bounds(summ, n, m, q0, tile_bytes, h);
  }
  Scale sc;
  if (kTrit && t != 0) {
    // with trits only block 0 needs M (for the result); the others need the
    // verdict, which the writing pass left in every partial: all 0xffffffff
    // for a refused tensor, otherwise the check pass's finite maxima
    __syncthreads();  // the tables
    sc.M = 0.0f;
    sc.U = 0.0f;
    sc.bad = partials[0] >= 0x7f800000u ? 1u : 0u;
  } else {
    sc = finish_scale(partials, np, s, s_scale);  // includes a barrier
  }
  if (t == 0 && threadIdx.x == 0) {
    ctrl->enc.err = sc.bad;
    ctrl->enc.scale = sc.M;
    host_put_result(hm.res, sc.bad, sc.M);
  }
  if (sc.bad) return;  // NaN/Inf or overflow: the buffer keeps acc, no stream
  const uint32_t lo = threadIdx.x * kBytes;
  const uint32_t cnt = lo < tile_bytes ? umin32(kBytes, tile_bytes - lo) : 0u;
  uint4 w = make_uint4(0u, 0u, 0u, 0u);  // the thread's quartic bytes [lo, lo + cnt)
  if (own) {
    w = pack_trit_words(h[0], s_lut);
  } else if (kTrit) {
    pack_trits(h, n, m, q0, tile_bytes, s_lut, sh.q);
  } else if (kPath == kPathVec) {
    if (summ)
      quantize_tile_vec_deferred<true>(r, n, m, sc, q0, tile_bytes, sh.q, s_fix, &sh.nfix,
                                       &sh.nneed, fix + (uint64_t)t * kFixCap, h);
    else
      quantize_tile_vec_deferred<false>(r, n, m, sc, q0, tile_bytes, sh.q, s_fix, &sh.nfix,
                                        &sh.nneed, fix + (uint64_t)t * kFixCap, h);
  } else {
    quantize_tile<kPath>(nullptr, r, n, m, sc, q0, tile_bytes, sh.q);
  }
  if (!own && cnt) w = *reinterpret_cast<const uint4*>(sh.q + lo);

  // ---- Section 3.3 from the tile's first non-121 byte on, from the gaps
  // between non-121 bytes: a max-scan over the threads' last non-121
  // positions gives each thread the previous one, a sum-scan of what each
  // thread emits gives its output offset (zre_scan.hpp: rs_gaps_len,
  // rs_gaps_emit); the thread with the tile's last non-121 byte adds the
  // trailing run's codes 255 to its length.
  // The mask of the thread's non-121 bytes is kept spread, bit 2i for byte
  // lo + i, the form the trits of a register-packed tile give directly.
  static_assert(kBytes == 16, "one uint4 of quartic bytes per thread");
  const uint32_t nz = own ? nonzero_mask_trits(h[0]) : (cnt ? nonzero_mask16_spread(w, cnt) : 0u);
  const uint32_t last = nz ? lo + (31u - (uint32_t)__builtin_clz(nz)) / 2u : 0u;
  const ScanU32 pm = block_scan_max_u32(nz ? last + 1u : 0u, sh.red);
  const int prev = (int)pm.excl - 1;  // the previous non-121 byte, -1 if none
  const bool tail = nz != 0u && last + 1u == pm.total;
  if (nz != 0u && prev < 0) sh.lead = lo + (uint32_t)__builtin_ctz(nz) / 2u;
  const uint32_t trail = tile_bytes - pm.total;  // 121s after the last non-121 byte
  const uint32_t mine = rs_gaps_len<2>(nz, lo, prev) + (tail ? trail / kRunMax : 0u);
  // every output byte that is not a remainder code or a non-121 byte is a
  // 255: fill the whole output with 255 first (the scan's barrier orders
  // it before the writes below), so runs only advance the offset
  static_assert(sizeof(sh.out) == 16 * (kThreads + 1), "one uint4 of output per thread, +1");
  reinterpret_cast<uint4*>(sh.out)[threadIdx.x] = make_uint4(~0u, ~0u, ~0u, ~0u);
  if (threadIdx.x == 0) reinterpret_cast<uint4*>(sh.out)[kThreads] = make_uint4(~0u, ~0u, ~0u, ~0u);
  const ScanU32 off = block_scan_u32(mine, sh.red2);
  uint32_t o = off.excl;
  auto put = [&](uint32_t c) {
    if (o < sizeof(sh.out)) sh.out[o] = (uint8_t)c;
    ++o;
  };
  const uint32_t w0 = w.x, w1 = w.y, w2 = w.z, w3 = w.w;
  rs_gaps_emit<2>(nz, lo, prev,
                  [w0, w1, w2, w3](uint32_t i) { return byte_of16(w0, w1, w2, w3, i); }, put,
                  [&](uint32_t k) { o += k; });
  // the slot holds at most the tile's own bytes; the clamp only keeps a
  // logic error inside the slot
  const uint32_t len = umin32(off.total, tile_bytes);
  __syncthreads();
  for (uint32_t i = 16u * threadIdx.x; i < len; i += 16u * kThreads)
    *reinterpret_cast<uint4*>(slots + q0 + i) = *reinterpret_cast<const uint4*>(sh.out + i);
  if (threadIdx.x == 0) {
    TileRec rec;
    if (pm.total == 0u) {  // all 121: one run
      rec.agg = rs_zero_run(tile_bytes).v;
      rec.lead = (uint16_t)tile_bytes;
      rec.len = 0u;
    } else {
      rec.agg = rs_combine(rs_zero_run(sh.lead), rs_make(0u, 0u, trail % kRunMax, off.total)).v;
      rec.lead = (uint16_t)sh.lead;
      rec.len = (uint16_t)len;
    }
    rec.nfix = umin32(sh.nfix, kFixCap);
    recs[t] = rec;
  }
}

// The first pass from trits with two waves per tile: each thread takes 32
// quartic bytes, twice what tlc_quant_encode_kernel's threads take, so the
// block scans, the scale's verdict and the record, which cost the same per
// thread, are spread over twice the bytes (this pass is bound by its vector
// instructions).  The same stream and records as tlc_quant_encode_kernel
// with trits: the thread's bytes are two halves of 16, each packed and
// masked as there, and the emitted-byte count and the emission take the
// halves in turn (a gap inside a half costs exactly one code).
constexpr int kTritThreads = 128;
constexpr int kTritWaves = kTritThreads / 64;
// Below this many tiles the grid is too small to hide the longer work per
// block, and four waves per tile are faster (on gfx950: 13,108 tiles 19.3
// against 23.0 us; a mix of 3,277- and 1,250-tile tensors 10.8 against 9.6).
constexpr uint32_t kTritTwoWaveMinTiles = 8192;
static_assert(kEncTile / kTritThreads == 32, "two uint4 of quartic bytes per thread");

__global__ __launch_bounds__(kTritThreads) void tlc_quant_encode_trits_kernel(
    uint64_t n, uint32_t m, float s, const uint32_t* __restrict__ partials, uint32_t np,
    uint8_t* __restrict__ slots, TileRec* __restrict__ recs, const uint8_t* __restrict__ trits,
    Ctrl* __restrict__ ctrl, HostMirror hm) {
  __shared__ EncShared sh;
  __shared__ uint32_t s_lut[5][256];
  __shared__ uint32_t s_scale[kTritWaves];  // block 0's reduction of M, read after its barrier
  const uint32_t t = blockIdx.x;
  const uint64_t q0 = (uint64_t)t * kEncTile;
  const uint32_t tile_bytes = (uint32_t)umin64(kEncTile, (uint64_t)m - q0);
  // an interior tile (whole, every value before n): each thread packs its
  // own 32 quartic bytes in registers; other tiles pack through sh.q
  const bool own = tile_bytes == (uint32_t)kEncTile && 4ull * m + q0 + kEncTile <= n;
  const uint32_t lo = threadIdx.x * 32u;
  uint32_t d[2][5];  // own tile: the trits of the thread's values, 16 per word
  uint32_t h[kEncTile / 4 / kTritThreads][5];
  if (own) {
    // 64 consecutive bits of the trit array per partition from bit
    // 2*(k*m + q0) + 64*tid on, from the aligned words at or after the one
    // holding the first; as in load_trit_words, the word past the last one
    // lies inside the trit area
    const uint32_t* tw = reinterpret_cast<const uint32_t*>(trits);
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      const uint64_t e0 = (uint64_t)k * m + q0;
      const uint32_t sh2 = 2u * (uint32_t)(e0 & 15u);
      const uint32_t* wp = tw + (e0 >> 4) + 2u * threadIdx.x;
      const uint32_t w0 = wp[0], w1 = wp[1], w2 = wp[2];
      d[0][k] = sh2 ? __builtin_amdgcn_alignbit(w1, w0, sh2) : w0;
      d[1][k] = sh2 ? __builtin_amdgcn_alignbit(w2, w1, sh2) : w1;
    }
  } else {
    load_trits<kTritThreads>(trits, n, m, q0, tile_bytes, h);
  }
  init_trit_luts<kTritThreads>(s_lut);
  Scale sc;
  if (t != 0) {
    // only block 0 needs M (for the result); the others need the verdict,
    // which the writing pass left in every partial: all 0xffffffff for a
    // refused tensor, otherwise the check pass's finite maxima
    __syncthreads();  // the tables
    sc.M = 0.0f;
    sc.U = 0.0f;
    sc.bad = partials[0] >= 0x7f800000u ? 1u : 0u;
  } else {
    // its own LDS words: the scans below reuse sh.red with no barrier between
    sc = finish_scale<kTritThreads>(partials, np, s, s_scale);  // includes a barrier
    if (threadIdx.x == 0) {
      ctrl->enc.err = sc.bad;
      ctrl->enc.scale = sc.M;
      host_put_result(hm.res, sc.bad, sc.M);
    }
  }
  if (sc.bad) return;  // NaN/Inf or overflow: the buffer keeps its values, no stream
  const uint32_t cnt = lo < tile_bytes ? umin32(32u, tile_bytes - lo) : 0u;
  uint4 w[2];
  uint32_t nz[2];  // non-121 bytes of each half, spread: bit 2i for byte i of the half
  if (own) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      w[hf] = pack_trit_words(d[hf], s_lut);
      nz[hf] = nonzero_mask_trits(d[hf]);
    }
  } else {
    pack_trits<kTritThreads>(h, n, m, q0, tile_bytes, s_lut, sh.q);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const uint32_t c = cnt > 16u * hf ? umin32(cnt - 16u * hf, 16u) : 0u;
      w[hf] = c ? *reinterpret_cast<const uint4*>(sh.q + lo + 16u * hf) : make_uint4(0, 0, 0, 0);
      nz[hf] = c ? nonzero_mask16_spread(w[hf], c) : 0u;
    }
  }

  // ---- Section 3.3 as in tlc_quant_encode_kernel, over the two halves
  const uint32_t last0 = nz[0] ? lo + (31u - (uint32_t)__builtin_clz(nz[0])) / 2u : 0u;
  const uint32_t last1 = nz[1] ? lo + 16u + (31u - (uint32_t)__builtin_clz(nz[1])) / 2u : 0u;
  const bool any = (nz[0] | nz[1]) != 0u;
  const uint32_t last = nz[1] ? last1 : last0;
  const ScanU32 pm = block_scan_max_u32<kTritWaves>(any ? last + 1u : 0u, sh.red);
  const int prev = (int)pm.excl - 1;  // the previous non-121 byte, -1 if none
  const int prev1 = nz[0] ? (int)last0 : prev;  // the same before the second half
  const bool tail = any && last + 1u == pm.total;
  if (any && prev < 0)
    sh.lead = nz[0] ? lo + (uint32_t)__builtin_ctz(nz[0]) / 2u
                    : lo + 16u + (uint32_t)__builtin_ctz(nz[1]) / 2u;
  const uint32_t trail = tile_bytes - pm.total;  // 121s after the last non-121 byte
  const uint32_t mine = rs_gaps_len<2>(nz[0], lo, prev) + rs_gaps_len<2>(nz[1], lo + 16u, prev1) +
                        (tail ? trail / kRunMax : 0u);
  static_assert(sizeof(sh.out) == 32 * kTritThreads + 16, "two uint4 of output per thread, +1");
  reinterpret_cast<uint4*>(sh.out)[2 * threadIdx.x] = make_uint4(~0u, ~0u, ~0u, ~0u);
  reinterpret_cast<uint4*>(sh.out)[2 * threadIdx.x + 1] = make_uint4(~0u, ~0u, ~0u, ~0u);
  if (threadIdx.x == 0)
    reinterpret_cast<uint4*>(sh.out)[2 * kTritThreads] = make_uint4(~0u, ~0u, ~0u, ~0u);
  const ScanU32 off = block_scan_u32<kTritWaves>(mine, sh.red2);
  uint32_t o = off.excl;
  auto put = [&](uint32_t c) {
    if (o < sizeof(sh.out)) sh.out[o] = (uint8_t)c;
    ++o;
  };
  auto fill = [&](uint32_t k) { o += k; };
  {
    const uint32_t a0 = w[0].x, a1 = w[0].y, a2 = w[0].z, a3 = w[0].w;
    rs_gaps_emit<2>(nz[0], lo, prev,
                    [a0, a1, a2, a3](uint32_t i) { return byte_of16(a0, a1, a2, a3, i); }, put,
                    fill);
    const uint32_t b0 = w[1].x, b1 = w[1].y, b2 = w[1].z, b3 = w[1].w;
    rs_gaps_emit<2>(nz[1], lo + 16u, prev1,
                    [b0, b1, b2, b3](uint32_t i) { return byte_of16(b0, b1, b2, b3, i); }, put,
                    fill);
  }
  // the slot holds at most the tile's own bytes; the clamp only keeps a
  // logic error inside the slot
  const uint32_t len = umin32(off.total, tile_bytes);
  __syncthreads();
  for (uint32_t i = 16u * threadIdx.x; i < len; i += 16u * kTritThreads)
    *reinterpret_cast<uint4*>(slots + q0 + i) = *reinterpret_cast<const uint4*>(sh.out + i);
  if (threadIdx.x == 0) {
    TileRec rec;
    if (pm.total == 0u) {  // all 121: one run
      rec.agg = rs_zero_run(tile_bytes).v;
      rec.lead = (uint16_t)tile_bytes;
      rec.len = 0u;
    } else {
      rec.agg = rs_combine(rs_zero_run(sh.lead), rs_make(0u, 0u, trail % kRunMax, off.total)).v;
      rec.lead = (uint16_t)sh.lead;
      rec.len = (uint16_t)len;
    }
    rec.nfix = 0u;
    recs[t] = rec;
  }
}

// Pass B: one wave per chunk of 64 tiles: every tile's prefix within its
// chunk (an ordered wave scan) and the chunk's summary.  The last block to
// finish (a count of finished blocks, each block's summaries released
// before its count) then scans the chunk summaries in place, each entry
// becoming its chunk's exclusive prefix, and clears the count for the next
// call.
constexpr uint32_t kChunkTiles = 64;

__global__ __launch_bounds__(kThreads) void tlc_zre_chunk_kernel(
    const TileRec* __restrict__ recs, uint32_t ntiles, uint64_t* __restrict__ local_pre,
    uint64_t* __restrict__ chunk_agg, Ctrl* __restrict__ ctrl) {
  __shared__ RunSum s_wave[kWaves];
  __shared__ uint32_t s_last;
  if (ctrl->enc.err) return;  // pass A refused the tensor (every block returns)
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint32_t nchunks = (ntiles + kChunkTiles - 1) / kChunkTiles;
  const uint32_t c = blockIdx.x * kWaves + wid;
  if (c < nchunks) {  // whole waves
    const uint32_t i = c * kChunkTiles + lane;
    RunSum a = rs_identity();
    if (i < ntiles) a.v = recs[i].agg;
    const RunSum incl = wave_incl_scan_rs(a);
    const RunSum ex = wave_prev_lane_rs(incl);
    if (i < ntiles) local_pre[i] = ex.v;
    if (lane == 63) chunk_agg[c] = incl.v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    s_last = atomicAdd(&ctrl->chunk_done, 1u) == gridDim.x - 1u ? 1u : 0u;
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  // thread j scans a run of consecutive chunks
  const uint32_t per = (nchunks + kThreads - 1) / kThreads;
  const uint32_t j0 = umin32(threadIdx.x * per, nchunks), j1 = umin32(j0 + per, nchunks);
  RunSum mine = rs_identity();
  for (uint32_t j = j0; j < j1; ++j) {
    RunSum a;
    a.v = chunk_agg[j];
    mine = rs_combine(mine, a);
  }
  const RunSum incl = wave_incl_scan_rs(mine);
  const RunSum ex = wave_prev_lane_rs(incl);
  if (lane == 63) s_wave[wid] = incl;
  __syncthreads();
  RunSum p = rs_identity();
  for (uint32_t w = 0; w < wid; ++w) p = rs_combine(p, s_wave[w]);
  p = rs_combine(p, ex);
  for (uint32_t j = j0; j < j1; ++j) {  // every load of the run came before these stores
    RunSum a;
    a.v = chunk_agg[j];
    chunk_agg[j] = p.v;
    p = rs_combine(p, a);
  }
  if (threadIdx.x == 0)
    __hip_atomic_store(&ctrl->chunk_done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Pass C, the compaction: one wave per tile.  Prefix = the chunk's prefix
// combined with the tile's prefix within the chunk; then the leading run's
// codes and the slot; the last tile also writes the remainder of a run that
// ends the stream and the stream length.  Every write is clamped to
// the m-byte output (the stream never exceeds m bytes; the clamp only
// contains a logic error).
__global__ __launch_bounds__(kThreads) void tlc_zre_compact_kernel(
    const TileRec* __restrict__ recs, const uint64_t* __restrict__ chunk_pre,
    const uint64_t* __restrict__ local_pre, const uint8_t* __restrict__ slots, uint32_t m,
    uint32_t ntiles, uint8_t* __restrict__ out, const uint2* __restrict__ fix,
    float* __restrict__ r, uint64_t n, Ctrl* __restrict__ ctrl, HostMirror hm) {
  if (ctrl->enc.err) return;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t t = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (t >= ntiles) return;  // whole waves; nothing below synchronises the block
  RunSum cp, lp;
  cp.v = chunk_pre[t / kChunkTiles];
  lp.v = local_pre[t];
  const RunSum P = rs_combine(cp, lp);
  const TileRec rec = recs[t];
  const uint64_t q0 = (uint64_t)t * kEncTile;
  const uint32_t tile_bytes = (uint32_t)umin64(kEncTile, (uint64_t)m - q0);
  const uint32_t off = rs_emitted(P);
  const uint32_t grown = rs_phase(P) + rec.lead;  // the open run after the leading 121s
  const uint32_t n255 = grown / kRunMax, rho = grown % kRunMax;
  const bool rest = rec.lead < tile_bytes;
  const uint32_t code = (rest && rho) ? 1u : 0u;
  for (uint32_t i = lane; i < n255; i += 64u)
    if (off + i < m) out[off + i] = (uint8_t)kFullChunk;
  if (code && lane == 0 && off + n255 < m) out[off + n255] = (uint8_t)rs_code(rho);
  if (rest) {
    const uint32_t at = off + n255 + code;
    const uint32_t len = umin32(rec.len, tile_bytes);
    // dword loads from the slot (4096-byte aligned, len <= 4096), byte stores
    for (uint32_t i = 4u * lane; i < len; i += 256u) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(slots + q0 + i);
#pragma unroll
      for (uint32_t b = 0; b < 4u; ++b)
        if (i + b < len && at + i + b < m) out[at + i + b] = (uint8_t)(w >> (8u * b));
    }
  }
  // the residuals the first pass left in the tile's fix list
  const uint2* tf = fix + (uint64_t)t * kFixCap;
  const uint32_t nf = umin32(rec.nfix, kFixCap);
  for (uint32_t i = lane; i < nf; i += 64u) {
    const uint2 f = tf[i];
    const uint32_t k = f.x / (uint32_t)kEncTile, p = f.x % (uint32_t)kEncTile;
    const uint64_t e = (uint64_t)k * m + q0 + p;
    if (k < 5u && p < tile_bytes && e < n) r[e] = __uint_as_float(f.y);
  }
  if (t + 1 == ntiles && lane == 0) {  // a run that ends the stream; the length
    RunSum a;
    a.v = rec.agg;
    const RunSum T = rs_combine(P, a);
    const uint32_t total = rs_total(T);
    if (rs_phase(T) && total >= 1u && total - 1u < m)
      out[total - 1u] = (uint8_t)rs_code(rs_phase(T));
    ctrl->enc.len = total;
    if (hm.res) host_put(&hm.res->len, total);
  }
}

// A small tensor in one pass: tiles taken in order from the ticket and
// chained by decoupled look-back (status slot = tile).  With few tiles the
// look-back rarely waits, and this saves the two small passes' launches.
// kX (the default error policy): partials are the check pass's, the buffer
// still holds the previous residual, and the tiles form acc = x + r
// themselves (no writing max pass before them).
template <int kPath, bool kX>
__global__ __launch_bounds__(kThreads) void tlc_quant_encode_chained_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n, uint32_t m, float s,
    const uint32_t* __restrict__ partials, uint32_t np, uint8_t* __restrict__ out,
    uint64_t* __restrict__ status, uint32_t ticket_base, uint32_t epoch,
    Ctrl* __restrict__ ctrl, HostMirror hm) {
  __shared__ EncShared sh;
  __shared__ uint32_t s_tile;
  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->enc_ticket) - ticket_base;
  const Scale sc = finish_scale(partials, np, s, sh.red);  // includes a barrier
  const uint32_t tile = s_tile;
  if (tile == 0 && threadIdx.x == 0) {
    ctrl->enc.err = sc.bad;
    ctrl->enc.scale = sc.M;
    host_put_result(hm.res, sc.bad, sc.M);
  }
  if (sc.bad) return;  // NaN/Inf or overflow: no stream (the buffer as it was, or acc)
  encode_tile<kPath, kX>(x, r, n, m, sc, tile, 0, out, status, epoch, ctrl, &ctrl->enc, hm.res,
                         hm.fault, sh);
}

// kX as for the chained kernel (partials: the check pass's).  The float4
// paths need x aligned like r (vec bit 2) when kX.
template <bool kX>
__global__ __launch_bounds__(kThreads) void tlc_quant_encode_batch_kernel(
    const EncDesc* __restrict__ descs, uint32_t count, const uint32_t* __restrict__ partials,
    EncResult* __restrict__ results, uint64_t* __restrict__ status, uint32_t ticket_base,
    uint32_t epoch, Ctrl* __restrict__ ctrl, HostMirror hm) {
  __shared__ EncShared sh;
  __shared__ uint32_t s_tile;
  if (threadIdx.x == 0) s_tile = take_ticket(&ctrl->enc_ticket) - ticket_base;
  __syncthreads();
  const uint32_t T = s_tile;
  const uint32_t t = find_desc(descs, count, T, [](const EncDesc& d) { return d.tile0; });
  const EncDesc d = descs[t];
  const Scale sc = finish_scale(partials + d.blk0, d.nblk, d.s, sh.red);
  const uint32_t lt = T - d.tile0;
  EncResult* hres = hm.res ? hm.res + t : nullptr;
  if (lt == 0 && threadIdx.x == 0) {
    results[t].err = sc.bad;
    results[t].scale = sc.M;
    host_put_result(hres, sc.bad, sc.M);
    if (sc.bad) {
      results[t].len = 0u;
      if (hres) host_put(&hres->len, 0u);
    }
  }
  if (sc.bad) return;  // this tensor is refused; the others go on
  const bool xal = !kX || (d.vec & 4u);
  if ((d.vec & 1u) && xal)
    encode_tile<kPathVec, kX>(d.x, d.r, d.n, d.m, sc, lt, d.tile0, d.out, status, epoch, ctrl,
                              &results[t], hres, hm.fault, sh);
  else if ((d.vec & 2u) && xal)
    encode_tile<kPathShift, kX>(d.x, d.r, d.n, d.m, sc, lt, d.tile0, d.out, status, epoch,
                                ctrl, &results[t], hres, hm.fault, sh);
  else
    encode_tile<kPathByte, kX>(d.x, d.r, d.n, d.m, sc, lt, d.tile0, d.out, status, epoch,
                               ctrl, &results[t], hres, hm.fault, sh);
}

// ---------------------------------------------------------------- comparison modes
// Quantization + quartic pack without zero-run encoding: the quartic bytes
// are the payload (m bytes), so tiles are independent and need no
// look-back.  kStoch selects stochastic 3-value quantization of x with
// Philox random words (no error feedback: r is not read or written);
// otherwise Eq. 2 on the accumulated buffer r with the residual write-back,
// exactly as in tlc_quant_encode_kernel (x is not read).
template <bool kVec, bool kStoch>
__global__ __launch_bounds__(kThreads) void tlc_quant_pack_kernel(
    const float* __restrict__ x, float* __restrict__ r, uint64_t n, uint32_t m, float s,
    uint64_t seed, uint64_t step, const uint32_t* __restrict__ partials, uint32_t np,
    uint8_t* __restrict__ out, Ctrl* __restrict__ ctrl) {
  __shared__ uint32_t red[kWaves];
  const Scale sc = finish_scale(partials, np, s, red);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctrl->enc.err = sc.bad;
    ctrl->enc.scale = sc.M;
    ctrl->enc.len = sc.bad ? 0u : m;
  }
  if (sc.bad) return;
  const uint64_t q0 = (uint64_t)blockIdx.x * kEncTile;
  const uint32_t tile_bytes = (uint32_t)umin64(kEncTile, (uint64_t)m - q0);
  if (kVec) {
    for (uint32_t g = threadIdx.x; g * 4u < tile_bytes; g += kThreads) {
      const uint64_t j = q0 + g * 4u;
      uint32_t w;
      if (!kStoch) {
        w = quantize_group4(nullptr, r, n, m, j, sc.M, sc.U);
      } else {
        uint32_t code[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int k = 0; k < 5; ++k) {
          const uint64_t e = k * m + j;  // a multiple of 4: one Philox call per slice
          const Philox4 rw = element_words(e >> 2, step, seed);
          if (e + 4 <= n) {
            const float4 a = ld_stream(x + e);
            code[0] = code[0] * 3u + stochastic_trit(a.x, sc.M, rw.v[0]);
            code[1] = code[1] * 3u + stochastic_trit(a.y, sc.M, rw.v[1]);
            code[2] = code[2] * 3u + stochastic_trit(a.z, sc.M, rw.v[2]);
            code[3] = code[3] * 3u + stochastic_trit(a.w, sc.M, rw.v[3]);
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
              code[c] = code[c] * 3u +
                        (e + c < n ? stochastic_trit(x[e + c], sc.M, rw.v[c]) : 0u);
          }
        }
        w = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) out[j + c] = (uint8_t)(w >> (8 * c));
    }
  } else {
    for (uint32_t lj = threadIdx.x; lj < tile_bytes; lj += kThreads) {
      const uint64_t j = q0 + lj;
      uint32_t code;
      if (!kStoch) {
        code = quantize_byte(nullptr, r, n, m, j, sc.M, sc.U);
      } else {
        code = 0u;
#pragma unroll
        for (int k = 0; k < 5; ++k) {
          const uint64_t e = k * m + j;
          uint32_t t = 0u;
          if (e < n) t = stochastic_trit(x[e], sc.M, element_words(e >> 2, step, seed).v[e & 3]);
          code = code * 3u + t;
        }
      }
      out[j] = (uint8_t)code;
    }
  }
}

// ---------------------------------------------------------------- launchers
static inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0u;
}

namespace {
uint32_t absmax_blocks(uint64_t n, bool vec) {
  const uint64_t items = vec ? (n >> 2) : n;
  uint64_t blocks = (items + kThreads * 4 - 1) / (kThreads * 4);
  return (uint32_t)(blocks < 1 ? 1 : (blocks > kAbsmaxMaxBlocks ? kAbsmaxMaxBlocks : blocks));
}
}  // namespace

hipError_t launch_absmax_check(const float* x, const float* r, uint64_t n, uint32_t* partials,
                               uint32_t* nblocks, hipStream_t st) {
  const bool vec = aligned16(x) && aligned16(r);
  const uint32_t blocks = absmax_blocks(n, vec);
  *nblocks = blocks;
  if (vec)
    launch_k(tlc_absmax_check_kernel<true>, blocks, kThreads, st, x, r, n, partials);
  else
    launch_k(tlc_absmax_check_kernel<false>, blocks, kThreads, st, x, r, n, partials);
  return hipGetLastError();
}

hipError_t launch_accum_absmax(const float* x, float* r, uint64_t n, uint32_t* partials,
                               uint32_t* nblocks, uint16_t* summ, const uint32_t* guard,
                               uint32_t guard_np, float s, bool trit, hipStream_t st) {
  const bool vec = aligned16(x) && (r == nullptr || aligned16(r));
  if (summ && !(vec && r)) return hipErrorInvalidValue;  // summaries need the float4 path
  if (trit && !(summ && guard)) return hipErrorInvalidValue;  // trits need M from the check
  const uint32_t blocks = absmax_blocks(n, vec);
  if (guard && guard_np != blocks) return hipErrorInvalidValue;  // same launch as the check
  *nblocks = blocks;
  if (trit) {
    launch_k(tlc_accum_quantize_kernel, blocks, kThreads, st,
        x, r, n, partials, reinterpret_cast<uint8_t*>(summ), guard, guard_np, s);
    return hipGetLastError();
  }
#define TLC_LAUNCH(V, R, S)                                                                 \
  launch_k(tlc_accum_absmax_kernel<V, R, S>, blocks, kThreads, st, x, r, n, partials, summ, guard, \
                                                                guard_np, s)
  if (r == nullptr) {  // no error buffer: max |x|
    if (aligned16(x)) TLC_LAUNCH(true, false, false); else TLC_LAUNCH(false, false, false);
  } else if (vec) {
    if (summ) TLC_LAUNCH(true, true, true); else TLC_LAUNCH(true, true, false);
  } else {
    TLC_LAUNCH(false, true, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

hipError_t launch_quant_encode(float* r, uint64_t n, uint32_t m, float s,
                               const uint32_t* partials, uint32_t npartials, uint8_t* slots,
                               TileRec* recs, uint2* fix, const uint16_t* summ, bool trit,
                               Ctrl* ctrl, HostMirror hm, hipStream_t st) {
  const uint32_t ntiles = (uint32_t)((m + kEncTile - 1) / kEncTile);
  const bool al = aligned16(r);
#define TLC_ARGS r, n, m, s, partials, npartials, slots, recs, fix, summ, ctrl, hm
  if (trit) {
    if (!summ) return hipErrorInvalidValue;
    if (ntiles >= kTritTwoWaveMinTiles)
      launch_k(tlc_quant_encode_trits_kernel, ntiles, kTritThreads, st, n, m, s, partials,
          npartials, slots, recs, reinterpret_cast<const uint8_t*>(summ), ctrl, hm);
    else
      launch_k(tlc_quant_encode_kernel<kPathVec, true>, ntiles, kThreads, st, TLC_ARGS);
  } else if (al && m % 4 == 0) {
    launch_k(tlc_quant_encode_kernel<kPathVec>, ntiles, kThreads, st, TLC_ARGS);
  } else {
    summ = nullptr;  // bounds serve the float4 slices only
    if (al)
      launch_k(tlc_quant_encode_kernel<kPathShift>, ntiles, kThreads, st, TLC_ARGS);
    else
      launch_k(tlc_quant_encode_kernel<kPathByte>, ntiles, kThreads, st, TLC_ARGS);
  }
#undef TLC_ARGS
  return hipGetLastError();
}

hipError_t launch_quant_encode_chained(const float* x, float* r, uint64_t n, uint32_t m,
                                       float s, const uint32_t* partials, uint32_t npartials,
                                       uint8_t* out, uint64_t* status, uint32_t ntiles,
                                       uint32_t ticket_base, uint32_t epoch, Ctrl* ctrl,
                                       HostMirror hm, hipStream_t st) {
  const bool fused = x != nullptr;
  const bool al = aligned16(r) && (!fused || aligned16(x));
#define TLC_LAUNCH(P, X)                                                                    \
  launch_k(tlc_quant_encode_chained_kernel<P, X>, ntiles, kThreads, st,                         \
      x, r, n, m, s, partials, npartials, out, status, ticket_base, epoch, ctrl, hm)
  if (al && m % 4 == 0) {
    if (fused) TLC_LAUNCH(kPathVec, true); else TLC_LAUNCH(kPathVec, false);
  } else if (al) {
    if (fused) TLC_LAUNCH(kPathShift, true); else TLC_LAUNCH(kPathShift, false);
  } else {
    if (fused) TLC_LAUNCH(kPathByte, true); else TLC_LAUNCH(kPathByte, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

hipError_t launch_zre_chunks(const TileRec* recs, uint32_t ntiles, uint64_t* local_pre,
                             uint64_t* chunk_agg, Ctrl* ctrl, hipStream_t st) {
  const uint32_t nchunks = (ntiles + kChunkTiles - 1) / kChunkTiles;
  launch_k(tlc_zre_chunk_kernel, (nchunks + kWaves - 1) / kWaves, kThreads, st,
      recs, ntiles, local_pre, chunk_agg, ctrl);
  return hipGetLastError();
}

hipError_t launch_zre_compact(const TileRec* recs, const uint64_t* chunk_pre,
                              const uint64_t* local_pre, const uint8_t* slots, uint32_t m,
                              uint8_t* out, const uint2* fix, float* r, uint64_t n, Ctrl* ctrl,
                              HostMirror hm, hipStream_t st) {
  const uint32_t ntiles = (uint32_t)((m + kEncTile - 1) / kEncTile);
  launch_k(tlc_zre_compact_kernel, (ntiles + kWaves - 1) / kWaves, kThreads, st,
      recs, chunk_pre, local_pre, slots, m, ntiles, out, fix, r, n, ctrl, hm);
  return hipGetLastError();
}

hipError_t launch_absmax_check_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_blocks, uint32_t* partials, hipStream_t st) {
  launch_k(tlc_absmax_check_batch_kernel, total_blocks, kThreads, st, descs, count, partials);
  return hipGetLastError();
}

hipError_t launch_accum_absmax_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_blocks, uint32_t* partials,
                                     const uint32_t* guard, hipStream_t st) {
  launch_k(tlc_accum_absmax_batch_kernel, total_blocks, kThreads, st, descs, count, partials,
                                                                   guard);
  return hipGetLastError();
}

hipError_t launch_quant_encode_batch(const EncDesc* descs, uint32_t count,
                                     uint32_t total_tiles, const uint32_t* partials,
                                     bool fused, EncResult* results, uint64_t* status,
                                     uint32_t ticket_base, uint32_t epoch, Ctrl* ctrl,
                                     HostMirror hm, hipStream_t st) {
  if (fused)
    launch_k(tlc_quant_encode_batch_kernel<true>, total_tiles, kThreads, st,
        descs, count, partials, results, status, ticket_base, epoch, ctrl, hm);
  else
    launch_k(tlc_quant_encode_batch_kernel<false>, total_tiles, kThreads, st,
        descs, count, partials, results, status, ticket_base, epoch, ctrl, hm);
  return hipGetLastError();
}

}  // namespace tlc

namespace tlc {

hipError_t launch_quant_pack(const float* x, float* r, uint64_t n, uint32_t m, float s,
                             int stochastic, uint64_t seed, uint64_t step,
                             const uint32_t* partials, uint32_t npartials, uint8_t* out,
                             Ctrl* ctrl, hipStream_t st) {
  const uint32_t blocks = (uint32_t)((m + kEncTile - 1) / kEncTile);
  const bool vec = (m % 4 == 0) && aligned16(stochastic ? x : r);
#define TLC_LAUNCH(V, S)                                                                      \
  launch_k(tlc_quant_pack_kernel<V, S>, blocks, kThreads, st, x, r, n, m, s, seed, step, partials, \
                                                           npartials, out, ctrl)
  if (stochastic) {
    if (vec) TLC_LAUNCH(true, true); else TLC_LAUNCH(false, true);
  } else {
    if (vec) TLC_LAUNCH(true, false); else TLC_LAUNCH(false, false);
  }
#undef TLC_LAUNCH
  return hipGetLastError();
}

}  // namespace tlc
