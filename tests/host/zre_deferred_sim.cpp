// Host-only simulation of the three-pass zero-run encoder:
//   pass A, per tile of `tile` bytes cut into threads of `per` bytes: L =
//     index of the tile's first non-121 byte (tile length if none); every
//     thread summarises its bytes at index >= L, the tile scans those
//     summaries, and each thread encodes its bytes from its own prefix
//     into the tile's slot (phase 0 at the first non-121 byte, so nothing
//     depends on earlier tiles); record = (summary of the whole tile, L,
//     slot length);
//   pass B: exclusive scan of the tile summaries in tile order;
//   pass C, per tile: with phase phi and output offset from its prefix,
//     write (phi + L) / 14 codes 255, then (if the tile has a non-121 byte)
//     the remainder code of (phi + L) mod 14 and the slot; after the last
//     tile, the remainder of a run that ends the stream.
// For PER <= 16 every thread's segment is also summarised and encoded from
// the mask of its non-121 bytes (rs_mask_summary, rs_mask_walk), which must
// agree with the byte-by-byte forms (exit 4, 5, 6 otherwise), and every
// tile is also encoded in the gap form (rs_gaps_len, rs_gaps_emit: output
// offsets from a sum over threads, the previous non-121 byte from a max),
// which must give the same slot and record (exit 7-10 otherwise), with the
// mask in its compact and its spread form alike (exit 11, 12 otherwise).
// Reads raw bytes on stdin, writes the encoded stream on stdout.
// Usage: zre_deferred_sim TILE PER < in > out
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../paper_1802_07389_amd/csrc/zre_scan.hpp"

using namespace tlc;

struct Rec {
  RunSum agg;
  uint32_t lead, len;
};

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  const size_t tile = std::strtoul(argv[1], nullptr, 10);
  const size_t per = std::strtoul(argv[2], nullptr, 10);
  if (!tile || !per || tile % per) return 2;
  std::vector<uint8_t> q;
  int ch;
  while ((ch = std::getchar()) != EOF) q.push_back((uint8_t)ch);
  const size_t m = q.size();
  const size_t ntiles = (m + tile - 1) / tile;
  std::vector<uint8_t> slots(ntiles * tile, 0xEE);
  std::vector<Rec> rec(ntiles);
  // pass A
  for (size_t t = 0; t < ntiles; ++t) {
    const size_t q0 = t * tile, tb = (q0 + tile <= m) ? tile : m - q0;
    size_t L = tb;
    for (size_t j = 0; j < tb; ++j)
      if (q[q0 + j] != kZeroGroup) {
        L = j;
        break;
      }
    RunSum pre = rs_identity();  // exclusive prefix of the thread, bytes >= L only
    for (size_t lo = 0; lo < tb; lo += per) {
      const size_t hi = lo + per < tb ? lo + per : tb;
      const size_t s0 = lo > L ? lo : L;
      const uint32_t o0 = rs_emitted(pre), phi0 = rs_phase(pre);
      uint32_t o = o0, phi = phi0;
      RunSum own = rs_identity();
      for (size_t j = s0; j < hi; ++j) {
        phi = rs_step(q[q0 + j], phi, [&](uint32_t b) { slots[t * tile + o++] = (uint8_t)b; });
        own = rs_combine(own, rs_byte(q[q0 + j]));
      }
      // the same segment from the mask of its non-121 bytes (segments of
      // at most 16 bytes): summary and bytes must agree
      if (per <= 16) {
        const uint32_t len = s0 < hi ? (uint32_t)(hi - s0) : 0u;
        uint32_t nz = 0u;
        for (uint32_t i = 0; i < len; ++i)
          if (q[q0 + s0 + i] != kZeroGroup) nz |= 1u << i;
        if (rs_mask_summary(nz, len).v != own.v) return 4;
        uint32_t o2 = o0;
        const uint32_t phi2 = rs_mask_walk(
            nz, len, phi0, [&](uint32_t i) { return (uint32_t)q[q0 + s0 + i]; },
            [&](uint32_t b) {
              if (o2 >= o || slots[t * tile + o2] != (uint8_t)b) std::exit(5);
              ++o2;
            });
        if (phi2 != phi || o2 != o) return 6;
      }
      pre = rs_combine(pre, own);
    }
    rec[t] = {rs_combine(rs_zero_run((uint32_t)L), pre), (uint32_t)L, rs_emitted(pre)};
    if (rec[t].len > tb) return 3;
    // the gap form (threads of `per` <= 16 bytes): previous non-121 byte by
    // an exclusive max over the threads' last ones, output offsets by an
    // exclusive sum of the threads' lengths; the thread with the tile's last
    // non-121 byte adds the trailing run's codes 255
    if (per <= 16) {
      std::vector<uint32_t> nzs, lens;
      int last_all = -1;
      for (size_t lo = 0; lo < tb; lo += per) {
        const size_t hi = lo + per < tb ? lo + per : tb;
        uint32_t nz = 0u;
        for (size_t j = lo; j < hi; ++j)
          if (q[q0 + j] != kZeroGroup) nz |= 1u << (j - lo);
        nzs.push_back(nz);
        if (nz) last_all = (int)(lo + 31 - __builtin_clz(nz));
      }
      std::vector<uint8_t> gslot;
      int prev = -1;
      uint32_t total = 0u;
      for (size_t ti = 0; ti < nzs.size(); ++ti) {
        const uint32_t lo = (uint32_t)(ti * per), nz = nzs[ti];
        const int last = nz ? (int)(lo + 31 - __builtin_clz(nz)) : -1;
        uint32_t len = rs_gaps_len(nz, lo, prev);
        // the spread form (bit 2i for byte lo + i) must agree
        uint32_t nz2 = 0u;
        for (uint32_t i = 0; i < 16u; ++i) nz2 |= ((nz >> i) & 1u) << (2u * i);
        if (rs_gaps_len<2>(nz2, lo, prev) != len) return 11;
        if (nz && last == last_all) len += (uint32_t)(tb - 1 - last) / kRunMax;
        const size_t before = gslot.size();
        auto fill = [&](uint32_t k) {
          for (uint32_t e = 0; e < k; ++e) gslot.push_back((uint8_t)kFullChunk);
        };
        std::vector<uint8_t> spread_out;
        rs_gaps_emit<2>(
            nz2, lo, prev, [&](uint32_t i) { return (uint32_t)q[q0 + lo + i]; },
            [&](uint32_t b) { spread_out.push_back((uint8_t)b); },
            [&](uint32_t k) { spread_out.insert(spread_out.end(), k, (uint8_t)kFullChunk); });
        rs_gaps_emit(
            nz, lo, prev, [&](uint32_t i) { return (uint32_t)q[q0 + lo + i]; },
            [&](uint32_t b) { gslot.push_back((uint8_t)b); }, fill);
        if (spread_out.size() != gslot.size() - before ||
            !std::equal(spread_out.begin(), spread_out.end(), gslot.begin() + before))
          return 12;
        if (nz && last == last_all) fill((uint32_t)(tb - 1 - last) / kRunMax);
        if (gslot.size() - before != len) return 7;
        total += len;
        if (nz) prev = last;
      }
      if (total != rec[t].len) return 8;
      for (uint32_t i = 0; i < total; ++i)
        if (gslot[i] != slots[t * tile + i]) return 9;
      const RunSum agg = last_all < 0 ? rs_zero_run((uint32_t)tb)
                                      : rs_combine(rs_zero_run((uint32_t)L),
                                                   rs_make(0u, 0u, (uint32_t)(tb - 1 - last_all) % kRunMax, total));
      if (agg.v != rec[t].agg.v) return 10;
    }
  }
  // pass B
  std::vector<RunSum> excl(ntiles);
  RunSum run = rs_identity();
  for (size_t t = 0; t < ntiles; ++t) {
    excl[t] = run;
    run = rs_combine(run, rec[t].agg);
  }
  const uint32_t total = m ? rs_total(run) : 0;
  // pass C
  std::vector<uint8_t> out(total, 0xEE);
  for (size_t t = 0; t < ntiles; ++t) {
    const size_t q0 = t * tile, tb = (q0 + tile <= m) ? tile : m - q0;
    const uint32_t phi = rs_phase(excl[t]);
    uint32_t o = rs_emitted(excl[t]);
    const uint32_t grown = phi + rec[t].lead;
    for (uint32_t e = 0; e < grown / kRunMax; ++e) out.at(o++) = (uint8_t)kFullChunk;
    if (rec[t].lead < tb) {
      if (grown % kRunMax) out.at(o++) = (uint8_t)rs_code(grown % kRunMax);
      for (uint32_t i = 0; i < rec[t].len; ++i) out.at(o++) = slots[t * tile + i];
    }
    if (t + 1 == ntiles && rs_phase(run)) out.at(total - 1) = (uint8_t)rs_code(rs_phase(run));
  }
  std::fwrite(out.data(), 1, out.size(), stdout);
  return 0;
}
