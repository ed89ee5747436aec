// Host-only simulation of the tiled zero-run encoder: the stream is cut into
// tiles of `tile` bytes and threads of `per` bytes; thread summaries are
// scanned inside a tile, tile prefixes are folded in order (what the
// decoupled look-back computes), and every thread encodes its bytes from its
// own prefix.  As in the kernel, a thread whose `per` bytes are all 121 uses
// the closed forms rs_zero_run / rs_zero_walk instead of the byte loop.
// Reads raw bytes on stdin and writes the encoded stream on stdout.
// Usage: zre_tiling_sim TILE PER < in > out
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../paper_1802_07389_amd/csrc/zre_scan.hpp"

using namespace tlc;

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  const size_t tile = std::strtoul(argv[1], nullptr, 10);
  const size_t per = std::strtoul(argv[2], nullptr, 10);
  if (!tile || !per || tile % per) return 2;
  std::vector<uint8_t> q;
  int c;
  while ((c = std::getchar()) != EOF) q.push_back((uint8_t)c);
  const size_t m = q.size();
  std::vector<uint8_t> out(m + 1, 0xEE);
  size_t ntiles = (m + tile - 1) / tile;
  // pass 1: tile aggregates (independent of every other tile)
  std::vector<RunSum> agg(ntiles);
  for (size_t t = 0; t < ntiles; ++t) {
    RunSum a = rs_identity();
    for (size_t j = t * tile; j < m && j < (t + 1) * tile; ++j)
      a = rs_combine(a, rs_byte(q[j]));
    agg[t] = a;
  }
  // pass 2: exclusive tile prefixes, then per-thread emission
  RunSum excl = rs_identity();
  uint32_t total_written = 0;
  for (size_t t = 0; t < ntiles; ++t) {
    RunSum thr = excl;
    for (size_t p = t * tile; p < (t + 1) * tile && p < m; p += per) {
      size_t cnt = (p + per <= m) ? per : m - p;
      bool zero = cnt == per;
      for (size_t j = p; j < p + cnt; ++j) zero = zero && q[j] == kZeroGroup;
      uint32_t o = rs_emitted(thr);
      uint32_t phi = rs_phase(thr);
      auto put = [&](uint32_t b) { out[o++] = (uint8_t)b; };
      phi = zero ? rs_zero_walk((uint32_t)cnt, phi, put) : rs_walk(&q[p], (uint32_t)cnt, phi, put);
      if (p + cnt == m && phi) out[o++] = (uint8_t)rs_code(phi);
      RunSum s = rs_identity();
      if (zero)
        s = rs_zero_run((uint32_t)cnt);
      else
        for (size_t j = p; j < p + cnt; ++j) s = rs_combine(s, rs_byte(q[j]));
      thr = rs_combine(thr, s);
      if (p + cnt == m) total_written = o;
    }
    excl = rs_combine(excl, agg[t]);
  }
  uint32_t total = m ? rs_total(excl) : 0;
  if (m && total != total_written) {
    std::fprintf(stderr, "length mismatch %u vs %u\n", total, total_written);
    return 1;
  }
  std::fwrite(out.data(), 1, total, stdout);
  return 0;
}
