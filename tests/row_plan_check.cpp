// Host check of the posterior's row plans (16-row blocks, both precisions) at
// every padded observation count the library accepts: each row block belongs
// to exactly one entry of a wave that exists, the block counts match the
// rows, the rows unpack in the order the kernels read them (shifting the
// packed words), and the four SIMDs carry equal work to within the largest
// row.  Prints one line per size and exits non-zero on a failure.
#include <cstdio>

#include "internal.h"

using namespace scoot;

static int check(int m_pad) {
  const int nb32 = m_pad / kBlk32, nb = m_pad / kBlk16, W = posterior_waves(nb32);
  int bad = 0, seen[64] = {0}, simd[4] = {0}, max_rows = 0;
  const RowPlan16 p = plan_rows16(nb, W);
  for (int e = 0; e < 8; ++e) {
    if (e >= W && p.nrows[e] != 0) ++bad;
    if (p.nrows[e] > kMaxRows16) ++bad;
    max_rows = p.nrows[e] > max_rows ? p.nrows[e] : max_rows;
    uint64_t lo = p.lo[e], hi = p.hi[e];
    int cost = 0, prev = -1;
    for (int q = 0; q < p.nrows[e]; ++q) {
      const int I = (int)(lo & ((1u << kRowBits16) - 1));
      if (I != plan16_row(p, e, q)) ++bad;
      if (I <= prev || I >= nb) ++bad;
      prev = I;
      ++seen[I < 64 ? I : 63];
      cost += I + 1;
      lo = (lo >> kRowBits16) | (hi << (64 - kRowBits16));
      hi >>= kRowBits16;
    }
    if (cost != p.blk_start[e + 1] - p.blk_start[e]) ++bad;
    simd[e % 4] += cost;
  }
  for (int I = 0; I < nb; ++I)
    if (seen[I] != 1) ++bad;
  if (p.blk_start[0] != 0 || p.blk_start[8] != nb * (nb + 1) / 2) ++bad;
  int lo_s = simd[0], hi_s = simd[0];
  for (int s : simd) {
    lo_s = s < lo_s ? s : lo_s;
    hi_s = s > hi_s ? s : hi_s;
  }
  if (hi_s - lo_s > nb) ++bad;
  std::printf("m_pad %3d blocks %2d waves %d rows/entry <= %2d simd work %d..%d%s\n", m_pad, nb, W, max_rows, lo_s,
              hi_s, bad ? "  BAD" : "");
  return bad;
}

int main() {
  int bad = 0;
  for (int m_pad = kBlk32; m_pad <= (SCOOT_MAX_OBS + kBlk32 - 1) / kBlk32 * kBlk32; m_pad += kBlk32)
    bad += check(m_pad);
  return bad ? 1 : 0;
}
