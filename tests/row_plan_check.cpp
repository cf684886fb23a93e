// Host check of the posterior's row plans (fp32: 32-row blocks, fp64: 16-row
// blocks) at every padded observation count the library accepts: each row
// block belongs to exactly one entry of a wave that exists, the block counts
// match the rows, the rows unpack in the order the kernels read them
// (shifting the packed words), and the four SIMDs carry equal work to within
// the largest row.  Prints one line per size and exits non-zero on a failure.
#include <cstdio>

#include "internal.h"

using namespace scoot;

static int check(int m_pad, bool fp64) {
  const int nb32 = m_pad / kBlk32, nb = fp64 ? m_pad / kBlk64 : nb32, W = posterior_waves(nb32);
  int bad = 0, seen[64] = {0}, simd[4] = {0}, max_rows = 0;
  RowPlan p32{};
  RowPlan64 p64{};
  if (fp64) p64 = plan_rows64(nb, W);
  else p32 = plan_rows(nb, W);
  const int32_t* nrows = fp64 ? p64.nrows : p32.nrows;
  const int32_t* start = fp64 ? p64.blk_start : p32.blk_start;
  for (int e = 0; e < 8; ++e) {
    if (e >= W && nrows[e] != 0) ++bad;
    if (nrows[e] > (fp64 ? kMaxRows64 : 64 / kRowBits)) ++bad;
    max_rows = nrows[e] > max_rows ? nrows[e] : max_rows;
    uint64_t lo = fp64 ? p64.lo[e] : p32.rows[e], hi = fp64 ? p64.hi[e] : 0;
    const int bits = fp64 ? kRowBits64 : kRowBits;
    int cost = 0, prev = -1;
    for (int q = 0; q < nrows[e]; ++q) {
      const int I = (int)(lo & ((1u << bits) - 1));
      if (fp64 && I != plan64_row(p64, e, q)) ++bad;
      if (I <= prev || I >= nb) ++bad;
      prev = I;
      ++seen[I < 64 ? I : 63];
      cost += I + 1;
      lo = (lo >> bits) | (bits < 64 ? hi << (64 - bits) : 0);
      hi >>= bits;
    }
    if (cost != start[e + 1] - start[e]) ++bad;
    simd[e % 4] += cost;
  }
  for (int I = 0; I < nb; ++I)
    if (seen[I] != 1) ++bad;
  if (start[0] != 0 || start[8] != nb * (nb + 1) / 2) ++bad;
  int lo_s = simd[0], hi_s = simd[0];
  for (int s : simd) {
    lo_s = s < lo_s ? s : lo_s;
    hi_s = s > hi_s ? s : hi_s;
  }
  if (hi_s - lo_s > nb) ++bad;
  std::printf("%s m_pad %3d blocks %2d waves %d rows/entry <= %2d simd work %d..%d%s\n", fp64 ? "fp64" : "fp32",
              m_pad, nb, W, max_rows, lo_s, hi_s, bad ? "  BAD" : "");
  return bad;
}

int main() {
  int bad = 0;
  for (int m_pad = kBlk32; m_pad <= (SCOOT_MAX_OBS + kBlk32 - 1) / kBlk32 * kBlk32; m_pad += kBlk32)
    bad += check(m_pad, false) + check(m_pad, true);
  return bad ? 1 : 0;
}
