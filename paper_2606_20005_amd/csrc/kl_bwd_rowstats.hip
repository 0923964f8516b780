// Launcher of the row-statistics prep of the dK kernel (kl_bwd_rowstats_kernel).
#include "kl_bwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

// One half-wave per 32-row tile (layout and arithmetic: see kl_bwd.hpp).
static __global__ void __launch_bounds__(kRowStatsTile * kRowStatsTilesPerBlock)
kl_bwd_rowstats_kernel(const float* __restrict__ kl, const float* __restrict__ lse_a,
                       const float* __restrict__ lse_b, const float* __restrict__ g, int NQ, int ntq,
                       long long tiles, float* __restrict__ stats, int* __restrict__ fold) {
  const int lane = threadIdx.x & 63, r = lane & 31;
  const long long T = (long long)blockIdx.x * kRowStatsTilesPerBlock + (threadIdx.x >> 5);
  const bool live = T < tiles;
  const long long bh = live ? T / ntq : 0;
  const int q = live ? (int)(T - bh * ntq) * kRowStatsTile + r : 0;
  RowStats s{0.f, 0.f, 0.f, 0.f};
  if (live && q < NQ) {
    const size_t ri = (size_t)bh * NQ + q;
    s = tile_row_stats(lse_a[ri], lse_b[ri], kl[ri], g ? g[ri] : 1.f, true);
  }
  const uint64_t neg = __builtin_amdgcn_ballot_w64(live && s.g < 0.f);
  const bool any_negative = ((neg >> (lane & 32)) & 0xffffffffull) != 0;   // this half-wave's tile
  if (!live) return;
  s = finish_tile_row_stats(s, any_negative);
  float* p = stats + (size_t)T * 4 * kRowStatsTile;
  p[0 * kRowStatsTile + r] = s.lsa2;
  p[1 * kRowStatsTile + r] = s.lsb2;
  p[2 * kRowStatsTile + r] = s.g;
  p[3 * kRowStatsTile + r] = s.dl;
  if (r == 0) fold[T] = any_negative ? 0 : 1;
}

static long long rowstats_tiles(int bh, int nq) { return (long long)bh * ((nq + kRowStatsTile - 1) / kRowStatsTile); }

size_t bwd_rowstats_floats(int bh, int nq) {
  const long long tiles = rowstats_tiles(bh, nq);
  return (size_t)tiles * 4 * kRowStatsTile + (size_t)tiles;   // the int flags take one float's room each
}

hipError_t launch_bwd_rowstats(BwdArgs& a, float* stats) {
  const int ntq = (a.NQ + kRowStatsTile - 1) / kRowStatsTile;
  const long long tiles = rowstats_tiles(a.BH, a.NQ);
  int* fold = reinterpret_cast<int*>(stats + (size_t)tiles * 4 * kRowStatsTile);
  const dim3 grid((unsigned)((tiles + kRowStatsTilesPerBlock - 1) / kRowStatsTilesPerBlock));
  hipLaunchKernelGGL(kl_bwd_rowstats_kernel, grid, dim3(kRowStatsTile * kRowStatsTilesPerBlock), 0, a.stream,
                     a.kl, a.lse_a, a.lse_b, a.g, a.NQ, ntq, tiles, stats, fold);
  a.pstats = stats;
  a.pfold = fold;
  return hipGetLastError();
}

}  // namespace streamkl
