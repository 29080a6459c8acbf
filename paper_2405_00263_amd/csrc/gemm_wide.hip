// Plans and launches of the matrix-core GEMM for hundreds of rows (kernel: gemm_wide.h).  This
// file is built with the VGPR form of the matrix-core instructions: its shapes keep their
// accumulators in the ordinary vector registers (the other form moved them between register
// files inside the loop).
#include "gemm_wide.h"

namespace clover {

bool plan_wide(int M, int ntiles, int nchunks, int mode, int max_splits, const int* seg_tiles, int nseg,
               GemmPlan& out) {
  if (M < WIDE_MIN_M || ntiles < 2 || ntiles % 2) return false;
  for (int s = 0; s < nseg; ++s)
    if (seg_tiles && seg_tiles[s] % 2) return false;  // tile pairs never straddle a segment
  if (mode == EP_QKV) {
    if (ntiles % (4 * kWideQkv.nb)) return false;
    out = make_wide(kWideQkv, M, ntiles, nchunks, 1);
    return true;
  }
  if (mode == EP_SWIGLU) {
    // 256-row workgroups (each weight tile read by two at 512 rows) while one round of
    // workgroups covers the grid; gate and up segments of equal length
    if (nseg != 2 || !seg_tiles || seg_tiles[0] != seg_tiles[1]) return false;
    const GemmPlan pl = make_wide(kWideSwiglu, M, ntiles, nchunks, 1);
    if ((long)pl.ngroups * pl.mchunks > WIDE_N_CU) return false;
    out = pl;
    return true;
  }
  if (mode != EP_PARTIAL) return false;
  // split-K projections whose unsplit grid covers at most half the compute units (the 7B
  // output and down projections at 512 rows: 4 splits)
  const GemmPlan one = make_wide(kWidePartial, M, ntiles, nchunks, 1);
  if ((long)one.ngroups * one.mchunks * 2 > WIDE_N_CU) return false;
  GemmPlan pl = one;
  for (int S = 2; S <= max_splits && (long)pl.ngroups * pl.mchunks * pl.S < WIDE_N_CU; ++S) {
    if ((nchunks + S - 1) / S < 8) break;  // keep each split several chunks long
    const GemmPlan q = make_wide(kWidePartial, M, ntiles, nchunks, S);
    if (q.S == S) pl = q;
  }
  out = pl;
  return true;
}

hipError_t launch_wide(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt) {
  if (p.mode == EP_SWIGLU) return launch_wide_acc(p, pl, st, lt);
  if (p.amax_part || (p.mode != EP_PARTIAL && p.mode != EP_QKV)) return hipErrorInvalidValue;
  if (p.mode == EP_QKV && pl.S != 1) return hipErrorInvalidValue;
  if (p.mode == EP_PARTIAL && !p.part) return hipErrorInvalidValue;
  const bool qkv = p.mode == EP_QKV;
  if (pl.mt == 2 && pl.tw == 3 && pl.ring == 4)
    return qkv ? launch_wide_shape<2, 3, 4, EP_QKV>(pl, p, st, lt) : launch_wide_shape<2, 3, 4, EP_PARTIAL>(pl, p, st, lt);
  if (pl.mt == 2 && pl.tw == 4 && pl.ring == 4)
    return qkv ? launch_wide_shape<2, 4, 4, EP_QKV>(pl, p, st, lt) : launch_wide_shape<2, 4, 4, EP_PARTIAL>(pl, p, st, lt);
  return hipErrorInvalidValue;
}

}  // namespace clover
