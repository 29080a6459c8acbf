// Launch of the 256-row SwiGLU shape of the matrix-core GEMM (kernel: gemm_wide.h).  Its 4 x 3
// accumulator blocks per wave (192 registers per lane) leave too few ordinary vector
// registers for the operands, so this file is built with the default form of the
// matrix-core instructions, which keeps accumulators in the accumulation registers.
#include "gemm_wide.h"

namespace clover {

hipError_t launch_wide_acc(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt) {
  if (p.mode != EP_SWIGLU || pl.S != 1 || !p.out_s || p.amax_part) return hipErrorInvalidValue;
  if (pl.mt == kWideSwiglu.mb && pl.tw == kWideSwiglu.nb && pl.ring == kWideSwiglu.nst)
    return launch_wide_shape<kWideSwiglu.mb, kWideSwiglu.nb, kWideSwiglu.nst, EP_SWIGLU>(pl, p, st, lt);
  return hipErrorInvalidValue;
}

}  // namespace clover
