// The fp64-contraction variants of the large-D matrix-core kernel
// (mfma_kernel<..., F64 = true> of k_mfma_kernel.h): sums, log-sum-exps and
// min / max with T formed on v_mfma_f64_16x16x4_f64 from fp64 operands and
// norms.  They run when the accuracy guard (SpreadGuard) finds the fp32
// expanded form's error bound above its budget, and always for the Laplacian
// forms and the squared distance's sums and extremes; launched beside the
// fp32 (or split bf16) kernel, exactly one of the two does the work.  Its own
// translation unit, so that it compiles beside k_mfma.hip.
#include "k_mfma_kernel.h"

namespace kred {
namespace {

// fp64 operands take twice the registers: one row block per wave from D = 128
template <int Q>
constexpr int rows_blocks64() { return Q >= 32 ? 1 : 2; }

template <int Q, int EPI, bool SP>
hipError_t launch_sum64(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  constexpr int RB = rows_blocks64<Q>();
  switch (a.EB) {
    case 1: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 1, 1, SP, true>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 2, 1, SP, true>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 4, 1, SP, true>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int Q, bool SP>
hipError_t launch_q64(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  constexpr int RB = rows_blocks64<Q>();
  switch (a.epi) {
    case 0: return launch_sum64<Q, 0, SP>(a, grid, s);
    case 1: return launch_sum64<Q, 1, SP>(a, grid, s);
    case 2: return launch_sum64<Q, 2, SP>(a, grid, s);
#define KRED_ONE64(EPV)                                                                        \
  case EPV:                                                                                    \
    hipLaunchKernelGGL((mfma_kernel<Q, RB, EPV, 1, 1, SP, true>), grid, dim3(256), 0, s, a);  \
    return hipGetLastError();
    KRED_ONE64(4) KRED_ONE64(5) KRED_ONE64(6) KRED_ONE64(7) KRED_ONE64(8) KRED_ONE64(9)
#undef KRED_ONE64
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

int mfma64_rows_per_block(int DP) { return 64 * (DP >= 128 ? 1 : 2); }

hipError_t launch_mfma64(const MfmaArgs& a, hipStream_t s) {
  const int rows = mfma64_rows_per_block(a.DP);
  const dim3 grid((unsigned)(mfma_row_groups(a, rows) * a.C));
  switch (a.DP) {
    case 32: return a.nr > 0 ? launch_q64<8, true>(a, grid, s) : launch_q64<8, false>(a, grid, s);
    case 64: return a.nr > 0 ? launch_q64<16, true>(a, grid, s) : launch_q64<16, false>(a, grid, s);
    case 128: return a.nr > 0 ? launch_q64<32, true>(a, grid, s) : launch_q64<32, false>(a, grid, s);
    case 256: return a.nr > 0 ? launch_q64<64, true>(a, grid, s) : launch_q64<64, false>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kred
