// bwd_launch.hip -- instantiations and launcher of the backward kernels:
// the row-delta kernel, then the dK/dV and dQ kernels (both read D).
#include "launch.hpp"

namespace mk {
namespace {

template <int D, bool CAUSAL>
hipError_t go(const BwdArgs& a, unsigned delta_blocks, unsigned dq_blocks, unsigned dkdv_blocks,
              hipStream_t st) {
  hipLaunchKernelGGL((bwd_delta_kernel<D>), dim3(delta_blocks), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (dkdv_blocks > 0) {
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, CAUSAL>), dim3(dkdv_blocks), dim3(256), 0, st, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((bwd_dq_kernel<D, CAUSAL>), dim3(dq_blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, unsigned delta_blocks, unsigned dq_blocks,
                      unsigned dkdv_blocks, int D, bool causal, hipStream_t st) {
  if (D == 128)
    return causal ? go<128, true>(a, delta_blocks, dq_blocks, dkdv_blocks, st)
                  : go<128, false>(a, delta_blocks, dq_blocks, dkdv_blocks, st);
  return causal ? go<64, true>(a, delta_blocks, dq_blocks, dkdv_blocks, st)
                : go<64, false>(a, delta_blocks, dq_blocks, dkdv_blocks, st);
}

}  // namespace mk
