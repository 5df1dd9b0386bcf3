// bwd_launch.hip -- instantiations and launcher of the backward kernels:
// the dQ kernel (which also writes D and LSE log2 e per row), then the
// dK/dV kernel (which reads them).
#include "launch.hpp"

namespace mk {
namespace {

template <int D, bool CAUSAL>
hipError_t go(const BwdArgs& a, unsigned dq_blocks, unsigned dkdv_blocks, hipStream_t st) {
  hipLaunchKernelGGL((bwd_dq_kernel<D, CAUSAL>), dim3(dq_blocks), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || dkdv_blocks == 0) return e;
  hipLaunchKernelGGL((bwd_dkdv_kernel<D, CAUSAL>), dim3(dkdv_blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, unsigned dq_blocks, unsigned dkdv_blocks, int D,
                      bool causal, hipStream_t st) {
  if (D == 128)
    return causal ? go<128, true>(a, dq_blocks, dkdv_blocks, st)
                  : go<128, false>(a, dq_blocks, dkdv_blocks, st);
  return causal ? go<64, true>(a, dq_blocks, dkdv_blocks, st)
                : go<64, false>(a, dq_blocks, dkdv_blocks, st);
}

}  // namespace mk
