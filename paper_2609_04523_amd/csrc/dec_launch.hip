// dec_launch.hip -- instantiations and launcher of the decode kernels.
#include "launch.hpp"

namespace mk {
namespace {

template <int D, int QB, bool PAGED>
void part(const DecArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((dec_part_kernel<D, QB, PAGED>), dim3(a.P), dim3(64), 0, st, a);
}

template <bool PAGED>
void parts(const DecArgs& a, int D, int qb, hipStream_t st) {
  if (D == 128) {
    if (qb == 1) part<128, 1, PAGED>(a, st);
    else if (qb == 2) part<128, 2, PAGED>(a, st);
    else part<128, 4, PAGED>(a, st);
  } else {
    if (qb == 1) part<64, 1, PAGED>(a, st);
    else part<64, 2, PAGED>(a, st);
  }
}

}  // namespace

hipError_t launch_decode(const DecArgs& a, int D, int qblocks, bool paged, hipStream_t st) {
  if (paged)
    parts<true>(a, D, qblocks, st);
  else
    parts<false>(a, D, qblocks, st);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned mblocks = (unsigned)((a.P + 3) / 4);  // one wave per part
  if (D == 128)
    hipLaunchKernelGGL(dec_close_kernel<128>, dim3(mblocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(dec_close_kernel<64>, dim3(mblocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace mk
