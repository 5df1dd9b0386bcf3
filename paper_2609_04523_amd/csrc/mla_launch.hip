// mla_launch.hip -- launcher of the MLA decode: the part kernel, then the
// decode merge kernel at the latent width.
#include "launch.hpp"
#include "mla_kernel.hpp"

namespace mk {

hipError_t launch_mla_decode(const DecArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(mla_part_kernel<MlaShape::H>, dim3(a.P), dim3(256), 0, st, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned mblocks = (unsigned)(((long long)a.B * a.Hq + 3) / 4);  // one wave per row
  hipLaunchKernelGGL(dec_merge_kernel<MlaShape::DC>, dim3(mblocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace mk
