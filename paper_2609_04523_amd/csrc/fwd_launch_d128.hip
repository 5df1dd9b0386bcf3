// fwd_launch_d128.hip -- dense forward launcher, head dim 128, and the
// head-dim dispatch.
#include "fwd_launch.hpp"

namespace mk {

hipError_t launch_fwd_d64(const FwdArgs& a, unsigned nblocks, bool causal, bool out_f32,
                          bool pos_scale, hipStream_t st);

hipError_t launch_fwd(const FwdArgs& a, unsigned nblocks, int D, bool causal, bool out_f32,
                      bool pos_scale, hipStream_t st) {
  if (D == 128) return fwd_detail::go_w<128, kFwdWaves>(a, nblocks, causal, out_f32, pos_scale, st);
  return launch_fwd_d64(a, nblocks, causal, out_f32, pos_scale, st);
}

}  // namespace mk
