// fwd_launch_d64.hip -- dense forward launcher, head dim 64.
#include "fwd_launch.hpp"

namespace mk {

hipError_t launch_fwd_d64(const FwdArgs& a, unsigned nblocks, bool causal, bool out_f32,
                          bool pos_scale, hipStream_t st) {
  return fwd_detail::go_w<64, kFwdWaves>(a, nblocks, causal, out_f32, pos_scale, st);
}

}  // namespace mk
