// fwd_launch.hpp -- the dense forward kernel's instantiations for one head
// dim; included by fwd_launch_d128.hip and fwd_launch_d64.hip.
#pragma once

#include "launch.hpp"

namespace mk {
namespace fwd_detail {

template <int D, bool CAUSAL, bool OUT_F32, bool POS, int WAVES>
hipError_t go(const FwdArgs& a, unsigned nblocks, hipStream_t st) {
  hipLaunchKernelGGL((fwd_kernel<D, CAUSAL, OUT_F32, kFwdQB, POS, false, WAVES>), dim3(nblocks),
                     dim3(FwdShape<D, kFwdQB, WAVES>::THREADS), 0, st, a);
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool OUT_F32, int WAVES>
hipError_t go_s(const FwdArgs& a, unsigned nblocks, bool pos, hipStream_t st) {
  return pos ? go<D, CAUSAL, OUT_F32, true, WAVES>(a, nblocks, st)
             : go<D, CAUSAL, OUT_F32, false, WAVES>(a, nblocks, st);
}

template <int D, int WAVES>
hipError_t go_w(const FwdArgs& a, unsigned nblocks, bool causal, bool out_f32, bool pos,
                hipStream_t st) {
  if (causal)
    return out_f32 ? go_s<D, true, true, WAVES>(a, nblocks, pos, st)
                   : go_s<D, true, false, WAVES>(a, nblocks, pos, st);
  return out_f32 ? go_s<D, false, true, WAVES>(a, nblocks, pos, st)
                 : go_s<D, false, false, WAVES>(a, nblocks, pos, st);
}



}  // namespace fwd_detail
}  // namespace mk
