// fwd_rpa_launch.hip -- instantiations and launcher of the forward kernel
// over packed ragged queries whose keys and values live in a paged cache
// (bf16 O).
#include "launch.hpp"

namespace mk {
namespace {

template <int D, bool CAUSAL, bool POS>
hipError_t go(const FwdArgs& a, unsigned nblocks, hipStream_t st) {
  hipLaunchKernelGGL((fwd_kernel<D, CAUSAL, false, kFwdQB, POS, true, kFwdWaves, true>),
                     dim3(nblocks), dim3(FwdShape<D, kFwdQB, kFwdWaves>::THREADS), 0, st, a);
  return hipGetLastError();
}

template <int D>
hipError_t go_d(const FwdArgs& a, unsigned nblocks, bool causal, bool pos, hipStream_t st) {
  if (causal) return pos ? go<D, true, true>(a, nblocks, st) : go<D, true, false>(a, nblocks, st);
  return pos ? go<D, false, true>(a, nblocks, st) : go<D, false, false>(a, nblocks, st);
}

}  // namespace

hipError_t launch_fwd_ragged_paged(const FwdArgs& a, unsigned nblocks, int D, bool causal,
                                   bool pos_scale, hipStream_t st) {
  return D == 128 ? go_d<128>(a, nblocks, causal, pos_scale, st)
                  : go_d<64>(a, nblocks, causal, pos_scale, st);
}

}  // namespace mk
