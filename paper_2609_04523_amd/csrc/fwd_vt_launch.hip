// fwd_vt_launch.hip -- the V^T pre-pass and the dense forward's VT
// instantiations (bf16 O, persistent grid).
#include "launch.hpp"
#include "vt_pack_kernel.hpp"

namespace mk {
namespace {

template <int D, bool CAUSAL, bool POS>
hipError_t go_vt(const FwdArgs& a, unsigned nblocks, hipStream_t st) {
  hipLaunchKernelGGL((fwd_kernel<D, CAUSAL, false, kFwdQB, POS, false, kFwdVtWaves, false, true, true>),
                     dim3(nblocks), dim3(FwdShape<D, kFwdQB, kFwdVtWaves>::THREADS), 0, st, a);
  return hipGetLastError();
}

template <int D>
hipError_t go_vt_d(const FwdArgs& a, unsigned nblocks, bool causal, bool pos, hipStream_t st) {
  if (causal) return pos ? go_vt<D, true, true>(a, nblocks, st) : go_vt<D, true, false>(a, nblocks, st);
  return pos ? go_vt<D, false, true>(a, nblocks, st) : go_vt<D, false, false>(a, nblocks, st);
}

}  // namespace

hipError_t launch_fwd_vt(const FwdArgs& a, unsigned nblocks, int D, bool causal, bool pos_scale,
                         unsigned pack_blocks, hipStream_t st) {
  VtPackArgs p;
  p.v = a.v;
  p.vt = const_cast<uint16_t*>(a.vt);
  p.kv_seqlens = a.kv_seqlens;
  p.Skv = a.Skv;
  p.vt_tiles = a.vt_tiles;
  p.Hkv = a.Hkv;
  p.ctr = a.ctr;
  p.ctr_init = (int)(nblocks / (unsigned)a.n_queues);
  p.n_queues = a.n_queues;
  if (D == 128)
    hipLaunchKernelGGL(vt_pack_kernel<128>, dim3(pack_blocks), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(vt_pack_kernel<64>, dim3(pack_blocks), dim3(256), 0, st, p);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return D == 128 ? go_vt_d<128>(a, nblocks, causal, pos_scale, st)
                  : go_vt_d<64>(a, nblocks, causal, pos_scale, st);
}

}  // namespace mk
