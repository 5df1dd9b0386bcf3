// launch.hpp -- host launchers of the kernel families, each in translation
// units of its own (fwd_launch_d128.hip, fwd_launch_d64.hip,
// fwd_varlen_launch.hip, fwd_vt_launch.hip, dec_launch.hip, bwd_launch.hip, mla_launch.hip) so that the library compiles in
// parallel.  Arguments are validated by the callers in mk_attn.hip; these
// only pick the instantiation and enqueue.
#pragma once

#include <hip/hip_runtime.h>

#include "bwd_kernel.hpp"
#include "decode_kernel.hpp"
#include "fwd_kernel.hpp"

namespace mk {

constexpr int kFwdQB = 1;     // 32-query blocks per wave in the forward kernel
constexpr int kFwdWaves = 4;  // waves per forward workgroup (128 query rows)
// waves per workgroup of the V^T forward (256 query rows sharing each K/V
// tile, one workgroup per compute unit)
constexpr int kFwdVtWaves = 8;

// Dense [B, H, S, D] forward: nblocks workgroups of the forward kernel.
hipError_t launch_fwd(const FwdArgs& a, unsigned nblocks, int D, bool causal, bool out_f32,
                      bool pos_scale, hipStream_t st);

// Dense forward through a V^T copy (bf16 O): the pack kernel writes
// a.vt (pack_blocks = B * Hkv * vt_tiles workgroups) and sets a.ctr's
// a.n_queues counters to nblocks / a.n_queues, then the forward (nblocks
// persistent workgroups of kFwdVtWaves waves, a multiple of a.n_queues and
// at most a.n_queues * a.per_queue) reads V from it.
hipError_t launch_fwd_vt(const FwdArgs& a, unsigned nblocks, int D, bool causal, bool pos_scale,
                         unsigned pack_blocks, hipStream_t st);

// Packed ragged forward (bf16 O).
hipError_t launch_fwd_varlen(const FwdArgs& a, unsigned nblocks, int D, bool causal,
                             bool pos_scale, hipStream_t st);

// Packed queries over a paged cache (bf16 O).
hipError_t launch_fwd_ragged_paged(const FwdArgs& a, unsigned nblocks, int D, bool causal,
                                   bool pos_scale, hipStream_t st);

// Decode: the part kernel (contiguous or paged cache) then the merge kernel.
hipError_t launch_decode(const DecArgs& a, int D, int qblocks, bool paged, hipStream_t st);

// Backward: the dQ kernel (it also writes the rows' D and LSE log2 e),
// then the dK/dV kernel (skipped when dkdv_blocks is 0).
hipError_t launch_bwd(const BwdArgs& a, unsigned dq_blocks, unsigned dkdv_blocks, int D,
                      bool causal, hipStream_t st);

// MLA decode (q [B, 16, 576], latent cache [B, Smax, 576] in kc, O
// [B, 16, 512]): the part kernel, then the merge kernel.
hipError_t launch_mla_decode(const DecArgs& a, hipStream_t st);

}  // namespace mk
