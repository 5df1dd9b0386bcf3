// mk_attn.hip -- host side of the C ABI declared in include/mk_attn.h.
//
// Validates arguments on the host, picks the kernel instantiation
// (head dim, causal flag, output type) and enqueues on the caller's
// stream.  No allocation, no synchronisation, no global mutable state.
#include <math.h>
#include <stdint.h>

#include "../../include/mk_attn.h"
#include "decode_kernel.hpp"
#include "fwd_kernel.hpp"

namespace {

constexpr int kVersion = 1;
constexpr int kFwdQB = 1;             // 32-query blocks per wave in the forward kernel
constexpr int kDefaultSplit = 384;    // decode keys per split (not a power of two: see decode_kernel.hpp)

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

template <int D, bool CAUSAL, bool OUT_F32, bool POS>
hipError_t launch_fwd(const mk::FwdArgs& a, unsigned nblocks, hipStream_t st) {
  hipLaunchKernelGGL((mk::fwd_kernel<D, CAUSAL, OUT_F32, kFwdQB, POS>), dim3(nblocks),
                     dim3(mk::FwdShape<D, kFwdQB>::THREADS), 0, st, a);
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool OUT_F32>
hipError_t launch_fwd_s(const mk::FwdArgs& a, unsigned nblocks, bool pos, hipStream_t st) {
  return pos ? launch_fwd<D, CAUSAL, OUT_F32, true>(a, nblocks, st)
             : launch_fwd<D, CAUSAL, OUT_F32, false>(a, nblocks, st);
}

template <int D>
hipError_t launch_fwd_d(const mk::FwdArgs& a, unsigned nblocks, bool causal, bool out_f32,
                        bool pos, hipStream_t st) {
  if (causal)
    return out_f32 ? launch_fwd_s<D, true, true>(a, nblocks, pos, st)
                   : launch_fwd_s<D, true, false>(a, nblocks, pos, st);
  return out_f32 ? launch_fwd_s<D, false, true>(a, nblocks, pos, st)
                 : launch_fwd_s<D, false, false>(a, nblocks, pos, st);
}

int fwd_impl(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int Sq, int Skv, int D, int causal, float scale, const int* kv_seqlens,
             void* stream, bool out_f32) {
  if (!q || !k || !v || !o) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Skv < 1 || D < 1) return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (causal != 0 && causal != 1) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  if (kv_seqlens && !aligned(kv_seqlens, 4)) return MK_ERR_ALIGN;
  const int BM = mk::FwdShape<128, kFwdQB>::BM;  // same for both head dims
  const long long n_qtiles = (Sq + BM - 1) / BM;
  const long long nblocks = n_qtiles * B * Hq;
  if (nblocks > 0x7fffffffLL) return MK_ERR_SHAPE;

  mk::FwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = o;
  a.lse = lse;
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Sq = Sq;
  a.Skv = Skv;
  a.n_qtiles = (int)n_qtiles;
  a.xcd_groups = ((B * Hkv) % 8 == 0) ? 1 : 0;
  a.scale_log2 = scale * mk::kLog2e;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool pos = scale > 0.f;
  hipError_t e = (D == 128) ? launch_fwd_d<128>(a, (unsigned)nblocks, causal, out_f32, pos, st)
                            : launch_fwd_d<64>(a, (unsigned)nblocks, causal, out_f32, pos, st);
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

struct DecLayout {
  int split, nsplit;
  size_t o_bytes, lse_off, total;
};

bool dec_layout(int B, int Hq, int Smax, int D, int split, DecLayout* out) {
  if (B < 1 || Hq < 1 || Smax < 1 || D < 1 || split < 0) return false;
  if (split == 0) split = kDefaultSplit;
  DecLayout l;
  l.split = split;
  l.nsplit = (Smax + split - 1) / split;
  l.o_bytes = (size_t)B * Hq * l.nsplit * D * sizeof(float);
  l.lse_off = round_up(l.o_bytes, 256);
  l.total = l.lse_off + round_up((size_t)B * Hq * l.nsplit * sizeof(float), 256);
  *out = l;
  return true;
}

}  // namespace

extern "C" {

int mk_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int Sq, int Skv, int D, int causal, float scale, const int* kv_seqlens,
                void* stream) {
  return fwd_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream,
                  false);
}

int mk_attn_fwd_o32(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                    int Hq, int Hkv, int Sq, int Skv, int D, int causal, float scale,
                    const int* kv_seqlens, void* stream) {
  return fwd_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream,
                  true);
}

size_t mk_attn_decode_workspace_bytes(int B, int Hq, int Smax, int D, int split) {
  DecLayout l;
  if (!dec_layout(B, Hq, Smax, D, split, &l)) return 0;
  return l.total;
}

int mk_attn_decode_default_split(void) { return kDefaultSplit; }

int mk_attn_decode(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                   int B, int Hq, int Hkv, int Smax, int D, float scale, const int* kv_seqlens,
                   int split, void* workspace, size_t workspace_bytes, void* stream) {
  if (!q || !k_cache || !v_cache || !o || !kv_seqlens) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || Smax < 1 || D < 1) return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (Hq / Hkv > 16) return MK_ERR_UNSUPPORTED;
  if (split < 0) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(o, 16) ||
      !aligned(kv_seqlens, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  DecLayout l;
  if (!dec_layout(B, Hq, Smax, D, split, &l)) return MK_ERR_SHAPE;
  if (!workspace || workspace_bytes < l.total) return MK_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MK_ERR_ALIGN;

  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  mk::DecArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.kc = static_cast<const uint16_t*>(k_cache);
  a.vc = static_cast<const uint16_t*>(v_cache);
  a.o_part = reinterpret_cast<float*>(ws);
  a.lse_part = reinterpret_cast<float*>(ws + l.lse_off);
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Smax = Smax;
  a.split = l.split;
  a.nsplit = l.nsplit;
  a.scale_log2 = scale * mk::kLog2e;
  const long long n_items = (long long)l.nsplit * Hkv * B;
  if (n_items > 0x7fffffffLL) return MK_ERR_SHAPE;
  const dim3 grid((unsigned)n_items);
  if (D == 128)
    hipLaunchKernelGGL(mk::dec_split_kernel<128>, grid, dim3(64), 0, st, a);
  else
    hipLaunchKernelGGL(mk::dec_split_kernel<64>, grid, dim3(64), 0, st, a);
  if (hipGetLastError() != hipSuccess) return MK_ERR_HIP;

  mk::CombArgs c;
  c.o_part = a.o_part;
  c.lse_part = a.lse_part;
  c.kv_seqlens = kv_seqlens;
  c.o = o;
  c.lse = lse;
  c.B = B;
  c.Hq = Hq;
  c.Smax = Smax;
  c.split = l.split;
  c.nsplit = l.nsplit;
  const unsigned cblocks = (unsigned)((B * Hq + 3) / 4);
  if (D == 128)
    hipLaunchKernelGGL(mk::dec_combine_kernel<128>, dim3(cblocks), dim3(256), 0, st, c);
  else
    hipLaunchKernelGGL(mk::dec_combine_kernel<64>, dim3(cblocks), dim3(256), 0, st, c);
  return hipGetLastError() == hipSuccess ? MK_OK : MK_ERR_HIP;
}

const char* mk_status_str(int status) {
  switch (status) {
    case MK_OK: return "MK_OK";
    case MK_ERR_NULL: return "MK_ERR_NULL: a required pointer is NULL";
    case MK_ERR_SHAPE: return "MK_ERR_SHAPE: invalid or too large sizes, or Hq % Hkv != 0";
    case MK_ERR_UNSUPPORTED: return "MK_ERR_UNSUPPORTED: head dim or group size not built";
    case MK_ERR_ALIGN: return "MK_ERR_ALIGN: a pointer is not aligned as required";
    case MK_ERR_WORKSPACE: return "MK_ERR_WORKSPACE: decode workspace missing or too small";
    case MK_ERR_HIP: return "MK_ERR_HIP: the HIP runtime refused a launch";
    case MK_ERR_ARG: return "MK_ERR_ARG: non-finite scale, bad causal flag or split";
    default: return "MK_ERR_UNKNOWN: not an mk_status value";
  }
}

int mk_attn_version(void) { return kVersion; }

}  // extern "C"
