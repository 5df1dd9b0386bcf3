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

constexpr int kVersion = 2;
constexpr int kFwdQB = 1;             // 32-query blocks per wave in the forward kernel
constexpr int kComputeUnits = 256;    // MI355X
constexpr int kLdsPerCu = 160 * 1024; // gfx950
constexpr int kMaxParts = 1 << 20;    // decode parts per call

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

// Decode workspace: o_part [P, 2, G, D] fp32, then lse_part [P, 2, G]
// fp32 at a 256-byte aligned offset.
struct DecLayout {
  int parts;
  size_t o_bytes, lse_off, total;
};

// ring-slot variant (16-byte Q chunks per 1 KB load) of a head dim and group
int dec_qblocks(int D, int G) {
  const int rows_per_kb = 512 / D;
  const int need = (G + rows_per_kb - 1) / rows_per_kb;
  return need <= 1 ? 1 : (need <= 2 ? 2 : 4);
}

int dec_lds_bytes(int D, int G) {
  return 3 * (2 * mk::kDecStageKeys * D * 2 + dec_qblocks(D, G) * 1024);
}

int dec_default_parts(int D, int G) {
  const int per_cu = kLdsPerCu / dec_lds_bytes(D, G);
  return kComputeUnits * (per_cu < 1 ? 1 : per_cu);
}

bool dec_layout(int Hq, int Hkv, int D, int n_parts, DecLayout* out) {
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || (D != 64 && D != 128)) return false;
  if (n_parts < 0 || n_parts > kMaxParts) return false;
  const int G = Hq / Hkv;
  if (G > 16) return false;
  DecLayout l;
  l.parts = n_parts == 0 ? dec_default_parts(D, G) : n_parts;
  l.o_bytes = (size_t)l.parts * 2 * G * D * sizeof(float);
  l.lse_off = round_up(l.o_bytes, 256);
  l.total = l.lse_off + round_up((size_t)l.parts * 2 * G * sizeof(float), 256);
  *out = l;
  return true;
}

template <int D, int QB>
void launch_dec(const mk::DecArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((mk::dec_part_kernel<D, QB>), dim3(a.P), dim3(64), 0, st, a);
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

size_t mk_attn_decode_workspace_bytes(int Hq, int Hkv, int D, int n_parts) {
  DecLayout l;
  if (!dec_layout(Hq, Hkv, D, n_parts, &l)) return 0;
  return l.total;
}

int mk_attn_decode_default_parts(int Hq, int Hkv, int D) {
  DecLayout l;
  if (!dec_layout(Hq, Hkv, D, 0, &l)) return 0;
  return l.parts;
}

int mk_attn_decode(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                   int B, int Hq, int Hkv, int Smax, int D, float scale, const int* kv_seqlens,
                   int n_parts, void* workspace, size_t workspace_bytes, void* stream) {
  if (!q || !k_cache || !v_cache || !o || !kv_seqlens) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || Smax < 1 || D < 1) return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  // stage indices and (batch, head) rows are 32-bit in the kernels
  const long long max_stages = (long long)B * Hkv * ((Smax + mk::kDecStageKeys - 1) /
                                                     mk::kDecStageKeys);
  if ((long long)B * Hq > 0x7fffffffLL || max_stages > 0x7fffffffLL) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (Hq / Hkv > 16) return MK_ERR_UNSUPPORTED;
  if (n_parts < 0 || n_parts > kMaxParts) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(o, 16) ||
      !aligned(kv_seqlens, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  DecLayout l;
  if (!dec_layout(Hq, Hkv, D, n_parts, &l)) return MK_ERR_SHAPE;
  if (!workspace || workspace_bytes < l.total) return MK_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MK_ERR_ALIGN;

  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  mk::DecArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.kc = static_cast<const uint16_t*>(k_cache);
  a.vc = static_cast<const uint16_t*>(v_cache);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.o_part = reinterpret_cast<float*>(ws);
  a.lse_part = reinterpret_cast<float*>(ws + l.lse_off);
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Smax = Smax;
  a.P = l.parts;
  a.scale_log2 = scale * mk::kLog2e;
  const int qb = dec_qblocks(D, Hq / Hkv);
  if (D == 128) {
    if (qb == 1) launch_dec<128, 1>(a, st);
    else if (qb == 2) launch_dec<128, 2>(a, st);
    else launch_dec<128, 4>(a, st);
  } else {
    if (qb == 1) launch_dec<64, 1>(a, st);
    else launch_dec<64, 2>(a, st);
  }
  if (hipGetLastError() != hipSuccess) return MK_ERR_HIP;
  const unsigned mblocks = (unsigned)(((long long)B * Hq + 3) / 4);  // one wave per row
  if (D == 128)
    hipLaunchKernelGGL(mk::dec_merge_kernel<128>, dim3(mblocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(mk::dec_merge_kernel<64>, dim3(mblocks), dim3(256), 0, st, a);
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
    case MK_ERR_ARG: return "MK_ERR_ARG: non-finite scale, bad causal flag or part count";
    default: return "MK_ERR_UNKNOWN: not an mk_status value";
  }
}

int mk_attn_version(void) { return kVersion; }

}  // extern "C"
