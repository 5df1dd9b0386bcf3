// mk_attn.hip -- host side of the C ABI declared in include/mk_attn.h.
//
// Validates arguments on the host, picks the kernel instantiation
// (head dim, causal flag, output type) and enqueues on the caller's
// stream.  No allocation and no synchronisation.  The only state is the
// per-device address of the fixed decode scratch (set once per device).
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "../../include/mk_attn.h"
#include "launch.hpp"
#include "mla_kernel.hpp"

namespace {

constexpr int kVersion = 10;
constexpr int kComputeUnits = 256;    // MI355X
constexpr int kLdsPerCu = 160 * 1024; // gfx950
constexpr int kMaxParts = 1 << 20;    // decode parts per call

// Scratch of the allocation-free decode entry point: a fixed device array,
// one copy on every GPU the library runs on, held until the process ends.
// Host code must never pass `scratch` itself to a kernel (on the host the
// name stands for a host-side shadow, not a device address): its device
// address is looked up once per device and kept in scratch_ptr.
constexpr size_t kScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
void* scratch_ptr[kMaxDevices];
hipError_t scratch_err[kMaxDevices];
std::once_flag scratch_once[kMaxDevices];

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace of mk_attn_fwd_ws: the V^T tiles, ceil(Skv / 64) tiles of
// 64 * D bf16 per (b, kv head), then the persistent forward's work-item
// counters (one per queue, 128 bytes apart).
constexpr size_t kFwdCtrBytes = 8 * 128;

size_t fwd_vt_tile_bytes(int B, int Hkv, int Skv, int D) {
  return (size_t)B * Hkv * (size_t)((Skv + 63) / 64) * 64 * D * 2;
}

size_t fwd_vt_bytes(int B, int Hkv, int Skv, int D) {
  if (B < 1 || Hkv < 1 || Skv < 1 || (D != 64 && D != 128)) return 0;
  return fwd_vt_tile_bytes(B, Hkv, Skv, D) + kFwdCtrBytes;
}

// vt: V^T workspace of mk_attn_fwd_ws (bf16 O), or null for the transposing path
int fwd_impl(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int Sq, int Skv, int D, int causal, float scale, const int* kv_seqlens,
             void* stream, bool out_f32, void* vt = nullptr) {
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
  const int BM = mk::FwdShape<128, mk::kFwdQB, mk::kFwdWaves>::BM;  // same for both head dims
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
  a.xcd_gp = ((B * Hkv) % 8 == 0) ? mk::xcd_group_pairs(Hq / Hkv, (int)n_qtiles) : 0;
  a.scale_log2 = scale * mk::kLog2e;
  a.cu_q = a.cu_k = nullptr;
  a.total_q = a.total_k = 0;
  a.block_table = nullptr;
  a.page_size = a.max_pages = a.n_pages = 0;
  a.ps_magic = 0;
  a.ps_shift = 0;
  a.tile_in_page = 0;
  a.vt = static_cast<const uint16_t*>(vt);
  a.vt_tiles = (Skv + 63) / 64;
  a.ctr = nullptr;
  a.n_queues = 1;
  a.per_queue = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool pos = scale > 0.f;
  if (vt) {
    // a persistent grid of kFwdVtWaves-wave workgroups, one per compute
    // unit, over per-XCD queues of work items (one queue when the K/V
    // heads do not divide evenly over the XCDs)
    const int BM_VT = mk::FwdShape<128, mk::kFwdQB, mk::kFwdVtWaves>::BM;
    const long long nq_vt = (Sq + BM_VT - 1) / BM_VT;
    a.n_qtiles = (int)nq_vt;
    // groups of two pairs: an XCD's queue then starts with the longest
    // q-tiles of both (its workgroups take items longest first)
    a.xcd_gp = ((B * Hkv) % 8 == 0) ? 2 : 0;
    const long long items = nq_vt * B * Hq;
    if (items > 0x7fffffffLL) return MK_ERR_SHAPE;
    a.n_queues = a.xcd_gp > 0 ? 8 : 1;
    a.per_queue = (int)(items / a.n_queues);
    const long long per_q_grid = std::min<long long>(a.per_queue, kComputeUnits / a.n_queues);
    a.ctr = reinterpret_cast<int*>(static_cast<char*>(vt) + fwd_vt_tile_bytes(B, Hkv, Skv, D));
    const long long pack_blocks = (long long)B * Hkv * a.vt_tiles;
    if (pack_blocks > 0x7fffffffLL) return MK_ERR_SHAPE;
    const hipError_t e = mk::launch_fwd_vt(a, (unsigned)(per_q_grid * a.n_queues), D, causal,
                                           pos, (unsigned)pack_blocks, st);
    return e == hipSuccess ? MK_OK : MK_ERR_HIP;
  }
  const hipError_t e = mk::launch_fwd(a, (unsigned)nblocks, D, causal, out_f32, pos, st);
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

// Decode workspace: o_part [P, 2, G, D] fp32, then lse_part [P, 2, G]
// fp32, then the parts' records of the cut pairs they close, int32 [P, 4],
// each region at a 256-byte aligned offset.
struct DecLayout {
  int parts;
  size_t o_bytes, lse_off, desc_off, total;
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
  l.desc_off = l.lse_off + round_up((size_t)l.parts * 2 * G * sizeof(float), 256);
  l.total = l.desc_off + round_up((size_t)l.parts * 4 * sizeof(int), 256);
  *out = l;
  return true;
}

// MLA decode workspace: o_part [P, 2, H, Dc] fp32, then lse_part [P, 2, H]
// at a 256-byte aligned offset; the default P is one part per compute unit
// (its four-wave workgroup holds 144 KB of LDS).
bool mla_layout(int H, int Dc, int n_parts, DecLayout* out) {
  if (H != mk::MlaShape::H || Dc != mk::MlaShape::DC) return false;
  if (n_parts < 0 || n_parts > kMaxParts) return false;
  DecLayout l;
  l.parts = n_parts == 0 ? kComputeUnits : n_parts;
  l.o_bytes = (size_t)l.parts * 2 * H * Dc * sizeof(float);
  l.lse_off = round_up(l.o_bytes, 256);
  l.desc_off = 0;  // the MLA merge needs no records
  l.total = l.lse_off + round_up((size_t)l.parts * 2 * H * sizeof(float), 256);
  *out = l;
  return true;
}

// Checks shared by both decode entry points (max_keys: keys a sequence can
// hold).
int dec_check(const void* q, const void* kc, const void* vc, const void* o, const float* lse,
              int B, int Hq, int Hkv, long long max_keys, int D, float scale,
              const int* kv_seqlens, int n_parts, const void* workspace, size_t workspace_bytes,
              DecLayout* l) {
  if (!q || !kc || !vc || !o || !kv_seqlens) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || max_keys < 1 || D < 1) return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  // stage indices, (batch, head) rows and key positions are 32-bit in the kernels
  const long long max_stages =
      (long long)B * Hkv * ((max_keys + mk::kDecStageKeys - 1) / mk::kDecStageKeys);
  if ((long long)B * Hq > 0x7fffffffLL || max_stages > 0x7fffffffLL || max_keys > 0x7fffffffLL)
    return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (Hq / Hkv > 16) return MK_ERR_UNSUPPORTED;
  if (n_parts < 0 || n_parts > kMaxParts) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(kc, 16) || !aligned(vc, 16) || !aligned(o, 16) ||
      !aligned(kv_seqlens, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  if (!dec_layout(Hq, Hkv, D, n_parts, l)) return MK_ERR_SHAPE;
  if (!workspace || workspace_bytes < l->total) return MK_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MK_ERR_ALIGN;
  return MK_OK;
}

mk::DecArgs dec_args(const void* q, const void* kc, const void* vc, void* o, float* lse, int B,
                     int Hq, int Hkv, int max_keys, float scale, const int* kv_seqlens,
                     const DecLayout& l, void* workspace) {
  char* ws = static_cast<char*>(workspace);
  mk::DecArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.kc = static_cast<const uint16_t*>(kc);
  a.vc = static_cast<const uint16_t*>(vc);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.o_part = reinterpret_cast<float*>(ws);
  a.lse_part = reinterpret_cast<float*>(ws + l.lse_off);
  a.close_desc = l.desc_off ? reinterpret_cast<int*>(ws + l.desc_off) : nullptr;
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Smax = max_keys;
  a.P = l.parts;
  a.scale_log2 = scale * mk::kLog2e;
  a.block_table = nullptr;
  a.page_size = a.max_pages = a.n_pages = 0;
  return a;
}

}  // namespace

extern "C" {

int mk_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int Sq, int Skv, int D, int causal, float scale, const int* kv_seqlens,
                void* stream) {
  return fwd_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream,
                  false);
}

int mk_attn_fwd_ws(const void* q, const void* k, const void* v, void* o, float* lse, int B,
                   int Hq, int Hkv, int Sq, int Skv, int D, int causal, float scale,
                   const int* kv_seqlens, void* workspace, size_t workspace_bytes,
                   void* stream) {
  if (!workspace) return MK_ERR_NULL;
  if (!aligned(workspace, 16)) return MK_ERR_ALIGN;
  const size_t need = fwd_vt_bytes(B, Hkv, Skv, D);
  if (need != 0 && workspace_bytes < need) return MK_ERR_ARG;
  return fwd_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream,
                  false, workspace);
}

size_t mk_attn_fwd_workspace_bytes(int B, int Hkv, int Skv, int D) {
  return fwd_vt_bytes(B, Hkv, Skv, D);
}

int mk_attn_fwd_o32(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                    int Hq, int Hkv, int Sq, int Skv, int D, int causal, float scale,
                    const int* kv_seqlens, void* stream) {
  return fwd_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Skv, D, causal, scale, kv_seqlens, stream,
                  true);
}

int mk_attn_fwd_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                       const int* cu_seqlens_q, const int* cu_seqlens_k, int B, int Hq,
                       int Hkv, int max_seqlen_q, int total_q, int total_k, int D, int causal,
                       float scale, void* stream) {
  if (!q || !k || !v || !o || !cu_seqlens_q || !cu_seqlens_k) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || max_seqlen_q < 1 || total_q < 1 || total_k < 1 || D < 1)
    return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (causal != 0 && causal != 1) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(cu_seqlens_q, 4) || !aligned(cu_seqlens_k, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  const int BM = mk::FwdShape<128, mk::kFwdQB, mk::kFwdWaves>::BM;
  const long long n_qtiles = (max_seqlen_q + BM - 1) / BM;
  const long long nblocks = n_qtiles * B * Hq;
  // workgroups of one launch; a key tile's rows (64 tokens of Hkv heads)
  // addressed with 32-bit offsets; B + 1 offsets per table
  if (nblocks > 0x7fffffffLL || (long long)Hkv * D * 2 * 64 > 0xffffffffLL || B > 0x7ffffffe)
    return MK_ERR_SHAPE;

  mk::FwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = o;
  a.lse = lse;
  a.kv_seqlens = nullptr;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Sq = max_seqlen_q;
  a.Skv = 0;
  a.n_qtiles = (int)n_qtiles;
  a.xcd_gp = 0;
  a.scale_log2 = scale * mk::kLog2e;
  a.cu_q = cu_seqlens_q;
  a.cu_k = cu_seqlens_k;
  a.total_q = total_q;
  a.total_k = total_k;
  a.block_table = nullptr;
  a.page_size = a.max_pages = a.n_pages = 0;
  a.ps_magic = 0;
  a.ps_shift = 0;
  a.tile_in_page = 0;
  a.vt = nullptr;
  a.vt_tiles = 0;
  a.ctr = nullptr;
  a.n_queues = 1;
  a.per_queue = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool pos = scale > 0.f;
  const hipError_t e = mk::launch_fwd_varlen(a, (unsigned)nblocks, D, causal, pos, st);
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

int mk_attn_fwd_ragged_paged(const void* q, const void* k_pages, const void* v_pages,
                             const int* block_table, void* o, float* lse,
                             const int* cu_seqlens_q, const int* kv_seqlens, int B, int Hq,
                             int Hkv, int max_seqlen_q, int total_q, int page_size,
                             int max_pages, int n_pages, int D, int causal, float scale,
                             void* stream) {
  if (!q || !k_pages || !v_pages || !block_table || !o || !cu_seqlens_q || !kv_seqlens)
    return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || max_seqlen_q < 1 || total_q < 1 || D < 1 ||
      page_size < 1 || max_pages < 1 || n_pages < 1)
    return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  // a wave's 1 KB block of a tile (4 or 8 key rows) must lie in one page
  if (page_size % 16 != 0) return MK_ERR_UNSUPPORTED;
  if (causal != 0 && causal != 1) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(o, 16) ||
      !aligned(cu_seqlens_q, 4) || !aligned(kv_seqlens, 4) || !aligned(block_table, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  const int BM = mk::FwdShape<128, mk::kFwdQB, mk::kFwdWaves>::BM;
  const long long n_qtiles = (max_seqlen_q + BM - 1) / BM;
  const long long nblocks = n_qtiles * B * Hq;
  // workgroups of one launch, key positions and table indices are 32-bit
  if (nblocks > 0x7fffffffLL || (long long)max_pages * page_size > 0x7fffffffLL ||
      (long long)B * max_pages > 0x7fffffffLL || B > 0x7ffffffe)
    return MK_ERR_SHAPE;

  mk::FwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_pages);
  a.v = static_cast<const uint16_t*>(v_pages);
  a.o = o;
  a.lse = lse;
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Sq = max_seqlen_q;
  a.Skv = 0;
  a.n_qtiles = (int)n_qtiles;
  a.xcd_gp = 0;
  a.scale_log2 = scale * mk::kLog2e;
  a.cu_q = cu_seqlens_q;
  a.cu_k = nullptr;
  a.total_q = total_q;
  a.total_k = 0;
  a.block_table = block_table;
  a.page_size = page_size;
  a.max_pages = max_pages;
  a.n_pages = n_pages;
  {
    int l = 0;  // ceil(log2 page_size)
    while ((1LL << l) < page_size) ++l;
    a.ps_shift = 31 + l;
    a.ps_magic = ((uint64_t)1 << a.ps_shift) / (uint64_t)page_size + 1;
  }
  a.tile_in_page = page_size % 64 == 0 ? 1 : 0;
  a.vt = nullptr;
  a.vt_tiles = 0;
  a.ctr = nullptr;
  a.n_queues = 1;
  a.per_queue = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool pos = scale > 0.f;
  const hipError_t e = mk::launch_fwd_ragged_paged(a, (unsigned)nblocks, D, causal, pos, st);
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

size_t mk_attn_mla_decode_workspace_bytes(int H, int Dc, int n_parts) {
  DecLayout l;
  if (!mla_layout(H, Dc, n_parts, &l)) return 0;
  return l.total;
}

int mk_attn_mla_decode(const void* q, const void* ckv, void* o, float* lse, int B, int H,
                       int Dc, int Dr, int Smax, float scale, const int* kv_seqlens,
                       int n_parts, void* workspace, size_t workspace_bytes, void* stream) {
  using S = mk::MlaShape;
  if (!q || !ckv || !o || !kv_seqlens) return MK_ERR_NULL;
  if (B < 1 || H < 1 || Dc < 1 || Dr < 0 || Smax < 1) return MK_ERR_SHAPE;
  const long long max_stages = (long long)B * ((Smax + mk::kDecStageKeys - 1) / mk::kDecStageKeys);
  if ((long long)B * H > 0x7fffffffLL || max_stages > 0x7fffffffLL) return MK_ERR_SHAPE;
  if (H != S::H || Dc != S::DC || Dr != S::DR) return MK_ERR_UNSUPPORTED;
  if (n_parts < 0 || n_parts > kMaxParts) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(ckv, 16) || !aligned(o, 16) || !aligned(kv_seqlens, 4))
    return MK_ERR_ALIGN;
  if (lse && !aligned(lse, 4)) return MK_ERR_ALIGN;
  DecLayout l;
  if (!mla_layout(H, Dc, n_parts, &l)) return MK_ERR_SHAPE;
  if (!workspace || workspace_bytes < l.total) return MK_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MK_ERR_ALIGN;
  // the cache is one kv head of rows of Dc + Dr values; the merge works at
  // the latent width
  mk::DecArgs a = dec_args(q, ckv, ckv, o, lse, B, H, 1, Smax, scale, kv_seqlens, l, workspace);
  const hipError_t e = mk::launch_mla_decode(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
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
  DecLayout l;
  const int rc = dec_check(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, D, scale, kv_seqlens,
                           n_parts, workspace, workspace_bytes, &l);
  if (rc != MK_OK) return rc;
  const mk::DecArgs a =
      dec_args(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, scale, kv_seqlens, l, workspace);
  const hipError_t e = mk::launch_decode(a, D, dec_qblocks(D, Hq / Hkv), false,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

int mk_attn_decode_noalloc(const void* q, const void* k_cache, const void* v_cache, void* o,
                           float* lse, int B, int Hq, int Hkv, int Smax, int D, float scale,
                           const int* kv_seqlens, int n_parts, void* stream) {
  // validate as mk_attn_decode would with a workspace of the scratch's size
  // (a stand-in address: nothing is launched unless every check passes)
  DecLayout l;
  int rc = dec_check(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, D, scale, kv_seqlens,
                     n_parts, reinterpret_cast<void*>(uintptr_t{256}), kScratchBytes, &l);
  if (rc == MK_ERR_WORKSPACE) return MK_ERR_SCRATCH;
  if (rc != MK_OK) return rc;
  // the device the work runs on: the stream's, which must be the current one
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return MK_ERR_HIP;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (st) {
    int sdev = -1;
    if (hipStreamGetDevice(st, &sdev) != hipSuccess) return MK_ERR_HIP;
    if (sdev != dev) return MK_ERR_ARG;
  }
  if (dev >= kMaxDevices) return MK_ERR_UNSUPPORTED;
  std::call_once(scratch_once[dev], [dev] {
    void* p = nullptr;
    scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    scratch_ptr[dev] = p;
  });
  if (scratch_err[dev] != hipSuccess || scratch_ptr[dev] == nullptr) return MK_ERR_HIP;
  const mk::DecArgs a = dec_args(q, k_cache, v_cache, o, lse, B, Hq, Hkv, Smax, scale,
                                 kv_seqlens, l, scratch_ptr[dev]);
  const hipError_t e = mk::launch_decode(a, D, dec_qblocks(D, Hq / Hkv), false, st);
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

size_t mk_attn_decode_noalloc_max_bytes(void) { return kScratchBytes; }

int mk_attn_decode_paged(const void* q, const void* k_pages, const void* v_pages,
                         const int* block_table, void* o, float* lse, int B, int Hq, int Hkv,
                         int page_size, int max_pages, int n_pages, int D, float scale,
                         const int* kv_seqlens, int n_parts, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (!block_table) return MK_ERR_NULL;
  if (page_size < 16 || page_size % 16 != 0 || max_pages < 1 || n_pages < 1)
    return MK_ERR_SHAPE;
  if ((long long)B * max_pages > 0x7fffffffLL) return MK_ERR_SHAPE;
  const long long max_keys = (long long)max_pages * page_size;
  DecLayout l;
  const int rc = dec_check(q, k_pages, v_pages, o, lse, B, Hq, Hkv, max_keys, D, scale,
                           kv_seqlens, n_parts, workspace, workspace_bytes, &l);
  if (rc != MK_OK) return rc;
  if (!aligned(block_table, 4)) return MK_ERR_ALIGN;
  mk::DecArgs a = dec_args(q, k_pages, v_pages, o, lse, B, Hq, Hkv, (int)max_keys, scale,
                           kv_seqlens, l, workspace);
  a.block_table = block_table;
  a.page_size = page_size;
  a.max_pages = max_pages;
  a.n_pages = n_pages;
  const hipError_t e = mk::launch_decode(a, D, dec_qblocks(D, Hq / Hkv), true,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

// Backward workspace: D and LSE log2(e), each [B, Hq, Sq rounded up to
// 128] fp32, the second at a 256-byte aligned offset.
size_t bwd_array_bytes(int B, int Hq, int Sq) {
  return round_up((size_t)B * Hq * round_up((size_t)Sq, 128) * sizeof(float), 256);
}

size_t mk_attn_bwd_workspace_bytes(int B, int Hq, int Sq) {
  if (B < 1 || Hq < 1 || Sq < 1) return 0;
  return 2 * bwd_array_bytes(B, Hq, Sq);
}

int mk_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                const float* lse, void* dq, void* dk, void* dv, int B, int Hq, int Hkv, int Sq,
                int Skv, int D, int causal, float scale, const int* kv_seqlens, void* workspace,
                size_t workspace_bytes, void* stream) {
  if (!q || !k || !v || !o || !dout || !lse || !dq || !dk || !dv) return MK_ERR_NULL;
  if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Skv < 1 || D < 1) return MK_ERR_SHAPE;
  if (Hq % Hkv != 0) return MK_ERR_SHAPE;
  if (D != 64 && D != 128) return MK_ERR_UNSUPPORTED;
  if (causal != 0 && causal != 1) return MK_ERR_ARG;
  if (!isfinite(scale)) return MK_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(dout, 16) || !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16) ||
      !aligned(lse, 4))
    return MK_ERR_ALIGN;
  if (kv_seqlens && !aligned(kv_seqlens, 4)) return MK_ERR_ALIGN;
  // workgroups of each launch
  const long long sq_pad = (Sq + 127) / 128 * 128;
  const long long dq_blocks = (long long)((Sq + 127) / 128) * B * Hq;
  const long long dkdv_blocks = (long long)((Skv + 127) / 128) * B * Hkv;
  if (dq_blocks > 0x7fffffffLL || dkdv_blocks > 0x7fffffffLL) return MK_ERR_SHAPE;
  const size_t need = mk_attn_bwd_workspace_bytes(B, Hq, Sq);
  if (!workspace || workspace_bytes < need) return MK_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MK_ERR_ALIGN;

  mk::BwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<const uint16_t*>(o);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dq = static_cast<uint16_t*>(dq);
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.delta = static_cast<float*>(workspace);
  a.lse2 = reinterpret_cast<float*>(static_cast<char*>(workspace) + bwd_array_bytes(B, Hq, Sq));
  a.sq_pad = (int)sq_pad;
  a.kv_seqlens = kv_seqlens;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Sq = Sq;
  a.Skv = Skv;
  a.n_qtiles = (Sq + 127) / 128;
  a.xcd_gp = ((B * Hkv) % 8 == 0) ? mk::xcd_group_pairs(Hq / Hkv, a.n_qtiles) : 0;
  a.n_kblocks = (Skv + 127) / 128;
  a.scale = scale;
  a.scale_log2 = scale * mk::kLog2e;
  const hipError_t e =
      mk::launch_bwd(a, (unsigned)dq_blocks, (unsigned)dkdv_blocks, D, causal != 0,
                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MK_OK : MK_ERR_HIP;
}

const char* mk_status_str(int status) {
  switch (status) {
    case MK_OK: return "MK_OK";
    case MK_ERR_NULL: return "MK_ERR_NULL: a required pointer is NULL";
    case MK_ERR_SHAPE: return "MK_ERR_SHAPE: invalid or too large sizes, or Hq % Hkv != 0";
    case MK_ERR_UNSUPPORTED: return "MK_ERR_UNSUPPORTED: head dim or group size not built";
    case MK_ERR_ALIGN: return "MK_ERR_ALIGN: a pointer is not aligned as required";
    case MK_ERR_WORKSPACE: return "MK_ERR_WORKSPACE: workspace missing or too small";
    case MK_ERR_HIP: return "MK_ERR_HIP: the HIP runtime refused a launch";
    case MK_ERR_ARG: return "MK_ERR_ARG: non-finite scale, bad causal flag or part count";
    case MK_ERR_SCRATCH:
      return "MK_ERR_SCRATCH: the request needs more decode scratch than the "
             "allocation-free entry point holds (use mk_attn_decode with a workspace)";
    default: return "MK_ERR_UNKNOWN: not an mk_status value";
  }
}

int mk_attn_version(void) { return kVersion; }

}  // extern "C"
