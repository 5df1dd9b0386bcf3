// mk_common.hpp -- device helpers shared by the gfx950 attention kernels.
//
// Register layouts of the CDNA4 matrix instructions used here (wave64):
//
//  v_mfma_f32_32x32x16_bf16  D[32x32] += A[32x16] * B[16x32]
//    A: lane l holds A[row = l%32][k-group l/32, 8 values]
//    B: lane l holds B[k-group l/32, 8 values][col = l%32]
//    D: lane l, register r holds D[row = 8*(r/4) + 4*(l/32) + r%4][col = l%32]
//
//  v_mfma_f32_16x16x32_bf16  D[16x16] += A[16x32] * B[32x16]
//    A: lane l holds A[row = l%16][k-group l/16, 8 values]
//    B: lane l holds B[k-group l/16, 8 values][col = l%16]
//    D: lane l, register r holds D[row = 4*(l/16) + r][col = l%16]
//
// A and B name their k-groups identically, so which 8 of the contraction
// indices a lane's k-group stands for is free, provided A and B agree.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the transcendental unit (v_exp_f32); 2^-inf = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 b) { return __builtin_bit_cast(u32x4, b); }

// Eight fp32 -> eight bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 to_bf16x8(float a0, float a1, float a2, float a3,
                                            float a4, float a5, float a6, float a7) {
  f32x8 f = {a0, a1, a2, a3, a4, a5, a6, a7};
  return __builtin_convertvector(f, bf16x8);
}

// fp32 -> bf16 bits, round to nearest even.
__device__ __forceinline__ uint16_t to_bf16_bits(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(uint16_t, h);
}

// Reductions between lane l and lane l^32 (v_permlane32_swap) and between
// lane l and lane l^16 (v_permlane16_swap).  Both lanes of a pair receive
// the same bits.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// 16 bytes global -> LDS without passing through registers
// (global_load_lds_dwordx4).  `lds` must be the same for the whole wave:
// lane l's 16 bytes land at lds + 16 l.
__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(
      (const void __attribute__((address_space(1)))*)g,
      (void __attribute__((address_space(3)))*)lds, 16, 0, 0);
}
// Same, with the destination given as a 32-bit LDS address.  The address is
// turned into an LDS pointer directly: going through a generic pointer
// would map LDS address 0 to the null pointer's LDS image (0xffffffff).
__device__ __forceinline__ void load_lds16_at(const void* g, uint32_t lds_addr) {
  __builtin_amdgcn_global_load_lds(
      (const void __attribute__((address_space(1)))*)g,
      (void __attribute__((address_space(3)))*)(uintptr_t)lds_addr, 16, 0, 0);
}

// The same load through a buffer resource: a wave-uniform base covering
// `bytes` (kept in scalar registers) plus a 32-bit lane offset, so no 64-bit
// address arithmetic runs on the vector unit.  Offsets at or past `bytes`
// read zeros instead of leaving the range.
// `soff` is a wave-uniform byte offset added to every lane's (it lives in a
// scalar register, so per-block offsets need no vector register each).
__device__ __forceinline__ void load_lds16_buf(const char* base, uint32_t bytes, uint32_t voff,
                                               uint32_t lds_addr, uint32_t soff = 0) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, (int)bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      rs, (__attribute__((address_space(3))) void*)(uintptr_t)lds_addr, 16, voff, soff, 0, 0);
}

// Workgroup barrier without the memory fence of __syncthreads() (which
// waits for every load of the wave, LDS-DMA loads of later stages
// included).  For callers that have already waited for what other waves
// will read -- their own LDS-DMA loads by vmcnt, their LDS reads by lgkmcnt
// -- so that loads issued for later stages stay in flight across it.
__device__ __forceinline__ void barrier_no_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(N): wait until at most N vector-memory operations of this
// wave are outstanding (expcnt and lgkmcnt untouched).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Transposing LDS read (ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane i names 4 consecutive bf16 of row i/4, columns 4(i%4)..+3,
// of a 4 x 16 block; lane j receives column j of the block, rows 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr16(const void* lds) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4*)(lds));
}

// Same, with the address given as a 32-bit LDS address (turned into an LDS
// pointer directly, see load_lds16_at).
__device__ __forceinline__ bf16x4 lds_read_tr16_at(uint32_t lds_addr) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4*)(uintptr_t)lds_addr);
}
// 16-byte LDS read at a 32-bit LDS address.
__device__ __forceinline__ u32x4 lds_read_b128_at(uint32_t lds_addr) {
  return *(const __attribute__((address_space(3))) u32x4*)(uintptr_t)lds_addr;
}

// The same read issued as inline assembly, so that the compiler's wait
// insertion does not tie it to in-flight LDS-DMA loads of other buffers.
// The result is NOT ready on return: pass it through lds_wait4() before
// use.  (LDS operations the compiler does not know about only make its
// own lgkmcnt waits more conservative.)
__device__ __forceinline__ u32x2 lds_read_tr16_async(uint32_t lds_addr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(lds_addr) : "memory");
  return r;
}
// Same, with a compile-time byte offset folded into the instruction.
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr16_async_off(uint32_t lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field is 16 bits");
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "i"(OFF)
               : "memory");
  return r;
}
// 16-byte LDS read issued as inline assembly (same contract as the
// transposing read above: pass the result through a tied wait before use).
template <int OFF>
__device__ __forceinline__ u32x4 lds_read_b128_async_off(uint32_t lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field is 16 bits");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "i"(OFF) : "memory");
  return r;
}
// s_waitcnt lgkmcnt(0) that the given registers depend on.
__device__ __forceinline__ void lds_wait_b128x4(u32x4& a, u32x4& b, u32x4& c, u32x4& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) :: "memory");
}
__device__ __forceinline__ void lds_wait_b128x2(u32x4& a, u32x4& b) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b) :: "memory");
}

// s_waitcnt lgkmcnt(N) for LDS reads issued as inline assembly: wait until
// at most N of this wave's LDS operations are outstanding (LDS operations
// complete in order).  Pass each destination register that must be ready
// through lds_ready() after it: the empty statement redefines the register
// after the wait, so no use of it can be scheduled before the wait
// (volatile statements keep their order).
template <int N>
__device__ __forceinline__ void lds_wait_lgkm() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
template <class T>
__device__ __forceinline__ void lds_ready(T& x) {
  asm volatile("" : "+v"(x));
}

// s_waitcnt lgkmcnt(0) that the four given registers depend on, so no use
// of them can be scheduled before the wait.
__device__ __forceinline__ void lds_wait4(u32x2& a, u32x2& b, u32x2& c, u32x2& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) :: "memory");
}

// 32-bit LDS address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) void*)p);
}

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// XOR swizzle of the 16-byte chunks of a K or V tile row in LDS (rows of
// D bf16 = D/8 chunks).  Row r's logical chunk c sits at physical chunk
// c ^ swz(r).  Sixteen consecutive rows read at one logical chunk hit
// sixteen different chunk positions (D = 128), and the transposing read's
// four rows x two adjacent chunks hit eight different positions.
template <int D>
__device__ __forceinline__ int chunk_swz(int r) {
  if (D == 128) return ((r & 7) << 1) | ((r >> 3) & 1);
  return ((r & 3) << 1) | ((r >> 2) & 1);
}

// The forward kernel's swizzle.  Its transposing reads fetch, per 32 lanes,
// 4 consecutive rows x 4 consecutive chunks; its K reads, per 16 lanes, 16
// consecutive rows x 1 chunk.  D = 128 (a row spans all 64 banks): the two
// high bits of the chunk index are XORed with r % 4 and the two low bits
// with (r / 4) % 4, so 4 rows land in 4 different chunk quads and 16 rows
// on 16 different chunks.  D = 64 (two rows share the 64 banks): rows of
// one parity must differ, so bit 2 takes (r / 2) % 2 and bits 0-1 take
// (r / 4) % 4.
template <int D>
__device__ __forceinline__ int fwd_swz(int r) {
  if (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// f(std::integral_constant<int, I>()) for I = A .. B-1, in order.
template <int A, int B, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (A < B) {
    f(std::integral_constant<int, A>());
    static_for<A + 1, B>(f);
  }
}

// a for P == 0, b otherwise (compile-time choice between two objects).
template <int P, class T>
__device__ __forceinline__ T& pick(T& a, T& b) {
  if constexpr (P == 0)
    return a;
  else
    return b;
}

// Work order of q-tile workgroups over (batch, kv head) pairs, for B * Hkv
// a multiple of 8.  Workgroup i runs on XCD i % 8 (the hardware deals
// workgroups to the XCDs in turn); XCD x takes pairs x, x + 8, ..., in
// groups of gp pairs, and within a group issues the q-tiles of all the
// group's query heads longest first.  A group is about as many q-tiles as
// one XCD holds at once, so the K/V rows of few pairs are live in that
// XCD's L2 at a time.  (gp at least the pairs per XCD: every pair of the
// XCD at once, q-tiles longest first.)
__device__ __forceinline__ void xcd_pair_map(int bid, int n_qtiles, int B, int Hkv, int G,
                                             int gp, int& qt, int& b, int& hq) {
  const int x = bid & 7, j = bid >> 3;
  const int n_pairs = (B * Hkv) >> 3;  // pairs on this XCD
  const int grp_items = gp * G * n_qtiles;
  const int grp = j / grp_items;
  const int gsz = min(gp, n_pairs - grp * gp);  // pairs in this group (the last may be short)
  int r = j - grp * grp_items;
  const int t = r / (gsz * G);  // q-tile rank, longest first
  r -= t * gsz * G;
  const int pl = r / G;
  const int p = x + 8 * (grp * gp + pl);
  qt = n_qtiles - 1 - t;
  b = p / Hkv;
  hq = (p - b * Hkv) * G + (r - pl * G);
}

// Pairs per group for xcd_pair_map: the q-tiles one XCD holds at once (32
// compute units, wg_per_cu workgroups each) over the q-tiles of one pair.
inline int xcd_group_pairs(int G, int n_qtiles, int wg_per_cu = 2) {
  const int gp = 32 * wg_per_cu / (G * n_qtiles);
  return gp < 1 ? 1 : gp;
}

__device__ __forceinline__ int clamp_len(int len, int hi) {
  return len < 0 ? 0 : (len > hi ? hi : len);
}

// Store x * acc^T as 32 bf16 rows of D values: acc[db][r] of lane
// (n, h) = l % 32, l / 32 is element (row n, column db*32 + 8 (r/4) + 4 h
// + r % 4).  The wave writes its rows to LDS at `stage` (32 rows x D bf16,
// 16-byte chunks XOR-swizzled by row) and reads them back 16 bytes per
// lane, 16 (D = 128) or 8 (D = 64) lanes per row (stage_rows_t), then
// stores them, row i at dst + i * stride (elements); rows >= n_rows are not
// stored (store_staged_rows).  x is per lane (its row's).
template <int D>
__device__ __forceinline__ void stage_rows_t(const f32x16 (&acc)[D / 32], float x,
                                             uint32_t stage, int n, int h, int lane,
                                             u32x4 (&rows)[D / 16]) {
  constexpr int CH = D / 8;  // 16-byte chunks per row
  constexpr int ROW_BYTES = D * 2;
  const int swz_w = n & (CH - 1);
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int c = db * 4 + r4;
      const u32x2 w = {(uint32_t)to_bf16_bits(acc[db][4 * r4] * x) |
                           ((uint32_t)to_bf16_bits(acc[db][4 * r4 + 1] * x) << 16),
                       (uint32_t)to_bf16_bits(acc[db][4 * r4 + 2] * x) |
                           ((uint32_t)to_bf16_bits(acc[db][4 * r4 + 3] * x) << 16)};
      const uint32_t ad = stage + n * ROW_BYTES + ((c ^ swz_w) << 4) + 8 * h;
      *(__attribute__((address_space(3))) u32x2*)(uintptr_t)ad = w;
    }
  constexpr int ROWS_PER_READ = 64 / CH;
#pragma unroll
  for (int i = 0; i < 32 / ROWS_PER_READ; ++i) {
    const int row = i * ROWS_PER_READ + lane / CH;
    const int c = lane % CH;
    const uint32_t ad = stage + row * ROW_BYTES + ((c ^ (row & (CH - 1))) << 4);
    rows[i] = *(const __attribute__((address_space(3))) u32x4*)(uintptr_t)ad;
  }
}

template <int D>
__device__ __forceinline__ void store_staged_rows(const u32x4 (&rows)[D / 16], int lane,
                                                  uint16_t* dst, size_t stride, int n_rows) {
  constexpr int CH = D / 8;
  constexpr int ROWS_PER_READ = 64 / CH;
#pragma unroll
  for (int i = 0; i < 32 / ROWS_PER_READ; ++i) {
    const int row = i * ROWS_PER_READ + lane / CH;
    const int c = lane % CH;
    if (row < n_rows) *reinterpret_cast<u32x4*>(dst + (size_t)row * stride + c * 8) = rows[i];
  }
}

template <int D>
__device__ __forceinline__ void store_rows_t(const f32x16 (&acc)[D / 32], float x,
                                             uint32_t stage, int n, int h, int lane,
                                             uint16_t* dst, size_t stride, int n_rows) {
  u32x4 rows[D / 16];
  stage_rows_t<D>(acc, x, stage, n, h, lane, rows);
  store_staged_rows<D>(rows, lane, dst, stride, n_rows);
}

}  // namespace mk
