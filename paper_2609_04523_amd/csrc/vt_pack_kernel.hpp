// vt_pack_kernel.hpp -- V^T tiles for the forward kernel's VT path.
//
// The forward forms O^T = V^T P^T with V^T as the MFMA A operand: a lane
// holds 8 consecutive k-values (keys) of one row (head dim).  From a
// row-major V tile those are a column, which only the transposing LDS read
// delivers, at half the LDS rate of a plain 16-byte read.  This pre-pass
// writes V once more, as tiles in the operand's own layout:
//
//   vt[b, g, kt, kc, d, 16]   (kt: 64-key tile, kc: 16-key chunk of it)
//
// Row (kc, d) holds v[b, g, 64 kt + 16 kc + key, d] for 16 keys in the
// order of the P^T operand: its k-group h takes keys 4 h + 0..3 and
// 8 + 4 h + 0..3 of the chunk (the 32x32 accumulator's row order), and the
// two 16-byte halves of a row are k-groups h ^ ((d / 8) % 2), which makes
// the forward's reads free of bank conflicts.  A tile is one contiguous
// block of D * 128 bytes.  Keys at or past the sequence's length (and the
// padding of the last tile) are zeros: the forward's mask gives them zero
// weight, and 0 * 0 = 0.
#pragma once

#include "mk_common.hpp"

namespace mk {

// key within a 16-key chunk at position e (0..7) of k-group h
__device__ __forceinline__ int vt_key(int h, int e) { return (e & 3) + 4 * h + 8 * (e >> 2); }

struct VtPackArgs {
  const uint16_t* v;       // [B, Hkv, Skv, D]
  uint16_t* vt;            // [B, Hkv, vt_tiles, 4, D, 16]
  const int* kv_seqlens;   // [B] or null (all Skv)
  int Skv, vt_tiles, Hkv;
  // the forward's work-item counters (FwdArgs::ctr), n_queues of them, each
  // set to ctr_init here, before the forward runs
  int* ctr;
  int ctr_init, n_queues;
};

// One workgroup per 64-key tile of one (b, kv head), B * Hkv * vt_tiles
// workgroups in (b, g)-major order: the tile's 64 V rows go to LDS (rows
// padded by 4 bytes against bank conflicts), then each thread gathers the
// 8 keys of one 16-byte piece of the V^T tile and the tile is written in
// order, 16 bytes per thread.
template <int D>
__global__ __launch_bounds__(256) void vt_pack_kernel(VtPackArgs a) {
  constexpr int BN = 64;
  constexpr int RB = D * 2;                // bytes per V row
  constexpr int PITCH = RB + 4;            // LDS bytes per key row
  constexpr int CH = D / 8;                // 16-byte chunks per V row
  __shared__ __attribute__((aligned(16))) uint8_t tile[BN * PITCH];
  const int bg = blockIdx.x / a.vt_tiles;  // b * Hkv + g
  const int kt = blockIdx.x - bg * a.vt_tiles;
  const int b = bg / a.Hkv;
  const int L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
  const uint16_t* v = a.v + (size_t)bg * a.Skv * D;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid < a.n_queues) a.ctr[32 * tid] = a.ctr_init;
#pragma unroll
  for (int i = tid; i < BN * CH; i += 256) {
    const int r = i / CH, c = i % CH;
    const int key = kt * BN + r;
    u32x4 w = {0u, 0u, 0u, 0u};
    if (key < L) w = *reinterpret_cast<const u32x4*>(v + (size_t)key * D + c * 8);
    uint32_t* dst = reinterpret_cast<uint32_t*>(tile + r * PITCH + c * 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) dst[j] = w[j];
  }
  __syncthreads();
  // piece i of the tile: chunk kc = i / (2 D), row d = (i / 2) % D, half i % 2
  uint16_t* out = a.vt + ((size_t)bg * a.vt_tiles + kt) * (BN * D);
#pragma unroll
  for (int i = tid; i < BN * D / 8; i += 256) {
    const int kc = i / (2 * D), d = (i / 2) % D;
    const int h = (i & 1) ^ ((d >> 3) & 1);
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k0 = 16 * kc + vt_key(h, 2 * j), k1 = 16 * kc + vt_key(h, 2 * j + 1);
      const uint32_t lo = *reinterpret_cast<const uint16_t*>(tile + k0 * PITCH + d * 2);
      const uint32_t hi = *reinterpret_cast<const uint16_t*>(tile + k1 * PITCH + d * 2);
      w[j] = lo | (hi << 16);
    }
    const u32x4 wv = {w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4*>(out + (size_t)i * 8) = wv;
  }
}

}  // namespace mk
