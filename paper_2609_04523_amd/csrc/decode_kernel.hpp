// decode_kernel.hpp -- split-KV decode attention for gfx950.
//
// Kernel 1 (dec_split_kernel): one workgroup per (split, kv head, batch).
// The G = Hq/Hkv query heads of the kv head are the columns of one
// 16x16x32 MFMA block, so every cached K/V byte is read once for all of
// them.  Keys of the split stream through LDS in coalesced 16-byte loads;
// each of the 4 waves takes 32 keys of a 128-key tile with its own online
// softmax state, and the waves are merged in LDS at the end.  The kernel
// writes the split's normalised output and its natural-log LSE.
//
// Kernel 2 (dec_combine_kernel): per (batch, query head), merge the splits
// by their log-sum-exp: LSE = log sum_s exp(LSE_s), O = sum_s
// exp(LSE_s - LSE) O_s.  Splits at or past the sequence end hold nothing
// and are not read.
#pragma once

#include "mk_common.hpp"

namespace mk {

struct DecArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  float* o_part;    // [B, Hq, nsplit, D]
  float* lse_part;  // [B, Hq, nsplit]
  const int* kv_seqlens;
  int B, Hq, Hkv, Smax, split, nsplit;
  float scale_log2;
};

struct CombArgs {
  const float* o_part;
  const float* lse_part;
  const int* kv_seqlens;
  void* o;     // [B, Hq, D] bf16
  float* lse;  // [B, Hq] or null
  int B, Hq, Smax, split, nsplit;
};

template <int D>
struct DecShape {
  static constexpr int WAVES = 4;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int BN = 128;                       // keys per LDS tile, 32 per wave
  static constexpr int CHUNKS = D / 8;                 // 16-byte chunks per row
  static constexpr int LOADS = BN * CHUNKS / THREADS;  // per thread per tensor
  static constexpr int VT_STRIDE = BN + 8;             // bf16 per transposed V row
  static constexpr int KSTEPS = D / 32;                // 16x16x32 steps over the head dim
  static constexpr int DBLK = D / 16;                  // 16-row blocks of O^T
};

template <int D>
__global__ __launch_bounds__(256, 2) void dec_split_kernel(DecArgs a) {
  using S = DecShape<D>;
  constexpr int BN = S::BN;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[D * S::VT_STRIDE];
  __shared__ float w_m[S::WAVES][16], w_l[S::WAVES][16];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;  // MFMA column (query head of the group) / row
  const int gq = lane >> 4;   // MFMA k-group

  const int sidx = blockIdx.x;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int G = a.Hq / a.Hkv;
  const int L = clamp_len(a.kv_seqlens[b], a.Smax);
  const int k_begin = sidx * a.split;
  if (k_begin >= L) return;  // empty split: nothing to write, the merge skips it
  const int k_end = min(k_begin + a.split, L);
  const int n_t = (k_end - k_begin + BN - 1) / BN;

  const size_t kv_off = ((size_t)b * a.Hkv + g) * (size_t)a.Smax * D;
  const uint16_t* __restrict__ kg = a.kc + kv_off;
  const uint16_t* __restrict__ vg = a.vc + kv_off;

  // Q^T fragments: column c16 is query head g*G + c16 (zero when c16 >= G).
  bf16x8 qf[S::KSTEPS];
#pragma unroll
  for (int s = 0; s < S::KSTEPS; ++s) {
    u32x4 u = {0u, 0u, 0u, 0u};
    if (c16 < G)
      u = *reinterpret_cast<const u32x4*>(a.q + ((size_t)b * a.Hq + g * G + c16) * D + s * 32 +
                                          gq * 8);
    qf[s] = as_bf16x8(u);
  }

  u32x4 kreg[S::LOADS], vreg[S::LOADS];
  auto load_tile = [&](int t) {
#pragma unroll
    for (int p = 0; p < S::LOADS; ++p) {
      const int c = tid + p * S::THREADS;
      const int key = c / S::CHUNKS;
      const int ch = c % S::CHUNKS;
      const int gk = k_begin + t * BN + key;
      u32x4 zk = {0u, 0u, 0u, 0u}, zv = {0u, 0u, 0u, 0u};
      if (gk < k_end) {
        zk = *reinterpret_cast<const u32x4*>(kg + (size_t)gk * D + ch * 8);
        zv = *reinterpret_cast<const u32x4*>(vg + (size_t)gk * D + ch * 8);
      }
      kreg[p] = zk;
      vreg[p] = zv;
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int p = 0; p < S::LOADS; ++p) {
      const int c = tid + p * S::THREADS;
      const int key = c / S::CHUNKS;
      const int ch = c % S::CHUNKS;
      *reinterpret_cast<u32x4*>(&k_lds[key * D + ((ch ^ (key & (S::CHUNKS - 1))) * 8)]) =
          kreg[p];
      const u32x4 vv = vreg[p];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        vt_lds[(ch * 8 + 2 * i) * S::VT_STRIDE + key] = (uint16_t)(vv[i] & 0xffffu);
        vt_lds[(ch * 8 + 2 * i + 1) * S::VT_STRIDE + key] = (uint16_t)(vv[i] >> 16);
      }
    }
  };

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o_acc[S::DBLK];
#pragma unroll
  for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) o_acc[db][r] = 0.f;

  load_tile(0);
  for (int t = 0; t < n_t; ++t) {
    store_tile();
    __syncthreads();
    if (t + 1 < n_t) load_tile(t + 1);
    const int kw0 = k_begin + t * BN + wave * 32;  // first key of this wave
    if (kw0 < k_end) {
      // S^T = K Q^T for the wave's 32 keys (two 16-key blocks).
      f32x4 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sacc[kb][r] = 0.f;
        const int row = wave * 32 + kb * 16 + c16;
#pragma unroll
        for (int s = 0; s < S::KSTEPS; ++s) {
          const int ch = 4 * s + gq;
          const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(
              &k_lds[row * D + ((ch ^ (row & (S::CHUNKS - 1))) * 8)]));
          sacc[kb] = mfma16(kf, qf[s], sacc[kb]);
        }
      }
      // Online softmax over the column (query head); lane holds 8 keys.
      float mx = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float x = sacc[kb][r] * a.scale_log2;
          if (kw0 + kb * 16 + 4 * gq + r >= k_end) x = kNegInf;
          sacc[kb][r] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = fast_exp2(m_run - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(sacc[kb][r] - m_use);
          sacc[kb][r] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 16, 64);
      rs += __shfl_xor(rs, 32, 64);
      l_run = l_run * alpha + rs;
      m_run = m_new;
      // P^T: k-group gq holds keys {4gq..4gq+3} and {16+4gq..16+4gq+3} of the wave.
      const bf16x8 pf = to_bf16x8(sacc[0][0], sacc[0][1], sacc[0][2], sacc[0][3], sacc[1][0],
                                  sacc[1][1], sacc[1][2], sacc[1][3]);
#pragma unroll
      for (int db = 0; db < S::DBLK; ++db) {
        const int d = db * 16 + c16;
        const uint16_t* vp = &vt_lds[d * S::VT_STRIDE + wave * 32 + 4 * gq];
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vp);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vp + 16);
        const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
#pragma unroll
        for (int r = 0; r < 4; ++r) o_acc[db][r] *= alpha;
        o_acc[db] = mfma16(as_bf16x8(w), pf, o_acc[db]);
      }
    }
    __syncthreads();
  }

  // Merge the four waves' states through LDS (reusing the K tile area).
  float* w_o = reinterpret_cast<float*>(k_lds);  // [WAVES][16 columns][D]
  if (gq == 0) {
    w_m[wave][c16] = m_run;
    w_l[wave][c16] = l_run;
  }
  if (c16 < G) {
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        w_o[(wave * 16 + c16) * D + db * 16 + 4 * gq + r] = o_acc[db][r];
  }
  __syncthreads();
  for (int it = tid; it < G * D; it += S::THREADS) {
    const int c = it / D;
    const int d = it - c * D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < S::WAVES; ++w) M = fmaxf(M, w_m[w][c]);
    float lsum = 0.f, acc = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < S::WAVES; ++w) {
        const float f = fast_exp2(w_m[w][c] - M);
        lsum += w_l[w][c] * f;
        acc += w_o[(w * 16 + c) * D + d] * f;
      }
    }
    const size_t pr = ((size_t)b * a.Hq + g * G + c) * a.nsplit + sidx;
    a.o_part[pr * D + d] = lsum > 0.f ? acc / lsum : 0.f;
    if (d == 0) a.lse_part[pr] = lsum > 0.f ? (M + log2f(lsum)) * kLn2 : kNegInf;
  }
}

template <int D>
__global__ __launch_bounds__(256) void dec_combine_kernel(CombArgs a) {
  constexpr int PER_LANE = D / 64;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, hq) row
  if (r >= a.B * a.Hq) return;
  const int b = r / a.Hq;
  const int L = clamp_len(a.kv_seqlens[b], a.Smax);
  const int ns = (L + a.split - 1) / a.split;  // splits holding keys
  const float* lp = a.lse_part + (size_t)r * a.nsplit;
  float M = kNegInf;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, lp[s]);
  float out[PER_LANE];
#pragma unroll
  for (int i = 0; i < PER_LANE; ++i) out[i] = 0.f;
  float lse = kNegInf;
  if (M != kNegInf) {
    float sum = 0.f;
    for (int s = 0; s < ns; ++s) sum += expf(lp[s] - M);
    lse = M + logf(sum);
    for (int s = 0; s < ns; ++s) {
      const float w = expf(lp[s] - lse);
      const float* op = a.o_part + ((size_t)r * a.nsplit + s) * D + lane * PER_LANE;
#pragma unroll
      for (int i = 0; i < PER_LANE; ++i) out[i] += w * op[i];
    }
  }
  uint16_t* o = static_cast<uint16_t*>(a.o) + (size_t)r * D + lane * PER_LANE;
  if (PER_LANE == 2) {
    *reinterpret_cast<uint32_t*>(o) =
        (uint32_t)to_bf16_bits(out[0]) | ((uint32_t)to_bf16_bits(out[PER_LANE - 1]) << 16);
  } else {
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) o[i] = to_bf16_bits(out[i]);
  }
  if (lane == 0 && a.lse) a.lse[r] = lse;
}

}  // namespace mk
