// fwd_kernel.hpp -- fused attention forward (prefill) for gfx950.
//
// One workgroup = 4 waves = BM query rows of one (batch, query head).  It
// streams the key/value tiles of the head's KV group (hq / (Hq/Hkv))
// through LDS, up to the causal diagonal, and keeps the softmax state and
// the output accumulator in registers (online softmax: exact rewrite of
// softmax(Q K^T * scale) V, folded tile by tile).
//
// Orientation.  Scores are formed transposed, S^T = K Q^T, with K as the
// MFMA A operand (rows = keys) and Q^T as the B operand (columns =
// queries).  A lane then owns one query column, so every softmax
// reduction is in-lane plus one exchange with lane l^32.  The output is
// formed as O^T = V^T P^T: P^T is the score accumulator converted to bf16
// in place (its key order is the accumulator's own row order), and V^T is
// read from a transposed LDS copy of the value tile.
#pragma once

#include "mk_common.hpp"

namespace mk {

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  void* o;
  float* lse;
  const int* kv_seqlens;
  int B, Hq, Hkv, Sq, Skv;
  int n_qtiles;
  int xcd_groups;     // 1: (batch, kv head) groups spread over the 8 XCDs
  float scale_log2;   // scale * log2(e)
};

template <int D, int QB>
struct FwdShape {
  static constexpr int WAVES = 4;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int BM = WAVES * 32 * QB;          // query rows per workgroup
  static constexpr int BN = 64;                       // keys per LDS tile
  static constexpr int KSTEPS = D / 16;               // MFMA steps over the head dim
  static constexpr int DBLK = D / 32;                 // 32-row output blocks of O^T
  static constexpr int CHUNKS = D / 8;                // 16-byte chunks per row
  static constexpr int VT_STRIDE = BN + 4;            // bf16 per transposed V row
  static constexpr int LOADS = BN * CHUNKS / THREADS; // 16-byte loads per thread per tensor
};

// Work-item order.  Longest causal q-tiles are issued first.  When the
// number of (batch, kv head) groups is a multiple of 8, consecutive
// workgroups on one XCD (dispatch is round-robin over the 8 XCDs) belong
// to the same group, so the query heads and q-tiles that re-read one K/V
// head share that XCD's L2.
__device__ __forceinline__ void fwd_map_block(int bid, const FwdArgs& a, int& qt, int& hq,
                                              int& b) {
  const int G = a.Hq / a.Hkv;
  if (a.xcd_groups) {
    const int x = bid & 7;
    const int j = bid >> 3;
    const int per = ((a.B * a.Hkv) >> 3) * G;  // items per XCD per q-tile
    const int t = j / per;
    const int rem = j - t * per;
    qt = a.n_qtiles - 1 - t;
    const int grp = x + 8 * (rem / G);
    b = grp / a.Hkv;
    hq = (grp - b * a.Hkv) * G + (rem % G);
  } else {
    const int per = a.B * a.Hq;
    const int t = bid / per;
    const int rem = bid - t * per;
    qt = a.n_qtiles - 1 - t;
    b = rem / a.Hq;
    hq = rem - b * a.Hq;
  }
}

template <int D, bool CAUSAL, bool OUT_F32, int QB>
__global__ __launch_bounds__(256, 1) void fwd_kernel(FwdArgs a) {
  using S = FwdShape<D, QB>;
  constexpr int BN = S::BN;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[2][D * S::VT_STRIDE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;  // MFMA column (query) / row (key) within a 32-block
  const int h = lane >> 5;  // MFMA k-group

  int qt, hq, b;
  fwd_map_block(blockIdx.x, a, qt, hq, b);
  const int G = a.Hq / a.Hkv;
  const int g = hq / G;
  const int L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
  const int off = L - a.Sq;  // bottom-right causal alignment
  const int q0 = qt * S::BM;
  const int q_end = min(q0 + S::BM, a.Sq);
  int n_keys = L;
  if (CAUSAL) n_keys = min(L, q_end + off);
  if (n_keys < 0) n_keys = 0;
  const int n_kt = (n_keys + BN - 1) / BN;

  const size_t q_row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
  const size_t kv_off = ((size_t)b * a.Hkv + g) * (size_t)a.Skv * D;
  const uint16_t* __restrict__ kg = a.k + kv_off;
  const uint16_t* __restrict__ vg = a.v + kv_off;

  // Q^T fragments: lane (column n, k-group h) holds q[row][16 s + 8 h .. +7].
  const int qw0 = q0 + wave * 32 * QB;
  bf16x8 qf[QB][S::KSTEPS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qw0 + qb * 32 + n;
#pragma unroll
    for (int s = 0; s < S::KSTEPS; ++s) {
      u32x4 u = {0u, 0u, 0u, 0u};
      if (row < a.Sq)
        u = *reinterpret_cast<const u32x4*>(a.q + (q_row0 + row) * D + s * 16 + h * 8);
      qf[qb][s] = as_bf16x8(u);
    }
  }

  // K/V tile staging through registers.
  u32x4 kreg[S::LOADS], vreg[S::LOADS];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int p = 0; p < S::LOADS; ++p) {
      const int c = tid + p * S::THREADS;
      const int key = c / S::CHUNKS;
      const int ch = c % S::CHUNKS;
      const int gk = kt * BN + key;
      u32x4 zk = {0u, 0u, 0u, 0u}, zv = {0u, 0u, 0u, 0u};
      if (gk < L) {
        zk = *reinterpret_cast<const u32x4*>(kg + (size_t)gk * D + ch * 8);
        zv = *reinterpret_cast<const u32x4*>(vg + (size_t)gk * D + ch * 8);
      }
      kreg[p] = zk;
      vreg[p] = zv;
    }
  };
  // K rows keep their layout with 16-byte chunks XOR-swizzled by row; V is
  // stored transposed ([d][key], padded rows) for the V^T operand.
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int p = 0; p < S::LOADS; ++p) {
      const int c = tid + p * S::THREADS;
      const int key = c / S::CHUNKS;
      const int ch = c % S::CHUNKS;
      *reinterpret_cast<u32x4*>(&k_lds[buf][key * D + ((ch ^ (key & (S::CHUNKS - 1))) * 8)]) =
          kreg[p];
      const u32x4 vv = vreg[p];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        vt_lds[buf][(ch * 8 + 2 * i) * S::VT_STRIDE + key] = (uint16_t)(vv[i] & 0xffffu);
        vt_lds[buf][(ch * 8 + 2 * i + 1) * S::VT_STRIDE + key] = (uint16_t)(vv[i] >> 16);
      }
    }
  };

  float m_run[QB], l_run[QB];
  f32x16 o_acc[QB][S::DBLK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = kNegInf;
    l_run[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o_acc[qb][db][r] = 0.f;
  }

  if (n_kt > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int kt = 0; kt < n_kt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < n_kt) load_tile(kt + 1);
    const int key0 = kt * BN;
    // A wave skips a tile whose keys all lie after its last query.
    bool active = qw0 < a.Sq;
    if (CAUSAL) active = active && key0 <= qw0 + 32 * QB - 1 + off;
    if (active) {
      // ---- S^T = K Q^T for the 64 keys of the tile ----
      f32x16 sacc[QB][2];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[qb][kb][r] = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int row = kb * 32 + n;
#pragma unroll
        for (int s = 0; s < S::KSTEPS; ++s) {
          const int ch = 2 * s + h;
          const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(
              &k_lds[buf][row * D + ((ch ^ (row & (S::CHUNKS - 1))) * 8)]));
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) sacc[qb][kb] = mfma32(kf, qf[qb][s], sacc[qb][kb]);
        }
      }
      // ---- online softmax, one query column per lane ----
      bf16x8 pf[QB][4];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int qrow = qw0 + qb * 32 + n;
        const bool need_mask =
            (key0 + BN > L) || (CAUSAL && key0 + BN - 1 > qw0 + qb * 32 + off);
        float mx = kNegInf;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float x = sacc[qb][kb][r] * a.scale_log2;
            if (need_mask) {
              const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
              if (key >= L || (CAUSAL && key > qrow + off)) x = kNegInf;
            }
            sacc[qb][kb][r] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, swap_halves(mx));
        const float m_new = fmaxf(m_run[qb], mx);
        const float m_use = (m_new == kNegInf) ? 0.f : m_new;
        const float alpha = fast_exp2(m_run[qb] - m_use);
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = fast_exp2(sacc[qb][kb][r] - m_use);
            sacc[qb][kb][r] = p;
            rs += p;
          }
        rs += swap_halves(rs);
        l_run[qb] = l_run[qb] * alpha + rs;
        m_run[qb] = m_new;
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o_acc[qb][db][r] *= alpha;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const f32x16 p = sacc[qb][kb];
          pf[qb][2 * kb] = to_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
          pf[qb][2 * kb + 1] = to_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
        }
      }
      // ---- O^T += V^T P^T over 16-key chunks ----
      // Chunk kc: lane (k-group h) holds P for keys 16 kc + {4h..4h+3, 8+4h..8+4h+3}.
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db) {
          const int d = db * 32 + n;
          const uint16_t* vp = &vt_lds[buf][d * S::VT_STRIDE + kc * 16 + 4 * h];
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vp);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vp + 8);
          const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
          const bf16x8 vf = as_bf16x8(w);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o_acc[qb][db] = mfma32(vf, pf[qb][kc], o_acc[qb][db]);
        }
      }
    }
    if (kt + 1 < n_kt) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: O = O_acc / l, LSE = ln 2 * (m + log2 l) ----
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qrow = qw0 + qb * 32 + n;
    if (qrow >= a.Sq) continue;
    const float lsum = l_run[qb];
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    const size_t obase = (q_row0 + qrow) * D;
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = db * 32 + 8 * r4 + 4 * h;
        const float v0 = o_acc[qb][db][4 * r4 + 0] * inv;
        const float v1 = o_acc[qb][db][4 * r4 + 1] * inv;
        const float v2 = o_acc[qb][db][4 * r4 + 2] * inv;
        const float v3 = o_acc[qb][db][4 * r4 + 3] * inv;
        if (OUT_F32) {
          const f32x4 w = {v0, v1, v2, v3};
          *reinterpret_cast<f32x4*>(static_cast<float*>(a.o) + obase + d) = w;
        } else {
          const u32x2 w = {(uint32_t)to_bf16_bits(v0) | ((uint32_t)to_bf16_bits(v1) << 16),
                           (uint32_t)to_bf16_bits(v2) | ((uint32_t)to_bf16_bits(v3) << 16)};
          *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.o) + obase + d) = w;
        }
      }
    if (h == 0 && a.lse)
      a.lse[q_row0 + qrow] = lsum > 0.f ? (m_run[qb] + log2f(lsum)) * kLn2 : kNegInf;
  }
}

}  // namespace mk
