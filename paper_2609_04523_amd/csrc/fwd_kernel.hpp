// fwd_kernel.hpp -- fused attention forward (prefill) for gfx950.
//
// One workgroup = 4 waves = BM query rows of one (batch, query head); wave w
// owns QB blocks of 32 consecutive rows.  The workgroup streams the 64-key
// K and V tiles of its KV head (hq / (Hq/Hkv)) from HBM straight into LDS
// (global_load_lds_dwordx4, double-buffered), up to the causal
// diagonal, and keeps the softmax state and the output accumulator in
// registers: online softmax, an exact rewrite of softmax(Q K^T * scale) V
// folded tile by tile.
//
// Orientation.  Scores are formed transposed, S^T = K Q^T, with K as the
// MFMA A operand (rows = keys) and Q^T as the B operand (columns =
// queries).  A lane then owns one query column, so the softmax row
// reductions are in-lane plus one exchange with lane l^32.  The output is
// O^T = V^T P^T: P^T is the score accumulator converted to bf16 in place
// (its key order is the accumulator's own row order), and the V^T operand
// is read from the row-major V tile with the transposing LDS read.
//
// Softmax bookkeeping (exp2 domain, c = scale * log2 e):
//   m    running row maximum of c*s, raised only when a tile's maximum
//        exceeds it by more than kRescaleSlack, so exp2(c*s - m) <= 2^8 and
//        the O accumulator is rescaled on few tiles;
//   l    running sum of the fp32 weights (each half-wave sums its own
//        keys; the halves are added at the end);
//   O    sum of bf16(weight) * V in fp32;
//   result O / l, LSE = ln 2 * (m + log2 l).
#pragma once

#include <type_traits>

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
  static constexpr int BM = WAVES * 32 * QB;              // query rows per workgroup
  static constexpr int BN = 64;                           // keys per LDS tile
  static constexpr int KSTEPS = D / 16;                   // MFMA steps over the head dim
  static constexpr int DBLK = D / 32;                     // 32-row blocks of O^T
  static constexpr int CHUNKS = D / 8;                    // 16-byte chunks per row
  static constexpr int ROWS_PER_KB = 512 / D;             // tile rows per 1 KB wave load
  static constexpr int BLOCKS_PER_WAVE = BN * D * 2 / 1024 / WAVES;
  static constexpr int LOADS_PER_TILE = 2 * BLOCKS_PER_WAVE;  // per thread, K and V
};

constexpr float kRescaleSlack = 8.0f;

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

// POS_SCALE: scale > 0, so the row maximum can be taken on raw scores and
// the scale folded into the exponent's FMA.  Otherwise scores are scaled
// first (scale 0 and negative scales).
template <int D, bool CAUSAL, bool OUT_F32, int QB, bool POS_SCALE>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdArgs a) {
  using S = FwdShape<D, QB>;
  constexpr int BN = S::BN;
  constexpr int TILE = BN * D;            // bf16 per tile per tensor
  constexpr int TILE_BYTES = TILE * 2;
  constexpr int ROW_BYTES = D * 2;
  constexpr int NK = 2 * S::KSTEPS;     // K fragment reads per tile
  constexpr int NV = 8 * S::DBLK;       // transposing V reads per tile
  constexpr int RW = 8;                 // LDS reads in flight
  static_assert(RW >= 2 && RW % 2 == 0 && RW <= NK && RW <= NV, "read window");
  __shared__ __attribute__((aligned(1024))) uint16_t k_lds[2][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_lds[2][TILE];

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
  const float c = a.scale_log2;

  const size_t q_row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
  const size_t kv_off = ((size_t)b * a.Hkv + g) * (size_t)a.Skv * D;
  const char* __restrict__ kg = reinterpret_cast<const char*>(a.k + kv_off);
  const char* __restrict__ vg = reinterpret_cast<const char*>(a.v + kv_off);

  // Q^T fragments: lane (column n, k-group h) holds q[row][16 s + 8 h .. +7].
  // Loaded before any K/V traffic so waiting for them waits for nothing else.
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

  // ---- tile loads: HBM -> LDS, one 1 KB wave-wide load per block ----
  // Block blk = 4 p + wave of a tile holds rows blk*ROWS_PER_KB + l/CHUNKS;
  // lane l fills physical chunk l % CHUNKS with logical chunk
  // (l % CHUNKS) ^ swz(row).  Rows past the sequence end re-read its last
  // row (finite data that the mask zeroes), so no load leaves [0, L).
  // The rows a lane loads are dma_row + ROW_STEP * p, and they all share
  // one swizzle (it depends on the row modulo 16 at D = 128 and on bits 1-3
  // of the row at D = 64, which the step leaves unchanged).
  constexpr int ROW_STEP = S::WAVES * S::ROWS_PER_KB;
  static_assert(ROW_STEP % 16 == 0, "row step must preserve the swizzle");
  const int dma_row = wave * S::ROWS_PER_KB + lane / S::CHUNKS;
  const int dma_ch = ((lane % S::CHUNKS) ^ fwd_swz<D>(dma_row)) * 16;  // byte offset
  const uint32_t k_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&k_lds[0][0]) + wave * 1024);
  const uint32_t v_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&v_lds[0][0]) + wave * 1024);
  auto issue_block = [&](int kt, auto buf_tag, auto p_tag) {
    constexpr int BUF = decltype(buf_tag)::value;
    constexpr int P = decltype(p_tag)::value;
    const int lim = L - 1 - kt * BN;  // last valid row of the tile
    const uint32_t goff = (uint32_t)(min(dma_row, lim - P * ROW_STEP) * ROW_BYTES + dma_ch) +
                          P * ROW_STEP * ROW_BYTES;
    const size_t toff = (size_t)kt * BN * ROW_BYTES;
    constexpr uint32_t lds_off = BUF * TILE_BYTES + P * S::WAVES * 1024;
    load_lds16_at(kg + toff + goff, k_lds_w + lds_off);
    load_lds16_at(vg + toff + goff, v_lds_w + lds_off);
  };
  auto issue_tile = [&](int kt, auto buf_tag) {
    static_for<0, S::BLOCKS_PER_WAVE>([&](auto p_tag) { issue_block(kt, buf_tag, p_tag); });
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

  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  if (n_kt > 0) issue_tile(0, B0());

  // Lane parts of the LDS read addresses (bytes within a tile).  K row
  // 32 kb + n: the swizzle of n + 32 kb equals that of n.  Transposing V
  // reads: rows 16 kc + 4 h + i/4 (+ 8), columns 32 db + 16 ((l/16) % 2) +
  // 4 (i % 4), i = l % 16; the swizzle does not depend on kc.
  uint32_t k_addr[S::KSTEPS];
#pragma unroll
  for (int s = 0; s < S::KSTEPS; ++s)
    k_addr[s] = lds_addr(&k_lds[0][0]) + n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
  uint32_t v_addr[S::DBLK][2];
  {
    const int tr_i = lane & 15;
    const int tr_row = 4 * h + (tr_i >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (tr_i & 3);
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int r = tr_row + 8 * hh;
        const int col = db * 32 + tr_col;
        v_addr[db][hh] = lds_addr(&v_lds[0][0]) + r * ROW_BYTES +
                         ((((col >> 3) ^ fwd_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }

  // One 64-key tile for this wave from LDS buffer BUF.  MASK: apply the
  // length / causal mask.
  auto tile = [&](auto mask_tag, auto buf_tag, int kt, auto&& qk_hook) {
    constexpr bool MASK = decltype(mask_tag)::value;
    constexpr int BUF = decltype(buf_tag)::value;
    const int key0 = kt * BN;
    // ---- S^T = K Q^T for the 64 keys of the tile ----
    // The tile's LDS reads form one stream: the NK K fragments (step s,
    // key block kb, alternating kb so that two accumulator chains are in
    // flight), then the NV transposing V reads in the order the P V
    // products consume them.  RW reads are kept in flight: consuming one
    // issues the next, so V's first reads are under way during the softmax.
    f32x16 sacc[QB][2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[qb][kb][r] = 0.f;
    u32x4 kr[NK];
    u32x2 vr[NV];
    auto issue_read = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      if constexpr (J < NK) {
        constexpr int OFF = BUF * TILE_BYTES + (J % 2) * 32 * ROW_BYTES;
        kr[J] = lds_read_b128_async_off<OFF>(k_addr[J / 2]);
      } else if constexpr (J < NK + NV) {
        constexpr int V = J - NK;        // (kc, db, hh) = V / (2 DBLK), V / 2 % DBLK, V % 2
        constexpr int OFF = BUF * TILE_BYTES + (V / (2 * S::DBLK)) * 16 * ROW_BYTES;
        vr[V] = lds_read_tr16_async_off<OFF>(v_addr[(V / 2) % S::DBLK][V % 2]);
      }
    };
    static_for<0, RW>(issue_read);
    static_for<0, NK>([&](auto i_tag) {
      constexpr int I = decltype(i_tag)::value;
      lds_wait_lgkm<RW - 1>();
      lds_ready(kr[I]);
      const bf16x8 kf = as_bf16x8(kr[I]);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        sacc[qb][I % 2] = mfma32(kf, qf[qb][I / 2], sacc[qb][I % 2]);
      issue_read(std::integral_constant<int, I + RW>());
      qk_hook(i_tag);
    });
    // ---- online softmax, one query column per lane ----
    bf16x8 pf[QB][4];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      if (!POS_SCALE) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[qb][kb][r] *= c;
      }
      if (MASK) {
        const int qrow = qw0 + qb * 32 + n;
        const int lim = min(L - 1, CAUSAL ? qrow + off : L - 1);  // last admissible key
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
            if (key > lim) sacc[qb][kb][r] = kNegInf;
          }
      }
      float mx = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[qb][kb][r]);
      mx = max_xor32(mx);
      if (POS_SCALE) mx *= c;
      if (__ballot(mx > m_run[qb] + kRescaleSlack)) {
        const float m_new = fmaxf(m_run[qb], mx);
        const float alpha = (m_new == kNegInf) ? 1.f : fast_exp2(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o_acc[qb][db][r] *= alpha;
      }
      const float m_use = (m_run[qb] == kNegInf) ? 0.f : m_run[qb];
      const float cc = POS_SCALE ? c : 1.f;
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(sacc[qb][kb][r], cc, -m_use));
          sacc[qb][kb][r] = p;
          rs += p;
        }
      l_run[qb] += rs;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const f32x16 p = sacc[qb][kb];
        pf[qb][2 * kb] = to_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
        pf[qb][2 * kb + 1] = to_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
      }
    }
    // ---- O^T += V^T P^T over 16-key chunks ----
    // Chunk kc: k-group h holds P for keys 16 kc + {4h..4h+3, 8+4h..8+4h+3};
    // the two transposing reads fetch V for exactly those keys, column d.
    // Product m = (kc, db) takes V reads 2m and 2m + 1 of the stream.
    static_for<0, NV / 2>([&](auto m_tag) {
      constexpr int M = decltype(m_tag)::value;
      constexpr int AHEAD = (RW < NV - 2 * M ? RW : NV - 2 * M) - 2;  // reads issued after 2M+1
      lds_wait_lgkm<AHEAD>();
      lds_ready(vr[2 * M]);
      lds_ready(vr[2 * M + 1]);
      const u32x4 w = {vr[2 * M][0], vr[2 * M][1], vr[2 * M + 1][0], vr[2 * M + 1][1]};
      const bf16x8 vf = as_bf16x8(w);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        o_acc[qb][M % S::DBLK] = mfma32(vf, pf[qb][M / S::DBLK], o_acc[qb][M % S::DBLK]);
      issue_read(std::integral_constant<int, NK + RW + 2 * M>());
      issue_read(std::integral_constant<int, NK + RW + 2 * M + 1>());
    });
  };

  // Tiles [0, n_free) need no mask for any row of this wave; tiles up to
  // n_live hold at least one admissible key for some row of the wave.
  const int w_first = qw0;                      // first query row of the wave
  const int w_last = min(qw0 + 32 * QB, a.Sq) - 1;
  int n_free = (CAUSAL ? min(L, w_first + off + 1) : L) / BN;
  int n_live = qw0 < a.Sq ? (CAUSAL ? min(L, w_last + off + 1) : L) : 0;
  n_live = (max(n_live, 0) + BN - 1) / BN;
  n_free = max(0, min(n_free, n_live));

  // Tile kt lives in buffer kt % 2; the loop is unrolled by two so the
  // buffer of every LDS access is a compile-time constant.  One barrier per
  // tile: once every wave has waited for its own loads of tile kt, the
  // barrier makes the whole tile visible and also proves that every wave
  // has finished tile kt - 1, so the loads of tile kt + 1 can go into that
  // buffer during tile kt, about a tile of compute ahead of their use.
  // The loads of tile kt + 1 are spread over the score products of tile
  // kt (one 1 KB block of K and of V per NK / BLOCKS_PER_WAVE products), so
  // no wave stalls on a burst of memory instructions.
  constexpr int QK_PER_BLOCK = NK / S::BLOCKS_PER_WAVE;
  static_assert(NK % S::BLOCKS_PER_WAVE == 0, "load spreading");
  auto step = [&](int kt, auto buf_tag, auto next_tag) {
    wait_vmcnt<0>();
    __syncthreads();
    const bool more = kt + 1 < n_kt;
    auto hook = [&](auto i_tag) {
      constexpr int I = decltype(i_tag)::value;
      if constexpr (I % QK_PER_BLOCK == QK_PER_BLOCK - 1)
        if (more) issue_block(kt + 1, next_tag, std::integral_constant<int, I / QK_PER_BLOCK>());
    };
    if (kt < n_free)
      tile(std::false_type(), buf_tag, kt, hook);
    else if (kt < n_live)
      tile(std::true_type(), buf_tag, kt, hook);
    else if (more)
      issue_tile(kt + 1, next_tag);
  };
  for (int kt = 0; kt < n_kt; kt += 2) {
    step(kt, B0(), B1());
    if (kt + 1 < n_kt) step(kt + 1, B1(), B0());
  }

  // ---- epilogue: O = O_acc / l, LSE = ln 2 * (m + log2 l) ----
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qrow = qw0 + qb * 32 + n;
    const float lsum = sum_xor32(l_run[qb]);
    if (qrow >= a.Sq) continue;
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
