// mla_kernel.hpp -- decode step of multi-head latent attention (absorbed
// form) for gfx950.
//
// Every query head reads the same cache row per key: its Dc = 512 latent
// values (the value, and the first part of the key) and Dr = 64 rotary
// values (the rest of the key).  With q [B, 16, 576] and the latent cache
// ckv [B, Smax, 576]:
//   s_hj = scale * q_h . ckv_j,   O_h = sum_j softmax(s_h)_j ckv_j[0:512].
// The stream of 32-key stages over the batch is cut into equal parts as in
// the plain decode (decode_kernel.hpp, one kv head), with its merge kernel
// for pieces cut by part boundaries.
//
// One workgroup of four waves per part.  A stage's 32 rows (36 KB) go
// HBM -> LDS with coalesced 1 KB LDS-DMA loads, three stages in a ring, and
// the 16 query rows of each piece into one of two Q buffers.  Every wave
// forms the whole S^T = K Q^T (32 keys x 16 heads, 16x16x32 MFMA over 576
// dims) and the online softmax, redundantly, and its own quarter of the
// output dims, O^T[128 w .. +127] += V^T P^T, so the output accumulators
// stay small; the matrix work is well below the time the stage takes to
// arrive.  Cache rows are 1152 bytes; their 16-byte chunks are XOR-swizzled
// by (row / 2) % 8 within groups of 8 chunks, which spreads the 16 rows of
// a K read over all 64 banks.
#pragma once

#include "decode_kernel.hpp"

namespace mk {

struct MlaShape {
  static constexpr int H = 16;                    // query heads
  static constexpr int DC = 512, DR = 64, DK = 576;
  static constexpr int ROW_BYTES = DK * 2;        // 1152
  static constexpr int BN = kDecStageKeys;        // 32 keys per stage
  static constexpr int SLOTS = 3;
  static constexpr int SLOT_BYTES = BN * ROW_BYTES;  // 36 KB
  static constexpr int Q_BYTES = H * ROW_BYTES;      // 18 KB
  static constexpr int KV_BLOCKS = SLOT_BYTES / 1024;  // 36 one-KB loads per stage
  static constexpr int Q_BLOCKS = Q_BYTES / 1024;      // 18
  static constexpr int WAVES = 4;
  static constexpr int KV_PER_WAVE = KV_BLOCKS / WAVES;                 // 9
  static constexpr int Q_PER_WAVE = (Q_BLOCKS + WAVES - 1) / WAVES;     // 5
  static constexpr int KSTEPS = DK / 32;          // 18
  static constexpr int DBLK_W = DC / 16 / WAVES;  // 8 output blocks of 16 dims per wave
  static constexpr int LDS_BYTES = SLOTS * SLOT_BYTES + 2 * Q_BYTES;  // 144 KB
  static_assert(KV_BLOCKS % WAVES == 0, "stage loads split evenly");
  static_assert(KV_PER_WAVE + Q_PER_WAVE < 64, "vmcnt range");
};

// Swizzle of 16-byte chunk c of cache row r (c ^ (r/2 % 8)).
__device__ __forceinline__ int mla_swz(int r) { return (r >> 1) & 7; }

// (A template, instantiated once, so that including this header in several
// translation units defines the kernel once.)
template <int H_>
__global__ __launch_bounds__(256, 1) void mla_part_kernel(DecArgs a) {
  using S = MlaShape;
  static_assert(H_ == S::H, "built for 16 query heads");
  constexpr int RB = S::ROW_BYTES;
  __shared__ __attribute__((aligned(1024))) char lds[S::LDS_BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int c16 = lane & 15;  // MFMA column (query head) / row (key)
  const int gq = lane >> 4;   // MFMA k-group
  const int w = blockIdx.x;

  // ---- this part's stages and the cursor at its first ----
  const SeqChunk first = seq_chunk(a, 0);
  const int T = dec_total(a, first);
  const int s0 = part_start(w, T, a.P);
  const int n_stages = part_start(w + 1, T, a.P) - s0;
  if (n_stages <= 0) return;
  DecCursor cur = dec_locate(a, first, s0);

  const uint32_t lds0 = lds_addr(lds);
  const uint32_t q_lds0 = lds0 + S::SLOTS * S::SLOT_BYTES;
  auto slot_addr = [&](int k) { return lds0 + (uint32_t)k * S::SLOT_BYTES; };

  // ---- loads.  LDS byte o = 1024 blk + 16 lane of a stage (or Q buffer)
  // is chunk (o % 1152) / 16 of row o / 1152, which holds logical chunk
  // p ^ swz(row).  Rows past the sequence end re-read its last row (the
  // mask zeroes their weight). ----
  auto issue_stage = [&](const DecCursor& c, uint32_t slot) {
    const int key0 = c.t * S::BN;
    const int lim = c.L - 1 - key0;
    const char* g = reinterpret_cast<const char*>(a.kc) +
                    ((size_t)c.b * a.Smax + key0) * RB;
    const uint32_t dst0 = __builtin_amdgcn_readfirstlane(slot);
#pragma unroll
    for (int i = 0; i < S::KV_PER_WAVE; ++i) {
      const int blk = wave + S::WAVES * i;
      const int o = blk * 1024 + 16 * lane;
      const int r = o / RB;
      const int p = (o - r * RB) >> 4;
      const int lc = p ^ mla_swz(r);
      load_lds16_buf(g, S::SLOT_BYTES, (uint32_t)(min(r, lim) * RB + lc * 16), dst0 + blk * 1024);
    }
  };
  auto issue_q = [&](int b, uint32_t qbuf) {
    const char* g = reinterpret_cast<const char*>(a.q) + (size_t)b * S::H * RB;
    const uint32_t dst0 = __builtin_amdgcn_readfirstlane(qbuf);
#pragma unroll
    for (int i = 0; i < S::Q_PER_WAVE; ++i) {
      const int blk = min(wave + S::WAVES * i, S::Q_BLOCKS - 1);  // waves 2, 3 repeat the last
      const int o = blk * 1024 + 16 * lane;
      const int r = o / RB;
      const int p = (o - r * RB) >> 4;
      const int lc = p ^ mla_swz(r);
      load_lds16_buf(g, S::Q_BYTES, (uint32_t)(r * RB + lc * 16), dst0 + blk * 1024);
    }
  };

  // ---- lane parts of the LDS read addresses ----
  // K row 16 kb + c16 (and Q row c16), logical chunk 4 s + gq: physical
  // chunk 8 (s / 2) + ((4 (s % 2) + gq) ^ swz), swz = swz(c16) for both.
  const int fz = mla_swz(c16);
  uint32_t k_lane[2][2], q_lane[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const uint32_t ch = (uint32_t)(((4 * par + gq) ^ fz) << 4);
    q_lane[par] = c16 * RB + ch;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) k_lane[kb][par] = (16 * kb + c16) * RB + ch;
  }
  // V (transposing): rows 4 gq + c16 / 4 (+ 16), columns 16 db + 4 (c16 % 4)
  // for this wave's blocks db = 8 wave + d: chunk 16 wave + 8 (d / 4) +
  // ((2 (d % 4) + (c16 % 4) / 2) ^ swz), byte 8 (c16 % 2) within it.
  uint32_t v_lane[4][2];
  {
    const int tr_row = 4 * gq + (c16 >> 2);
    const int fv = mla_swz(tr_row);  // rows r and r + 16 share it
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        v_lane[j][hh] = (tr_row + 16 * hh) * RB + wave * 256 +
                        ((((2 * j + ((c16 & 3) >> 1)) ^ fv)) << 4) + 8 * (c16 & 1);
  }

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o_acc[S::DBLK_W];
#pragma unroll
  for (int db = 0; db < S::DBLK_W; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) o_acc[db][r] = 0.f;
  bf16x8 qf[S::KSTEPS];
  const float c = a.scale_log2;

  // Q^T fragments of the piece from Q buffer qbuf: column c16 = query head.
  auto load_q = [&](uint32_t qbuf) {
    u32x4 x[S::KSTEPS];
    static_for<0, S::KSTEPS>([&](auto s_tag) {
      constexpr int s = decltype(s_tag)::value;
      x[s] = lds_read_b128_async_off<128 * (s / 2)>(qbuf + q_lane[s % 2]);
    });
    lds_wait_lgkm<0>();
#pragma unroll
    for (int s = 0; s < S::KSTEPS; ++s) {
      lds_ready(x[s]);
      qf[s] = as_bf16x8(x[s]);
    }
  };

  // One stage.  The LDS reads form one stream -- the 36 K fragments (step
  // s, then key block kb, so the two blocks' accumulation chains
  // interleave), then the 16 transposing V reads (block d, low / high
  // keys) -- kept RW reads ahead of their use and waited for by count, so
  // the V reads are in flight during the softmax.
  constexpr int NK = 2 * S::KSTEPS, NV = 2 * S::DBLK_W, TOT = NK + NV, RW = 8;
  auto consume = [&](const DecCursor& cc, uint32_t slot) {
    const int key0 = cc.t * S::BN;
    u32x4 kr[NK];
    u32x2 vr[NV];
    const uint32_t kb0[2] = {slot + k_lane[0][0], slot + k_lane[0][1]};
    const uint32_t kb1[2] = {slot + k_lane[1][0], slot + k_lane[1][1]};
    auto issue_read = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      if constexpr (J < NK) {
        constexpr int KB = J % 2, ST = J / 2;
        kr[J] = lds_read_b128_async_off<128 * (ST / 2)>(KB == 0 ? kb0[ST % 2] : kb1[ST % 2]);
      } else if constexpr (J < TOT) {
        constexpr int V = J - NK, D = V / 2, HH = V % 2;
        vr[V] = lds_read_tr16_async_off<128 * (D / 4)>(slot + v_lane[D % 4][HH]);
      }
    };
    static_for<0, RW>(issue_read);
    // S^T = K Q^T: lane holds keys 16 kb + 4 gq + r of head c16
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) sacc[kb][r] = 0.f;
    static_for<0, NK>([&](auto i_tag) {
      constexpr int I = decltype(i_tag)::value;
      constexpr int AHEAD = (I + RW < TOT ? I + RW : TOT) - I - 1;
      lds_wait_lgkm<AHEAD>();
      lds_ready(kr[I]);
      sacc[I % 2] = mfma16(as_bf16x8(kr[I]), qf[I / 2], sacc[I % 2]);
      issue_read(std::integral_constant<int, I + RW>());
    });
    // online softmax over the keys of head c16 (every wave the same)
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = sacc[kb][r] * c;
        if (key0 + kb * 16 + 4 * gq + r >= cc.L) x = kNegInf;
        sacc[kb][r] = x;
        mx = fmaxf(mx, x);
      }
    mx = max_xor32(max_xor16(mx));
    if (__ballot(mx > m_run + kDecRescaleSlack)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = (m_new == kNegInf) ? 1.f : fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < S::DBLK_W; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) o_acc[db][r] *= alpha;
    }
    const float m_use = (m_run == kNegInf) ? 0.f : m_run;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = fast_exp2(sacc[kb][r] - m_use);
        sacc[kb][r] = p;
        l_run += p;
      }
    // P^T: k-group gq holds keys {4 gq .. +3} and {16 + 4 gq .. +3}
    const bf16x8 pf = to_bf16x8(sacc[0][0], sacc[0][1], sacc[0][2], sacc[0][3], sacc[1][0],
                                sacc[1][1], sacc[1][2], sacc[1][3]);
    // O^T[this wave's dims] += V^T P^T
    static_for<0, S::DBLK_W>([&](auto d_tag) {
      constexpr int d = decltype(d_tag)::value;
      constexpr int BASE = NK + 2 * d;  // stream index of its low read
      constexpr int AHEAD = (BASE + RW < TOT ? BASE + RW : TOT) - (BASE + 1) - 1;
      lds_wait_lgkm<AHEAD>();
      lds_ready(vr[2 * d]);
      lds_ready(vr[2 * d + 1]);
      const u32x4 wv = {vr[2 * d][0], vr[2 * d][1], vr[2 * d + 1][0], vr[2 * d + 1][1]};
      o_acc[d] = mfma16(as_bf16x8(wv), pf, o_acc[d]);
      issue_read(std::integral_constant<int, BASE + RW>());
      issue_read(std::integral_constant<int, BASE + RW + 1>());
    });
  };

  // End of a piece: a whole sequence goes to O and LSE, a cut piece to the
  // part's workspace slot 0 (its first piece) or 1 (its last).
  auto finish_piece = [&](const DecCursor& cc, bool whole, int slot_i) {
    const float lsum = sum_xor32(sum_xor16(l_run));  // add the four k-groups
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    const float lse_v = lsum > 0.f ? (m_run + log2f(lsum)) * kLn2 : kNegInf;
    const int dim0 = wave * (S::DC / S::WAVES) + 4 * gq;
    if (whole) {
      const size_t row = (size_t)cc.b * S::H + c16;
      uint16_t* o = a.o + row * S::DC + dim0;
#pragma unroll
      for (int db = 0; db < S::DBLK_W; ++db) {
        const u32x2 wv = {(uint32_t)to_bf16_bits(o_acc[db][0] * inv) |
                              ((uint32_t)to_bf16_bits(o_acc[db][1] * inv) << 16),
                          (uint32_t)to_bf16_bits(o_acc[db][2] * inv) |
                              ((uint32_t)to_bf16_bits(o_acc[db][3] * inv) << 16)};
        *reinterpret_cast<u32x2*>(o + db * 16) = wv;
      }
      if (wave == 0 && gq == 0 && a.lse) a.lse[row] = lse_v;
    } else {
      const size_t pr = ((size_t)w * 2 + slot_i) * S::H + c16;
#pragma unroll
      for (int db = 0; db < S::DBLK_W; ++db) {
        const f32x4 wv = {o_acc[db][0] * inv, o_acc[db][1] * inv, o_acc[db][2] * inv,
                          o_acc[db][3] * inv};
        *reinterpret_cast<f32x4*>(a.o_part + pr * S::DC + dim0 + db * 16) = wv;
      }
      if (wave == 0 && gq == 0) a.lse_part[pr] = lse_v;
    }
    m_run = kNegInf;
    l_run = 0.f;
#pragma unroll
    for (int db = 0; db < S::DBLK_W; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) o_acc[db][r] = 0.f;
  };

  // ---- pipeline.  Stage j sits in slot j % 3, piece k's Q rows in Q
  // buffer k % 2.  Iteration j first issues stage j + 2 into the slot of
  // stage j - 1 (every wave left it at the barrier that ended iteration
  // j - 1), so three stages are in flight while the wave waits for stage j;
  // after a barrier (every wave's part of stage j has landed) a new piece's
  // Q rows are copied to registers and stage j is consumed; a barrier then
  // marks slot j % 3 and the Q copy done, and the Q rows of the piece that
  // stage j + 2 starts, if any, go out into the Q buffer of two pieces back.
  // Issue order: Q(0), DMA(0), DMA(1), Q(1), then per iteration DMA(j + 2),
  // Q(j + 2): the loads after stage j's (and its Q's) are DMA(j + 1),
  // Q(j + 1) and DMA(j + 2). ----
  constexpr int LKV = S::KV_PER_WAVE, LQ = S::Q_PER_WAVE;
  auto starts_piece = [](const DecCursor& c) { return c.t == 0; };
  DecCursor iss = cur;  // cursor of the last issued stage
  int iss_piece = 0;    // piece index of the last issued stage
  issue_q(cur.b, q_lds0);
  issue_stage(iss, slot_addr(0));
  bool q1 = false;  // stage j + 1 brought Q rows
  if (n_stages > 1) {
    dec_advance(iss, a);
    issue_stage(iss, slot_addr(1));
    if (starts_piece(iss)) {
      ++iss_piece;
      issue_q(iss.b, q_lds0 + (uint32_t)(iss_piece & 1) * S::Q_BYTES);
      q1 = true;
    }
  }
  bool piece_from_pair_start = cur.t == 0;
  bool first_piece = true;
  int piece = 0;
  int slot_c = 0;
  bool new_piece = true;  // stage j starts a piece
  for (int j = 0; j < n_stages; ++j) {
    const bool more2 = j + 2 < n_stages;
    if (more2) {
      dec_advance(iss, a);
      issue_stage(iss, slot_addr(slot_c == 0 ? 2 : slot_c - 1));
      if (q1)
        wait_vmcnt<2 * LKV + LQ>();
      else
        wait_vmcnt<2 * LKV>();
    } else if (j + 1 < n_stages) {
      if (q1)
        wait_vmcnt<LKV + LQ>();
      else
        wait_vmcnt<LKV>();
    } else {
      wait_vmcnt<0>();
    }
    barrier_no_fence();
    if (new_piece) load_q(q_lds0 + (uint32_t)(piece & 1) * S::Q_BYTES);
    consume(cur, slot_addr(slot_c));
    const bool pair_end = cur.t + 1 == cur.nt;
    if (pair_end || j + 1 == n_stages) {
      finish_piece(cur, piece_from_pair_start && pair_end, first_piece ? 0 : 1);
      first_piece = false;
      piece_from_pair_start = true;
    }
    lds_wait_lgkm<0>();
    barrier_no_fence();
    // Q rows of the piece stage j + 2 starts, into the buffer of piece
    // iss_piece - 2, whose rows every wave copied before the barrier
    bool q2 = false;
    if (more2 && starts_piece(iss)) {
      ++iss_piece;
      issue_q(iss.b, q_lds0 + (uint32_t)(iss_piece & 1) * S::Q_BYTES);
      q2 = true;
    }
    slot_c = slot_c == 2 ? 0 : slot_c + 1;
    new_piece = j + 1 < n_stages && pair_end;
    if (pair_end) ++piece;
    q1 = q2;
    if (j + 1 < n_stages) dec_advance(cur, a);
  }
}

}  // namespace mk
