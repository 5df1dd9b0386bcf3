// decode_kernel.hpp -- split-KV decode attention for gfx950, with the
// splits cut so that every wave streams the same number of cache bytes.
//
// The keys of every (batch, kv head) pair are cut into 32-key stages and
// the stages of all pairs are laid end to end, pair after pair (pair
// b * Hkv + g, its stages t = 0 .. ceil(L_b / 32) - 1).  This stream of T
// stages is cut into P equal parts, part w holding stages
// [floor(w T / P), floor((w + 1) T / P)), and each part is one single-wave
// workgroup.  However ragged the sequence lengths, the waves finish
// together; a split-per-sequence grid instead leaves the waves of short
// sequences idle while the long ones drain.
//
// Kernel 1 (dec_part_kernel).  A wave walks its part stage by stage, across
// pair boundaries, with two stages in flight: each stage's K rows, V rows
// and the pair's G query rows go HBM -> LDS with coalesced 1 KB wave loads
// (global_load_lds_dwordx4) into one of three private ring slots.  The G
// query heads of the pair are the columns of 16x16x32 MFMA blocks, so each
// cached byte is read once for all of them.  Every LDS read is inline
// assembly waited on right before its use, so no loaded register lives
// across an iteration.  Per piece of a pair the wave keeps an online
// softmax.  A pair lying wholly inside the part is written straight to O
// and LSE.  A piece cut by a part boundary (only a part's first and last
// piece can be) is one split of split-KV attention: its normalised output
// and natural-log LSE go to the part's workspace slot 0 (first piece) or 1
// (last piece).
//
// Paged cache (PAGED): K and V live in a pool of pages [n_pages, Hkv,
// page_size, D]; block_table [B, max_pages] lists the pages of sequence b
// in key order.  Pages hold a multiple of 16 keys, so each 16-key half of
// a stage lies in one page: the stage's two page numbers come through the
// scalar cache (consecutive entries of one table row share its lines) and
// each lane's 16-byte row chunk is addressed in its half's page.  The
// stream, the pieces and the merge are those of the contiguous cache.
//
// Kernel 2 (dec_close_kernel), one wave per part: the part that closes a
// cut pair (holds its last piece) recorded where the pair's pieces lie, and
// its wave merges them by log-sum-exp, LSE = log sum_i exp(LSE_i),
// O = sum_i exp(LSE_i - LSE) O_i, into the pair's G rows; sequences without
// keys get O = 0, LSE = -inf; every other row is left alone.  (The MLA
// decode merges with dec_merge_kernel, one wave per row.)
#pragma once

#include "mk_common.hpp"

namespace mk {

constexpr float kDecRescaleSlack = 8.0f;
constexpr int kDecStageKeys = 32;

struct DecArgs {
  const uint16_t* q;        // [B, Hq, D] bf16
  const uint16_t* kc;       // [B, Hkv, Smax, D] bf16
  const uint16_t* vc;
  uint16_t* o;              // [B, Hq, D] bf16
  float* lse;               // [B, Hq] or null
  float* o_part;            // [P, 2, G, D]
  float* lse_part;          // [P, 2, G]
  int* close_desc;          // [P, 4]: the cut pair a part closes (see dec_part_kernel)
  const int* kv_seqlens;    // [B]
  int B, Hq, Hkv, Smax, P;  // paged: Smax = max_pages * page_size
  float scale_log2;
  // paged cache only: kc / vc are page pools [n_pages, Hkv, page_size, D]
  const int* block_table;   // [B, max_pages]
  int page_size, max_pages, n_pages;
};

__device__ __forceinline__ int dec_stages_of_len(int L) {
  return (L + kDecStageKeys - 1) / kDecStageKeys;
}

__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

// First stage of part w, floor(w T / P), for T < 2^31 stages in
// P <= 2^20 parts.  w T is exact in double and the quotient is correctly
// rounded; when w T / P is not an integer its distance to the next
// integer (>= 1/P >= 2^-20) exceeds half an ulp of any value below 2^31
// (<= 2^-22), so the floor of the rounded quotient is the exact floor.
__device__ __forceinline__ int part_start(int w, int T, int P) {
  return (int)floor((double)w * (double)T / (double)P);
}

// Owner of stage s (0 <= s < T): the largest part w with
// floor(w T / P) <= s, i.e. w T < (s + 1) P, which is
// ceil((s + 1) P / T) - 1 (in [0, P - 1] since s + 1 <= T).  The ceiling is
// exact by the argument of part_start: (s + 1) P is exact in double, and a
// non-integer quotient lies >= 1/T >= 2^-31 from an integer while half an
// ulp of a value <= P <= 2^20 is <= 2^-33.
__device__ __forceinline__ int part_of(int s, int T, int P) {
  return (int)ceil((double)(s + 1) * (double)P / (double)T) - 1;
}

// Stage counts of sequences b0 + lane (0 past B) and their inclusive scan.
struct SeqChunk {
  int len, nt, incl;  // clamped length, its stages, inclusive scan of stages
};
__device__ __forceinline__ SeqChunk seq_chunk(const DecArgs& a, int b0) {
  const int b = b0 + (int)(threadIdx.x & 63);
  SeqChunk c;
  c.len = b < a.B ? clamp_len(a.kv_seqlens[b], a.Smax) : 0;
  c.nt = dec_stages_of_len(c.len);
  c.incl = wave_incl_scan(c.nt);
  return c;
}

// Value of lane j, known to the compiler as wave-uniform (a shuffle's
// result is not), so that what is computed from it stays in scalar
// registers and loads through it go through the scalar cache.
__device__ __forceinline__ int lane_value(int x, int j) {
  return __builtin_amdgcn_readfirstlane(__shfl(x, j, 64));
}

// Total stages T = Hkv * sum_b ceil(L_b / 32).
__device__ __forceinline__ int dec_total(const DecArgs& a, const SeqChunk& first) {
  int sum = lane_value(first.incl, 63);
  for (int b0 = 64; b0 < a.B; b0 += 64) sum += lane_value(seq_chunk(a, b0).incl, 63);
  return a.Hkv * sum;
}

// Length of sequence b for a wave-uniform b, read through the scalar cache
// (s_load): a vector load here would make the compiler wait for every
// cache load in flight before its use.
__device__ __forceinline__ int seq_len_uniform(const DecArgs& a, int b) {
  const __attribute__((address_space(4))) int* lens =
      (const __attribute__((address_space(4))) int*)a.kv_seqlens;
  return clamp_len(lens[b], a.Smax);
}

// Position of a wave in the stage stream.
struct DecCursor {
  int b, g, t;  // sequence, kv head, stage within the pair
  int nt;       // stages of each pair of sequence b
  int L;        // clamped length of sequence b
};

// Cursor at stage s (0 <= s < T): the sequence whose pairs hold s.
__device__ __forceinline__ DecCursor dec_locate(const DecArgs& a, const SeqChunk& first, int s) {
  int carry = 0;  // stages per kv head of the sequences before the chunk
  for (int b0 = 0; b0 < a.B; b0 += 64) {
    const SeqChunk c = b0 == 0 ? first : seq_chunk(a, b0);
    const int lo = a.Hkv * (carry + c.incl - c.nt);
    const unsigned long long hit = __ballot(s >= lo && s < lo + a.Hkv * c.nt);
    if (hit) {
      const int j = __builtin_ctzll(hit);
      DecCursor r;
      r.b = b0 + j;
      r.nt = lane_value(c.nt, j);
      r.L = lane_value(c.len, j);
      const int rem = s - lane_value(lo, j);  // < Hkv * nt
      r.g = rem / r.nt;
      r.t = rem - r.g * r.nt;
      return r;
    }
    carry += lane_value(c.incl, 63);
  }
  return DecCursor{0, 0, 0, 0, 0};  // not reached for s < T
}

// Next stage of the stream; callers never step past its end, so a
// following sequence with keys exists when the last pair of b is left.
__device__ __forceinline__ void dec_advance(DecCursor& c, const DecArgs& a) {
  if (++c.t < c.nt) return;
  c.t = 0;
  if (++c.g < a.Hkv) return;
  c.g = 0;
  do {
    ++c.b;
    c.L = seq_len_uniform(a, c.b);
  } while (c.L == 0);
  c.nt = dec_stages_of_len(c.L);
}

template <int D, int QBLOCKS>
struct DecShape {
  static constexpr int BN = kDecStageKeys;             // keys per stage
  static constexpr int STAGES = 3;                     // LDS ring slots
  static constexpr int CHUNKS = D / 8;                 // 16-byte chunks per row
  static constexpr int ROW_BYTES = D * 2;
  static constexpr int ROWS_PER_KB = 512 / D;          // rows per 1 KB wave load
  static constexpr int KV_BLOCKS = BN * ROW_BYTES / 1024;
  static constexpr int LOADS_PER_STAGE = 2 * KV_BLOCKS + QBLOCKS;
  static constexpr int KSTEPS = D / 32;                // 16x16x32 steps over the head dim
  static constexpr int DBLK = D / 16;                  // 16-row blocks of O^T
  static constexpr int TILE_BYTES = BN * ROW_BYTES;    // one tensor, one stage
  static constexpr int Q_OFF = 2 * TILE_BYTES;         // the pair's Q rows follow K and V
  static constexpr int SLOT_BYTES = 2 * TILE_BYTES + QBLOCKS * 1024;
  static constexpr int LDS_BYTES = STAGES * SLOT_BYTES;
  static constexpr int MAX_G = QBLOCKS * ROWS_PER_KB;  // query heads per kv head
  static_assert(MAX_G <= 16, "one 16-column MFMA block of query heads");
  static_assert(2 * LOADS_PER_STAGE < 64, "vmcnt range");
};

// Page holding table position pi of sequence b (wave-uniform, through the
// scalar cache), clamped into the pool.
__device__ __forceinline__ int page_uniform(const DecArgs& a, int b, int pi) {
  const __attribute__((address_space(4))) int* bt =
      (const __attribute__((address_space(4))) int*)a.block_table;
  const int p = bt[(size_t)b * a.max_pages + pi];
  return p < 0 ? 0 : (p >= a.n_pages ? a.n_pages - 1 : p);
}

template <int D, int QBLOCKS, bool PAGED>
__global__ __launch_bounds__(64) void dec_part_kernel(DecArgs a) {
  using S = DecShape<D, QBLOCKS>;
  constexpr int BN = S::BN;
  constexpr int RB = S::ROW_BYTES;
  __shared__ __attribute__((aligned(1024))) char kv_lds[S::LDS_BYTES];

  const int lane = threadIdx.x;
  const int c16 = lane & 15;  // MFMA column (query head of the group) / row (key)
  const int gq = lane >> 4;   // MFMA k-group
  const int G = a.Hq / a.Hkv;
  const int w = blockIdx.x;

  // ---- this part's stages [s0, s0 + n_stages) and the cursor at s0 ----
  const SeqChunk first = seq_chunk(a, 0);
  const int T = dec_total(a, first);
  const int s0 = part_start(w, T, a.P);
  const int n_stages = part_start(w + 1, T, a.P) - s0;
  // A part whose first piece ends a pair that began in an earlier part
  // closes that cut pair: it records the pair's first output row, the part
  // holding the pair's first stage and that piece's slot there, and T, so
  // that the merge kernel needs no stream geometry.  Every part writes its
  // record (flag bit 1 clear when it closes nothing).
  DecCursor cur = {0, 0, 0, 0, 0};
  int rec[4] = {0, 0, 0, T};
  if (n_stages > 0) {
    cur = dec_locate(a, first, s0);
    if (cur.t > 0 && cur.nt - cur.t <= n_stages) {
      const int A = s0 - cur.t;  // the pair's first stage
      const int w0 = part_of(A, T, a.P);
      rec[0] = cur.b * a.Hq + cur.g * G;
      rec[1] = w0;
      rec[2] = 2 | (A > part_start(w0, T, a.P) ? 1 : 0);
    }
  }
  if (lane == 0) {
    const u32x4 r = {(uint32_t)rec[0], (uint32_t)rec[1], (uint32_t)rec[2], (uint32_t)rec[3]};
    *reinterpret_cast<u32x4*>(a.close_desc + 4 * w) = r;
  }
  if (n_stages <= 0) return;

  // ---- stage loads: slot <- K rows, V rows, then the pair's Q rows, each
  // row's 16-byte chunks XOR-swizzled.  K/V rows past the sequence end
  // re-read its last row (the mask zeroes their weight) and Q rows past G
  // re-read row G-1, so no load leaves the caller's valid data.
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(kv_lds));
  const int dma_row = lane / S::CHUNKS;
  auto issue = [&](const DecCursor& c, uint32_t slot) {
    const int key0 = c.t * BN;
    const int lim = c.L - 1 - key0;  // last valid row of the stage
    if constexpr (PAGED) {
      // pages of rows [0, 16) and [16, 32) (the second is the first when the
      // stage ends in its first half)
      const int ps = a.page_size;
      const int pi0 = key0 / ps;
      const int pi1 = min(key0 + 16, c.L - 1) / ps;
      const size_t head0 = ((size_t)page_uniform(a, c.b, pi0) * a.Hkv + c.g) * ps;
      const size_t head1 = ((size_t)page_uniform(a, c.b, pi1) * a.Hkv + c.g) * ps;
      const int first0 = pi0 * ps, first1 = pi1 * ps;  // first key of each page
#pragma unroll
      for (int blk = 0; blk < S::KV_BLOCKS; ++blk) {
        const int r = dma_row + blk * S::ROWS_PER_KB;
        const int ch = ((lane % S::CHUNKS) ^ chunk_swz<D>(r)) * 16;
        const int rr = min(r, lim);
        const bool hi = rr >= 16;
        const size_t row = (hi ? head1 : head0) + (size_t)(key0 + rr - (hi ? first1 : first0));
        const size_t goff = row * RB + ch;
        load_lds16_at(reinterpret_cast<const char*>(a.kc) + goff, slot + blk * 1024);
        load_lds16_at(reinterpret_cast<const char*>(a.vc) + goff,
                      slot + S::TILE_BYTES + blk * 1024);
      }
    } else {
      const size_t kv_off = (((size_t)c.b * a.Hkv + c.g) * (size_t)a.Smax + key0) * RB;
      const char* kt_g = reinterpret_cast<const char*>(a.kc) + kv_off;
      const char* vt_g = reinterpret_cast<const char*>(a.vc) + kv_off;
#pragma unroll
      for (int blk = 0; blk < S::KV_BLOCKS; ++blk) {
        const int r = dma_row + blk * S::ROWS_PER_KB;
        const int ch = ((lane % S::CHUNKS) ^ chunk_swz<D>(r)) * 16;
        const uint32_t goff = (uint32_t)(min(r, lim) * RB + ch);
        load_lds16_buf(kt_g, S::TILE_BYTES, goff, slot + blk * 1024);
        load_lds16_buf(vt_g, S::TILE_BYTES, goff, slot + S::TILE_BYTES + blk * 1024);
      }
    }
    const char* q_g = reinterpret_cast<const char*>(a.q) + ((size_t)c.b * a.Hq + c.g * G) * RB;
#pragma unroll
    for (int blk = 0; blk < QBLOCKS; ++blk) {
      const int r = dma_row + blk * S::ROWS_PER_KB;
      const int ch = ((lane % S::CHUNKS) ^ chunk_swz<D>(r)) * 16;
      load_lds16_buf(q_g, (uint32_t)(G * RB), (uint32_t)(min(r, G - 1) * RB + ch),
                     slot + S::Q_OFF + blk * 1024);
    }
  };

  // ---- lane parts of the LDS read addresses within a slot ----
  // K: row 16 kb + c16, logical chunk 4 s + gq.  Q: row min(c16, G-1),
  // same chunks (columns c16 >= G are zeroed after the read).
  // V (transposing): rows 4 gq + c16/4 (+ 16), columns 16 db + 4 (c16 % 4).
  uint32_t k_addr[2][S::KSTEPS], q_addr[S::KSTEPS];
  const int q_row = min(c16, G - 1);
#pragma unroll
  for (int s = 0; s < S::KSTEPS; ++s) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int r = kb * 16 + c16;
      k_addr[kb][s] = r * RB + (((4 * s + gq) ^ chunk_swz<D>(r)) << 4);
    }
    q_addr[s] = S::Q_OFF + q_row * RB + (((4 * s + gq) ^ chunk_swz<D>(q_row)) << 4);
  }
  uint32_t v_addr[S::DBLK][2];
  {
    const int tr_row = 4 * gq + (c16 >> 2);
    const int tr_col = 4 * (c16 & 3);
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int r = tr_row + 16 * hh;
        const int col = db * 16 + tr_col;
        v_addr[db][hh] = S::TILE_BYTES + r * RB +
                         ((((col >> 3) ^ chunk_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o_acc[S::DBLK];
#pragma unroll
  for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) o_acc[db][r] = 0.f;
  const float c = a.scale_log2;

  auto consume = [&](const DecCursor& cc, uint32_t slot) {
    const int key0 = cc.t * BN;
    // Q^T fragments: column c16 is query head g*G + c16 (zero for c16 >= G).
    u32x4 qr[S::KSTEPS];
#pragma unroll
    for (int s = 0; s < S::KSTEPS; ++s) qr[s] = lds_read_b128_async_off<0>(slot + q_addr[s]);
    static_assert(S::KSTEPS == 2 || S::KSTEPS == 4, "head dim 64 or 128");
    if constexpr (S::KSTEPS == 4)
      lds_wait_b128x4(qr[0], qr[1], qr[2], qr[3]);
    else
      lds_wait_b128x2(qr[0], qr[1]);
    bf16x8 qf[S::KSTEPS];
#pragma unroll
    for (int s = 0; s < S::KSTEPS; ++s) {
      const u32x4 zero = {0u, 0u, 0u, 0u};
      qf[s] = as_bf16x8(c16 < G ? qr[s] : zero);
    }
    // S^T = K Q^T for the 32 keys of the stage (two 16-key blocks).
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      u32x4 kf[S::KSTEPS];
#pragma unroll
      for (int s = 0; s < S::KSTEPS; ++s) kf[s] = lds_read_b128_async_off<0>(slot + k_addr[kb][s]);
      if constexpr (S::KSTEPS == 4)
        lds_wait_b128x4(kf[0], kf[1], kf[2], kf[3]);
      else
        lds_wait_b128x2(kf[0], kf[1]);
#pragma unroll
      for (int r = 0; r < 4; ++r) sacc[kb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < S::KSTEPS; ++s) sacc[kb] = mfma16(as_bf16x8(kf[s]), qf[s], sacc[kb]);
    }
    // Online softmax over the column (query head); lane holds keys
    // 16 kb + 4 gq + r of the stage.
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
      for (int db = 0; db < S::DBLK; ++db)
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
    // P^T: k-group gq holds keys {4gq..4gq+3} and {16+4gq..16+4gq+3}.
    const bf16x8 pf = to_bf16x8(sacc[0][0], sacc[0][1], sacc[0][2], sacc[0][3], sacc[1][0],
                                sacc[1][1], sacc[1][2], sacc[1][3]);
#pragma unroll
    for (int db0 = 0; db0 < S::DBLK; db0 += 2) {
      u32x2 vr[2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) vr[j][hh] = lds_read_tr16_async(slot + v_addr[db0 + j][hh]);
      lds_wait4(vr[0][0], vr[0][1], vr[1][0], vr[1][1]);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const u32x4 wv = {vr[j][0][0], vr[j][0][1], vr[j][1][0], vr[j][1][1]};
        o_acc[db0 + j] = mfma16(as_bf16x8(wv), pf, o_acc[db0 + j]);
      }
    }
  };

  // End of a piece: a whole pair goes to O and LSE, a cut piece to the
  // part's workspace slot 0 (its first piece) or 1 (its last); then the
  // softmax state restarts.
  auto finish_piece = [&](const DecCursor& cc, bool whole, int slot_i) {
    const float lsum = sum_xor32(sum_xor16(l_run));  // add the four k-groups
    if (c16 < G) {
      const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
      const float lse_v = lsum > 0.f ? (m_run + log2f(lsum)) * kLn2 : kNegInf;
      if (whole) {
        const size_t row = (size_t)cc.b * a.Hq + cc.g * G + c16;
        uint16_t* o = a.o + row * D + 4 * gq;
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db) {
          const u32x2 wv = {(uint32_t)to_bf16_bits(o_acc[db][0] * inv) |
                                ((uint32_t)to_bf16_bits(o_acc[db][1] * inv) << 16),
                            (uint32_t)to_bf16_bits(o_acc[db][2] * inv) |
                                ((uint32_t)to_bf16_bits(o_acc[db][3] * inv) << 16)};
          *reinterpret_cast<u32x2*>(o + db * 16) = wv;
        }
        if (gq == 0 && a.lse) a.lse[row] = lse_v;
      } else {
        const size_t pr = ((size_t)w * 2 + slot_i) * G + c16;
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db) {
          const f32x4 wv = {o_acc[db][0] * inv, o_acc[db][1] * inv, o_acc[db][2] * inv,
                            o_acc[db][3] * inv};
          *reinterpret_cast<f32x4*>(a.o_part + pr * D + db * 16 + 4 * gq) = wv;
        }
        if (gq == 0) a.lse_part[pr] = lse_v;
      }
    }
    m_run = kNegInf;
    l_run = 0.f;
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) o_acc[db][r] = 0.f;
  };

  // ---- pipeline: stage j sits in ring slot j % 3 and is issued two
  // stages ahead of its use ----
  static_assert(S::STAGES == 3, "the wait counts below assume two stages ahead");
  auto slot_addr = [&](int k) { return lds0 + (uint32_t)k * S::SLOT_BYTES; };
  DecCursor iss = cur;  // cursor of the last issued stage
  issue(iss, slot_addr(0));
  if (n_stages > 1) {
    dec_advance(iss, a);
    issue(iss, slot_addr(1));
  }
  bool piece_from_pair_start = cur.t == 0;
  bool first_piece = true;
  int slot_c = 0;  // ring slot of stage j
  for (int j = 0; j < n_stages; ++j) {
    // Before stage j is read only the stages issued after it may still be
    // loading.  Slot (j+2) % 3 held stage j-1, whose reads completed in the
    // previous iteration.
    if (j + 2 < n_stages) {
      dec_advance(iss, a);
      issue(iss, slot_addr(slot_c == 0 ? 2 : slot_c - 1));
      wait_vmcnt<2 * S::LOADS_PER_STAGE>();
    } else if (j + 1 < n_stages) {
      wait_vmcnt<S::LOADS_PER_STAGE>();
    } else {
      wait_vmcnt<0>();
    }
    consume(cur, slot_addr(slot_c));
    slot_c = slot_c == 2 ? 0 : slot_c + 1;
    const bool pair_end = cur.t + 1 == cur.nt;
    if (pair_end || j + 1 == n_stages) {
      finish_piece(cur, piece_from_pair_start && pair_end, first_piece ? 0 : 1);
      first_piece = false;
      piece_from_pair_start = true;
    }
    if (j + 1 < n_stages) dec_advance(cur, a);
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// One wave per (batch, query head) row.  After the stream geometry (one
// round of length loads), every load the merge needs -- the LSEs of the
// row's pieces (lane i: piece i) and the partial outputs of its first
// CHUNK pieces (lanes: head dims) -- is issued before any is used, so a
// cut row costs about two memory round trips and an uncut row one.
// N consecutive floats (N * 4 bytes aligned to min(16, N * 4)) into x.
template <int N>
__device__ __forceinline__ void load_row_part(const float* p, float (&x)[N]) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int j = 0; j < N / 4; ++j) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(p + 4 * j);
#pragma unroll
      for (int k = 0; k < 4; ++k) x[4 * j + k] = v[k];
    }
  } else {
#pragma unroll
    for (int k = 0; k < N; ++k) x[k] = p[k];
  }
}

template <int D>
__global__ __launch_bounds__(256) void dec_merge_kernel(DecArgs a) {
  constexpr int PER_LANE = D / 64;
  // pieces whose partial outputs are loaded together (fewer at wide rows,
  // to bound the registers they take)
  constexpr int CHUNK = PER_LANE > 2 ? 8 : 16;
  const int lane = threadIdx.x & 63;
  // b * Hq + hq (wave-uniform: scalar registers, scalar loads)
  const int row = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= a.B * a.Hq) return;
  const int b = row / a.Hq;
  const int hq = row - b * a.Hq;
  const int G = a.Hq / a.Hkv;
  const int g = hq / G;
  const int h = hq - g * G;
  const SeqChunk first = seq_chunk(a, 0);
  const int L = seq_len_uniform(a, b);
  uint16_t* o = a.o + (size_t)row * D + lane * PER_LANE;
  if (L == 0) {
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) o[i] = 0;
    if (lane == 0 && a.lse) a.lse[row] = kNegInf;
    return;
  }
  // stages [A, A + nt) of pair (b, g): A = Hkv * (stages per kv head of
  // the sequences before b) + g * nt
  const int T = dec_total(a, first);
  int before = 0;
  for (int b0 = 0; b0 < b; b0 += 64) {
    const SeqChunk c = b0 == 0 ? first : seq_chunk(a, b0);
    const int k = b - b0 - 1;  // last sequence of the chunk before b
    before += lane_value(c.incl, k < 63 ? k : 63);
  }
  const int nt = dec_stages_of_len(L);
  const int A = a.Hkv * before + g * nt;
  const int wa = part_of(A, T, a.P);
  const int we = part_of(A + nt - 1, T, a.P);
  if (wa == we) return;  // one part held the whole pair and wrote it
  // Piece i of the pair lies in part wa + i.  The first is part wa's last
  // piece (slot 1) unless that part starts with the pair; every later one
  // starts its part (slot 0).  Parts without stages hold no piece.
  const int n_pc = we - wa + 1;
  const int slot_a = A > part_start(wa, T, a.P) ? 1 : 0;
  auto entry = [&](int i) {
    const int w = wa + i;
    return ((size_t)w * 2 + (i == 0 ? slot_a : 0)) * G + h;
  };
  // with T >= P every part holds at least floor(T / P) >= 1 stages
  const bool all_hold = T >= a.P;
  auto holds = [&](int i) {
    const int w = wa + i;
    return all_hold || part_start(w, T, a.P) < part_start(w + 1, T, a.P);
  };
  const bool lane_holds = lane < n_pc && holds(lane);
  const unsigned long long held = __ballot(lane_holds);  // pieces 0..63
  const float ls0 = lane_holds ? a.lse_part[entry(lane)] : kNegInf;
  // The first CHUNK pieces' partial outputs, loaded together.  A piece that
  // is not held gets weight 0 below; its load reads piece 0 (always held:
  // its part contains the pair's first stage), so every load is a plain
  // vector load with no branch around it.
  float part[CHUNK][PER_LANE];
#pragma unroll
  for (int i = 0; i < CHUNK; ++i) {
    const bool use = (held >> i) & 1;
    load_row_part<PER_LANE>(a.o_part + entry(use ? i : 0) * D + lane * PER_LANE, part[i]);
  }
  float M = ls0;
  for (int i = 64 + lane; i < n_pc; i += 64)
    if (holds(i)) M = fmaxf(M, a.lse_part[entry(i)]);
  M = wave_max(M);
  float sum = expf(ls0 - M);
  for (int i = 64 + lane; i < n_pc; i += 64)
    if (holds(i)) sum += expf(a.lse_part[entry(i)] - M);
  const float lse = M + logf(wave_sum(sum));
  const float w_lane = expf(ls0 - lse);  // weight of piece `lane` (0 if none)
  float out[PER_LANE];
#pragma unroll
  for (int k = 0; k < PER_LANE; ++k) out[k] = 0.f;
#pragma unroll
  for (int i = 0; i < CHUNK; ++i) {
    const float wt = __shfl(w_lane, i, 64);
#pragma unroll
    for (int k = 0; k < PER_LANE; ++k) out[k] += wt * part[i][k];
  }
  for (int i = CHUNK; i < n_pc; ++i) {
    if (!(i < 64 ? (held >> i) & 1 : holds(i))) continue;
    const float wt = expf(a.lse_part[entry(i)] - lse);
#pragma unroll
    for (int k = 0; k < PER_LANE; ++k) out[k] += wt * a.o_part[entry(i) * D + lane * PER_LANE + k];
  }
#pragma unroll
  for (int k = 0; k < PER_LANE; ++k) o[k] = to_bf16_bits(out[k]);
  if (lane == 0 && a.lse) a.lse[row] = lse;
}


// One wave per part w (see kernel 2 above).  Each lane takes 16-byte
// chunks of the pair's G x D block of outputs (chunk c: head 4c / D, head
// dims 4c % D .. +3) and merges the pieces online, in order, eight at a
// time with all their loads issued before any is used:
//   M' = max(M, LSE_i),  S = S 2^.. + exp(LSE_i - M'),  acc likewise,
// then O = acc / S and LSE = M' + log S.
template <int D>
__global__ __launch_bounds__(256) void dec_close_kernel(DecArgs a) {
  constexpr int BATCH = 8;  // pieces whose loads are issued together
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (w >= a.P) return;
  const int G = a.Hq / a.Hkv;
  // the record, through the scalar cache
  const __attribute__((address_space(4))) int* rp =
      (const __attribute__((address_space(4))) int*)(a.close_desc + 4 * w);
  const int row0 = rp[0], w0 = rp[1], flags = rp[2], T = rp[3];

  // sequences without keys: b = w, w + P, ...
  for (int b = w; b < a.B; b += a.P) {
    if (seq_len_uniform(a, b) != 0) continue;
    uint16_t* o = a.o + (size_t)b * a.Hq * D;
    for (int i = lane; i < a.Hq * D / 8; i += 64)
      *reinterpret_cast<u32x4*>(o + 8 * i) = u32x4{0u, 0u, 0u, 0u};
    if (a.lse)
      for (int i = lane; i < a.Hq; i += 64) a.lse[(size_t)b * a.Hq + i] = kNegInf;
  }
  if (!(flags & 2)) return;

  // pieces: i = 0 in part w0 (slot flags & 1), i >= 1 in part w0 + i
  // (slot 0); with fewer stages than parts some parts hold none
  const int n_pc = w - w0 + 1;
  const int slot_a = flags & 1;
  const bool all_hold = T >= a.P;
  auto entry = [&](int i) {  // (part, slot) row of piece i in the workspace
    return (size_t)(w0 + i) * 2 + (i == 0 ? slot_a : 0);
  };
  auto holds = [&](int i) {
    const int p = w0 + i;
    return all_hold || part_start(p, T, a.P) < part_start(p + 1, T, a.P);
  };
  const int n_chunks = G * D / 4;
  for (int c = lane; c < n_chunks; c += 64) {
    const int h = (4 * c) / D;
    const int d0 = 4 * c - h * D;
    float M = kNegInf, S = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int i0 = 0; i0 < n_pc; i0 += BATCH) {
      float ls[BATCH];
      f32x4 ov[BATCH];
#pragma unroll
      for (int j = 0; j < BATCH; ++j) {
        // a piece past the pair or in an empty part reads piece 0 and
        // weighs nothing
        const bool use = i0 + j < n_pc && holds(i0 + j);
        const size_t e = entry(use ? i0 + j : 0) * G + h;
        ls[j] = a.lse_part[e];
        ov[j] = *reinterpret_cast<const f32x4*>(a.o_part + e * D + d0);
        if (!use) ls[j] = kNegInf;
      }
#pragma unroll
      for (int j = 0; j < BATCH; ++j) {
        const float m_new = fmaxf(M, ls[j]);
        if (m_new == kNegInf) continue;  // nothing weighed yet
        const float f_old = __expf(M - m_new);
        const float f_new = __expf(ls[j] - m_new);
        S = S * f_old + f_new;
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[k] = acc[k] * f_old + f_new * ov[j][k];
        M = m_new;
      }
    }
    const float inv = S > 0.f ? 1.f / S : 0.f;
    const u32x2 wv = {(uint32_t)to_bf16_bits(acc[0] * inv) |
                          ((uint32_t)to_bf16_bits(acc[1] * inv) << 16),
                      (uint32_t)to_bf16_bits(acc[2] * inv) |
                          ((uint32_t)to_bf16_bits(acc[3] * inv) << 16)};
    *reinterpret_cast<u32x2*>(a.o + (size_t)(row0 + h) * D + d0) = wv;
    if (d0 == 0 && a.lse) a.lse[row0 + h] = S > 0.f ? M + logf(S) : kNegInf;
  }
}

}  // namespace mk
