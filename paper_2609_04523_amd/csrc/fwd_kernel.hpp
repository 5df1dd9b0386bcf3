// fwd_kernel.hpp -- fused attention forward (prefill) for gfx950.
//
// A work item = BM query rows (a q-tile) of one (batch, query head), taken
// by one workgroup of WAVES waves (4; 8 on the V^T path); wave w owns QB
// blocks of 32 consecutive rows.  The workgroup streams the 64-key K and V
// tiles of its KV head (hq / (Hq/Hkv)) from HBM straight into LDS (LDS-DMA
// loads, double-buffered), up to the causal diagonal, and keeps the softmax
// state and the output accumulator in registers: online softmax, an exact
// rewrite of softmax(Q K^T * scale) V folded tile by tile.  A workgroup
// takes one item (its own index), or with PERSIST works through queues of
// items.
//
// Orientation.  Scores are formed transposed, S^T = K Q^T, with K as the
// MFMA A operand (rows = keys) and Q^T as the B operand (columns =
// queries).  A lane then owns one query column, so the softmax row
// reductions are in-lane plus one exchange with lane l^32.  The output is
// O^T = V^T P^T: P^T is the score accumulator converted to bf16 in place
// (its key order is the accumulator's own row order), and the V^T operand
// is read from the row-major V tile with the transposing LDS read -- or,
// with VT, from a copy of V that a pre-pass wrote tile by tile in the
// operand's own layout, with plain 16-byte LDS reads (which the LDS serves
// at twice the rate of the transposing ones).
//
// Softmax bookkeeping (exp2 domain, c = scale * log2 e):
//   m    running row maximum of c*s, raised only when a tile's maximum
//        exceeds it by more than kRescaleSlack, so exp2(c*s - m) <= 2^8 and
//        the O accumulator is rescaled on few tiles.  The first tile and
//        masked tiles take their row maximum; the other tiles are weighed
//        against m directly, and one whose weights sum past 2^8 in any lane
//        (scores that rose steeply) is formed again against its maximum;
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
  int xcd_gp;         // > 0: xcd_pair_map order with groups of xcd_gp pairs; 0: plain order
  float scale_log2;   // scale * log2(e)
  // packed ragged batches only: q, o [total_q, Hq, D], k, v [total_k, Hkv, D],
  // sequence b = query tokens [cu_q[b], cu_q[b+1]), keys [cu_k[b], cu_k[b+1]),
  // lse [Hq, total_q]; Sq is then the largest query length
  const int* cu_q;
  const int* cu_k;
  int total_q, total_k;
  // packed queries over a paged cache (PAGED) only: k, v are page pools
  // [n_pages, Hkv, page_size, D]; key j of sequence b is row j % page_size
  // of page block_table[b][j / page_size]; sequence b has kv_seqlens[b] keys
  const int* block_table;
  int page_size, max_pages, n_pages;
  // r / page_size = (r * ps_magic) >> ps_shift for 0 <= r < 2^31
  // (ps_magic = floor(2^ps_shift / page_size) + 1, ps_shift = 31 +
  // ceil(log2 page_size): exact for 31-bit dividends)
  uint64_t ps_magic;
  int ps_shift;
  int tile_in_page;  // page_size % 64 == 0: a 64-key tile lies in one page
  // VT only: the V^T tiles of vt_pack_kernel, [B, Hkv, vt_tiles, 4, D, 16]
  // bf16 (vt_tiles = ceil(Skv / 64))
  const uint16_t* vt;
  int vt_tiles;
  // PERSIST only: work-item queues.  Queue x (x < n_queues) holds the items
  // bid = n_queues * i + x, i < per_queue, in fwd_map_block's order; its
  // counter ctr[32 x] (set to the grid's share per queue before the launch:
  // workgroup bid takes item bid first) hands out i.
  int* ctr;
  int n_queues, per_queue;
};

// Tokens [start, end) of sequence b from cumulative offsets, clamped into
// [0, total] and non-decreasing, so no offset can lead outside the tensor.
__device__ __forceinline__ void fwd_seq_range(const int* cu, int b, int total, int& start,
                                              int& len) {
  const int s0 = clamp_len(cu[b], total);
  const int s1 = clamp_len(cu[b + 1], total);
  start = s0;
  len = s1 > s0 ? s1 - s0 : 0;
}

template <int D, int QB, int WAVES_ = 4>
struct FwdShape {
  static constexpr int WAVES = WAVES_;
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
// A tile whose weights were formed against the running maximum without its
// own is accepted when every lane's share of each row's weights sums to at
// most 2^kRescaleSlack (so no weight exceeds it); otherwise its scores are
// formed again and the tile is weighed against their maximum.
constexpr float kSumLimit = 256.0f;

// Work-item order.  Longest causal q-tiles are issued first.  When the
// number of (batch, kv head) pairs is a multiple of 8, the pairs are placed
// on the XCDs (xcd_pair_map), so the query heads and q-tiles that re-read
// one K/V head share that XCD's L2.
__device__ __forceinline__ void fwd_map_block(int bid, const FwdArgs& a, int& qt, int& hq,
                                              int& b) {
  if (a.xcd_gp > 0) {
    xcd_pair_map(bid, a.n_qtiles, a.B, a.Hkv, a.Hq / a.Hkv, a.xcd_gp, qt, b, hq);
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
// first (scale 0 and negative scales).  VARLEN: a packed ragged batch (see
// FwdArgs); only where rows live changes, the tile pipeline is the same.
// PAGED (with VARLEN): the keys and values of the packed queries' sequences
// come from a paged cache; each wave's 1 KB block of a tile is 4 (D = 128)
// or 8 (D = 64) consecutive key rows, which lie in one page since pages
// hold a multiple of 16 keys, so the page of every block is one table
// entry, read through the scalar cache at the start of the step.
// VT (dense batches only): the V tiles come from the pre-pass's V^T tiles
// (contiguous 64-key blocks of D * 128 bytes, copied to LDS as they are) and
// the products read them with ds_read_b128.
// PERSIST (with VT): a grid of one workgroup per compute unit works through
// the items of FwdArgs' queues: workgroup bid first takes item bid, then
// items of its own queue (the K/V heads its XCD holds), then of the others
// once its own is empty, so XCDs that run ahead take over the rest of the
// slower ones' work.  The next item's Q and first K tile are loaded while
// the current one's output goes out, through an LDS area of its own.
template <int D, bool CAUSAL, bool OUT_F32, int QB, bool POS_SCALE, bool VARLEN, int WAVES,
          bool PAGED = false, bool VT = false, bool PERSIST = false>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void fwd_kernel(FwdArgs a) {
  static_assert(VARLEN || !PAGED, "the paged cache is read by the packed forward");
  static_assert(!(VT && VARLEN), "the V^T copy is made for dense batches");
  static_assert(!PERSIST || (VT && !OUT_F32), "the persistent grid runs the V^T path");
  using S = FwdShape<D, QB, WAVES>;
  constexpr int BN = S::BN;
  constexpr int TILE = BN * D;            // bf16 per tile per tensor
  constexpr int TILE_BYTES = TILE * 2;
  constexpr int ROW_BYTES = D * 2;
  constexpr int NK = 2 * S::KSTEPS;     // K fragment reads per tile
  constexpr int RPP = VT ? 1 : 2;       // LDS reads per V^T operand
  constexpr int NV = 4 * RPP * S::DBLK;  // V reads per tile
  // LDS reads in flight (fewer where the registers are needed elsewhere;
  // the V^T path's 16-byte V reads need half as many for the same bytes)
  constexpr int RW = POS_SCALE && !PAGED && !VT ? 8 : 4;
  static_assert(RW >= 2 && RW % 2 == 0 && RW <= NK && RW <= NV, "read window");
  // K tile buffers 0 and 1, then V tile buffers 0 and 1, contiguous (the
  // epilogue stages the output rows of all waves through them)
  __shared__ __attribute__((aligned(1024))) uint16_t kv_lds[4][TILE];
  uint16_t(*const k_lds)[TILE] = kv_lds;
  uint16_t(*const v_lds)[TILE] = kv_lds + 2;
  static_assert(S::WAVES * 32 * QB * D * 2 <= 4 * TILE_BYTES, "output staging fits the tiles");
  // PERSIST: the output rows' staging area (each wave its own 32 rows), and
  // the next work item as claimed by thread 0, by item parity
  __shared__ __attribute__((aligned(16))) uint16_t o_stage[PERSIST ? S::WAVES * 32 * D : 8];
  __shared__ int next_item[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;  // MFMA column (query) / row (key) within a 32-block
  const int h = lane >> 5;  // MFMA k-group

  const int G = a.Hq / a.Hkv;
  // The work item: query tile qt of (b, hq), kv head g.  Where its rows
  // live: query / output row i at q_base + i * q_stride (elements), key /
  // value row j at byte j * kv_stride from kg / vg, LSE of row i at
  // lse_base[i].
  int qt, hq, b, g, Sq, L;
  const uint16_t* q_base;
  size_t o_base, q_stride, kv_stride;
  float* lse_base;
  const char* kg;
  const char* vg;
  int off, q0, n_kt, n_full, qw0, n_free, n_live;
  // Sets the item's geometry; false when the item holds no query rows (a
  // q-tile past its sequence's queries in a packed batch).
  auto setup = [&](int bid) -> bool {
    fwd_map_block(bid, a, qt, hq, b);
    g = hq / G;
    lse_base = a.lse;
    if constexpr (VARLEN) {
      int qs, ks = 0;
      fwd_seq_range(a.cu_q, b, a.total_q, qs, Sq);
      if constexpr (PAGED)
        L = clamp_len(a.kv_seqlens[b], a.max_pages * a.page_size);
      else
        fwd_seq_range(a.cu_k, b, a.total_k, ks, L);
      if (qt * S::BM >= Sq) return false;  // past this sequence's queries
      o_base = ((size_t)qs * a.Hq + hq) * D;
      q_stride = (size_t)a.Hq * D;
      if (lse_base) lse_base += (size_t)hq * a.total_q + qs;
      if constexpr (PAGED) {
        // rows of one head inside a page are consecutive; kg / vg point at
        // head g of page 0 (page p adds p * Hkv * page_size rows)
        kv_stride = ROW_BYTES;
        const size_t kv_off = (size_t)g * a.page_size * D;
        kg = reinterpret_cast<const char*>(a.k + kv_off);
        vg = reinterpret_cast<const char*>(a.v + kv_off);
      } else {
        kv_stride = (size_t)a.Hkv * ROW_BYTES;
        const size_t kv_off = ((size_t)ks * a.Hkv + g) * D;
        kg = reinterpret_cast<const char*>(a.k + kv_off);
        vg = reinterpret_cast<const char*>(a.v + kv_off);
      }
    } else {
      Sq = a.Sq;
      L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
      const size_t q_row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
      o_base = q_row0 * D;
      q_stride = D;
      kv_stride = ROW_BYTES;
      if (lse_base) lse_base += q_row0;
      const size_t kv_off = ((size_t)b * a.Hkv + g) * (size_t)a.Skv * D;
      kg = reinterpret_cast<const char*>(a.k + kv_off);
      vg = reinterpret_cast<const char*>(
          VT ? a.vt + ((size_t)b * a.Hkv + g) * a.vt_tiles * (size_t)TILE : a.v + kv_off);
    }
    q_base = a.q + o_base;
    off = L - Sq;  // bottom-right causal alignment
    q0 = qt * S::BM;
    const int q_end = min(q0 + S::BM, Sq);
    int n_keys = L;
    if (CAUSAL) n_keys = min(L, q_end + off);
    if (n_keys < 0) n_keys = 0;
    n_kt = (n_keys + BN - 1) / BN;
    n_full = L / BN;  // tiles that lie wholly inside the sequence
    qw0 = q0 + wave * 32 * QB;
    // Tiles [0, n_free) need no mask for any row of this wave; tiles up to
    // n_live hold at least one admissible key for some row of the wave.
    const int w_first = qw0;  // first query row of the wave
    const int w_last = min(qw0 + 32 * QB, Sq) - 1;
    n_free = (CAUSAL ? min(L, w_first + off + 1) : L) / BN;
    n_live = qw0 < Sq ? (CAUSAL ? min(L, w_last + off + 1) : L) : 0;
    n_live = (max(n_live, 0) + BN - 1) / BN;
    n_free = max(0, min(n_free, n_live));
    return true;
  };
  if (!setup(blockIdx.x)) return;  // (the whole workgroup)
  const float c = a.scale_log2;

  // Q^T fragments: lane (column n, k-group h) holds q[row][16 s + 8 h .. +7].
  // Loaded before any K/V traffic so waiting for them waits for nothing else.
  bf16x8 qf[QB][S::KSTEPS];
  auto load_q = [&]() {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int row = qw0 + qb * 32 + n;
#pragma unroll
      for (int s = 0; s < S::KSTEPS; ++s) {
        u32x4 u = {0u, 0u, 0u, 0u};
        if (row < Sq)
          u = *reinterpret_cast<const u32x4*>(q_base + row * q_stride + s * 16 + h * 8);
        qf[qb][s] = as_bf16x8(u);
      }
    }
  };
  load_q();

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
  // Block p of tile kt of one tensor (K or V) into LDS buffer BUF.  FULL:
  // the tile lies inside the sequence, so no row needs clamping: the load
  // goes through a buffer resource on the tile with the lane offset
  // full_off and the block's (wave-uniform) offset p * ROW_STEP rows.
  const uint32_t full_off = (uint32_t)(dma_row * kv_stride + dma_ch);
  // PAGED: byte offset, from kg / vg, of key row r (the same in every lane)
  // of this sequence: row r % page_size of its page, the table entry read
  // through the scalar cache and clamped into the pool.
  auto page_row = [&](int r) -> size_t {
    const uint32_t ru = (uint32_t)__builtin_amdgcn_readfirstlane(r);
    const uint32_t pi = (uint32_t)(((uint64_t)ru * a.ps_magic) >> a.ps_shift);  // ru / page_size
    const __attribute__((address_space(4))) int* bt =
        (const __attribute__((address_space(4))) int*)(a.block_table + (size_t)b * a.max_pages);
    int pg = bt[pi];
    pg = pg < 0 ? 0 : (pg >= a.n_pages ? a.n_pages - 1 : pg);
    return ((size_t)pg * a.Hkv * a.page_size + (ru - pi * (uint32_t)a.page_size)) * ROW_BYTES;
  };
  // PAGED: a lane's byte offset within its wave's block (row, then chunk)
  const uint32_t paged_lane_off = (uint32_t)((lane / S::CHUNKS) * ROW_BYTES + dma_ch);
  // PAGED: first row this wave reads for block p of tile kt (its own block,
  // or the sequence's last row when the block lies wholly past it)
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // the same in every lane
  auto block_row = [&](int kt, int p) {
    const int r0 = kt * BN + (p * S::WAVES + wave_u) * S::ROWS_PER_KB;
    return r0 < L ? r0 : L - 1;
  };
  auto issue_rows = [&](const char* g, uint32_t lds_w, int kt, auto buf_tag, auto p_tag,
                        auto full_tag, size_t page_off = 0) {
    constexpr int BUF = decltype(buf_tag)::value;
    constexpr int P = decltype(p_tag)::value;
    constexpr uint32_t lds_off = BUF * TILE_BYTES + P * S::WAVES * 1024;
    if constexpr (PAGED) {
      // page_off = page_row(block_row(kt, P)): the wave's block through a
      // buffer resource on its rows in the page; a lane's row within the
      // block is clamped to the sequence's last row
      const char* blk = g + page_off;
      if constexpr (decltype(full_tag)::value) {
        load_lds16_buf(blk, S::ROWS_PER_KB * ROW_BYTES, paged_lane_off, lds_w + lds_off);
      } else {
        const int r0 = kt * BN + (P * S::WAVES + wave) * S::ROWS_PER_KB;
        const int lr = r0 < L ? min(lane / S::CHUNKS, L - 1 - r0) : 0;
        load_lds16_buf(blk, S::ROWS_PER_KB * ROW_BYTES, (uint32_t)(lr * ROW_BYTES + dma_ch),
                       lds_w + lds_off);
      }
      return;
    }
    // kt is the same in every lane; saying so keeps the tile address, and so
    // the load's buffer resource, in scalar registers
    const char* tile = g + (size_t)__builtin_amdgcn_readfirstlane(kt) * BN * kv_stride;
    if constexpr (decltype(full_tag)::value) {
      load_lds16_buf(tile, (uint32_t)(BN * kv_stride), full_off, lds_w + lds_off,
                     (uint32_t)(P * ROW_STEP * kv_stride));
    } else {
      const int lim = L - 1 - kt * BN;  // last valid row of the tile
      const uint32_t goff = (uint32_t)(min(dma_row, lim - P * ROW_STEP) * kv_stride + dma_ch) +
                            (uint32_t)(P * ROW_STEP * kv_stride);
      load_lds16_at(tile + goff, lds_w + lds_off);
    }
  };

  // VT: block p (1 KB at byte 1024 (4 p + wave)) of V^T tile kt into V
  // buffer BUF: the tile is contiguous and padded in the copy, so the
  // block is a plain 1 KB copy with no clamping.
  auto issue_vt = [&](int kt, auto buf_tag, auto p_tag) {
    constexpr int BUF = decltype(buf_tag)::value;
    constexpr int P = decltype(p_tag)::value;
    constexpr uint32_t lds_off = BUF * TILE_BYTES + P * S::WAVES * 1024;
    const char* tile = vg + (size_t)__builtin_amdgcn_readfirstlane(kt) * TILE_BYTES;
    load_lds16_buf(tile, TILE_BYTES, (uint32_t)(wave * 1024 + lane * 16), v_lds_w + lds_off,
                   (uint32_t)(P * S::WAVES * 1024));
  };

  float m_run[QB], l_run[QB];
  f32x16 o_acc[QB][S::DBLK];

  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  // the item's first K tile into K buffer 0
  auto issue_k0 = [&]() {
    if (n_kt > 0)
      static_for<0, S::BLOCKS_PER_WAVE>([&](auto p_tag) {
        issue_rows(kg, k_lds_w, 0, B0(), p_tag, std::false_type(),
                   PAGED ? page_row(block_row(0, decltype(p_tag)::value)) : 0);
      });
  };
  issue_k0();

  // Lane parts of the LDS read addresses (bytes within a tile).  K row
  // 32 kb + n: the swizzle of n + 32 kb equals that of n.  Transposing V
  // reads: rows 16 kc + 4 h + i/4 (+ 8), columns 32 db + 16 ((l/16) % 2) +
  // 4 (i % 4), i = l % 16; the swizzle does not depend on kc.
  uint32_t k_addr[S::KSTEPS];
#pragma unroll
  for (int s = 0; s < S::KSTEPS; ++s)
    k_addr[s] = lds_addr(&k_lds[0][0]) + n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
  // VT: a V^T tile is [4 key chunks][D head dims][16 keys]; the operand of
  // key chunk kc and head dims 32 db + n is the 16-byte half h ^ ((n / 8) % 2)
  // of row (kc, 32 db + n) (the halves of rows 8..15 of every 16 swapped, so
  // 16 lanes of one k-group hit 64 distinct banks).
  const uint32_t vt_addr = lds_addr(&v_lds[0][0]) + n * 32 + ((h ^ ((n >> 3) & 1)) << 4);
  uint32_t v_addr[S::DBLK][2];
  if constexpr (!VT) {
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

  // Scores (fp32) and weights (bf16 P^T fragments) of even and odd tiles.
  // Step t forms the scores of tile t, turns those of tile t - 1 into
  // weights and adds the weights of tile t - 2 times V into O.
  f32x16 s_even[QB][2], s_odd[QB][2];
  u32x4 p_even[QB][4], p_odd[QB][4];  // bf16 bits (carried as integers)
  float m_use[QB];  // exponent offset of the weights being formed

  // Step t (t = 0 .. n_kt + 1) of the pipeline, for one wave:
  //   A  PV (2 <= t <= n_live + 1): O += P(t-2) V(t-2) on the matrix cores,
  //      with the weights of tile t - 1 (first half of its keys) formed in
  //      between; HEAD: tile t - 1 first gets its row maximum (MASK: the
  //      length / causal mask too) and the lazy rescale, whose factor
  //      reaches O once the products of tile t - 2 are in;
  //   B  QK (t < n_live): S(t) = K(t) Q^T, with the second half of the
  //      weights of tile t - 1 formed in between;
  //   then the check of tile t - 1's weights (EX: 1 <= t <= n_live).
  // Every product thus has about one exponential and three other vector
  // operations beside it, so the vector work of a wave runs under its own
  // matrix work.  K(t) sits in K buffer t % 2 and V(t - 2) in V buffer t % 2;
  // the step loads K(t + 1) and V(t - 1) into the other two, spread over
  // its first products.  STEADY: both loads are due, both tiles lie inside
  // the sequence and the step has both phases without a head, so the loads
  // go out unconditionally and the products form one schedulable block.
  auto step = [&](int t, auto par_tag, auto qk_tag, auto ex_tag, auto pv_tag, auto head_tag,
                  auto mask_tag, auto steady_tag) {
    constexpr int PAR = decltype(par_tag)::value;
    constexpr bool QK = decltype(qk_tag)::value;
    constexpr bool EX = decltype(ex_tag)::value;
    constexpr bool PV = decltype(pv_tag)::value;
    constexpr bool HEAD = decltype(head_tag)::value;
    constexpr bool MASK = decltype(mask_tag)::value;
    constexpr bool STEADY = decltype(steady_tag)::value;
    static_assert(EX || !HEAD, "a head belongs to a tile being weighed");
    auto& s_new = pick<PAR>(s_even, s_odd);      // S(t)
    auto& s_old = pick<1 - PAR>(s_even, s_odd);  // S(t - 1), turned into weights
    auto& p_new = pick<1 - PAR>(p_even, p_odd);  // P(t - 1)
    auto& p_old = pick<PAR>(p_even, p_odd);      // P(t - 2)
    const int tw = t - 1;                        // the tile being weighed
    // A step that forms no scores (no weights) still gives the array a
    // value: otherwise the contents of two steps back would stay live
    // through every step, since the compiler cannot see that no later step
    // reads them.
    if constexpr (!QK) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s_new[qb][kb][r] = 0.f;
    }
    if constexpr (!EX) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) p_new[qb][kc] = u32x4{0u, 0u, 0u, 0u};
    }
    const bool load_k = t + 1 < n_kt;
    const bool load_v = t >= 1 && t - 1 < n_kt;
    // PAGED: the pages of this step's blocks, looked up before any LDS read
    // is in flight (so the wait for them waits for nothing else)
    size_t pk_off[S::BLOCKS_PER_WAVE], pv_off[S::BLOCKS_PER_WAVE];
    if constexpr (PAGED) {
      if (a.tile_in_page) {
        // one entry per tile: a block's rows follow the tile's first row
        const size_t k0 = (STEADY || load_k) ? page_row((t + 1) * BN) : 0;
        const size_t v0 = (STEADY || load_v) ? page_row((t - 1) * BN) : 0;
#pragma unroll
        for (int p = 0; p < S::BLOCKS_PER_WAVE; ++p) {
          pk_off[p] = k0 + (size_t)(block_row(t + 1, p) - (t + 1) * BN) * ROW_BYTES;
          pv_off[p] = v0 + (size_t)(block_row(t - 1, p) - (t - 1) * BN) * ROW_BYTES;
        }
      } else {
#pragma unroll
        for (int p = 0; p < S::BLOCKS_PER_WAVE; ++p) {
          pk_off[p] = (STEADY || load_k) ? page_row(block_row(t + 1, p)) : 0;
          pv_off[p] = (STEADY || load_v) ? page_row(block_row(t - 1, p)) : 0;
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    auto load_block = [&](auto p_tag) {
      using NB_ = std::integral_constant<int, 1 - PAR>;
      constexpr int P_ = decltype(p_tag)::value;
      if (STEADY || load_k)
        issue_rows(kg, k_lds_w, t + 1, NB_(), p_tag, steady_tag, PAGED ? pk_off[P_] : 0);
      if constexpr (VT) {
        if (STEADY || load_v) issue_vt(t - 1, NB_(), p_tag);
      } else {
        if (STEADY || load_v)
          issue_rows(vg, v_lds_w, t - 1, NB_(), p_tag, steady_tag, PAGED ? pv_off[P_] : 0);
      }
    };

    // ---- LDS read stream: the NV V reads of tile t - 2 in the order the
    // products consume them (RPP per product), then the NK K fragments of
    // tile t (key block kb, then step s).  RS reads are kept in flight:
    // consuming one issues the next. ----
    constexpr int NVS = PV ? NV : 0;
    constexpr int NKS = QK ? NK : 0;
    constexpr int TOT = NVS + NKS;
    constexpr int RS = RW < TOT ? RW : TOT;
    std::conditional_t<VT, u32x4, u32x2> vr[NV];
    u32x4 kr[NK];
    auto issue_read = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      if constexpr (J < NVS && VT) {
        // product J: key chunk J / DBLK, head dims 32 (J % DBLK) ..
        constexpr int OFF = PAR * TILE_BYTES + (J / S::DBLK) * D * 32 + (J % S::DBLK) * 32 * 32;
        vr[J] = lds_read_b128_async_off<OFF>(vt_addr);
      } else if constexpr (J < NVS) {
        constexpr int OFF = PAR * TILE_BYTES + (J / (2 * S::DBLK)) * 16 * ROW_BYTES;
        vr[J] = lds_read_tr16_async_off<OFF>(v_addr[(J / 2) % S::DBLK][J % 2]);
      } else if constexpr (J < TOT) {
        constexpr int K = J - NVS;
        constexpr int OFF = PAR * TILE_BYTES + (K / S::KSTEPS) * 32 * ROW_BYTES;
        kr[K] = lds_read_b128_async_off<OFF>(k_addr[K % S::KSTEPS]);
      }
    };
    static_for<0, RS>(issue_read);

    // ---- weights of tile t - 1: chunk kc = keys 16 kc .. 16 kc + 15
    // (accumulator rows 8 (kc % 2) .. +7 of key block kc / 2) ----
    const float cc = POS_SCALE ? c : 1.f;
    float l_tile[QB];  // this lane's share of the row sums of tile t - 1
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l_tile[qb] = 0.f;
    auto exp_one = [&](auto kc_tag, auto e_tag) {
      constexpr int KC = decltype(kc_tag)::value;
      constexpr int R = 8 * (KC % 2) + decltype(e_tag)::value;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        s_old[qb][KC / 2][R] = fast_exp2(fmaf(s_old[qb][KC / 2][R], cc, -m_use[qb]));
    };
    auto exp_finish = [&](auto kc_tag) {
      constexpr int KC = decltype(kc_tag)::value;
      constexpr int R = 8 * (KC % 2);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const f32x16& x = s_old[qb][KC / 2];
        l_tile[qb] += ((x[R] + x[R + 1]) + (x[R + 2] + x[R + 3])) +
                      ((x[R + 4] + x[R + 5]) + (x[R + 6] + x[R + 7]));
        p_new[qb][KC] = as_u32x4(to_bf16x8(x[R], x[R + 1], x[R + 2], x[R + 3], x[R + 4],
                                           x[R + 5], x[R + 6], x[R + 7]));
      }
    };
    // exponential i (0 .. 15) of half H (chunks 2H, 2H + 1), and the chunk's
    // fragment after its last one
    auto exp_item = [&](auto h_tag, auto i_tag) {
      constexpr int H = decltype(h_tag)::value;
      constexpr int I = decltype(i_tag)::value;
      using KC_ = std::integral_constant<int, 2 * H + I / 8>;
      exp_one(KC_(), std::integral_constant<int, I % 8>());
      if constexpr (I % 8 == 7) exp_finish(KC_());
    };

    // ---- head of tile t - 1: scale (scale <= 0), mask, row maximum in
    // eight parts, then the lazy rescale of the running state.  The rescale
    // factor of O is applied once the products of tile t - 2 are in. ----
    float mx0[QB], mx1[QB], alpha_o[QB];
    bool rescale_o = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) mx0[qb] = mx1[qb] = kNegInf;
    auto head_part = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      constexpr int KB = J / 4, R0 = 4 * (J % 4);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int r = R0; r < R0 + 4; ++r) {
          if (!POS_SCALE) s_old[qb][KB][r] *= c;
          if (MASK) {
            const int qrow = qw0 + qb * 32 + n;
            const int lim = min(L - 1, CAUSAL ? qrow + off : L - 1);  // last admissible key
            // The lane's key tw BN + 4 h + o, o = 32 KB + 8 (r / 4) + r % 4.
            // Two spellings of the same test: comparing o (an inline
            // constant) with lim - tw BN - 4 h keeps no per-register key
            // offsets, which the register allocator needs on the VT path
            // and does worse with on the other.
            if constexpr (VT) {
              if (KB * 32 + 8 * (r >> 2) + (r & 3) > lim - tw * BN - 4 * h)
                s_old[qb][KB][r] = kNegInf;
            } else {
              const int key = tw * BN + KB * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
              if (key > lim) s_old[qb][KB][r] = kNegInf;
            }
          }
        }
        float& mx = KB == 0 ? mx0[qb] : mx1[qb];
        mx = fmaxf(fmaxf(mx, s_old[qb][KB][R0]), s_old[qb][KB][R0 + 1]);
        mx = fmaxf(fmaxf(mx, s_old[qb][KB][R0 + 2]), s_old[qb][KB][R0 + 3]);
      }
    };
    auto head_end = [&]() {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = max_xor32(fmaxf(mx0[qb], mx1[qb]));
        if (POS_SCALE) mx *= c;
        alpha_o[qb] = 1.f;
        if (__ballot(mx > m_run[qb] + kRescaleSlack)) {
          const float m_new = fmaxf(m_run[qb], mx);
          const float alpha = (m_new == kNegInf) ? 1.f : fast_exp2(m_run[qb] - m_new);
          m_run[qb] = m_new;
          l_run[qb] *= alpha;
          alpha_o[qb] = alpha;
          rescale_o = true;
        }
        m_use[qb] = (m_run[qb] == kNegInf) ? 0.f : m_run[qb];
      }
    };

    // ---- phase A: O += P(t-2) V(t-2), the head and the first half of the
    // weights of tile t - 1 in between ----
    constexpr bool LOADS_A = PV;  // the loads go out during the first products
    if constexpr (PV) {
      constexpr int NP = NV / RPP;  // products: (kc, db) = (m / DBLK, m % DBLK)
      static_assert(NP == 16 || NP == 8, "products per phase");
      constexpr int PER_LOAD = NP / S::BLOCKS_PER_WAVE;
      static_for<0, NP>([&](auto m_tag) {
        constexpr int M = decltype(m_tag)::value;
        // reads still in flight once those of product M are in
        constexpr int AHEAD = (RS < TOT - RPP * M ? RS : TOT - RPP * M) - RPP;
        lds_wait_lgkm<AHEAD>();
        bf16x8 vf;
        if constexpr (VT) {
          lds_ready(vr[M]);
          vf = as_bf16x8(vr[M]);
        } else {
          lds_ready(vr[2 * M]);
          lds_ready(vr[2 * M + 1]);
          const u32x4 w = {vr[2 * M][0], vr[2 * M][1], vr[2 * M + 1][0], vr[2 * M + 1][1]};
          vf = as_bf16x8(w);
        }
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o_acc[qb][M % S::DBLK] =
              mfma32(vf, as_bf16x8(p_old[qb][M / S::DBLK]), o_acc[qb][M % S::DBLK]);
        static_for<0, RPP>([&](auto i_tag) {
          issue_read(std::integral_constant<int, RPP * M + decltype(i_tag)::value + RS>());
        });
        if constexpr (M % PER_LOAD == 0) load_block(std::integral_constant<int, M / PER_LOAD>());
        if constexpr (EX) {
          if constexpr (HEAD) {
            // the first half of the products carries the head's eight
            // parts, the second half the sixteen exponentials
            constexpr int NH = NP / 2, HPP = 8 / NH, EPP = 16 / (NP - NH);
            if constexpr (M < NH) {
              static_for<0, HPP>([&](auto j_tag) {
                head_part(std::integral_constant<int, HPP * M + decltype(j_tag)::value>());
              });
              if constexpr (M == NH - 1) head_end();
            } else {
              static_for<0, EPP>([&](auto e_tag) {
                exp_item(std::integral_constant<int, 0>(),
                         std::integral_constant<int, EPP * (M - NH) + decltype(e_tag)::value>());
              });
            }
          } else {
            constexpr int EPP = 16 / NP;
            static_for<0, EPP>([&](auto e_tag) {
              exp_item(std::integral_constant<int, 0>(),
                       std::integral_constant<int, EPP * M + decltype(e_tag)::value>());
            });
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (HEAD) {
        if (rescale_o) {
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
              for (int r = 0; r < 16; ++r) o_acc[qb][db][r] *= alpha_o[qb];
        }
      }
    } else if constexpr (EX) {
      // t = 1: no product has reached O yet, so O needs no rescale
      if constexpr (HEAD) {
        static_for<0, 8>(head_part);
        head_end();
      }
      static_for<0, 16>([&](auto i_tag) { exp_item(std::integral_constant<int, 0>(), i_tag); });
    }

    // ---- phase B: S(t) = K(t) Q^T, the second half of the weights in
    // between ----
    if constexpr (QK) {
      static_assert(NK == 16 || NK == 8, "products per phase");
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s_new[qb][kb][r] = 0.f;
      constexpr int PER_LOAD = NK / S::BLOCKS_PER_WAVE;
      constexpr int EPP = 16 / NK;  // exponentials per product
      static_for<0, NK>([&](auto i_tag) {
        constexpr int I = decltype(i_tag)::value;
        constexpr int KB = I / S::KSTEPS, ST = I % S::KSTEPS;
        constexpr int J = NVS + I;  // position in the read stream
        constexpr int AHEAD = (J + RS < TOT ? RS : TOT - J) - 1;
        lds_wait_lgkm<AHEAD>();
        lds_ready(kr[I]);
        const bf16x8 kf = as_bf16x8(kr[I]);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s_new[qb][KB] = mfma32(kf, qf[qb][ST], s_new[qb][KB]);
        issue_read(std::integral_constant<int, J + RS>());
        if constexpr (!LOADS_A && I % PER_LOAD == PER_LOAD - 1)
          load_block(std::integral_constant<int, I / PER_LOAD>());
        if constexpr (EX)
          static_for<0, EPP>([&](auto e_tag) {
            exp_item(std::integral_constant<int, 1>(),
                     std::integral_constant<int, EPP * I + decltype(e_tag)::value>());
          });
        __builtin_amdgcn_sched_barrier(0);
      });
    } else {
      if constexpr (!LOADS_A) static_for<0, S::BLOCKS_PER_WAVE>(load_block);
      if constexpr (EX)
        static_for<0, 16>([&](auto i_tag) { exp_item(std::integral_constant<int, 1>(), i_tag); });
    }

    // ---- the weights of tile t - 1 are complete.  Rows whose sums overran
    // kSumLimit (a tile weighed without its own maximum whose scores rose
    // well above the running one) get the tile's scores again, from K in
    // global memory (its LDS buffer is being refilled by now), a lazy
    // rescale to the exact maximum, and new weights.  O holds tiles up to
    // t - 2 here, so its rescale is immediate.  Then the sums join the
    // running ones. ----
    // the rescale to the exact maximum of re-formed scores S(t - 1) (in
    // s_old) and the tile's new weights
    auto settle_tail = [&](int qb) {
      float mx = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s_old[qb][kb][r]);
      mx = max_xor32(mx) * c;
      const float m_new = fmaxf(m_run[qb], mx);
      const float alpha = (m_new == kNegInf) ? 1.f : fast_exp2(m_run[qb] - m_new);
      m_run[qb] = m_new;
      l_run[qb] *= alpha;
#pragma unroll
      for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o_acc[qb][db][r] *= alpha;
      m_use[qb] = (m_new == kNegInf) ? 0.f : m_new;
      l_tile[qb] = 0.f;
      static_for<0, 4>([&](auto kc_tag) {
        constexpr int KC = decltype(kc_tag)::value;
        constexpr int R = 8 * (KC % 2);
        f32x16& x = s_old[qb][KC / 2];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[R + e] = fast_exp2(fmaf(x[R + e], c, -m_use[qb]));
        l_tile[qb] += ((x[R] + x[R + 1]) + (x[R + 2] + x[R + 3])) +
                      ((x[R + 4] + x[R + 5]) + (x[R + 6] + x[R + 7]));
        p_new[qb][KC] = as_u32x4(to_bf16x8(x[R], x[R + 1], x[R + 2], x[R + 3], x[R + 4],
                                           x[R + 5], x[R + 6], x[R + 7]));
      });
    };
    if constexpr (EX) {
      if constexpr (POS_SCALE && !HEAD) {
        // only tiles 1 .. n_free - 1 are weighed without their maximum; they
        // lie wholly inside the sequence, so their K rows can be read again
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          if (__ballot(l_tile[qb] > kSumLimit)) {
            // (the base is made wave-uniform explicitly: a resource in vector
            // registers would need a loop over its distinct values)
            const uintptr_t base = (uintptr_t)(kg + (size_t)tw * BN * kv_stride);
            const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)base);
            const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
            const __amdgpu_buffer_rsrc_t rows = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<char*>(((uintptr_t)hi << 32) | lo), 0, (int)(BN * kv_stride),
                0x00020000);
            // lane part of the fragment offsets in a vector register, the
            // rest (wave-uniform) in the scalar offset
            const uint32_t lane_off = (uint32_t)(n * kv_stride + 16 * h);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
              for (int r = 0; r < 16; ++r) s_old[qb][kb][r] = 0.f;
#pragma unroll
              for (int st = 0; st < S::KSTEPS; ++st) {
                const u32x4 u = __builtin_amdgcn_raw_buffer_load_b128(
                    rows, lane_off, (uint32_t)(32 * kb * kv_stride + 32 * st), 0);
                s_old[qb][kb] = mfma32(as_bf16x8(u), qf[qb][st], s_old[qb][kb]);
                __builtin_amdgcn_sched_barrier(0);  // one fragment in registers at a time
              }
            }
            settle_tail(qb);
          }
        }
      }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) l_run[qb] += l_tile[qb];
    }
  };

  // One barrier per step: once every wave has waited for its own loads,
  // the barrier makes K(t) and V(t - 2) visible and proves that every wave
  // has finished step t - 1, whose buffers the step's loads overwrite.
  using T1 = std::true_type;
  using F0 = std::false_type;
  // PERSIST: thread 0 claims the next index of its own queue two steps
  // before an item's last (the atomic's return is waited for with that
  // step's tile loads) and keeps a mask of the queues it has found empty.
  const int own_q = PERSIST ? (int)(blockIdx.x % (unsigned)a.n_queues) : 0;
  int pending = 0;
  unsigned drained = 0;
  auto run_step = [&](int t, auto par_tag) {
    wait_vmcnt<0>();
    __syncthreads();
    if constexpr (PERSIST) {
      if (t == max(n_kt - 1, 0) && tid == 0)
        pending = ((drained >> own_q) & 1u) ? a.per_queue : atomicAdd(a.ctr + 32 * own_q, 1);
    }
    const bool qk = t < n_live;
    const bool ex = t >= 1 && t <= n_live;
    const bool pv = t >= 2 && t <= n_live + 1;
    // tile t - 1 gets its maximum: the first tile, masked tiles, and every
    // tile when the scale is not positive or the keys come from pages (a
    // tile weighed against the running maximum may have to be formed again
    // from K, which the paged path does not do)
    const bool mask = t - 1 >= n_free;
    const bool head = !POS_SCALE || PAGED || t == 1 || mask;
    if (qk && ex && pv) {
      if (!head) {
        if (t + 1 < n_full)
          step(t, par_tag, T1(), T1(), T1(), F0(), F0(), T1());
        else
          step(t, par_tag, T1(), T1(), T1(), F0(), F0(), F0());
      } else if (mask) {
        step(t, par_tag, T1(), T1(), T1(), T1(), T1(), F0());
      } else if (PAGED && t + 1 < n_full) {
        step(t, par_tag, T1(), T1(), T1(), T1(), F0(), T1());
      } else {
        step(t, par_tag, T1(), T1(), T1(), T1(), F0(), F0());
      }
    } else if (qk && ex) {  // t = 1
      if (mask)
        step(t, par_tag, T1(), T1(), F0(), T1(), T1(), F0());
      else
        step(t, par_tag, T1(), T1(), F0(), T1(), F0(), F0());
    } else if (qk) {  // t = 0
      step(t, par_tag, T1(), F0(), F0(), F0(), F0(), F0());
    } else if (ex && pv) {  // t = n_live
      if (!head)
        step(t, par_tag, F0(), T1(), T1(), F0(), F0(), F0());
      else if (mask)
        step(t, par_tag, F0(), T1(), T1(), T1(), T1(), F0());
      else
        step(t, par_tag, F0(), T1(), T1(), T1(), F0(), F0());
    } else if (ex) {  // t = 1 = n_live
      if (mask)
        step(t, par_tag, F0(), T1(), F0(), T1(), T1(), F0());
      else
        step(t, par_tag, F0(), T1(), F0(), T1(), F0(), F0());
    } else if (pv) {  // t = n_live + 1
      step(t, par_tag, F0(), F0(), T1(), F0(), F0(), F0());
    } else {
      step(t, par_tag, F0(), F0(), F0(), F0(), F0(), F0());
    }
  };
  for (int par_item = 0;; par_item ^= 1) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      m_run[qb] = kNegInf;
      l_run[qb] = 0.f;
      m_use[qb] = 0.f;
#pragma unroll
      for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o_acc[qb][db][r] = 0.f;
    }
    // (an item without tiles claims here)
    if constexpr (PERSIST) {
      if (n_kt == 0 && tid == 0)
        pending = ((drained >> own_q) & 1u) ? a.per_queue : atomicAdd(a.ctr + 32 * own_q, 1);
    }
    if (n_kt > 0) {
      for (int t = 0; t <= n_kt + 1; t += 2) {
        run_step(t, B0());
        if (t + 1 <= n_kt + 1) run_step(t + 1, B1());
      }
    }

    // PERSIST: the next item (-1: none left), from the own queue, else from
    // the others in turn.  Past the barrier every wave is done with the K
    // buffers, so the next item's first K tile can go into buffer 0 while
    // this item's output is written.
    int next = -1;
    if constexpr (PERSIST) {
      if (tid == 0) {
        int nb = -1;
        if (pending < a.per_queue) {
          nb = pending * a.n_queues + own_q;
        } else {
          drained |= 1u << own_q;
          for (int k = 1; k < a.n_queues && nb < 0; ++k) {
            const int x = (own_q + k) % a.n_queues;
            if ((drained >> x) & 1u) continue;
            const int i = atomicAdd(a.ctr + 32 * x, 1);
            if (i < a.per_queue)
              nb = i * a.n_queues + x;
            else
              drained |= 1u << x;
          }
        }
        next_item[par_item] = nb;
      }
      __syncthreads();
      // the same in every lane: saying so keeps the item's geometry in
      // scalar registers
      next = __builtin_amdgcn_readfirstlane(next_item[par_item]);
    }
    const size_t e_o_base = o_base;  // where the finished item's rows go
    float* const e_lse = lse_base;
    const int e_qw0 = qw0, e_Sq = Sq;

    // ---- epilogue: O = O_acc / l, LSE = ln 2 * (m + log2 l).  bf16 O is
    // staged through LDS (the now free K buffers, or PERSIST's own area) so
    // that the stores are whole rows; fp32 O goes out 16 bytes per lane
    // directly.  PERSIST: the next item's loads are issued between the LDS
    // round trip and the stores (LDS reads issued after LDS-DMA loads would
    // wait for them). ----
    if constexpr (!OUT_F32 && !PERSIST) __syncthreads();
    // the lane's indices formed anew here (an opaque copy of the thread
    // index), so that the output addresses, which do not change from item
    // to item, are not computed once and held in registers through the
    // item's tiles
    int tid_e = tid;
    asm volatile("" : "+v"(tid_e));
    const int lane_e = tid_e & 63, n_e = lane_e & 31, h_e = lane_e >> 5;
    const uint32_t stage =
        (PERSIST ? lds_addr(&o_stage[0]) : lds_addr(&k_lds[0][0])) + wave * 32 * ROW_BYTES;
    float lsum[QB];
    u32x4 rows[QB][OUT_F32 ? 1 : D / 16];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      lsum[qb] = sum_xor32(l_run[qb]);
      if constexpr (!OUT_F32)
        stage_rows_t<D>(o_acc[qb], lsum[qb] > 0.f ? 1.f / lsum[qb] : 0.f, stage, n_e, h_e,
                        lane_e, rows[qb]);
    }
    if constexpr (PERSIST) {
      if (next >= 0) {
        setup(next);
        load_q();
        issue_k0();
      }
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qrow = e_qw0 + qb * 32 + n_e;
      if constexpr (!OUT_F32) {
        store_staged_rows<D>(rows[qb], lane_e,
                             static_cast<uint16_t*>(a.o) + e_o_base + (e_qw0 + qb * 32) * q_stride,
                             q_stride, e_Sq - (e_qw0 + qb * 32));
      }
      if (qrow >= e_Sq) continue;
      if constexpr (OUT_F32) {
        const float inv = lsum[qb] > 0.f ? 1.f / lsum[qb] : 0.f;
        const size_t obase = e_o_base + qrow * q_stride;
#pragma unroll
        for (int db = 0; db < S::DBLK; ++db)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            const int d = db * 32 + 8 * r4 + 4 * h_e;
            const f32x4 w = {o_acc[qb][db][4 * r4 + 0] * inv, o_acc[qb][db][4 * r4 + 1] * inv,
                             o_acc[qb][db][4 * r4 + 2] * inv, o_acc[qb][db][4 * r4 + 3] * inv};
            *reinterpret_cast<f32x4*>(static_cast<float*>(a.o) + obase + d) = w;
          }
      }
      if (h_e == 0 && e_lse)
        e_lse[qrow] = lsum[qb] > 0.f ? (m_run[qb] + log2f(lsum[qb])) * kLn2 : kNegInf;
    }
    if (next < 0) break;
  }
}

}  // namespace mk
