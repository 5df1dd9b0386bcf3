// bwd_kernel.hpp -- attention backward for gfx950: gradients of the output
// with respect to q, k and v (the LSE output is taken as not
// differentiated).
//
// With P = softmax(scale * q k^T) over the valid keys (the forward's masks)
// and dO = dL/dO:
//   dV_j  = sum_i P_ij dO_i                 (dK, dV summed over the query
//   dP_ij = dO_i . v_j                        heads of the kv head)
//   D_i   = sum_j P_ij dP_ij = dO_i . O_i
//   dS_ij = P_ij (dP_ij - D_i)
//   dQ_i  = scale * sum_j dS_ij k_j,   dK_j = scale * sum_i dS_ij q_i
// P is recomputed from the forward's LSE, P_ij = exp(scale s_ij - LSE_i),
// so no attention matrix is stored.
//
// Two kernels on one stream:
//   bwd_dq_kernel     one workgroup per 128 query rows of one (b, hq),
//                     shaped like the forward: K and V 64-key tiles stream
//                     through LDS, each wave keeps its 32 rows' Q and dO in
//                     registers and accumulates dQ^T = K^T dS^T; it first
//                     forms D_i = dO_i . O_i and LSE_i log2 e of its rows
//                     and writes them to the workspace;
//   bwd_dkdv_kernel   (after it) one workgroup per 128 keys of one (b, kv head): each
//                     wave keeps its 32 keys' K and V in registers, the Q,
//                     dO, LSE and D tiles of every query head of the group
//                     stream through LDS, and dK^T = Q^T dS, dV^T = dO^T P
//                     accumulate without atomics (deterministic).
// All products are bf16 MFMA with fp32 accumulation; P and dS enter them
// as bf16.
#pragma once

#include "mk_common.hpp"

namespace mk {

struct BwdArgs {
  const uint16_t* q;     // [B, Hq, Sq, D]
  const uint16_t* k;     // [B, Hkv, Skv, D]
  const uint16_t* v;
  const uint16_t* o;     // forward output [B, Hq, Sq, D]
  const uint16_t* dout;  // dL/dO [B, Hq, Sq, D]
  const float* lse;      // forward LSE [B, Hq, Sq] (natural log)
  uint16_t* dq;          // [B, Hq, Sq, D] bf16 (written)
  uint16_t* dk;          // [B, Hkv, Skv, D] bf16 (written)
  uint16_t* dv;
  float* delta;          // workspace [B, Hq, sq_pad]: D_i (0 on padding rows)
  float* lse2;           // workspace [B, Hq, sq_pad]: LSE_i log2(e); +inf on rows
                         // without keys and on padding rows, so that P = 0 there
  const int* kv_seqlens;
  int B, Hq, Hkv, Sq, Skv;
  int sq_pad;            // Sq rounded up to a multiple of 128
  int n_qtiles;          // dQ kernel: ceil(Sq / 128)
  int xcd_gp;            // dQ kernel: > 0 xcd_pair_map order (groups of xcd_gp pairs)
  int n_kblocks;         // dK/dV kernel: ceil(Skv / 128)
  float scale;
  float scale_log2;      // scale * log2(e)
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// P of one element: 2^(s c - LSE log2 e), 0 where masked (lse2 = +inf on
// rows without keys gives 0 by itself).
__device__ __forceinline__ float bwd_prob(float s, float c, float lse2, bool valid) {
  const float p = fast_exp2(fmaf(s, c, -lse2));
  return valid ? p : 0.f;
}

// ---------------------------------------------------------------------------
// dQ: workgroup = 4 waves x 32 query rows of one (b, hq); 64-key K/V tiles.
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void bwd_dq_kernel(BwdArgs a) {
  constexpr int WAVES = 4, BM = 128, BN = 64;
  constexpr int KSTEPS = D / 16, DBLK = D / 32, CHUNKS = D / 8;
  constexpr int ROW_BYTES = D * 2, TILE = BN * D, TILE_BYTES = TILE * 2;
  constexpr int ROWS_PER_KB = 512 / D;
  constexpr int BLOCKS_PER_WAVE = BN * D * 2 / 1024 / WAVES;
  constexpr int LOADS_PER_TILE = 2 * BLOCKS_PER_WAVE;
  // K tiles in buffers 0 and 1, V tiles in 2 and 3
  __shared__ __attribute__((aligned(1024))) uint16_t kv_lds[4][TILE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  // longest query tiles first; pairs placed on the XCDs when possible
  int qt, b, hq;
  if (a.xcd_gp > 0) {
    xcd_pair_map(blockIdx.x, a.n_qtiles, a.B, a.Hkv, a.Hq / a.Hkv, a.xcd_gp, qt, b, hq);
  } else {
    const int per = a.B * a.Hq;
    const int t_ = blockIdx.x / per;
    const int rem = blockIdx.x - t_ * per;
    qt = a.n_qtiles - 1 - t_;
    b = rem / a.Hq;
    hq = rem - b * a.Hq;
  }
  const int g = hq / (a.Hq / a.Hkv);
  const int L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
  const int off = L - a.Sq;
  const int q0 = qt * BM;
  const int q_end = min(q0 + BM, a.Sq);
  int n_keys = CAUSAL ? min(L, q_end + off) : L;
  if (n_keys < 0) n_keys = 0;
  const int n_kt = (n_keys + BN - 1) / BN;
  const float c = a.scale_log2;

  const size_t row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
  const char* kg = reinterpret_cast<const char*>(a.k + ((size_t)b * a.Hkv + g) * (size_t)a.Skv * D);
  const char* vg = reinterpret_cast<const char*>(a.v + ((size_t)b * a.Hkv + g) * (size_t)a.Skv * D);

  // this lane's query row, its Q^T and dO^T fragments, LSE and D
  const int qrow = q0 + wave * 32 + n;
  const bool row_ok = qrow < a.Sq;
  bf16x8 qf[KSTEPS], df[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s) {
    u32x4 u = {0u, 0u, 0u, 0u}, w = {0u, 0u, 0u, 0u};
    if (row_ok) {
      u = *reinterpret_cast<const u32x4*>(a.q + (row0 + qrow) * D + s * 16 + h * 8);
      w = *reinterpret_cast<const u32x4*>(a.dout + (row0 + qrow) * D + s * 16 + h * 8);
    }
    qf[s] = as_bf16x8(u);
    df[s] = as_bf16x8(w);
  }
  // D_i = dO_i . O_i (this lane's half of the row, then its partner lane's
  // half) and LSE_i log2 e, kept for this kernel and written to the
  // workspace for the dK/dV kernel, which runs next; padding rows (past Sq)
  // and rows without keys get D = 0 and +inf, so that P vanishes there.
  const size_t prow = ((size_t)b * a.Hq + hq) * (size_t)a.sq_pad + qrow;  // qrow < sq_pad
  float dl = 0.f, lse2 = __builtin_inff();
  {
    float part = 0.f;
    if (row_ok) {
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const u32x4 ov = *reinterpret_cast<const u32x4*>(a.o + (row0 + qrow) * D + s * 16 + h * 8);
        const u32x4 dv = as_u32x4(df[s]);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          part = fmaf(bf16_lo(ov[w]), bf16_lo(dv[w]), part);
          part = fmaf(bf16_hi(ov[w]), bf16_hi(dv[w]), part);
        }
      }
      const float lse = a.lse[row0 + qrow];
      lse2 = lse == kNegInf ? __builtin_inff() : lse * kLog2e;
    }
    dl = part + __shfl_xor(part, 32, 64);
    if (h == 0) {
      a.delta[prow] = dl;
      a.lse2[prow] = lse2;
    }
  }
  const int lim = CAUSAL ? min(L - 1, qrow + off) : L - 1;  // last key this row sees

  // tile loads, as in the forward kernel
  constexpr int ROW_STEP = WAVES * ROWS_PER_KB;
  const int dma_row = wave * ROWS_PER_KB + lane / CHUNKS;
  const int dma_ch = ((lane % CHUNKS) ^ fwd_swz<D>(dma_row)) * 16;
  const uint32_t k0 = lds_addr(&kv_lds[0][0]);
  const uint32_t k_lds_w = __builtin_amdgcn_readfirstlane(k0 + wave * 1024);
  const uint32_t v_lds_w = __builtin_amdgcn_readfirstlane(k0 + 2 * TILE_BYTES + wave * 1024);
  auto issue_tile = [&](int kt, int buf) {
    const int tlim = L - 1 - kt * BN;
#pragma unroll
    for (int p = 0; p < BLOCKS_PER_WAVE; ++p) {
      const uint32_t goff = (uint32_t)(min(dma_row + p * ROW_STEP, tlim) * ROW_BYTES + dma_ch);
      const size_t toff = (size_t)kt * BN * ROW_BYTES;
      const uint32_t lds_off = buf * TILE_BYTES + p * WAVES * 1024;
      load_lds16_buf(kg + toff, TILE_BYTES, goff, k_lds_w + lds_off);
      load_lds16_buf(vg + toff, TILE_BYTES, goff, v_lds_w + lds_off);
    }
  };

  // LDS read addresses (in K buffer 0; the buffer, the key block and V are
  // immediate offsets): K / V rows (A operand, 32 keys x 8 head dims) and
  // transposing K^T reads (A operand of dQ^T = K^T dS^T)
  uint32_t kr_addr[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    kr_addr[s] = k0 + n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
  uint32_t kt_addr[DBLK][2];
  {
    const int tr_i = lane & 15;
    const int tr_row = 4 * h + (tr_i >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (tr_i & 3);
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int r = tr_row + 8 * hh;
        const int col = db * 32 + tr_col;
        kt_addr[db][hh] =
            k0 + r * ROW_BYTES + ((((col >> 3) ^ fwd_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }

  f32x16 acc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  // One 64-key tile in buffer BUF.  Its LDS reads form one stream -- the
  // K and V fragments of the score products (key block kb, step s, K then
  // V), then the transposing K reads of dQ^T (chunk kc, block db, low /
  // high rows) -- kept RW reads ahead of their use and waited for by count.
  constexpr int NA = 4 * KSTEPS, NC = 8 * DBLK, TOT = NA + NC, RW = 6;
  auto tile = [&](int kt, auto buf_tag) {
    constexpr int BUF = decltype(buf_tag)::value;
    if (kt + 1 < n_kt)
      wait_vmcnt<LOADS_PER_TILE>();
    else
      wait_vmcnt<0>();
    __syncthreads();
    const int key0 = kt * BN;
    u32x4 ar[NA];
    u32x2 cr[NC];
    auto issue = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      if constexpr (J < NA) {
        constexpr int KB = J / (2 * KSTEPS), ST = (J / 2) % KSTEPS, W = J % 2;
        constexpr int OFF = (2 * W + BUF) * TILE_BYTES + KB * 32 * ROW_BYTES;
        ar[J] = lds_read_b128_async_off<OFF>(kr_addr[ST]);
      } else if constexpr (J < TOT) {
        constexpr int C = J - NA, KC = C / (2 * DBLK), DB = (C / 2) % DBLK, HH = C % 2;
        constexpr int OFF = BUF * TILE_BYTES + KC * 16 * ROW_BYTES;
        cr[C] = lds_read_tr16_async_off<OFF>(kt_addr[DB][HH]);
      }
    };
    static_for<0, RW>(issue);
    // S^T = K Q^T and dP^T = V dO^T for the tile's two 32-key blocks, then
    // dQ^T += K^T dS^T over its four 16-key chunks.  The elements of dS^T =
    // P^T (dP^T - D) (bf16; chunk kc = rows 8 (kc % 2) .. +7 of key block
    // kc / 2) of key block 0 are formed beside the products of key block 1,
    // those of key block 1 beside the dQ^T products of chunks 0 and 1, so
    // the vector work runs under the matrix work.  Each product's result
    // passes through an empty volatile statement, which keeps the product
    // in its scheduling group (the compiler would otherwise gather the
    // products into one block).
    f32x16 st[2], dpt[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) st[kb][r] = dpt[kb][r] = 0.f;
    float e[4][8];
    bf16x8 dsf[4];
    auto elem = [&](auto i_tag) {  // element I: chunk I / 8, its row I % 8
      constexpr int I = decltype(i_tag)::value;
      constexpr int KC = I / 8, J = I % 8, R = 8 * (KC % 2) + J;
      const int key = key0 + (KC / 2) * 32 + 8 * (R >> 2) + 4 * h + (R & 3);
      const float p = bwd_prob(st[KC / 2][R], c, lse2, key <= lim);
      e[KC][J] = p * (dpt[KC / 2][R] - dl);
      if constexpr (J == 7)
        dsf[KC] = to_bf16x8(e[KC][0], e[KC][1], e[KC][2], e[KC][3], e[KC][4], e[KC][5],
                            e[KC][6], e[KC][7]);
    };
    constexpr int EPA = 32 / NA;  // elements of key block 0 per product of key block 1
    static_for<0, NA>([&](auto i_tag) {
      constexpr int I = decltype(i_tag)::value;
      constexpr int KB = I / (2 * KSTEPS), ST = (I / 2) % KSTEPS;
      constexpr int AHEAD = (I + RW < TOT ? I + RW : TOT) - I - 1;
      lds_wait_lgkm<AHEAD>();
      lds_ready(ar[I]);
      if constexpr (I % 2 == 0) {
        st[KB] = mfma32(as_bf16x8(ar[I]), qf[ST], st[KB]);
        asm volatile("" : "+v"(st[KB]));
      } else {
        dpt[KB] = mfma32(as_bf16x8(ar[I]), df[ST], dpt[KB]);
        asm volatile("" : "+v"(dpt[KB]));
      }
      issue(std::integral_constant<int, I + RW>());
      if constexpr (I >= NA / 2)
        static_for<0, EPA>([&](auto e_tag) {
          elem(std::integral_constant<int, EPA * (I - NA / 2) + decltype(e_tag)::value>());
        });
      __builtin_amdgcn_sched_barrier(0);
    });
    constexpr int EPC = 16 / (2 * DBLK);  // elements of key block 1 per dQ^T product
    static_for<0, 4 * DBLK>([&](auto m_tag) {
      constexpr int M = decltype(m_tag)::value;  // (kc, db) = (M / DBLK, M % DBLK)
      constexpr int BASE = NA + 2 * M;
      constexpr int AHEAD = (BASE + RW < TOT ? BASE + RW : TOT) - (BASE + 1) - 1;
      lds_wait_lgkm<AHEAD>();
      lds_ready(cr[2 * M]);
      lds_ready(cr[2 * M + 1]);
      const u32x4 w = {cr[2 * M][0], cr[2 * M][1], cr[2 * M + 1][0], cr[2 * M + 1][1]};
      acc[M % DBLK] = mfma32(as_bf16x8(w), dsf[M / DBLK], acc[M % DBLK]);
      asm volatile("" : "+v"(acc[M % DBLK]));
      issue(std::integral_constant<int, BASE + RW>());
      issue(std::integral_constant<int, BASE + RW + 1>());
      if constexpr (M < 2 * DBLK)
        static_for<0, EPC>([&](auto e_tag) {
          elem(std::integral_constant<int, 16 + EPC * M + decltype(e_tag)::value>());
        });
      __builtin_amdgcn_sched_barrier(0);
    });
    __syncthreads();
    if (kt + 2 < n_kt) issue_tile(kt + 2, BUF);
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  if (n_kt > 0) issue_tile(0, 0);
  if (n_kt > 1) issue_tile(1, 1);
  for (int kt = 0; kt < n_kt; kt += 2) {
    tile(kt, B0());
    if (kt + 1 < n_kt) tile(kt + 1, B1());
  }

  // dQ = scale * acc^T (lane (query n, k-group h) holds head dims
  // db*32 + 8 (r/4) + 4 h + r % 4), staged through the K buffers so that
  // the stores are whole rows
  __syncthreads();
  store_rows_t<D>(acc, a.scale, k0 + wave * 32 * ROW_BYTES, n, h, lane,
                  a.dq + (row0 + q0 + wave * 32) * D, D, a.Sq - (q0 + wave * 32));
}

template <int D>
struct DkdvShape {
  static constexpr int WAVES = 4, BK = 128, BQ = 64, NBUF = 4;
  static constexpr int KSTEPS = D / 16, DBLK = D / 32, CHUNKS = D / 8;
  static constexpr int ROW_BYTES = D * 2, TILE_BYTES = BQ * ROW_BYTES;
  static constexpr int BUF_BYTES = 2 * TILE_BYTES;  // Q tile, then dO tile
  static constexpr int ROWS_PER_KB = 512 / D;
  static constexpr int BLOCKS_PER_WAVE = TILE_BYTES / 1024 / WAVES;  // per tensor
  static constexpr int ROW_STEP = WAVES * ROWS_PER_KB;
  static constexpr int RL_BYTES = 2 * BQ * 4;  // lse2 row, then D row, per buffer
  static constexpr int RW = 8;                 // LDS reads kept in flight
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(BwdArgs a) {
  using S = DkdvShape<D>;
  constexpr int KSTEPS = S::KSTEPS, DBLK = S::DBLK, ROW_BYTES = S::ROW_BYTES;
  constexpr int TILE_BYTES = S::TILE_BYTES, NBUF = S::NBUF, BQ = S::BQ;
  static_assert(S::ROW_STEP % 16 == 0, "row step must preserve the swizzle");
  __shared__ __attribute__((aligned(1024))) uint8_t qd_lds[NBUF * S::BUF_BYTES];
  __shared__ __attribute__((aligned(512))) uint8_t rl_lds[NBUF * S::RL_BYTES];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  // Workgroup order: groups of GS (batch, kv head) pairs, about as many
  // key blocks as run at once (256 compute units, one workgroup each), so
  // the key blocks that read the same Q and dO rows run together; within a
  // group key blocks ascend (under the causal mask the first blocks are
  // seen by the most query rows), and the pairs of a group alternate, so
  // that pair j stays on one XCD (launch order i goes to XCD i % 8).
  const int BH = a.B * a.Hkv, nkb = a.n_kblocks;
  const int GS = max(8, 256 / nkb / 8 * 8);
  const int grp = blockIdx.x / (GS * nkb);
  const int in_grp = blockIdx.x - grp * GS * nkb;
  const int gs = min(GS, BH - grp * GS);
  const int kblk = in_grp / gs;
  const int rem = grp * GS + (in_grp - kblk * gs);
  const int b = rem / a.Hkv, g = rem - (rem / a.Hkv) * a.Hkv;
  const int G = a.Hq / a.Hkv;
  const int L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
  const int off = L - a.Sq;
  const int k0 = kblk * S::BK;
  const int kw0 = k0 + wave * 32;  // this wave's first key
  const int key = kw0 + n;         // this lane's key (MFMA column)
  const float c = a.scale_log2;

  // query tiles that can see a key of the block
  int q_first = CAUSAL ? max(0, k0 - off) : 0;
  if (k0 >= L) q_first = a.Sq;  // no valid key: nothing to accumulate
  const int qt_first = q_first / BQ;
  const int n_qt = q_first < a.Sq ? (a.Sq + BQ - 1) / BQ - qt_first : 0;
  const int n_it = G * n_qt;

  // K and V of this wave's keys as B operands (lane = key column, k-group
  // h = head dims 16 s + 8 h .. +7); keys past the sequence read its last
  // row (their gradients are replaced by zeros at the end)
  const size_t kvh = ((size_t)b * a.Hkv + g) * (size_t)a.Skv;
  const int krow = min(key, L > 0 ? L - 1 : 0);
  bf16x8 kf[KSTEPS], vf[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s) {
    u32x4 u = {0u, 0u, 0u, 0u}, w = {0u, 0u, 0u, 0u};
    if (L > 0) {
      u = *reinterpret_cast<const u32x4*>(a.k + (kvh + krow) * D + s * 16 + h * 8);
      w = *reinterpret_cast<const u32x4*>(a.v + (kvh + krow) * D + s * 16 + h * 8);
    }
    kf[s] = as_bf16x8(u);
    vf[s] = as_bf16x8(w);
  }

  // ---- tile loads: Q and dO rows of tile `it` into ring buffer `buf`
  // (rows past Sq repeat row Sq - 1; their lse2 = +inf zeroes them), and
  // the lse2 row (even waves) or the D row (odd waves, the same bytes
  // twice), one dword per lane.  Tiles past the last are clamped to it, so
  // every wave issues the same loads every tile and no branch is needed.
  const int dma_row = wave * S::ROWS_PER_KB + lane / S::CHUNKS;
  const int dma_ch = ((lane % S::CHUNKS) ^ fwd_swz<D>(dma_row)) * 16;
  const uint32_t qd_base = lds_addr(&qd_lds[0]);
  const uint32_t rl_base = lds_addr(&rl_lds[0]);
  const uint32_t qd_w = __builtin_amdgcn_readfirstlane(qd_base + wave * 1024);
  struct TileSrc {
    const char* qg;
    const char* dg;
    const float* rows;
    int tlim;  // last valid row of the tile
    uint32_t lbuf, rdst;
  };
  auto tile_src = [&](int it, int buf) {
    it = min(it, n_it - 1);
    const int hq = g * G + it / n_qt;
    const int q0 = (qt_first + it % n_qt) * BQ;
    const size_t row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
    const size_t prow = ((size_t)b * a.Hq + hq) * (size_t)a.sq_pad + q0;
    TileSrc t;
    t.qg = reinterpret_cast<const char*>(a.q + (row0 + q0) * D);
    t.dg = reinterpret_cast<const char*>(a.dout + (row0 + q0) * D);
    t.rows = ((wave & 1) ? a.delta : a.lse2) + prow;
    t.tlim = a.Sq - 1 - q0;
    t.lbuf = qd_w + buf * S::BUF_BYTES;
    t.rdst = __builtin_amdgcn_readfirstlane(rl_base + buf * S::RL_BYTES + (wave & 1) * BQ * 4);
    return t;
  };
  auto issue_block = [&](const TileSrc& t, int p) {
    const uint32_t goff = (uint32_t)(min(dma_row + p * S::ROW_STEP, t.tlim) * ROW_BYTES + dma_ch);
    load_lds16_buf(t.qg, TILE_BYTES, goff, t.lbuf + p * S::WAVES * 1024);
    load_lds16_buf(t.dg, TILE_BYTES, goff, t.lbuf + TILE_BYTES + p * S::WAVES * 1024);
  };
  auto issue_rows = [&](const TileSrc& t) {
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(t.rows + lane),
                                     (void __attribute__((address_space(3)))*)(uintptr_t)t.rdst,
                                     4, 0, 0);
  };
  // vector-memory operations per tile and wave
  constexpr int LPT = 2 * S::BLOCKS_PER_WAVE + 1;

  // ---- LDS read addresses (the ring buffer's offset is folded in and
  // moved on per tile) ----
  // Q / dO fragment s of row n + 32 ch: Q at qa[s] + 32 ch rows, dO one
  // tile further
  uint32_t qa[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    qa[s] = qd_base + n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
  // transposing reads: rows 4 h + i/4 (+ 8), columns 32 db + 16 ((l/16) % 2)
  // + 4 (i % 4), i = l % 16
  uint32_t qt[DBLK][2];
  {
    const int tr_i = lane & 15;
    const int tr_row = 4 * h + (tr_i >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (tr_i & 3);
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int r = tr_row + 8 * hh;
        const int col = db * 32 + tr_col;
        qt[db][hh] = qd_base + r * ROW_BYTES + ((((col >> 3) ^ fwd_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }
  // lse2 / D of rows 32 ch + 8 j + 4 h .. +3
  uint32_t la = rl_base + 16 * h;

  f32x16 dk_acc[DBLK], dv_acc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk_acc[db][r] = dv_acc[db][r] = 0.f;

  f32x16 sacc[2][2];  // [chunk][S, dP]
  u32x4 lv[8];        // lse2 (j = 0..3) and D (4 + j) of the chunk B works on
  bf16x8 pf[2], dsf[2];
  int diag = 0;       // key - off - (first row of the chunk) - 4 h

  // One pipeline step: A(chunk ACH of the tile the fragment addresses point
  // at) with B(chunk BCH) on the vector ALU in between, then C(chunk BCH),
  // then the lse2 / D reads for chunk LCH (read by the next step's B).  -1:
  // no such part.  Elements with diag > 8 (r/4) + r % 4 are masked.
  // mid() runs between A and C (while C's first reads are in flight), and
  // dma(M) after C's M-th pair of products.
  auto step = [&](auto ach_tag, auto bch_tag, auto lch_tag, auto&& mid, auto&& dma) {
    constexpr int ACH = decltype(ach_tag)::value;
    constexpr int BCH = decltype(bch_tag)::value;
    constexpr int LCH = decltype(lch_tag)::value;
    constexpr int NA = ACH >= 0 ? 2 * KSTEPS : 0;
    constexpr int NC = BCH >= 0 ? 8 * DBLK : 0;
    constexpr int NL = LCH >= 0 ? 8 : 0;
    constexpr int TOT = NA + NC + NL;
    constexpr int RS = S::RW < TOT ? S::RW : TOT;
    static_assert(RS >= 4 || NC == 0, "C consumes four reads at a time");
    u32x4 ar[NA > 0 ? NA : 1];
    u32x2 cr[NC > 0 ? NC : 1];
    // item J of the read stream: A fragments (Q s, dO s for s = 0, 1, ..),
    // then C's transposing reads (kc, db, dO lo / hi, Q lo / hi), then the
    // lse2 / D rows of chunk LCH
    auto issue = [&](auto j_tag) {
      constexpr int J = decltype(j_tag)::value;
      if constexpr (J < NA) {
        constexpr int OFF = (J % 2) * TILE_BYTES + (ACH > 0 ? ACH : 0) * 32 * ROW_BYTES;
        ar[J] = lds_read_b128_async_off<OFF>(qa[J / 2]);
      } else if constexpr (J < NA + NC) {
        constexpr int C = J - NA;
        constexpr int KC = C / (4 * DBLK), DB = (C / 4) % DBLK, W = C % 4;
        constexpr int OFF = (W < 2 ? TILE_BYTES : 0) + ((BCH > 0 ? BCH : 0) * 32 + KC * 16) * ROW_BYTES;
        cr[C] = lds_read_tr16_async_off<OFF>(qt[DB][W % 2]);
      } else if constexpr (J < TOT) {
        constexpr int Lx = J - NA - NC;
        constexpr int OFF = (Lx / 4) * BQ * 4 + (LCH > 0 ? LCH : 0) * 128 + (Lx % 4) * 32;
        lv[Lx] = lds_read_b128_async_off<OFF>(la);
      }
    };
    static_for<0, RS>(issue);

    // B: element r of chunk BCH (row 8 (r/4) + 4 h + r % 4 of the chunk)
    float pe[8], de[8];
    auto b_elem = [&](auto r_tag) {
      constexpr int R = decltype(r_tag)::value;
      if constexpr (BCH >= 0) {
        const float sv = sacc[BCH > 0 ? 1 : 0][0][R];
        const float dp = sacc[BCH > 0 ? 1 : 0][1][R];
        const float l2 = __uint_as_float(lv[R / 4][R % 4]);
        const float dl = __uint_as_float(lv[4 + R / 4][R % 4]);
        float p = fast_exp2(fmaf(sv, c, -l2));
        p = diag <= 8 * (R / 4) + (R % 4) ? p : 0.f;
        pe[R % 8] = p;
        de[R % 8] = p * (dp - dl);
        if constexpr (R % 8 == 7) {
          pf[R / 8] = to_bf16x8(pe[0], pe[1], pe[2], pe[3], pe[4], pe[5], pe[6], pe[7]);
          dsf[R / 8] = to_bf16x8(de[0], de[1], de[2], de[3], de[4], de[5], de[6], de[7]);
        }
      }
    };

    if constexpr (NA > 0) {
      constexpr int AC = ACH > 0 ? 1 : 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[AC][0][r] = sacc[AC][1][r] = 0.f;
      constexpr int EPM = 16 / NA;  // B elements per product
      static_for<0, NA>([&](auto i_tag) {
        constexpr int I = decltype(i_tag)::value;
        constexpr int AHEAD = (I + RS < TOT ? I + RS : TOT) - I - 1;
        lds_wait_lgkm<AHEAD>();
        lds_ready(ar[I]);
        if constexpr (I == 0 && BCH >= 0) {
          // the lse2 / D reads were issued before this step's
#pragma unroll
          for (int l = 0; l < 8; ++l) lds_ready(lv[l]);
        }
        if constexpr (I % 2 == 0)
          sacc[AC][0] = mfma32(as_bf16x8(ar[I]), kf[I / 2], sacc[AC][0]);  // S
        else
          sacc[AC][1] = mfma32(as_bf16x8(ar[I]), vf[I / 2], sacc[AC][1]);  // dP
        // The product's result passes through an empty volatile statement,
        // which keeps the product in this group: otherwise the compiler
        // sinks all of A's products below B's vector work, and the two no
        // longer overlap.
        asm volatile("" : "+a"(sacc[AC][I % 2]));
        issue(std::integral_constant<int, I + RS>());
        static_for<0, EPM>([&](auto e_tag) {
          b_elem(std::integral_constant<int, I * EPM + decltype(e_tag)::value>());
        });
        __builtin_amdgcn_sched_barrier(0);
      });
    } else if constexpr (BCH >= 0) {
      lds_wait_lgkm<RS>();
#pragma unroll
      for (int l = 0; l < 8; ++l) lds_ready(lv[l]);
      static_for<0, 16>(b_elem);
      __builtin_amdgcn_sched_barrier(0);
    }

    mid();

    if constexpr (NC > 0) {
      static_for<0, 2 * DBLK>([&](auto m_tag) {
        constexpr int M = decltype(m_tag)::value;  // (kc, db) = (M / DBLK, M % DBLK)
        constexpr int BASE = NA + 4 * M;           // stream index of its first read
        constexpr int AHEAD = (BASE + RS < TOT ? BASE + RS : TOT) - (BASE + 3) - 1;
        static_assert(AHEAD >= 0, "read window");
        lds_wait_lgkm<AHEAD>();
        u32x2& d0 = cr[4 * M];
        u32x2& d1 = cr[4 * M + 1];
        u32x2& q0r = cr[4 * M + 2];
        u32x2& q1r = cr[4 * M + 3];
        lds_ready(d0);
        lds_ready(d1);
        lds_ready(q0r);
        lds_ready(q1r);
        const bf16x8 dt = as_bf16x8(u32x4{d0[0], d0[1], d1[0], d1[1]});
        const bf16x8 qtf = as_bf16x8(u32x4{q0r[0], q0r[1], q1r[0], q1r[1]});
        dv_acc[M % DBLK] = mfma32(dt, pf[M / DBLK], dv_acc[M % DBLK]);
        dk_acc[M % DBLK] = mfma32(qtf, dsf[M / DBLK], dk_acc[M % DBLK]);
        static_for<0, 4>([&](auto e_tag) {
          issue(std::integral_constant<int, BASE + RS + decltype(e_tag)::value>());
        });
        dma(m_tag);
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    // remaining reads of the stream (the lse2 / D rows for the next step)
    static_for<NA + NC + RS, TOT>(issue);
  };

  using N1 = std::integral_constant<int, -1>;
  using C0 = std::integral_constant<int, 0>;
  using C1 = std::integral_constant<int, 1>;

  auto none = [&]() {};
  auto no_dma = [&](auto) {};
  if (n_it > 0) {
    static_for<0, NBUF - 1>([&](auto i_tag) {
      constexpr int I = decltype(i_tag)::value;
      const TileSrc t = tile_src(I, I);
      static_for<0, S::BLOCKS_PER_WAVE>([&](auto p_tag) { issue_block(t, p_tag); });
      issue_rows(t);
    });
    wait_vmcnt<(NBUF - 2) * LPT>();  // tile 0
    __syncthreads();
    step(C0(), N1(), C0(), none, no_dma);  // A(tile 0, chunk 0), lse2 / D of chunk 0
  }
  const uint32_t ring = NBUF * S::BUF_BYTES;
  // C's pairs of products between two Q / dO blocks of the next load
  constexpr int PAIRS_PER_BLOCK = 2 * DBLK / S::BLOCKS_PER_WAVE;
  static_assert(PAIRS_PER_BLOCK >= 2 && 2 * DBLK % S::BLOCKS_PER_WAVE == 0, "load spacing");
  for (int it = 0; it < n_it; ++it) {
    const int buf = it % NBUF;
    // ring offset from this tile's buffer to the next one's
    const int adv = buf == NBUF - 1 ? (int)S::BUF_BYTES - (int)ring : S::BUF_BYTES;
    const int adv_rl = buf == NBUF - 1 ? S::RL_BYTES - NBUF * S::RL_BYTES : S::RL_BYTES;
    const int q0 = (qt_first + it % n_qt) * BQ;
    const bool m0 = CAUSAL && q0 + off < kw0 + 31;
    const bool m1 = CAUSAL && q0 + 32 + off < kw0 + 31;

    // chunk 0: A(chunk 1) with B(chunk 0), C(chunk 0), rows of chunk 1.
    // Between A and C: tile it + 1 must have landed, and every wave must be
    // done with tile it - 1, whose buffer then takes tile it + NBUF - 1
    // (loaded during C; C's reads of tile it are already in flight).
    // The loop body has no branch around the steps: a branch would make
    // the compiler move the accumulators between register files at every
    // product.  So the mask is always applied (an unmasked chunk gets a
    // threshold every element passes), tiles past the last are loaded
    // clamped, and the last tile's second step also forms A of a tile that
    // does not exist (in-bounds reads of a stale ring buffer, never used).
    diag = m0 ? key - off - q0 - 4 * h : -0x40000000;
    TileSrc nxt;
    auto mid = [&]() {
      wait_vmcnt<LPT>();
      __syncthreads();
      nxt = tile_src(it + NBUF - 1, (it + NBUF - 1) % NBUF);
    };
    auto dma = [&](auto m_tag) {
      constexpr int M = decltype(m_tag)::value;
      if constexpr (M % PAIRS_PER_BLOCK == 0) issue_block(nxt, M / PAIRS_PER_BLOCK);
      if constexpr (M == 1) issue_rows(nxt);
    };
    step(C1(), C0(), C1(), mid, dma);
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) qa[s] += adv;
    la += adv_rl;

    // chunk 1: A(next tile, chunk 0) with B(chunk 1), C(chunk 1), rows of
    // the next tile's chunk 0
    diag = m1 ? key - off - q0 - 32 - 4 * h : -0x40000000;
    step(C0(), C1(), C0(), none, no_dma);
    // the transposing reads move on once C of chunk 1 is done
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
      qt[db][0] += adv;
      qt[db][1] += adv;
    }
  }
  wait_vmcnt<0>();  // loads of clamped tiles past the last

  // dK = scale * dk_acc^T, dV = dv_acc^T, staged through LDS so that the
  // stores are whole rows: lane (key n, k-group h) holds head dims
  // db*32 + 8 (r/4) + 4 h + r % 4 of its key; keys past the sequence get
  // zeros.  The ring is free once every wave is past its last read.
  __syncthreads();
  const uint32_t stage = qd_base + wave * 2 * 32 * ROW_BYTES;
  const bool kvalid = key < L;
  store_rows_t<D>(dk_acc, kvalid ? a.scale : 0.f, stage, n, h, lane,
                  a.dk + (kvh + kw0) * D, D, a.Skv - kw0);
  store_rows_t<D>(dv_acc, kvalid ? 1.f : 0.f, stage + 32 * ROW_BYTES, n, h, lane,
                  a.dv + (kvh + kw0) * D, D, a.Skv - kw0);
}

}  // namespace mk
