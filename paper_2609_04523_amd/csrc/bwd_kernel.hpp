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
// Three kernels on one stream:
//   bwd_delta_kernel  D_i from the forward's O and dO (16 lanes per row);
//   bwd_dq_kernel     one workgroup per 128 query rows of one (b, hq),
//                     shaped like the forward: K and V 64-key tiles stream
//                     through LDS, each wave keeps its 32 rows' Q and dO in
//                     registers and accumulates dQ^T = K^T dS^T;
//   bwd_dkdv_kernel   one workgroup per 128 keys of one (b, kv head): each
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
  float* delta;          // workspace [B, Hq, Sq]: D_i
  const int* kv_seqlens;
  int B, Hq, Hkv, Sq, Skv;
  int n_qtiles;          // dQ kernel: ceil(Sq / 128)
  int n_kblocks;         // dK/dV kernel: ceil(Skv / 128)
  float scale;
  float scale_log2;      // scale * log2(e)
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// D_i = dO_i . O_i, 16 lanes per row of D bf16 values.
template <int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(BwdArgs a) {
  constexpr int LPR = 16;
  constexpr int WORDS = D / LPR / 2;  // 32-bit words (bf16 pairs) per lane
  const long long rows = (long long)a.B * a.Hq * a.Sq;
  const long long row = (long long)blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
  const int part = threadIdx.x % LPR;
  float acc = 0.f;
  if (row < rows) {
    const uint32_t* o = reinterpret_cast<const uint32_t*>(a.o + row * D) + part * WORDS;
    const uint32_t* d = reinterpret_cast<const uint32_t*>(a.dout + row * D) + part * WORDS;
#pragma unroll
    for (int w = 0; w < WORDS; ++w) {
      const uint32_t x = o[w], y = d[w];
      acc = fmaf(bf16_lo(x), bf16_lo(y), acc);
      acc = fmaf(bf16_hi(x), bf16_hi(y), acc);
    }
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (row < rows && part == 0) a.delta[row] = acc;
}

// P and the validity of one element; lse2 = LSE * log2 e of the row.
__device__ __forceinline__ float bwd_prob(float s, float c, float lse, bool valid) {
  const float p = fast_exp2(fmaf(s, c, -lse * kLog2e));
  return (valid && lse != kNegInf) ? p : 0.f;
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
  __shared__ __attribute__((aligned(1024))) uint16_t k_lds[2][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_lds[2][TILE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  // longest query tiles first
  const int per = a.B * a.Hq;
  const int t_ = blockIdx.x / per;
  const int rem = blockIdx.x - t_ * per;
  const int qt = a.n_qtiles - 1 - t_;
  const int b = rem / a.Hq, hq = rem - (rem / a.Hq) * a.Hq;
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
  const float lse = row_ok ? a.lse[row0 + qrow] : kNegInf;
  const float dl = row_ok ? a.delta[row0 + qrow] : 0.f;
  const int lim = CAUSAL ? min(L - 1, qrow + off) : L - 1;  // last key this row sees

  // tile loads, as in the forward kernel
  constexpr int ROW_STEP = WAVES * ROWS_PER_KB;
  const int dma_row = wave * ROWS_PER_KB + lane / CHUNKS;
  const int dma_ch = ((lane % CHUNKS) ^ fwd_swz<D>(dma_row)) * 16;
  const uint32_t k_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&k_lds[0][0]) + wave * 1024);
  const uint32_t v_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&v_lds[0][0]) + wave * 1024);
  auto issue_tile = [&](int kt, int buf) {
    const int tlim = L - 1 - kt * BN;
#pragma unroll
    for (int p = 0; p < BLOCKS_PER_WAVE; ++p) {
      const uint32_t goff = (uint32_t)(min(dma_row + p * ROW_STEP, tlim) * ROW_BYTES + dma_ch);
      const size_t toff = (size_t)kt * BN * ROW_BYTES;
      const uint32_t lds_off = buf * TILE_BYTES + p * WAVES * 1024;
      load_lds16_at(kg + toff + goff, k_lds_w + lds_off);
      load_lds16_at(vg + toff + goff, v_lds_w + lds_off);
    }
  };

  // LDS read addresses: K / V rows (A operand, 32 keys x 8 head dims) and
  // transposing K^T reads (A operand of dQ^T = K^T dS^T)
  uint32_t kr_addr[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    kr_addr[s] = n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
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
        kt_addr[db][hh] = r * ROW_BYTES + ((((col >> 3) ^ fwd_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }
  const uint32_t k0 = lds_addr(&k_lds[0][0]), v0 = lds_addr(&v_lds[0][0]);

  f32x16 acc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  if (n_kt > 0) issue_tile(0, 0);
  if (n_kt > 1) issue_tile(1, 1);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < n_kt)
      wait_vmcnt<LOADS_PER_TILE>();
    else
      wait_vmcnt<0>();
    __syncthreads();
    const uint32_t kb_base = k0 + buf * TILE_BYTES, vb_base = v0 + buf * TILE_BYTES;
    const int key0 = kt * BN;
    // S^T = K Q^T and dP^T = V dO^T for the tile's two 32-key blocks
    f32x16 st[2], dpt[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) st[kb][r] = dpt[kb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const uint32_t ad = kr_addr[s] + kb * 32 * ROW_BYTES;
        const bf16x8 kf = as_bf16x8(lds_read_b128_at(kb_base + ad));
        const bf16x8 vf = as_bf16x8(lds_read_b128_at(vb_base + ad));
        st[kb] = mfma32(kf, qf[s], st[kb]);
        dpt[kb] = mfma32(vf, df[s], dpt[kb]);
      }
    }
    // dS^T = P^T (dP^T - D) as bf16, 16-key chunk kc = rows 8 (kc % 2) .. +7
    // of key block kc / 2
    bf16x8 dsf[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      float e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = 8 * (kc % 2) + j;
        const int key = key0 + (kc / 2) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        const float p = bwd_prob(st[kc / 2][r], c, lse, key <= lim);
        e[j] = p * (dpt[kc / 2][r] - dl);
      }
      dsf[kc] = to_bf16x8(e[0], e[1], e[2], e[3], e[4], e[5], e[6], e[7]);
    }
    // dQ^T += K^T dS^T over the four 16-key chunks
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
#pragma unroll
      for (int db = 0; db < DBLK; ++db) {
        const uint32_t base = kb_base + kc * 16 * ROW_BYTES;
        const bf16x4 lo = lds_read_tr16_at(base + kt_addr[db][0]);
        const bf16x4 hi = lds_read_tr16_at(base + kt_addr[db][1]);
        acc[db] = mfma32(cat(lo, hi), dsf[kc], acc[db]);
      }
    }
    __syncthreads();
    if (kt + 2 < n_kt) issue_tile(kt + 2, buf);
  }

  // dQ = scale * acc^T: lane (query n, k-group h) holds head dims
  // db*32 + 8 (r/4) + 4 h + r % 4
  if (row_ok) {
    uint16_t* dst = a.dq + (row0 + qrow) * D;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = db * 32 + 8 * r4 + 4 * h;
        const u32x2 w = {(uint32_t)to_bf16_bits(acc[db][4 * r4 + 0] * a.scale) |
                             ((uint32_t)to_bf16_bits(acc[db][4 * r4 + 1] * a.scale) << 16),
                         (uint32_t)to_bf16_bits(acc[db][4 * r4 + 2] * a.scale) |
                             ((uint32_t)to_bf16_bits(acc[db][4 * r4 + 3] * a.scale) << 16)};
        *reinterpret_cast<u32x2*>(dst + d) = w;
      }
  }
}

// ---------------------------------------------------------------------------
// dK, dV: workgroup = 4 waves x 32 keys of one (b, kv head); 64-row tiles of
// Q, dO (and their LSE, D) of every query head of the group.
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(BwdArgs a) {
  constexpr int WAVES = 4, BK = 128, BQ = 64;
  constexpr int KSTEPS = D / 16, DBLK = D / 32, CHUNKS = D / 8;
  constexpr int ROW_BYTES = D * 2, TILE = BQ * D, TILE_BYTES = TILE * 2;
  constexpr int ROWS_PER_KB = 512 / D;
  constexpr int BLOCKS_PER_WAVE = BQ * D * 2 / 1024 / WAVES;
  // per thread per tile: Q and dO blocks, plus one dword of LSE or D on
  // waves 0 and 1
  __shared__ __attribute__((aligned(1024))) uint16_t q_lds[2][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t do_lds[2][TILE];
  __shared__ __attribute__((aligned(256))) float lse_lds[2][BQ];
  __shared__ __attribute__((aligned(256))) float dl_lds[2][BQ];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  // key blocks in ascending order: under the causal mask the first blocks
  // are seen by the most query rows
  const int per = a.B * a.Hkv;
  const int kblk = blockIdx.x / per;
  const int rem = blockIdx.x - kblk * per;
  const int b = rem / a.Hkv, g = rem - (rem / a.Hkv) * a.Hkv;
  const int G = a.Hq / a.Hkv;
  const int L = a.kv_seqlens ? clamp_len(a.kv_seqlens[b], a.Skv) : a.Skv;
  const int off = L - a.Sq;
  const int k0 = kblk * BK;
  const int kw0 = k0 + wave * 32;  // this wave's first key
  const int key = kw0 + n;         // this lane's key (MFMA column)
  const float c = a.scale_log2;

  // query tiles that can see a key of the block
  int q_first = CAUSAL ? max(0, k0 - off) : 0;
  if (k0 >= L) q_first = a.Sq;  // no valid key: nothing to accumulate
  const int qt_first = q_first / BQ;
  const int n_qt = q_first < a.Sq ? (a.Sq + BQ - 1) / BQ - qt_first : 0;
  const int n_it = G * n_qt;

  // K^T and V^T fragments of this wave's keys (B operand: lane = key
  // column, k-group h = head dims 16 s + 8 h .. +7); rows past the
  // sequence read its last row (their gradients are masked to zero)
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

  // tile loads: Q and dO rows like the forward's K/V tiles; LSE by wave 0
  // and D by wave 1, one dword per lane
  constexpr int ROW_STEP = WAVES * ROWS_PER_KB;
  const int dma_row = wave * ROWS_PER_KB + lane / CHUNKS;
  const int dma_ch = ((lane % CHUNKS) ^ fwd_swz<D>(dma_row)) * 16;
  const uint32_t q_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&q_lds[0][0]) + wave * 1024);
  const uint32_t do_lds_w = __builtin_amdgcn_readfirstlane(lds_addr(&do_lds[0][0]) + wave * 1024);
  const uint32_t lse_lds0 = __builtin_amdgcn_readfirstlane(lds_addr(&lse_lds[0][0]));
  const uint32_t dl_lds0 = __builtin_amdgcn_readfirstlane(lds_addr(&dl_lds[0][0]));
  auto issue_tile = [&](int it, int buf) {
    const int hq = g * G + it / n_qt;
    const int q0 = (qt_first + it % n_qt) * BQ;
    const size_t row0 = ((size_t)b * a.Hq + hq) * (size_t)a.Sq;
    const int tlim = a.Sq - 1 - q0;  // last valid row of the tile
    const char* qg = reinterpret_cast<const char*>(a.q + (row0 + q0) * D);
    const char* dg = reinterpret_cast<const char*>(a.dout + (row0 + q0) * D);
#pragma unroll
    for (int p = 0; p < BLOCKS_PER_WAVE; ++p) {
      const uint32_t goff = (uint32_t)(min(dma_row + p * ROW_STEP, tlim) * ROW_BYTES + dma_ch);
      const uint32_t lds_off = buf * TILE_BYTES + p * WAVES * 1024;
      load_lds16_at(qg + goff, q_lds_w + lds_off);
      load_lds16_at(dg + goff, do_lds_w + lds_off);
    }
    if (wave < 2) {
      const float* src = (wave == 0 ? a.lse : a.delta) + row0 + q0 + min(lane, tlim);
      const uint32_t dst = (wave == 0 ? lse_lds0 : dl_lds0) + buf * BQ * 4;
      __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                       (void __attribute__((address_space(3)))*)(uintptr_t)dst,
                                       4, 0, 0);
    }
  };

  // LDS read addresses: Q / dO rows (A operand: row = query, 8 head dims)
  // and transposing Q^T / dO^T reads (A operand of dK^T, dV^T)
  uint32_t qr_addr[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    qr_addr[s] = n * ROW_BYTES + (((2 * s + h) ^ fwd_swz<D>(n)) << 4);
  uint32_t qt_addr[DBLK][2];
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
        qt_addr[db][hh] = r * ROW_BYTES + ((((col >> 3) ^ fwd_swz<D>(r)) << 4) | ((col & 7) * 2));
      }
  }
  const uint32_t ql0 = lds_addr(&q_lds[0][0]), dol0 = lds_addr(&do_lds[0][0]);

  f32x16 dk_acc[DBLK], dv_acc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk_acc[db][r] = dv_acc[db][r] = 0.f;

  if (n_it > 0) issue_tile(0, 0);
  if (n_it > 1) issue_tile(1, 1);
  for (int it = 0; it < n_it; ++it) {
    const int buf = it & 1;
    if (it + 1 < n_it) {
      // the next tile's loads may still be in flight
      if (wave < 2)
        wait_vmcnt<2 * BLOCKS_PER_WAVE + 1>();
      else
        wait_vmcnt<2 * BLOCKS_PER_WAVE>();
    } else {
      wait_vmcnt<0>();
    }
    __syncthreads();
    const int q0 = (qt_first + it % n_qt) * BQ;
    // rows of this tile this wave's keys can be seen by
    const bool live = !CAUSAL || q0 + BQ - 1 + off >= kw0;
    if (live) {
      const uint32_t qb_base = ql0 + buf * TILE_BYTES, db_base = dol0 + buf * TILE_BYTES;
      const float* lse_t = &lse_lds[buf][0];
      const float* dl_t = &dl_lds[buf][0];
#pragma unroll
      for (int ch = 0; ch < BQ / 32; ++ch) {
        // S = Q K^T and dP = dO V^T for query rows 32 ch .. +31
        f32x16 sq, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) sq[r] = dp[r] = 0.f;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
          const uint32_t ad = qr_addr[s] + ch * 32 * ROW_BYTES;
          const bf16x8 qa = as_bf16x8(lds_read_b128_at(qb_base + ad));
          const bf16x8 da = as_bf16x8(lds_read_b128_at(db_base + ad));
          sq = mfma32(qa, kf[s], sq);
          dp = mfma32(da, vf[s], dp);
        }
        // P and dS; element r is query row 32 ch + 8 (r/4) + 4 h + r % 4
        bf16x8 pf[2], dsf[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          float pe[8], de[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int r = 8 * kc + j;
            const int qr = ch * 32 + 8 * (r >> 2) + 4 * h + (r & 3);  // row within the tile
            const int qabs = q0 + qr;
            const bool valid = qabs < a.Sq && key < L && (!CAUSAL || key <= qabs + off);
            const float p = bwd_prob(sq[r], c, lse_t[qr], valid);
            pe[j] = p;
            de[j] = p * (dp[r] - dl_t[qr]);
          }
          pf[kc] = to_bf16x8(pe[0], pe[1], pe[2], pe[3], pe[4], pe[5], pe[6], pe[7]);
          dsf[kc] = to_bf16x8(de[0], de[1], de[2], de[3], de[4], de[5], de[6], de[7]);
        }
        // dV^T += dO^T P and dK^T += Q^T dS over the two 16-row chunks
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          const uint32_t roff = (ch * 32 + kc * 16) * ROW_BYTES;
#pragma unroll
          for (int db = 0; db < DBLK; ++db) {
            const bf16x4 dlo = lds_read_tr16_at(db_base + roff + qt_addr[db][0]);
            const bf16x4 dhi = lds_read_tr16_at(db_base + roff + qt_addr[db][1]);
            dv_acc[db] = mfma32(cat(dlo, dhi), pf[kc], dv_acc[db]);
            const bf16x4 qlo = lds_read_tr16_at(qb_base + roff + qt_addr[db][0]);
            const bf16x4 qhi = lds_read_tr16_at(qb_base + roff + qt_addr[db][1]);
            dk_acc[db] = mfma32(cat(qlo, qhi), dsf[kc], dk_acc[db]);
          }
        }
      }
    }
    __syncthreads();
    if (it + 2 < n_it) issue_tile(it + 2, buf);
  }

  // dK = scale * dk_acc^T, dV = dv_acc^T: lane (key n, k-group h) holds
  // head dims db*32 + 8 (r/4) + 4 h + r % 4 of its key
  if (key < a.Skv) {
    uint16_t* dkr = a.dk + (kvh + key) * D;
    uint16_t* dvr = a.dv + (kvh + key) * D;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = db * 32 + 8 * r4 + 4 * h;
        const u32x2 wk = {(uint32_t)to_bf16_bits(dk_acc[db][4 * r4 + 0] * a.scale) |
                              ((uint32_t)to_bf16_bits(dk_acc[db][4 * r4 + 1] * a.scale) << 16),
                          (uint32_t)to_bf16_bits(dk_acc[db][4 * r4 + 2] * a.scale) |
                              ((uint32_t)to_bf16_bits(dk_acc[db][4 * r4 + 3] * a.scale) << 16)};
        const u32x2 wv = {(uint32_t)to_bf16_bits(dv_acc[db][4 * r4 + 0]) |
                              ((uint32_t)to_bf16_bits(dv_acc[db][4 * r4 + 1]) << 16),
                          (uint32_t)to_bf16_bits(dv_acc[db][4 * r4 + 2]) |
                              ((uint32_t)to_bf16_bits(dv_acc[db][4 * r4 + 3]) << 16)};
        *reinterpret_cast<u32x2*>(dkr + d) = wk;
        *reinterpret_cast<u32x2*>(dvr + d) = wv;
      }
  }
}

}  // namespace mk
