// decode_kernel.hpp -- split-KV decode attention for gfx950.
//
// Kernel 1 (dec_split_kernel): one single-wave workgroup per (split, kv
// head, batch).  The G = Hq/Hkv query heads of the kv head are the columns
// of 16x16x32 MFMA blocks, so every cached K/V byte is read once for all
// of them.  The wave streams its split 32 keys per stage through a private
// ring of STAGES LDS slots, loading K and V HBM -> LDS with coalesced 1 KB
// wave loads (global_load_lds_dwordx4) STAGES-1 stages ahead of use; no
// barrier is needed since no other wave touches its LDS.  All LDS reads are
// issued as inline assembly and waited on right before use, so no loaded
// register lives across an iteration (the compiler's own waits would
// otherwise serialise the prefetch).  The wave keeps its own online-softmax
// state and writes the split's normalised output and natural-log LSE.
//
// Kernel 2 (dec_combine_kernel): per (batch, query head), merge the splits
// by their log-sum-exp: LSE = log sum_s exp(LSE_s), O = sum_s
// exp(LSE_s - LSE) O_s.  Splits at or past the sequence end hold nothing
// and are not read.
#pragma once

#include <type_traits>

#include "mk_common.hpp"

namespace mk {

constexpr float kDecRescaleSlack = 8.0f;

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
  static constexpr int BN = 32;                        // keys per stage
  static constexpr int STAGES = 3;                     // LDS ring slots
  static constexpr int CHUNKS = D / 8;                 // 16-byte chunks per row
  static constexpr int ROW_BYTES = D * 2;
  static constexpr int ROWS_PER_KB = 512 / D;          // rows per 1 KB wave load
  static constexpr int BLOCKS = BN * ROW_BYTES / 1024; // 1 KB loads per tensor per stage
  static constexpr int LOADS_PER_STAGE = 2 * BLOCKS;   // K and V
  static constexpr int KSTEPS = D / 32;                // 16x16x32 steps over the head dim
  static constexpr int DBLK = D / 16;                  // 16-row blocks of O^T
  static constexpr int TILE_BYTES = BN * ROW_BYTES;    // one tensor, one stage
  static constexpr int SLOT_BYTES = 2 * TILE_BYTES;    // K then V
};

template <int D>
__global__ __launch_bounds__(64) void dec_split_kernel(DecArgs a) {
  using S = DecShape<D>;
  constexpr int BN = S::BN;
  constexpr int RB = S::ROW_BYTES;
  __shared__ __attribute__((aligned(1024))) char kv_lds[S::STAGES * S::SLOT_BYTES];

  const int lane = threadIdx.x;
  const int c16 = lane & 15;  // MFMA column (query head of the group) / row (key)
  const int gq = lane >> 4;   // MFMA k-group

  // Work item order: the split index varies slowest.  Workgroups are
  // dealt round-robin to the 8 XCDs, so the XCD of an item is set by its
  // (batch, kv head) pair and not by the split index; the low splits,
  // which every sequence has, are spread over all XCDs instead of piling
  // onto the few that a split-fastest order would give them.
  const int n_gb = a.B * a.Hkv;
  const int sidx = blockIdx.x / n_gb;
  const int gb = blockIdx.x - sidx * n_gb;
  const int b = gb / a.Hkv;
  const int g = gb - b * a.Hkv;
  const int G = a.Hq / a.Hkv;
  const int L = clamp_len(a.kv_seqlens[b], a.Smax);
  const int k_begin = sidx * a.split;
  if (k_begin >= L) return;  // empty split: nothing to write, the merge skips it
  const int k_end = min(k_begin + a.split, L);
  const int n_t = (k_end - k_begin + BN - 1) / BN;
  // The split's stages are walked starting at a per-workgroup rotation, so
  // that workgroups running together do not stream addresses that agree
  // modulo large powers of two.  The order of the stages does not change
  // the result beyond rounding.
  const int rot = (int)(((unsigned)(b * 131 + g * 37 + sidx * 7)) % (unsigned)n_t);
  auto stage_key0 = [&](int t) {
    int u = t + rot;
    if (u >= n_t) u -= n_t;
    return k_begin + u * BN;
  };

  const size_t kv_off = ((size_t)b * a.Hkv + g) * (size_t)a.Smax * D;
  const char* __restrict__ kg = reinterpret_cast<const char*>(a.kc + kv_off);
  const char* __restrict__ vg = reinterpret_cast<const char*>(a.vc + kv_off);

  // Q^T fragments: column c16 is query head g*G + c16 (zero when c16 >= G);
  // loaded before any cache traffic so that waiting for them waits for
  // nothing else.
  bf16x8 qf[S::KSTEPS];
#pragma unroll
  for (int s = 0; s < S::KSTEPS; ++s) {
    u32x4 u = {0u, 0u, 0u, 0u};
    if (c16 < G)
      u = *reinterpret_cast<const u32x4*>(a.q + ((size_t)b * a.Hq + g * G + c16) * D + s * 32 +
                                          gq * 8);
    qf[s] = as_bf16x8(u);
  }

  // Stage t -> ring slot t % STAGES: K rows, then V rows, each tile row
  // blk*ROWS_PER_KB + l/CHUNKS with its 16-byte chunks XOR-swizzled.  Rows
  // past the split end re-read its last row (the mask zeroes their
  // weight), so no load leaves the valid keys [0, L).
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(kv_lds));
  const int dma_row = lane / S::CHUNKS;
  constexpr int ROW_STEP = S::ROWS_PER_KB;  // rows per 1 KB block
  auto issue = [&](int t) {
    const uint32_t slot = lds0 + (uint32_t)(t % S::STAGES) * S::SLOT_BYTES;
    const int key0 = stage_key0(t);
    const int lim = k_end - 1 - key0;  // last valid row of the stage
    const char* kt_g = kg + (size_t)key0 * RB;
    const char* vt_g = vg + (size_t)key0 * RB;
#pragma unroll
    for (int blk = 0; blk < S::BLOCKS; ++blk) {
      const int row = min(dma_row + blk * ROW_STEP, lim);
      const int ch = ((lane % S::CHUNKS) ^ chunk_swz<D>(dma_row + blk * ROW_STEP)) * 16;
      const uint32_t goff = (uint32_t)(row * RB + ch);
      load_lds16_at(kt_g + goff, slot + blk * 1024);
      load_lds16_at(vt_g + goff, slot + S::TILE_BYTES + blk * 1024);
    }
  };

  // Lane parts of the LDS read addresses within a slot.  K: row 16 kb +
  // c16, logical chunk 4 s + gq.  V (transposing): rows 4 gq + c16/4 (+ 16),
  // columns 16 db + 4 (c16 % 4).
  uint32_t k_addr[2][S::KSTEPS];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int s = 0; s < S::KSTEPS; ++s) {
      const int r = kb * 16 + c16;
      k_addr[kb][s] = r * RB + (((4 * s + gq) ^ chunk_swz<D>(r)) << 4);
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

  auto consume = [&](int t) {
    const uint32_t slot = lds0 + (uint32_t)(t % S::STAGES) * S::SLOT_BYTES;
    const int key0 = stage_key0(t);
    // S^T = K Q^T for the 32 keys of the stage (two 16-key blocks).
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      u32x4 kf[S::KSTEPS];
#pragma unroll
      for (int s = 0; s < S::KSTEPS; ++s) kf[s] = lds_read_b128_async_off<0>(slot + k_addr[kb][s]);
      static_assert(S::KSTEPS == 2 || S::KSTEPS == 4, "head dim 64 or 128");
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
    // 16 kb + 4 gq + r.
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = sacc[kb][r] * c;
        if (key0 + kb * 16 + 4 * gq + r >= k_end) x = kNegInf;
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
        const u32x4 w = {vr[j][0][0], vr[j][0][1], vr[j][1][0], vr[j][1][1]};
        o_acc[db0 + j] = mfma16(as_bf16x8(w), pf, o_acc[db0 + j]);
      }
    }
  };

  static_assert(S::STAGES == 3, "the wait counts below assume two stages ahead");
  issue(0);
  if (1 < n_t) issue(1);
  for (int t = 0; t < n_t; ++t) {
    // Before stage t is read, only the stages issued after it may still be
    // loading.  Slot (t+2) % 3 held stage t-1, whose reads all completed
    // in the previous iteration.
    if (t + 2 < n_t) {
      issue(t + 2);
      wait_vmcnt<2 * S::LOADS_PER_STAGE>();
    } else if (t + 1 < n_t) {
      wait_vmcnt<S::LOADS_PER_STAGE>();
    } else {
      wait_vmcnt<0>();
    }
    consume(t);
  }

  // l: each k-group summed its own keys; add the four groups.
  const float lsum = sum_xor32(sum_xor16(l_run));
  if (c16 < G) {
    const size_t pr = ((size_t)b * a.Hq + g * G + c16) * a.nsplit + sidx;
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
    for (int db = 0; db < S::DBLK; ++db) {
      const f32x4 w = {o_acc[db][0] * inv, o_acc[db][1] * inv, o_acc[db][2] * inv,
                       o_acc[db][3] * inv};
      *reinterpret_cast<f32x4*>(a.o_part + pr * D + db * 16 + 4 * gq) = w;
    }
    if (gq == 0) a.lse_part[pr] = lsum > 0.f ? (m_run + log2f(lsum)) * kLn2 : kNegInf;
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

// One wave per (batch, query head) row.  Every load the row needs (its
// length, the split LSEs, the partial outputs of up to 16 splits) is issued
// before any of them is used, so the kernel costs about one memory round
// trip: lanes take the splits for the max / sum, then the head dims for the
// weighted sum of partial outputs.
template <int D>
__global__ __launch_bounds__(256) void dec_combine_kernel(CombArgs a) {
  constexpr int PER_LANE = D / 64;
  constexpr int CHUNK = 16;  // splits whose partial outputs are loaded together
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, hq) row
  if (r >= a.B * a.Hq) return;
  const int b = r / a.Hq;
  const float* lp = a.lse_part + (size_t)r * a.nsplit;
  const float* op = a.o_part + (size_t)r * a.nsplit * D + lane * PER_LANE;
  const int len = a.kv_seqlens[b];
  float ls[(64 + 63) / 64];
  ls[0] = lane < a.nsplit ? lp[lane] : kNegInf;
  float part[CHUNK][PER_LANE];
#pragma unroll
  for (int s = 0; s < CHUNK; ++s)
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) part[s][i] = s < a.nsplit ? op[(size_t)s * D + i] : 0.f;

  const int L = clamp_len(len, a.Smax);
  const int ns = (L + a.split - 1) / a.split;  // splits holding keys
  // max over the valid splits (lanes beyond 64 splits loop)
  float M = lane < ns ? ls[0] : kNegInf;
  for (int s = 64 + lane; s < ns; s += 64) M = fmaxf(M, lp[s]);
  M = wave_max(M);
  float out[PER_LANE];
#pragma unroll
  for (int i = 0; i < PER_LANE; ++i) out[i] = 0.f;
  float lse = kNegInf;
  if (M != kNegInf) {
    float sum = lane < ns ? expf(ls[0] - M) : 0.f;
    for (int s = 64 + lane; s < ns; s += 64) sum += expf(lp[s] - M);
    lse = M + logf(wave_sum(sum));
    // weight of split s, taken from the lane that loaded its LSE
    const float w_lane = lane < ns ? expf(ls[0] - lse) : 0.f;
#pragma unroll
    for (int s = 0; s < CHUNK; ++s) {
      const float w = __shfl(w_lane, s, 64);
      if (s < ns)
#pragma unroll
        for (int i = 0; i < PER_LANE; ++i) out[i] += w * part[s][i];
    }
    for (int s = CHUNK; s < ns; ++s) {
      const float w = expf(lp[s] - lse);
#pragma unroll
      for (int i = 0; i < PER_LANE; ++i) out[i] += w * op[(size_t)s * D + i];
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
