/*
 * mk_attn.h -- C ABI of the MI355X (gfx950) fused attention library.
 *
 * The operation is the attention forward of the paper's "Flash Attention"
 * and "GQA Attention" workloads (Table 2; tolerances in Table 4,
 * Appendix A), the one-token decode step of its "Paged Attention" /
 * "Ragged Paged Attention" family (Table 2) over a contiguous or paged
 * cache, packed ragged batches, the backward, and the decode step of its
 * "MLA Attention" workload:
 *
 *   O = softmax(Q K^T * scale + mask) V,   LSE = log(sum_j exp(s_j))
 *
 * with grouped heads (query head hq reads key/value head hq / (Hq/Hkv)),
 * causal masking aligned bottom-right (query i of Sq sits at absolute
 * position i + L_b - Sq, and sees keys j <= that position), per-sequence
 * key lengths L_b, and a natural-log LSE over the scaled, masked scores.
 * Fully masked rows give O = 0 and LSE = -inf.
 *
 * Conventions shared by every entry point:
 *   - All tensors live in device memory, are contiguous with the last
 *     dimension fastest, and are owned by the caller.  The library never
 *     allocates, frees or synchronises; every call only enqueues kernels
 *     on `stream` (a hipStream_t; NULL means the default stream) and
 *     returns.
 *   - bf16 tensors are passed as `const void*` (IEEE bfloat16 bits).
 *   - Every pointer must be 16-byte aligned (lse: 4-byte aligned).
 *   - Arguments are validated on the host before anything is enqueued;
 *     a non-zero mk_status is returned and nothing is launched.  Errors
 *     raised while kernels run surface at the caller's next
 *     synchronisation, as for any HIP call.
 *   - `kv_seqlens` lives on the device, so the host cannot check it; the
 *     kernels clamp each length into [0, Skv] (decode: [0, Smax]).  This
 *     follows the paper's robustness fix for ragged paged attention
 *     (Section 3.4): a bad length never produces an out-of-range slice.
 *   - Supported head dims: D = 64 and D = 128.
 *   - The library is stateless and thread-safe.
 */
#ifndef MK_ATTN_H
#define MK_ATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MK_OK = 0,
    MK_ERR_NULL = 1,        /* a required pointer is NULL */
    MK_ERR_SHAPE = 2,       /* a size is < 1, Hq % Hkv != 0, or too large */
    MK_ERR_UNSUPPORTED = 3, /* head dim / group size this library does not build */
    MK_ERR_ALIGN = 4,       /* a pointer is not aligned as required */
    MK_ERR_WORKSPACE = 5,   /* workspace missing or too small */
    MK_ERR_HIP = 6,         /* the HIP runtime refused a launch */
    MK_ERR_ARG = 7,         /* non-finite scale, bad causal flag or part count */
    MK_ERR_SCRATCH = 8      /* more decode scratch needed than the fixed array holds */
} mk_status;

/*
 * Attention forward (prefill, or any Sq <= Skv).
 *   q    [B, Hq,  Sq,  D] bf16
 *   k, v [B, Hkv, Skv, D] bf16
 *   o    [B, Hq,  Sq,  D] bf16 (written)
 *   lse  [B, Hq,  Sq]     fp32 natural-log LSE (written), or NULL to skip
 *   B, Hq, Hkv, Sq, Skv >= 1, Hq % Hkv == 0, D in {64, 128}
 *   causal      0 or 1 (bottom-right aligned, see above)
 *   scale       finite multiplier of q.k (usually 1/sqrt(D)); 0 is legal
 *   kv_seqlens  device int32 [B] valid key count per sequence, or NULL
 *               for Skv everywhere; clamped into [0, Skv] on the device
 *   stream      hipStream_t or NULL
 * Returns MK_OK or an mk_status; asynchronous on `stream`.
 */
int mk_attn_fwd(const void *q, const void *k, const void *v, void *o, float *lse,
                int B, int Hq, int Hkv, int Sq, int Skv, int D,
                int causal, float scale, const int *kv_seqlens, void *stream);

/*
 * Same as mk_attn_fwd, but o is fp32 [B, Hq, Sq, D]: the output is not
 * rounded to bf16, so the kernel's own error can be seen in isolation.
 */
int mk_attn_fwd_o32(const void *q, const void *k, const void *v, float *o, float *lse,
                    int B, int Hq, int Hkv, int Sq, int Skv, int D,
                    int causal, float scale, const int *kv_seqlens, void *stream);

/*
 * Same computation and result as mk_attn_fwd (bitwise: the same products
 * in the same order), with V read through a copy that the call first
 * writes into `workspace`: V^T in 64-key tiles laid out as the matrix
 * cores take it, so the forward reads its V operand from LDS with plain
 * 16-byte reads instead of transposing ones.  The copy costs one read and
 * one write of V (4 * B * Hkv * Skv * D bytes of HBM traffic), which pays
 * where each key tile is used by many query tiles (long causal sequences,
 * grouped query heads).  The forward itself runs as one workgroup per
 * compute unit, each taking 256-row query tiles from counters at the end
 * of the workspace until none are left (the K/V heads' tiles grouped by
 * XCD, so each XCD's L2 holds the heads it works on).
 *   workspace        device memory of at least
 *                    mk_attn_fwd_workspace_bytes(B, Hkv, Skv, D) bytes,
 *                    16-byte aligned, owned by the caller; overwritten by
 *                    the call (calls that share it on different streams
 *                    race)
 *   other arguments  as mk_attn_fwd (bf16 O)
 * Returns MK_OK or an mk_status (MK_ERR_NULL for a null workspace,
 * MK_ERR_ARG when it is smaller than required, MK_ERR_ALIGN when it is not
 * 16-byte aligned); asynchronous on `stream`.
 */
int mk_attn_fwd_ws(const void *q, const void *k, const void *v, void *o, float *lse,
                   int B, int Hq, int Hkv, int Sq, int Skv, int D,
                   int causal, float scale, const int *kv_seqlens,
                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * Workspace bytes mk_attn_fwd_ws needs: B * Hkv * ceil(Skv / 64) * 64 * D
 * * 2 for the V^T tiles, plus 1024 for the work-item counters of its
 * persistent grid.  Returns 0 for arguments mk_attn_fwd_ws would reject as
 * a shape (B, Hkv, Skv < 1, D not 64 or 128).
 */
size_t mk_attn_fwd_workspace_bytes(int B, int Hkv, int Skv, int D);

/*
 * Forward over a packed batch of variable-length sequences (the ragged
 * batches of the paper's "Ragged Paged Attention" workload, Table 2): each
 * sequence is attended on its own, with the same computation as
 * mk_attn_fwd.  Sequences with one query token are decode steps, so prefill
 * chunks and decode tokens can share one call.
 *   q, o   [total_q, Hq, D] bf16, token-major (a token's Hq heads adjacent);
 *          o is written only at rows some sequence owns
 *   k, v   [total_k, Hkv, D] bf16
 *   lse    [Hq, total_q] fp32 natural-log LSE (written at owned rows), or
 *          NULL to skip
 *   cu_seqlens_q, cu_seqlens_k  device int32 [B + 1]: sequence b owns query
 *          tokens [cu_seqlens_q[b], cu_seqlens_q[b + 1]) and key tokens
 *          [cu_seqlens_k[b], cu_seqlens_k[b + 1]); each offset is clamped
 *          into [0, total] on the device and a decreasing pair gives an empty
 *          range, so no offset makes the kernel leave the tensors.
 *          Sequences must not share query rows (their writes would race).
 *   max_seqlen_q  at least every sequence's query count: the grid covers
 *          that many rows per sequence, and rows past it are not computed
 *   causal 0 or 1; causal is bottom-right per sequence: query i of a
 *          sequence with Sq queries and Skv keys sees keys j <= i + Skv - Sq
 *          (its queries are its last Sq tokens)
 *   B, Hq, Hkv, max_seqlen_q, total_q, total_k >= 1, Hq % Hkv == 0,
 *   D in {64, 128}; scale, stream as mk_attn_fwd
 * Returns MK_OK or an mk_status; asynchronous on `stream`.
 */
int mk_attn_fwd_varlen(const void *q, const void *k, const void *v, void *o, float *lse,
                       const int *cu_seqlens_q, const int *cu_seqlens_k, int B, int Hq,
                       int Hkv, int max_seqlen_q, int total_q, int total_k, int D,
                       int causal, float scale, void *stream);

/*
 * Ragged paged attention (the paper's "Ragged Paged Attention" workload,
 * Table 2; length clamps as in Section 3.4): a packed batch of query
 * chunks of many sequences -- decode tokens, prefill chunks and whole
 * prompts in one call -- attending to their sequences' keys and values in
 * a paged cache.  Sequence b's Sq_b query tokens are its last positions,
 * and its keys (including the new tokens', already written to the cache)
 * are the first L_b rows its block table lists.
 *   q, o            [total_q, Hq, D] bf16, token-major; o written only at
 *                   rows some sequence owns
 *   k_pages, v_pages  [n_pages, Hkv, page_size, D] bf16 page pools; key j
 *                   of sequence b, kv head g, is row j % page_size of page
 *                   block_table[b][j / page_size], head g
 *   block_table     device int32 [B, max_pages]; an entry outside
 *                   [0, n_pages) is read as the nearest valid page;
 *                   entries at or past ceil(L_b / page_size) are not read
 *   lse             [Hq, total_q] fp32 natural-log LSE (written at owned
 *                   rows), or NULL to skip
 *   cu_seqlens_q    device int32 [B + 1]: sequence b owns query tokens
 *                   [cu_seqlens_q[b], cu_seqlens_q[b + 1]) (offsets clamped
 *                   into [0, total_q], a decreasing pair is empty);
 *                   sequences must not share query rows
 *   kv_seqlens      device int32 [B]: L_b, clamped into
 *                   [0, max_pages * page_size]
 *   max_seqlen_q    at least every sequence's query count (rows past it are
 *                   not computed)
 *   causal          0 or 1; causal is bottom-right per sequence: query i
 *                   sees keys j <= i + L_b - Sq_b
 *   page_size       keys per page, a positive multiple of 16
 *                   (MK_ERR_UNSUPPORTED otherwise)
 *   B, Hq, Hkv, max_seqlen_q, total_q, max_pages, n_pages >= 1,
 *   Hq % Hkv == 0, D in {64, 128}; max_pages * page_size and
 *   B * max_pages must fit in 31 bits (MK_ERR_SHAPE); scale, stream as
 *   mk_attn_fwd.
 * The result is mk_attn_fwd_varlen's on the keys and values gathered from
 * the pages, up to rounding (every tile here takes its own row maximum;
 * the results are bitwise equal unless a tile's scaled scores rise more
 * than 8 (log2 units) above the earlier tiles' maximum).  Returns MK_OK or
 * an mk_status; asynchronous on `stream`.
 */
int mk_attn_fwd_ragged_paged(const void *q, const void *k_pages, const void *v_pages,
                             const int *block_table, void *o, float *lse,
                             const int *cu_seqlens_q, const int *kv_seqlens, int B, int Hq,
                             int Hkv, int max_seqlen_q, int total_q, int page_size,
                             int max_pages, int n_pages, int D, int causal, float scale,
                             void *stream);

/*
 * Decode step: one query token per sequence against a key/value cache
 * (the decode step of the paper's paged-attention workloads, Table 2),
 * computed as split-KV attention whose per-split results are merged by
 * their log-sum-exp.  The splits are cut so that every wave streams the
 * same number of cache bytes: the keys of all (batch, kv head) pairs, in
 * 32-key stages, are laid end to end (pair b * Hkv + g after pair
 * b * Hkv + g - 1) and this stream is cut into n_parts equal parts, one
 * wave each.  A pair that lies inside one part is attended and written by
 * that wave alone; a pair cut by part boundaries is attended piecewise and
 * its pieces are merged by a second kernel, one wave per part, in which
 * the part holding the pair's last piece merges it.  Two kernels on
 * `stream`.
 *   q                 [B, Hq, D] bf16
 *   k_cache, v_cache  [B, Hkv, Smax, D] bf16; positions >= L_b are never read
 *   o                 [B, Hq, D] bf16 (written)
 *   lse               [B, Hq] fp32 natural-log LSE (written), or NULL to skip
 *   kv_seqlens        device int32 [B] (required), clamped into [0, Smax];
 *                     query (b, hq) attends to keys [0, L_b); L_b = 0 gives
 *                     O = 0, LSE = -inf
 *   Hq / Hkv must be at most 16; B * Hq and B * Hkv * ceil(Smax / 32) must
 *   fit in 31 bits (MK_ERR_SHAPE otherwise).
 *   n_parts           waves the key stream is cut into, 1 .. 2^20
 *                     (0 = mk_attn_decode_default_parts(Hq, Hkv, D));
 *                     any value gives the same result up to rounding.
 *                     There is no "keys per split" argument: the stream's
 *                     length depends on kv_seqlens, which lives on the
 *                     device, so keys per part are fixed inside the kernel
 *                     (about 32 * Hkv * sum_b ceil(L_b / 32) / n_parts).
 *   Groups wider than 16 query heads per kv head (Hq / Hkv > 16) return
 *   MK_ERR_UNSUPPORTED: a pair's query heads are the columns of one
 *   16-wide matrix-core block.
 *   workspace         device buffer, 256-byte aligned, of workspace_bytes >=
 *                     mk_attn_decode_workspace_bytes(Hq, Hkv, D, n_parts);
 *                     its contents need no initialisation and are left
 *                     undefined
 * The workspace must not be shared by calls that may overlap in time.
 */
int mk_attn_decode(const void *q, const void *k_cache, const void *v_cache, void *o,
                   float *lse, int B, int Hq, int Hkv, int Smax, int D, float scale,
                   const int *kv_seqlens, int n_parts, void *workspace,
                   size_t workspace_bytes, void *stream);

/*
 * Decode step that allocates nothing, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): mk_attn_decode with the workspace
 * taken from a fixed device array inside the library (16 MiB, one copy per
 * GPU, held until the process ends) instead of a caller's buffer.
 *   Arguments as mk_attn_decode, without workspace and workspace_bytes.
 *   The stream must belong to the current device (MK_ERR_ARG otherwise).
 *   The first call on a device looks up that device's copy of the array
 *   (hipGetSymbolAddress, with the device current); make it outside any
 *   graph capture.  No call allocates or frees memory.
 *   Returns MK_ERR_SCRATCH when mk_attn_decode_workspace_bytes(Hq, Hkv, D,
 *   n_parts) exceeds mk_attn_decode_noalloc_max_bytes(); nothing is
 *   launched then.
 * Every call on one GPU shares that GPU's array, and the array keeps the
 * last call's contents (nothing in it needs clearing: each call writes
 * every entry it reads).  Calls that may overlap in time on one GPU (on
 * different streams, or from different threads) race on it: serialise
 * them.  The result is mk_attn_decode's bit for bit.
 */
int mk_attn_decode_noalloc(const void *q, const void *k_cache, const void *v_cache, void *o,
                           float *lse, int B, int Hq, int Hkv, int Smax, int D, float scale,
                           const int *kv_seqlens, int n_parts, void *stream);

/* Bytes of the fixed array mk_attn_decode_noalloc uses (16 MiB). */
size_t mk_attn_decode_noalloc_max_bytes(void);

/*
 * Decode step over a paged key/value cache (the paper's "Paged Attention"
 * workload, Table 2): the same split-KV computation as mk_attn_decode, with
 * the cache held in fixed-size pages that a block table lists per sequence.
 *   q                 [B, Hq, D] bf16
 *   k_pages, v_pages  [n_pages, Hkv, page_size, D] bf16 page pools; key j
 *                     of sequence b, kv head g, is row j % page_size of
 *                     page block_table[b][j / page_size], head g
 *   block_table       device int32 [B, max_pages] (required); an entry
 *                     outside [0, n_pages) is read as the nearest valid
 *                     page (it cannot make the kernel leave the pool);
 *                     entries at or past ceil(L_b / page_size) are not read
 *   o, lse            as mk_attn_decode
 *   page_size         keys per page, a positive multiple of 16
 *   max_pages         table columns; lengths are clamped into
 *                     [0, max_pages * page_size]
 *   n_pages           pages in each pool (>= 1)
 *   kv_seqlens, n_parts, workspace, workspace_bytes, stream: as
 *                     mk_attn_decode (the same workspace size)
 * B * max_pages and max_pages * page_size must fit in 31 bits, as must the
 * stage count B * Hkv * ceil(max_pages * page_size / 32) (MK_ERR_SHAPE).
 * The result is mk_attn_decode's on the contiguous cache that gathers each
 * sequence's pages in table order (up to rounding: bitwise the same).
 */
int mk_attn_decode_paged(const void *q, const void *k_pages, const void *v_pages,
                         const int *block_table, void *o, float *lse, int B, int Hq,
                         int Hkv, int page_size, int max_pages, int n_pages, int D,
                         float scale, const int *kv_seqlens, int n_parts,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * Bytes of decode workspace for these sizes: per part, two partial outputs
 * [2, G, D] fp32 (the part's first and last piece, G = Hq / Hkv), their
 * LSEs [2, G] fp32, and an int32 [4] record of the cut pair the part
 * closes, the three regions 256-byte aligned.  n_parts = 0 selects the
 * default.  Independent of B and Smax.  Returns 0 for invalid sizes.
 */
size_t mk_attn_decode_workspace_bytes(int Hq, int Hkv, int D, int n_parts);

/*
 * Parts used when n_parts = 0: 256 compute units times the single-wave
 * workgroups one compute unit holds at once (bounded by LDS), or 0 for
 * invalid sizes.
 */
int mk_attn_decode_default_parts(int Hq, int Hkv, int D);

/*
 * Attention backward: gradients of a scalar loss L with respect to q, k
 * and v, given dout = dL/dO of the forward above (same q, k, v, masks,
 * scale and kv_seqlens).  The LSE output is taken as not differentiated.
 * From the derivative of softmax (the standard identity the paper's
 * "Flash Attention" workload family relies on, Table 2), with
 * P_ij = exp(scale s_ij - LSE_i) over the valid keys:
 *   dV_j = sum_i P_ij dO_i,   dP_ij = dO_i . v_j,   D_i = dO_i . O_i,
 *   dS_ij = P_ij (dP_ij - D_i),
 *   dQ_i = scale sum_j dS_ij k_j,   dK_j = scale sum_i dS_ij q_i,
 * dK and dV summed over the Hq / Hkv query heads of each kv head.
 *   q, o, dout   [B, Hq,  Sq,  D] bf16; o is the forward's output
 *   k, v         [B, Hkv, Skv, D] bf16
 *   lse          [B, Hq,  Sq] fp32, the forward's LSE (required)
 *   dq           [B, Hq,  Sq,  D] bf16 (written)
 *   dk, dv       [B, Hkv, Skv, D] bf16 (written; keys no row sees get 0)
 *   workspace    device memory of at least mk_attn_bwd_workspace_bytes()
 *                bytes, 256-byte aligned, owned by the caller; holds D_i
 *                and LSE_i log2 e during the call (written by it, so no
 *                clearing is needed) and may be reused after it returns.
 * Rows without a valid key give dq = 0.  Products run in bf16 with fp32
 * accumulation; P and dS enter them rounded to bf16.  The result is
 * deterministic (no atomics).  Outputs may not alias inputs.
 * Errors as mk_attn_fwd; MK_ERR_WORKSPACE when the workspace is missing or
 * too small.
 */
int mk_attn_bwd(const void *q, const void *k, const void *v, const void *o, const void *dout,
                const float *lse, void *dq, void *dk, void *dv, int B, int Hq, int Hkv,
                int Sq, int Skv, int D, int causal, float scale, const int *kv_seqlens,
                void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of backward workspace: two arrays of B * Hq * round_up(Sq, 128)
 * fp32 (D_i and LSE_i log2 e), each rounded up to 256 bytes; 0 for invalid
 * sizes. */
size_t mk_attn_bwd_workspace_bytes(int B, int Hq, int Sq);

/*
 * Decode step of multi-head latent attention in its absorbed form (the
 * "MLA Attention" workload of Table 2; the paper gives no shapes, this
 * library builds H = 16 query heads -- one eighth of a 128-head model,
 * the rest on other GPUs -- with Dc = 512 latent and Dr = 64 rotary
 * values).  Every head reads the same cache row per key: all Dc + Dr
 * values enter the score, the first Dc values are the value:
 *   L_b = clamp(kv_seqlens[b], 0, Smax)
 *   s_hj = scale * q[b,h,:] . ckv[b,j,:]                  (j < L_b)
 *   O[b,h,:] = sum_j softmax(s_h)_j ckv[b,j,0:Dc],  LSE[b,h] = log sum_j exp(s_hj)
 * L_b = 0 gives O = 0 and LSE = -inf.
 *   q     [B, H, Dc + Dr] bf16 (the latent part already multiplied into
 *         the latent space)
 *   ckv   [B, Smax, Dc + Dr] bf16 latent cache (rows past L_b never read)
 *   o     [B, H, Dc] bf16 (written);  lse [B, H] fp32 or NULL
 *   kv_seqlens [B] int32, device, required
 *   n_parts, workspace: as mk_attn_decode (the key stream of all sequences
 *         is cut into n_parts equal parts; 0 selects one per compute unit);
 *         size from mk_attn_mla_decode_workspace_bytes().
 * MK_ERR_UNSUPPORTED unless H = 16, Dc = 512, Dr = 64.  Other errors as
 * mk_attn_decode.
 */
int mk_attn_mla_decode(const void *q, const void *ckv, void *o, float *lse, int B, int H,
                       int Dc, int Dr, int Smax, float scale, const int *kv_seqlens,
                       int n_parts, void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of MLA decode workspace: per part two partial outputs [2, H, Dc]
 * fp32 and their LSEs [2, H] fp32, the two regions 256-byte aligned;
 * n_parts = 0 selects the default.  Returns 0 for unsupported sizes. */
size_t mk_attn_mla_decode_workspace_bytes(int H, int Dc, int n_parts);

/* Static string naming a status code ("MK_OK", ...); never NULL. */
const char *mk_status_str(int status);

/* ABI version of this header (incremented on incompatible change). */
int mk_attn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MK_ATTN_H */
