/*
 * mk_attn.h -- C ABI of the MI355X (gfx950) fused attention library.
 *
 * The operation is the attention forward of the paper's "Flash Attention"
 * and "GQA Attention" workloads (Table 2; tolerances in Table 4,
 * Appendix A), and the one-token decode step of its "Paged Attention" /
 * "Ragged Paged Attention" family (Table 2) over a contiguous cache:
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
    MK_ERR_WORKSPACE = 5,   /* decode workspace missing or too small */
    MK_ERR_HIP = 6,         /* the HIP runtime refused a launch */
    MK_ERR_ARG = 7          /* non-finite scale, bad causal flag or split */
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
 * Bytes of caller-owned device workspace mk_attn_decode needs for these
 * sizes: per-split partial outputs [B, Hq, nsplit, D] fp32 and their
 * LSEs [B, Hq, nsplit] fp32, nsplit = ceil(Smax / split), each region
 * 256-byte aligned.  split = 0 selects the library default (the value
 * mk_attn_decode would use).  Returns 0 for invalid sizes.
 */
size_t mk_attn_decode_workspace_bytes(int B, int Hq, int Smax, int D, int split);

/*
 * Decode step: one query token per sequence against a key/value cache,
 * split along the keys, each split attended on its own, and the splits
 * merged by their log-sum-exp (two kernels on `stream`).
 *   q                 [B, Hq, D] bf16
 *   k_cache, v_cache  [B, Hkv, Smax, D] bf16; positions >= L_b are never read
 *   o                 [B, Hq, D] bf16 (written)
 *   lse               [B, Hq] fp32 (written), or NULL to skip
 *   kv_seqlens        device int32 [B] (required), clamped into [0, Smax];
 *                     query (b, hq) attends to keys [0, L_b)
 *   Hq / Hkv must be at most 16.
 *   split             keys per split, a multiple of 64 (0 = default)
 *   workspace         device buffer of workspace_bytes >=
 *                     mk_attn_decode_workspace_bytes(B, Hq, Smax, D, split)
 * The workspace must not be shared by overlapping calls.
 */
int mk_attn_decode(const void *q, const void *k_cache, const void *v_cache, void *o,
                   float *lse, int B, int Hq, int Hkv, int Smax, int D, float scale,
                   const int *kv_seqlens, int split, void *workspace,
                   size_t workspace_bytes, void *stream);

/* Default keys per split used when split = 0. */
int mk_attn_decode_default_split(void);

/* Static string naming a status code ("MK_OK", ...); never NULL. */
const char *mk_status_str(int status);

/* ABI version of this header (incremented on incompatible change). */
int mk_attn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MK_ATTN_H */
