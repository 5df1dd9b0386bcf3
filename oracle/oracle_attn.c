/*
 * oracle_attn.c -- plain fp64 CPU oracle for causal grouped-query
 * scaled-dot-product attention (forward), its split-KV decode form,
 * decode over a paged cache (the "Paged Attention" workload of Table 2),
 * the forward over packed variable-length sequences, the same over a paged
 * cache (the "Ragged Paged Attention" workload of Table 2), the backward
 * (gradients of the output with respect to q, k and v), and the decode
 * step of multi-head latent attention (the "MLA Attention" workload).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the GPU path is
 * measured against; it is loaded by the test suite, by the smoke check and
 * by the benchmark's CPU-baseline leg, and by nothing else.  It shares no
 * code, header, table or helper with the HIP library.
 *
 * What it computes.  The paper names the operation only as workloads (the
 * "Flash Attention" and "GQA Attention" rows of Table 2, tolerances in
 * Table 4 of Appendix A) and states the correctness criterion as agreement
 * with an unoptimised reference (Section 3.1).  Flash/online-softmax
 * tiling and split-KV with a log-sum-exp merge are exact rewrites of the
 * plain definition in real arithmetic, so the oracle is the plain
 * definition, evaluated in double precision on the exact bf16 inputs:
 *
 *   G   = Hq / Hkv,  g = hq / G                       (grouped heads)
 *   L_b = clamp(kv_seqlens ? kv_seqlens[b] : Skv, 0, Skv)
 *   off = L_b - Sq                                    (bottom-right causal)
 *   J_i = { j : 0 <= j < L_b and (!causal or j <= i + off) }
 *   s_j = scale * sum_d q[b,hq,i,d] * k[b,g,j,d]
 *   m   = max_j s_j ;  w_j = exp(s_j - m) ;  l = sum_j w_j
 *   O[b,hq,i,d] = sum_j (w_j / l) * v[b,g,j,d]
 *   LSE[b,hq,i] = m + log(l)                          (natural log)
 *   J_i empty  =>  O = 0, LSE = -inf
 *
 * The clamp of L_b follows the robustness fix described in Section 3.4
 * (clamped lengths so that no slice size can go negative).
 *
 * Layouts (all contiguous, last dimension fastest):
 *   q [B,Hq,Sq,D], k/v [B,Hkv,Skv,D] as raw bf16 bit patterns (uint16),
 *   o [B,Hq,R,D] double, lse [B,Hq,R] double, where R = Sq or the number
 *   of sampled rows.
 *
 * Pins: every function here is checked by the CPU test tier against brute
 * force on tiny inputs, closed forms (scale 0, one key, equal V rows,
 * causal row 0), invariants (rows of P sum to 1, GQA equals MHA with
 * repeated K/V heads, decode equals the last prefill row, split-combine
 * equals unsplit, paged decode equals decode on the cache gathered through
 * the block table, a packed ragged batch equals each of its sequences run
 * alone, the ragged paged forward equals the packed forward over keys
 * gathered from the pages and the paged decode for one-token sequences,
 * the backward equals central finite differences of an independent
 * forward, MLA decode equals a decode over the same rows used as K and as
 * zero-padded V) and hand-derived values stored under tests/golden/.
 *
 * Build: plain C11, no -ffast-math, libm only (gcc -O2 -shared -fPIC).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* bf16 is the top half of an IEEE binary32; widening is exact. */
static double bf16_bits_to_double(uint16_t bits)
{
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int clamp_len(int len, int hi)
{
    if (len < 0) return 0;
    if (len > hi) return hi;
    return len;
}

/* Row of key j of sequence b, kv head g, in a page pool
   [n_pages, Hkv, page_size, D] (see oracle_decode_paged). */
static size_t paged_row(const int32_t *block_table, int b, int max_pages,
                        int n_pages, int page_size, int Hkv, int g, int j)
{
    int page = block_table[(size_t)b * max_pages + j / page_size];
    if (page < 0) page = 0;
    if (page > n_pages - 1) page = n_pages - 1;
    return ((size_t)page * Hkv + g) * page_size + (size_t)(j % page_size);
}

/* ------------------------------------------------------------------ */
/* One query row of the plain definition.                              */
/* ------------------------------------------------------------------ */

/*
 * q_row: D bf16 values; k_head, v_head: Skv x D bf16 values of the key /
 * value head the query head maps to.  Keys j in [0, n_valid) are the
 * valid set J (a prefix of the key axis in every case this oracle
 * handles: causal masking and length masking both cut a prefix).
 * s_buf: scratch of at least n_valid doubles.
 * Writes D outputs to o_row and the natural-log LSE to *lse_out.
 */
static void attend_row(const uint16_t *q_row, const uint16_t *k_head,
                       const uint16_t *v_head, int D, int n_valid,
                       double scale, double *s_buf, double *o_row,
                       double *lse_out)
{
    if (n_valid <= 0) {
        for (int d = 0; d < D; ++d) o_row[d] = 0.0;
        *lse_out = -INFINITY;
        return;
    }
    /* scores */
    for (int j = 0; j < n_valid; ++j) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
            dot += bf16_bits_to_double(q_row[d]) *
                   bf16_bits_to_double(k_head[(size_t)j * D + d]);
        s_buf[j] = scale * dot;
    }
    /* max, then weights and their sum (two-pass softmax) */
    double m = s_buf[0];
    for (int j = 1; j < n_valid; ++j)
        if (s_buf[j] > m) m = s_buf[j];
    double l = 0.0;
    for (int j = 0; j < n_valid; ++j) {
        s_buf[j] = exp(s_buf[j] - m);
        l += s_buf[j];
    }
    /* weighted sum of value rows */
    for (int d = 0; d < D; ++d) o_row[d] = 0.0;
    for (int j = 0; j < n_valid; ++j) {
        double p = s_buf[j] / l;
        for (int d = 0; d < D; ++d)
            o_row[d] += p * bf16_bits_to_double(v_head[(size_t)j * D + d]);
    }
    *lse_out = m + log(l);
}

/* ------------------------------------------------------------------ */
/* Prefill / general forward                                           */
/* ------------------------------------------------------------------ */

typedef struct {
    const uint16_t *q, *k, *v;
    int B, Hq, Hkv, Sq, Skv, D, causal;
    double scale;
    const int32_t *kv_seqlens; /* host array [B] or NULL */
    const int32_t *rows;       /* host array [B*Hq*nrows] or NULL */
    int nrows;                 /* rows per (b, hq) */
    double *o, *lse;
    /* work split */
    long long n_items;
    int n_threads;
    int tid;
} fwd_job;

static void *fwd_worker(void *arg)
{
    fwd_job *job = (fwd_job *)arg;
    double *s_buf = (double *)malloc(sizeof(double) * (size_t)(job->Skv > 0 ? job->Skv : 1));
    if (!s_buf) return (void *)1;
    const int G = job->Hq / job->Hkv;
    const int D = job->D;
    for (long long it = job->tid; it < job->n_items; it += job->n_threads) {
        /* item = ((b * Hq) + hq) * nrows + r */
        long long r = it % job->nrows;
        long long bh = it / job->nrows;
        int hq = (int)(bh % job->Hq);
        int b = (int)(bh / job->Hq);
        int g = hq / G;
        int i = job->rows ? job->rows[it] : (int)r;
        int L = clamp_len(job->kv_seqlens ? job->kv_seqlens[b] : job->Skv, job->Skv);
        int n_valid = L;
        if (job->causal) {
            int off = L - job->Sq;
            int last = i + off; /* largest admissible key index */
            if (last + 1 < n_valid) n_valid = last + 1;
            if (n_valid < 0) n_valid = 0;
        }
        const uint16_t *q_row = job->q + (((size_t)b * job->Hq + hq) * job->Sq + i) * D;
        const uint16_t *k_head = job->k + ((size_t)b * job->Hkv + g) * (size_t)job->Skv * D;
        const uint16_t *v_head = job->v + ((size_t)b * job->Hkv + g) * (size_t)job->Skv * D;
        attend_row(q_row, k_head, v_head, D, n_valid, job->scale, s_buf,
                   job->o + (size_t)it * D, job->lse + it);
    }
    free(s_buf);
    return NULL;
}

static int run_jobs(fwd_job *proto, int n_threads)
{
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t th[256];
    fwd_job jobs[256];
    int started = 0, rc = 0;
    for (int t = 0; t < n_threads; ++t) {
        jobs[t] = *proto;
        jobs[t].n_threads = n_threads;
        jobs[t].tid = t;
    }
    if (n_threads == 1) return fwd_worker(&jobs[0]) ? -5 : 0;
    for (int t = 0; t < n_threads; ++t) {
        if (pthread_create(&th[t], NULL, fwd_worker, &jobs[t]) != 0) { rc = -6; break; }
        ++started;
    }
    for (int t = 0; t < started; ++t) {
        void *ret = NULL;
        pthread_join(th[t], &ret);
        if (ret) rc = -5;
    }
    return rc;
}

/*
 * Attention forward by the plain definition above.
 * rows == NULL: every query row, nrows must equal Sq, outputs [B,Hq,Sq,(D)].
 * rows != NULL: rows[(b*Hq + hq)*nrows + r] is the r-th query row computed
 *               for head (b, hq); outputs [B,Hq,nrows,(D)].
 * Returns 0 on success, a negative code on bad arguments.
 */
int oracle_attn_fwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                    int B, int Hq, int Hkv, int Sq, int Skv, int D,
                    int causal, double scale, const int32_t *kv_seqlens,
                    const int32_t *rows, int nrows, double *o, double *lse,
                    int n_threads)
{
    if (!q || !k || !v || !o || !lse) return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Skv < 1 || D < 1) return -2;
    if (Hq % Hkv != 0) return -3;
    if (!rows) nrows = Sq;
    if (nrows < 1) return -4;
    if (rows) {
        for (long long t = 0; t < (long long)B * Hq * nrows; ++t)
            if (rows[t] < 0 || rows[t] >= Sq) return -4;
    }
    fwd_job job;
    memset(&job, 0, sizeof job);
    job.q = q; job.k = k; job.v = v;
    job.B = B; job.Hq = Hq; job.Hkv = Hkv; job.Sq = Sq; job.Skv = Skv; job.D = D;
    job.causal = causal ? 1 : 0;
    job.scale = scale;
    job.kv_seqlens = kv_seqlens;
    job.rows = rows;
    job.nrows = nrows;
    job.o = o; job.lse = lse;
    job.n_items = (long long)B * Hq * nrows;
    return run_jobs(&job, n_threads);
}

/*
 * The normalised attention weights P[b,hq,i,j] = w_j / l (0 outside J_i),
 * for the rows-sum-to-one pin.  p: [B,Hq,Sq,Skv] doubles.  Single thread;
 * meant for small shapes.
 */
int oracle_attn_probs(const uint16_t *q, const uint16_t *k, int B, int Hq,
                      int Hkv, int Sq, int Skv, int D, int causal,
                      double scale, const int32_t *kv_seqlens, double *p)
{
    if (!q || !k || !p) return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Skv < 1 || D < 1) return -2;
    if (Hq % Hkv != 0) return -3;
    const int G = Hq / Hkv;
    double *s = (double *)malloc(sizeof(double) * (size_t)Skv);
    if (!s) return -5;
    for (int b = 0; b < B; ++b)
        for (int hq = 0; hq < Hq; ++hq)
            for (int i = 0; i < Sq; ++i) {
                int g = hq / G;
                int L = clamp_len(kv_seqlens ? kv_seqlens[b] : Skv, Skv);
                int n_valid = L;
                if (causal) {
                    int last = i + (L - Sq);
                    if (last + 1 < n_valid) n_valid = last + 1;
                    if (n_valid < 0) n_valid = 0;
                }
                double *prow = p + (((size_t)b * Hq + hq) * Sq + i) * (size_t)Skv;
                for (int j = 0; j < Skv; ++j) prow[j] = 0.0;
                if (n_valid == 0) continue;
                const uint16_t *q_row = q + (((size_t)b * Hq + hq) * Sq + i) * D;
                const uint16_t *k_head = k + ((size_t)b * Hkv + g) * (size_t)Skv * D;
                for (int j = 0; j < n_valid; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += bf16_bits_to_double(q_row[d]) *
                               bf16_bits_to_double(k_head[(size_t)j * D + d]);
                    s[j] = scale * dot;
                }
                double m = s[0];
                for (int j = 1; j < n_valid; ++j) if (s[j] > m) m = s[j];
                double l = 0.0;
                for (int j = 0; j < n_valid; ++j) l += exp(s[j] - m);
                for (int j = 0; j < n_valid; ++j) prow[j] = exp(s[j] - m) / l;
            }
    free(s);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Decode: one query token per sequence over a length-masked cache     */
/* ------------------------------------------------------------------ */

/*
 * q [B,Hq,D], k_cache/v_cache [B,Hkv,Smax,D], kv_seqlens [B] (required).
 * Query (b, hq) attends to every key j < clamp(kv_seqlens[b], 0, Smax).
 * o [B,Hq,D], lse [B,Hq].
 */
int oracle_decode(const uint16_t *q, const uint16_t *k_cache,
                  const uint16_t *v_cache, int B, int Hq, int Hkv, int Smax,
                  int D, double scale, const int32_t *kv_seqlens, double *o,
                  double *lse, int n_threads)
{
    if (!kv_seqlens) return -1;
    /* A decode step is the forward with one query row per sequence whose
       admissible keys are the whole valid prefix: run it non-causally
       under the length mask. */
    return oracle_attn_fwd(q, k_cache, v_cache, B, Hq, Hkv, 1, Smax, D, 0,
                           scale, kv_seqlens, NULL, 1, o, lse, n_threads);
}

/*
 * Merge per-split partial results by their log-sum-exp (the split-KV
 * decode's final step).  o_part [R,nsplit,D] holds each split's own
 * normalised output, lse_part [R,nsplit] its natural-log LSE (-inf for an
 * empty split).  For each r:
 *   M = max_s lse_s ;  LSE = M + log(sum_s exp(lse_s - M))
 *   O = sum_s exp(lse_s - LSE) * O_s
 * and O = 0, LSE = -inf when every split is empty.
 */
int oracle_lse_combine(const double *o_part, const double *lse_part, int R,
                       int nsplit, int D, double *o, double *lse)
{
    if (!o_part || !lse_part || !o || !lse) return -1;
    if (R < 1 || nsplit < 1 || D < 1) return -2;
    for (int r = 0; r < R; ++r) {
        const double *ls = lse_part + (size_t)r * nsplit;
        double M = -INFINITY;
        for (int s = 0; s < nsplit; ++s) if (ls[s] > M) M = ls[s];
        double *orow = o + (size_t)r * D;
        for (int d = 0; d < D; ++d) orow[d] = 0.0;
        if (M == -INFINITY) { lse[r] = -INFINITY; continue; }
        double sum = 0.0;
        for (int s = 0; s < nsplit; ++s) sum += exp(ls[s] - M);
        double L = M + log(sum);
        lse[r] = L;
        for (int s = 0; s < nsplit; ++s) {
            if (ls[s] == -INFINITY) continue;
            double w = exp(ls[s] - L);
            const double *op = o_part + ((size_t)r * nsplit + s) * D;
            for (int d = 0; d < D; ++d) orow[d] += w * op[d];
        }
    }
    return 0;
}

/*
 * Split-KV decode carried out step by step: keys of sequence b are cut
 * into consecutive splits of `split` keys, each split is attended on its
 * own (plain definition restricted to the split), and the partials are
 * merged with oracle_lse_combine.  nsplit = ceil(Smax / split).
 * o_part [B,Hq,nsplit,D] and lse_part [B,Hq,nsplit] receive the partials.
 */
int oracle_decode_split(const uint16_t *q, const uint16_t *k_cache,
                        const uint16_t *v_cache, int B, int Hq, int Hkv,
                        int Smax, int D, double scale,
                        const int32_t *kv_seqlens, int split, double *o_part,
                        double *lse_part, double *o, double *lse)
{
    if (!q || !k_cache || !v_cache || !kv_seqlens || !o_part || !lse_part || !o || !lse)
        return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Smax < 1 || D < 1 || split < 1) return -2;
    if (Hq % Hkv != 0) return -3;
    const int G = Hq / Hkv;
    const int nsplit = (Smax + split - 1) / split;
    double *s_buf = (double *)malloc(sizeof(double) * (size_t)split);
    if (!s_buf) return -5;
    for (int b = 0; b < B; ++b) {
        int L = clamp_len(kv_seqlens[b], Smax);
        for (int hq = 0; hq < Hq; ++hq) {
            int g = hq / G;
            const uint16_t *q_row = q + ((size_t)b * Hq + hq) * D;
            for (int sp = 0; sp < nsplit; ++sp) {
                int j0 = sp * split;
                int n = L - j0;
                if (n > split) n = split;
                if (n < 0) n = 0;
                const uint16_t *k_head = k_cache + (((size_t)b * Hkv + g) * Smax + j0) * D;
                const uint16_t *v_head = v_cache + (((size_t)b * Hkv + g) * Smax + j0) * D;
                size_t pr = ((size_t)b * Hq + hq) * nsplit + sp;
                attend_row(q_row, k_head, v_head, D, n, scale, s_buf,
                           o_part + pr * D, lse_part + pr);
            }
        }
    }
    free(s_buf);
    return oracle_lse_combine(o_part, lse_part, B * Hq, nsplit, D, o, lse);
}

/* ------------------------------------------------------------------ */
/* Paged decode: the cache is a pool of fixed-size pages               */
/* ------------------------------------------------------------------ */

/*
 * k_pages / v_pages [n_pages, Hkv, page_size, D]; block_table
 * [B, max_pages] lists the pages of sequence b in key order, so key j of
 * sequence b is row j % page_size of page block_table[b][j / page_size].
 * The length clamps to [0, max_pages * page_size]; a table entry outside
 * [0, n_pages) is read as the nearest valid page (the same clamp the
 * lengths get: no lookup may leave the pool).  Then the plain decode
 * definition, written out here with its own loops:
 *   s_j = scale * q[b,hq,:] . k(j),  w_j = exp(s_j - max s),
 *   O = sum_j (w_j / sum w) v(j),    LSE = max s + log(sum w).
 * o [B,Hq,D], lse [B,Hq].
 */
int oracle_decode_paged(const uint16_t *q, const uint16_t *k_pages,
                        const uint16_t *v_pages, const int32_t *block_table,
                        int B, int Hq, int Hkv, int page_size, int max_pages,
                        int n_pages, int D, double scale,
                        const int32_t *kv_seqlens, double *o, double *lse)
{
    if (!q || !k_pages || !v_pages || !block_table || !kv_seqlens || !o || !lse)
        return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || page_size < 1 ||
        max_pages < 1 || n_pages < 1 || D < 1)
        return -2;
    const int G = Hq / Hkv;
    const int max_keys = max_pages * page_size;
    double *s = malloc((size_t)max_keys * sizeof *s);
    if (!s) return -3;
    for (int b = 0; b < B; ++b) {
        const int L = clamp_len(kv_seqlens[b], max_keys);
        for (int hq = 0; hq < Hq; ++hq) {
            const int g = hq / G;
            const uint16_t *q_row = q + ((size_t)b * Hq + hq) * D;
            double *o_row = o + ((size_t)b * Hq + hq) * D;
            if (L == 0) {
                for (int d = 0; d < D; ++d) o_row[d] = 0.0;
                lse[(size_t)b * Hq + hq] = -INFINITY;
                continue;
            }
            double m = -INFINITY;
            for (int j = 0; j < L; ++j) {
                const size_t krow = paged_row(block_table, b, max_pages, n_pages,
                                              page_size, Hkv, g, j);
                double dot = 0.0;
                for (int d = 0; d < D; ++d)
                    dot += bf16_bits_to_double(q_row[d]) *
                           bf16_bits_to_double(k_pages[krow * D + d]);
                s[j] = scale * dot;
                if (s[j] > m) m = s[j];
            }
            double l = 0.0;
            for (int j = 0; j < L; ++j) {
                s[j] = exp(s[j] - m);
                l += s[j];
            }
            for (int d = 0; d < D; ++d) o_row[d] = 0.0;
            for (int j = 0; j < L; ++j) {
                const size_t vrow = paged_row(block_table, b, max_pages, n_pages,
                                              page_size, Hkv, g, j);
                const double p = s[j] / l;
                for (int d = 0; d < D; ++d)
                    o_row[d] += p * bf16_bits_to_double(v_pages[vrow * D + d]);
            }
            lse[(size_t)b * Hq + hq] = m + log(l);
        }
    }
    free(s);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Variable-length (ragged) forward over packed sequences              */
/* ------------------------------------------------------------------ */

/* Clamped [start, end) of sequence b from cumulative offsets cu[0..B]. */
static void seq_range(const int32_t *cu, int b, int total, int *start, int *end)
{
    int s0 = cu[b], s1 = cu[b + 1];
    if (s0 < 0) s0 = 0;
    if (s0 > total) s0 = total;
    if (s1 < s0) s1 = s0;
    if (s1 > total) s1 = total;
    *start = s0;
    *end = s1;
}

/*
 * Packed layout, token-major with the heads inside a token: q and o
 * [total_q, Hq, D], k and v [total_k, Hkv, D].  Sequence b owns query
 * tokens [cu_q[b], cu_q[b+1]) and key tokens [cu_k[b], cu_k[b+1]) (offsets
 * clamped into [0, total] and made non-decreasing).  Query row i of
 * sequence b, head hq, attends to its sequence's keys j < Skv_b, and when
 * causal only to j <= i + Skv_b - Sq_b (bottom-right alignment, so a
 * sequence whose queries are its last tokens -- a chunk of a longer prompt
 * or a single decode token -- sees every earlier key).  The plain
 * definition per row, written out here with strided rows:
 *   s_j = scale * q . k_j,  O = sum_j softmax(s)_j v_j,  LSE = log sum exp s.
 * lse [Hq, total_q].  Rows no sequence owns are not written.
 */
int oracle_attn_fwd_varlen(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                           const int32_t *cu_q, const int32_t *cu_k, int B, int Hq,
                           int Hkv, int total_q, int total_k, int D, int causal,
                           double scale, double *o, double *lse)
{
    if (!q || !k || !v || !cu_q || !cu_k || !o || !lse) return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || D < 1 || total_q < 0 ||
        total_k < 0 || (causal != 0 && causal != 1))
        return -2;
    const int G = Hq / Hkv;
    double *s = malloc(sizeof(double) * (size_t)(total_k > 0 ? total_k : 1));
    if (!s) return -3;
    for (int b = 0; b < B; ++b) {
        int q0, q1, k0, k1;
        seq_range(cu_q, b, total_q, &q0, &q1);
        seq_range(cu_k, b, total_k, &k0, &k1);
        const int Sq = q1 - q0, Skv = k1 - k0;
        for (int hq = 0; hq < Hq; ++hq) {
            const int g = hq / G;
            for (int i = 0; i < Sq; ++i) {
                const uint16_t *q_row = q + ((size_t)(q0 + i) * Hq + hq) * D;
                double *o_row = o + ((size_t)(q0 + i) * Hq + hq) * D;
                double *lse_row = lse + (size_t)hq * total_q + (q0 + i);
                int n_valid = Skv;
                if (causal && i + Skv - Sq + 1 < n_valid) n_valid = i + Skv - Sq + 1;
                if (n_valid <= 0) {
                    for (int d = 0; d < D; ++d) o_row[d] = 0.0;
                    *lse_row = -INFINITY;
                    continue;
                }
                double m = -INFINITY;
                for (int j = 0; j < n_valid; ++j) {
                    const uint16_t *k_row = k + ((size_t)(k0 + j) * Hkv + g) * D;
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += bf16_bits_to_double(q_row[d]) * bf16_bits_to_double(k_row[d]);
                    s[j] = scale * dot;
                    if (s[j] > m) m = s[j];
                }
                double l = 0.0;
                for (int j = 0; j < n_valid; ++j) {
                    s[j] = exp(s[j] - m);
                    l += s[j];
                }
                for (int d = 0; d < D; ++d) o_row[d] = 0.0;
                for (int j = 0; j < n_valid; ++j) {
                    const uint16_t *v_row = v + ((size_t)(k0 + j) * Hkv + g) * D;
                    const double p = s[j] / l;
                    for (int d = 0; d < D; ++d) o_row[d] += p * bf16_bits_to_double(v_row[d]);
                }
                *lse_row = m + log(l);
            }
        }
    }
    free(s);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Ragged paged forward: packed queries over a paged key/value cache    */
/* ------------------------------------------------------------------ */

/*
 * The "Ragged Paged Attention" workload of Table 2 (prefill chunks and
 * decode tokens of many sequences in one call, the keys in a paged cache),
 * with the length clamps of Section 3.4.  Sequence b owns query tokens
 * [cu_q[b], cu_q[b+1]) of the packed q [total_q, Hq, D] (offsets clamped
 * into [0, total_q] and made non-decreasing) and L_b = clamp(kv_seqlens[b],
 * 0, max_pages * page_size) keys; key j of sequence b, kv head g, is row
 * j % page_size of page block_table[b][j / page_size] of the pools
 * k_pages / v_pages [n_pages, Hkv, page_size, D] (an entry outside
 * [0, n_pages) read as the nearest valid page).  The Sq_b queries are the
 * sequence's last positions: query row i attends to keys j < L_b, and when
 * causal only to j <= i + L_b - Sq_b.  The plain definition per row,
 * written out with its own loops:
 *   s_j = scale * q . k_j,  O = sum_j softmax(s)_j v_j,  LSE = log sum exp s,
 * no valid key -> O = 0, LSE = -inf.  o [total_q, Hq, D] double, lse
 * [Hq, total_q] double; rows no sequence owns are not written.
 */
int oracle_attn_fwd_ragged_paged(const uint16_t *q, const uint16_t *k_pages,
                                 const uint16_t *v_pages, const int32_t *cu_q,
                                 const int32_t *kv_seqlens, const int32_t *block_table,
                                 int B, int Hq, int Hkv, int total_q, int page_size,
                                 int max_pages, int n_pages, int D, int causal,
                                 double scale, double *o, double *lse)
{
    if (!q || !k_pages || !v_pages || !cu_q || !kv_seqlens || !block_table || !o || !lse)
        return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || total_q < 0 || page_size < 1 ||
        max_pages < 1 || n_pages < 1 || D < 1 || (causal != 0 && causal != 1))
        return -2;
    const int G = Hq / Hkv;
    const int max_keys = max_pages * page_size;
    double *s = malloc((size_t)max_keys * sizeof *s);
    if (!s) return -3;
    for (int b = 0; b < B; ++b) {
        int q0, q1;
        seq_range(cu_q, b, total_q, &q0, &q1);
        const int Sq = q1 - q0;
        const int L = clamp_len(kv_seqlens[b], max_keys);
        for (int hq = 0; hq < Hq; ++hq) {
            const int g = hq / G;
            for (int i = 0; i < Sq; ++i) {
                const uint16_t *q_row = q + ((size_t)(q0 + i) * Hq + hq) * D;
                double *o_row = o + ((size_t)(q0 + i) * Hq + hq) * D;
                double *lse_row = &lse[(size_t)hq * total_q + q0 + i];
                int n_valid = L;
                if (causal && i + L - Sq + 1 < n_valid) n_valid = i + L - Sq + 1;
                if (n_valid <= 0) {
                    for (int d = 0; d < D; ++d) o_row[d] = 0.0;
                    *lse_row = -INFINITY;
                    continue;
                }
                double m = -INFINITY;
                for (int j = 0; j < n_valid; ++j) {
                    const size_t krow = paged_row(block_table, b, max_pages, n_pages,
                                                  page_size, Hkv, g, j);
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += bf16_bits_to_double(q_row[d]) *
                               bf16_bits_to_double(k_pages[krow * D + d]);
                    s[j] = scale * dot;
                    if (s[j] > m) m = s[j];
                }
                double l = 0.0;
                for (int j = 0; j < n_valid; ++j) {
                    s[j] = exp(s[j] - m);
                    l += s[j];
                }
                for (int d = 0; d < D; ++d) o_row[d] = 0.0;
                for (int j = 0; j < n_valid; ++j) {
                    const size_t vrow = paged_row(block_table, b, max_pages, n_pages,
                                                  page_size, Hkv, g, j);
                    const double p = s[j] / l;
                    for (int d = 0; d < D; ++d)
                        o_row[d] += p * bf16_bits_to_double(v_pages[vrow * D + d]);
                }
                *lse_row = m + log(l);
            }
        }
    }
    free(s);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Backward: gradients of the output with respect to q, k, v            */
/* ------------------------------------------------------------------ */

/*
 * Given do = dL/dO for the forward of oracle_attn_fwd (same layouts and
 * masks; the LSE output is taken as not differentiated), the gradients of
 * L with respect to q, k and v, from the derivative of softmax: with
 * P_ij = softmax_j(s_i) over the valid keys,
 *   dV_j  = sum_i P_ij dO_i               (summed over the query heads of
 *   dP_ij = dO_i . v_j                      the kv head for dK and dV)
 *   D_i   = sum_j P_ij dP_ij
 *   dS_ij = P_ij (dP_ij - D_i)
 *   dQ_i  = scale * sum_j dS_ij k_j
 *   dK_j  = scale * sum_i dS_ij q_i
 * Rows without valid keys contribute nothing; keys no row sees get zero.
 * dq [B,Hq,Sq,D], dk, dv [B,Hkv,Skv,D], all double.
 */
int oracle_attn_bwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                    const uint16_t *dout, int B, int Hq, int Hkv, int Sq, int Skv, int D,
                    int causal, double scale, const int32_t *kv_seqlens, double *dq,
                    double *dk, double *dv)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || Sq < 1 || Skv < 1 || D < 1 ||
        (causal != 0 && causal != 1))
        return -2;
    const int G = Hq / Hkv;
    double *p = malloc(sizeof(double) * (size_t)Skv);
    double *dp = malloc(sizeof(double) * (size_t)Skv);
    if (!p || !dp) { free(p); free(dp); return -3; }
    memset(dq, 0, sizeof(double) * (size_t)B * Hq * Sq * D);
    memset(dk, 0, sizeof(double) * (size_t)B * Hkv * Skv * D);
    memset(dv, 0, sizeof(double) * (size_t)B * Hkv * Skv * D);
    for (int b = 0; b < B; ++b) {
        const int L = clamp_len(kv_seqlens ? kv_seqlens[b] : Skv, Skv);
        for (int hq = 0; hq < Hq; ++hq) {
            const int g = hq / G;
            const size_t kv0 = ((size_t)b * Hkv + g) * (size_t)Skv * D;
            for (int i = 0; i < Sq; ++i) {
                int n = L;
                if (causal && i + L - Sq + 1 < n) n = i + L - Sq + 1;
                if (n <= 0) continue;
                const size_t qi = (((size_t)b * Hq + hq) * Sq + i) * D;
                /* probabilities of row i */
                double m = -INFINITY;
                for (int j = 0; j < n; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += bf16_bits_to_double(q[qi + d]) *
                               bf16_bits_to_double(k[kv0 + (size_t)j * D + d]);
                    p[j] = scale * dot;
                    if (p[j] > m) m = p[j];
                }
                double z = 0.0;
                for (int j = 0; j < n; ++j) {
                    p[j] = exp(p[j] - m);
                    z += p[j];
                }
                for (int j = 0; j < n; ++j) p[j] /= z;
                /* dP_ij, D_i */
                double delta = 0.0;
                for (int j = 0; j < n; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += bf16_bits_to_double(dout[qi + d]) *
                               bf16_bits_to_double(v[kv0 + (size_t)j * D + d]);
                    dp[j] = dot;
                    delta += p[j] * dot;
                }
                for (int j = 0; j < n; ++j) {
                    const double ds = p[j] * (dp[j] - delta);
                    for (int d = 0; d < D; ++d) {
                        dv[kv0 + (size_t)j * D + d] += p[j] * bf16_bits_to_double(dout[qi + d]);
                        dq[qi + d] += scale * ds * bf16_bits_to_double(k[kv0 + (size_t)j * D + d]);
                        dk[kv0 + (size_t)j * D + d] += scale * ds * bf16_bits_to_double(q[qi + d]);
                    }
                }
            }
        }
    }
    free(p);
    free(dp);
    return 0;
}

/* ------------------------------------------------------------------ */
/* MLA decode: a shared latent cache with a latent and a rotary part    */
/* ------------------------------------------------------------------ */

/*
 * One decode step of multi-head latent attention in its absorbed form (the
 * "MLA Attention" workload of Table 2; the paper gives no shapes).  Every
 * query head reads the same cache row per key: its first Dc values are the
 * latent vector, which serves as the value, and the last Dr values the
 * rotary key part.  The query head carries the matching Dc + Dr values (the
 * latent part already multiplied into the latent space).  For each b, h:
 *   L   = clamp(kv_seqlens[b], 0, Smax)
 *   s_j = scale * sum_{d < Dc+Dr} q[b,h,d] * ckv[b,j,d]        (j < L)
 *   O[b,h,e] = sum_j softmax(s)_j * ckv[b,j,e]                 (e < Dc)
 *   LSE[b,h] = log sum_j exp(s_j) ;  L = 0 -> O = 0, LSE = -inf
 * q [B,H,Dc+Dr], ckv [B,Smax,Dc+Dr] bf16 bits; o [B,H,Dc], lse [B,H] double.
 */
int oracle_mla_decode(const uint16_t *q, const uint16_t *ckv, int B, int H,
                      int Dc, int Dr, int Smax, double scale,
                      const int32_t *kv_seqlens, double *o, double *lse)
{
    if (!q || !ckv || !kv_seqlens || !o || !lse) return -1;
    if (B < 1 || H < 1 || Dc < 1 || Dr < 0 || Smax < 1) return -2;
    const int Dk = Dc + Dr;
    double *s = (double *)malloc(sizeof(double) * (size_t)Smax);
    if (!s) return -3;
    for (int b = 0; b < B; ++b) {
        const int L = clamp_len(kv_seqlens[b], Smax);
        const uint16_t *cache = ckv + (size_t)b * Smax * Dk;
        for (int h = 0; h < H; ++h) {
            const uint16_t *q_row = q + ((size_t)b * H + h) * Dk;
            double *o_row = o + ((size_t)b * H + h) * Dc;
            for (int e = 0; e < Dc; ++e) o_row[e] = 0.0;
            if (L == 0) { lse[(size_t)b * H + h] = -INFINITY; continue; }
            double m = -INFINITY;
            for (int j = 0; j < L; ++j) {
                double dot = 0.0;
                for (int d = 0; d < Dk; ++d)
                    dot += bf16_bits_to_double(q_row[d]) *
                           bf16_bits_to_double(cache[(size_t)j * Dk + d]);
                s[j] = scale * dot;
                if (s[j] > m) m = s[j];
            }
            double l = 0.0;
            for (int j = 0; j < L; ++j) { s[j] = exp(s[j] - m); l += s[j]; }
            for (int j = 0; j < L; ++j) {
                const double p = s[j] / l;
                for (int e = 0; e < Dc; ++e)
                    o_row[e] += p * bf16_bits_to_double(cache[(size_t)j * Dk + e]);
            }
            lse[(size_t)b * H + h] = m + log(l);
        }
    }
    free(s);
    return 0;
}

int oracle_version(void) { return 6; }
