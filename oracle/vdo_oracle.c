/*
 * vdo_oracle.c -- fp64 CPU oracle for batched single-token paged GQA decode
 * attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or helper with the HIP
 * library; it reads the same bytes through its own page walk.
 *
 * What it computes (the plain definition, no blocking, no fusion):
 *   The decode step of a served model attends, for every running request, the
 *   newest query token to all N_kv tokens held in the request's KV cache; the
 *   paper names these quantities N_req and N_kv and says the attention layer's
 *   work and KV-cache reads scale with N_kv (EcoPred, Sec. 5.4, Eq. pred-itl).
 *   The cache is paged in the PagedAttention sense (Sec. 2.1).  For request b
 *   with L_b cached tokens and query head h:
 *       g      = floor(h / G),  G = Hq / Hkv           (grouped-query heads)
 *       s_t    = scale * sum_d q[b][h][d] * k_t[d]       t = 0 .. L_b-1
 *       w_t    = exp(s_t - max_u s_u)
 *       out[d] = sum_t w_t v_t[d] / sum_t w_t
 *   where k_t, v_t are row (slot t mod S) of physical page
 *   page_table[b][t / S], KV head g.  L_b = 0 gives out = 0.
 *
 * Layouts (little-endian, row-major, element = raw bf16 bit pattern):
 *   q          uint16 [B][Hq][D]
 *   k_pages    uint16 [num_pages][S][Hkv][D]     v_pages: same
 *   page_table int32  [B][max_pages_per_seq]     entries past ceil(L_b/S) unused
 *   seq_lens   int32  [B]
 *   out        double [B][Hq][D]
 *
 * Precision: bf16 is widened exactly (bits << 16 -> float -> double); the
 * scale is the float the GPU receives, widened; every sum is a plain
 * ascending fp64 loop.  Softmax is max-subtracted so exp never overflows.
 *
 * Parity status: pinned by the not-gpu tests (brute force, L = 1, constant V,
 * shift invariance, page-permutation invariance, closed forms, GQA vs
 * duplicated MHA, one-hot, float64 SDPA of a library; the gather and the KV
 * append by direct indexing of the pools).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double vdo_bf16_to_f64(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Attention for one (request b, query head h); scores[] has room for L. */
static void vdo_one_head(const uint16_t *q, const uint16_t *k_pages,
                         const uint16_t *v_pages, const int32_t *page_table,
                         int L, int b, int h, int n_q_heads, int n_kv_heads,
                         int head_dim, int page_size, double scale,
                         int max_pages_per_seq, double *scores, double *out)
{
    const int G = n_q_heads / n_kv_heads;
    const int g = h / G;
    const size_t row = (size_t)n_kv_heads * head_dim;   /* one token's row */
    const size_t page = (size_t)page_size * row;        /* one page */
    const uint16_t *qh = q + ((size_t)b * n_q_heads + h) * head_dim;

    for (int d = 0; d < head_dim; ++d)
        out[d] = 0.0;
    if (L <= 0)
        return;

    /* scores */
    double m = -INFINITY;
    for (int t = 0; t < L; ++t) {
        const int32_t p = page_table[(size_t)b * max_pages_per_seq + t / page_size];
        const uint16_t *kt = k_pages + (size_t)p * page +
                             (size_t)(t % page_size) * row + (size_t)g * head_dim;
        double dot = 0.0;
        for (int d = 0; d < head_dim; ++d)
            dot += vdo_bf16_to_f64(qh[d]) * vdo_bf16_to_f64(kt[d]);
        scores[t] = scale * dot;
        if (scores[t] > m)
            m = scores[t];
    }

    /* weights and normaliser */
    double z = 0.0;
    for (int t = 0; t < L; ++t) {
        scores[t] = exp(scores[t] - m);
        z += scores[t];
    }

    /* weighted sum of value rows */
    for (int t = 0; t < L; ++t) {
        const int32_t p = page_table[(size_t)b * max_pages_per_seq + t / page_size];
        const uint16_t *vt = v_pages + (size_t)p * page +
                             (size_t)(t % page_size) * row + (size_t)g * head_dim;
        for (int d = 0; d < head_dim; ++d)
            out[d] += scores[t] * vdo_bf16_to_f64(vt[d]);
    }
    for (int d = 0; d < head_dim; ++d)
        out[d] /= z;
}

static int vdo_check_dims(int num_seqs, int n_q_heads, int n_kv_heads,
                          int head_dim, int page_size, int max_pages_per_seq)
{
    if (num_seqs < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 ||
        page_size <= 0 || max_pages_per_seq < 0)
        return 1;
    if (n_q_heads % n_kv_heads != 0)
        return 1;
    return 0;
}

/*
 * Full output.  nthreads <= 0 uses the OpenMP default.  Returns 0 on success,
 * 1 on bad dimensions, 2 if a scratch allocation fails.
 */
int vdo_decode_attn_f64(const uint16_t *q, const uint16_t *k_pages,
                        const uint16_t *v_pages, const int32_t *page_table,
                        const int32_t *seq_lens, double *out, int num_seqs,
                        int n_q_heads, int n_kv_heads, int head_dim,
                        int page_size, float scale, int max_pages_per_seq,
                        int nthreads)
{
    if (vdo_check_dims(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                       max_pages_per_seq))
        return 1;
    const long n_pairs = (long)num_seqs * n_q_heads;
    int failed = 0;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(|: failed)
#endif
    for (long i = 0; i < n_pairs; ++i) {
        const int b = (int)(i / n_q_heads), h = (int)(i % n_q_heads);
        const int L = seq_lens[b];
        double *scores = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
        if (!scores) {
            failed |= 1;
            continue;
        }
        vdo_one_head(q, k_pages, v_pages, page_table, L, b, h, n_q_heads,
                     n_kv_heads, head_dim, page_size, (double)scale,
                     max_pages_per_seq, scores, out + (size_t)i * head_dim);
        free(scores);
    }
    return failed ? 2 : 0;
}

/*
 * Selected outputs only: for k in [0, n_sel), computes the head_dim outputs of
 * (sel_b[k], sel_h[k]) into out[k][head_dim].  Used where the full output is
 * too slow to compute on the CPU.
 */
int vdo_decode_attn_rows_f64(const uint16_t *q, const uint16_t *k_pages,
                             const uint16_t *v_pages, const int32_t *page_table,
                             const int32_t *seq_lens, const int32_t *sel_b,
                             const int32_t *sel_h, int n_sel, double *out,
                             int num_seqs, int n_q_heads, int n_kv_heads,
                             int head_dim, int page_size, float scale,
                             int max_pages_per_seq, int nthreads)
{
    if (vdo_check_dims(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                       max_pages_per_seq) || n_sel < 0)
        return 1;
    for (int k = 0; k < n_sel; ++k)
        if (sel_b[k] < 0 || sel_b[k] >= num_seqs || sel_h[k] < 0 ||
            sel_h[k] >= n_q_heads)
            return 1;
    int failed = 0;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(|: failed)
#endif
    for (int k = 0; k < n_sel; ++k) {
        const int b = sel_b[k];
        const int L = seq_lens[b];
        double *scores = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
        if (!scores) {
            failed |= 1;
            continue;
        }
        vdo_one_head(q, k_pages, v_pages, page_table, L, b, sel_h[k], n_q_heads,
                     n_kv_heads, head_dim, page_size, (double)scale,
                     max_pages_per_seq, scores, out + (size_t)k * head_dim);
        free(scores);
    }
    return failed ? 2 : 0;
}

/*
 * Host gather through the page table: writes every cached K and V row of
 * every request, in logical token order, to k_out / v_out
 * (uint16 [sum_b L_b][Hkv][D]).  Pure byte copies.
 */
int vdo_gather(const uint16_t *k_pages, const uint16_t *v_pages,
               const int32_t *page_table, const int32_t *seq_lens,
               uint16_t *k_out, uint16_t *v_out, int num_seqs, int n_kv_heads,
               int head_dim, int page_size, int max_pages_per_seq)
{
    if (num_seqs < 0 || n_kv_heads <= 0 || head_dim <= 0 || page_size <= 0)
        return 1;
    const size_t row = (size_t)n_kv_heads * head_dim;
    size_t dst = 0;
    for (int b = 0; b < num_seqs; ++b) {
        for (int t = 0; t < seq_lens[b]; ++t) {
            const int32_t p = page_table[(size_t)b * max_pages_per_seq + t / page_size];
            const size_t src = (size_t)p * page_size * row + (size_t)(t % page_size) * row;
            memcpy(k_out + dst, k_pages + src, row * sizeof(uint16_t));
            memcpy(v_out + dst, v_pages + src, row * sizeof(uint16_t));
            dst += row;
        }
    }
    return 0;
}

/*
 * Append one token per request: copy k_new[b] / v_new[b] (uint16
 * [B][Hkv][D]) into row (pos mod S) of page page_table[b][pos / S] of the
 * pools, pos = positions[b]; requests with pos < 0 or pos >= max_pages * S
 * are skipped.  Pure byte copies.
 */
int vdo_kv_append(const uint16_t *k_new, const uint16_t *v_new, uint16_t *k_pages,
                  uint16_t *v_pages, const int32_t *page_table, const int32_t *positions,
                  int num_seqs, int n_kv_heads, int head_dim, int page_size,
                  int max_pages_per_seq)
{
    if (num_seqs < 0 || n_kv_heads <= 0 || head_dim <= 0 || page_size <= 0)
        return 1;
    const size_t row = (size_t)n_kv_heads * head_dim;
    for (int b = 0; b < num_seqs; ++b) {
        const int pos = positions[b];
        if (pos < 0 || pos >= max_pages_per_seq * page_size)
            continue;
        const int32_t p = page_table[(size_t)b * max_pages_per_seq + pos / page_size];
        const size_t dst = (size_t)p * page_size * row + (size_t)(pos % page_size) * row;
        memcpy(k_pages + dst, k_new + (size_t)b * row, row * sizeof(uint16_t));
        memcpy(v_pages + dst, v_new + (size_t)b * row, row * sizeof(uint16_t));
    }
    return 0;
}

/*
 * Dense projection of a decode step: y[m][n] = sum_k x[m][k] * w[n][k] for
 * x uint16 (bf16) [M][K] and w uint16 (bf16) [N][K] (the layout of a linear
 * layer's weight), y double [M][N]; plain ascending fp64 sums.  The paper's
 * decode latency model charges these GEMMs to N_req (Sec. 5.4, Eq.
 * pred-itl) and ties their latency steps to tile quantisation (Sec. 3.3).
 */
int vdo_gemm_f64(const uint16_t *x, const uint16_t *w, double *y, int M, int N, int K,
                 int nthreads)
{
    if (M < 0 || N < 0 || K < 0)
        return 1;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(static) num_threads(nthreads)
#endif
    for (long i = 0; i < (long)M * N; ++i) {
        const int m = (int)(i / N), n = (int)(i % N);
        double acc = 0.0;
        for (int k = 0; k < K; ++k)
            acc += vdo_bf16_to_f64(x[(size_t)m * K + k]) * vdo_bf16_to_f64(w[(size_t)n * K + k]);
        y[i] = acc;
    }
    return 0;
}

/* Max-subtracted softmax of n scores (exposed so tests can pin it alone). */
void vdo_softmax_f64(const double *s, int n, double *w)
{
    double m = -INFINITY, z = 0.0;
    for (int i = 0; i < n; ++i)
        if (s[i] > m)
            m = s[i];
    for (int i = 0; i < n; ++i) {
        w[i] = exp(s[i] - m);
        z += w[i];
    }
    for (int i = 0; i < n; ++i)
        w[i] /= z;
}

/* Number of OpenMP threads a default parallel region uses (1 without OpenMP). */
int vdo_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
