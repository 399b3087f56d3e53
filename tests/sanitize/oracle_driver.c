/* The oracle under AddressSanitizer / UndefinedBehaviorSanitizer (CPU test
 * infrastructure).  Exact-size allocations, so any read or write outside an
 * input is reported; the checks are closed forms that hold exactly. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int vdo_decode_attn_f64(const uint16_t *, const uint16_t *, const uint16_t *, const int32_t *,
                        const int32_t *, double *, int, int, int, int, int, float, int, int);
int vdo_decode_attn_rows_f64(const uint16_t *, const uint16_t *, const uint16_t *, const int32_t *,
                             const int32_t *, const int32_t *, const int32_t *, int, double *, int,
                             int, int, int, int, float, int, int);
int vdo_gather(const uint16_t *, const uint16_t *, const int32_t *, const int32_t *, uint16_t *,
               uint16_t *, int, int, int, int, int);
int vdo_kv_append(const uint16_t *, const uint16_t *, uint16_t *, uint16_t *, const int32_t *,
                  const int32_t *, int, int, int, int, int);
int vdo_gemm_f64(const uint16_t *, const uint16_t *, double *, int, int, int, int);
void vdo_softmax_f64(const double *, int, double *);

enum { B = 4, HQ = 4, HKV = 2, D = 128, S = 16, MAXP = 3 };

static int failures = 0;
#define CHECK(c, ...) do { if (!(c)) { fprintf(stderr, __VA_ARGS__); fputc('\n', stderr); ++failures; } } while (0)

static uint16_t bf16_of(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);   /* values below are exact in bf16 */
}

static double f_of(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static uint32_t lcg = 12345u;
static float small_value(void)
{
    lcg = lcg * 1664525u + 1013904223u;
    return (float)((int)(lcg >> 24) - 128) / 64.0f;   /* multiples of 1/64 in [-2, 2) */
}

int main(void)
{
    const int32_t lens[B] = {1, 17, 0, 40};
    int P[B], npages = 0;
    for (int b = 0; b < B; ++b) {
        P[b] = (lens[b] + S - 1) / S;
        npages += P[b];
    }
    const int pool = npages + 1;   /* plus a spare page */
    const size_t row = (size_t)HKV * D, page = (size_t)S * row;
    int32_t *pt = malloc(sizeof(int32_t) * B * MAXP);
    int32_t *sl = malloc(sizeof(lens));
    memcpy(sl, lens, sizeof(lens));
    for (int b = 0, next = npages - 1; b < B; ++b)   /* pages dealt in reverse */
        for (int j = 0; j < MAXP; ++j)
            pt[b * MAXP + j] = j < P[b] ? next-- : npages;
    uint16_t *q = malloc(sizeof(uint16_t) * B * HQ * D);
    uint16_t *k = malloc(sizeof(uint16_t) * pool * page);
    uint16_t *v = malloc(sizeof(uint16_t) * pool * page);
    for (size_t i = 0; i < (size_t)B * HQ * D; ++i) q[i] = bf16_of(small_value());
    for (size_t i = 0; i < pool * page; ++i) k[i] = bf16_of(small_value());
    /* constant V per KV head: out = c_g for every non-empty request */
    for (size_t p = 0; p < (size_t)pool; ++p)
        for (int s = 0; s < S; ++s)
            for (int g = 0; g < HKV; ++g)
                for (int d = 0; d < D; ++d)
                    v[p * page + s * row + g * D + d] = bf16_of((float)(g + 1) * 0.5f - (float)d / 64.0f);

    double *out = malloc(sizeof(double) * B * HQ * D);
    const float scale = 0.08838834764831845f;
    CHECK(vdo_decode_attn_f64(q, k, v, pt, sl, out, B, HQ, HKV, D, S, scale, MAXP, 1) == 0, "attn rc");
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < HQ; ++h)
            for (int d = 0; d < D; ++d) {
                const int g = h / (HQ / HKV);
                const double want = lens[b] ? f_of(bf16_of((float)(g + 1) * 0.5f - (float)d / 64.0f)) : 0.0;
                const double got = out[((size_t)b * HQ + h) * D + d];
                CHECK(fabs(got - want) <= 1e-12, "constant V b %d h %d d %d: %g vs %g", b, h, d, got, want);
            }

    /* L = 1 with random V: out = that row */
    for (size_t i = 0; i < pool * page; ++i) v[i] = bf16_of(small_value());
    CHECK(vdo_decode_attn_f64(q, k, v, pt, sl, out, B, HQ, HKV, D, S, scale, MAXP, 1) == 0, "attn rc");
    for (int h = 0; h < HQ; ++h)
        for (int d = 0; d < D; ++d) {
            const double want = f_of(v[(size_t)pt[0] * page + (h / 2) * D + d]);
            CHECK(out[(size_t)h * D + d] == want, "L=1 h %d d %d", h, d);
        }

    /* selected rows equal the full result */
    const int32_t selb[3] = {3, 1, 2}, selh[3] = {0, 3, 1};
    double *rows = malloc(sizeof(double) * 3 * D);
    CHECK(vdo_decode_attn_rows_f64(q, k, v, pt, sl, selb, selh, 3, rows, B, HQ, HKV, D, S, scale,
                                   MAXP, 1) == 0, "rows rc");
    for (int i = 0; i < 3; ++i)
        for (int d = 0; d < D; ++d)
            CHECK(rows[i * D + d] == out[((size_t)selb[i] * HQ + selh[i]) * D + d], "row %d d %d", i, d);

    /* gather: direct indexing */
    int ntok = 0;
    for (int b = 0; b < B; ++b) ntok += lens[b];
    uint16_t *ko = malloc(sizeof(uint16_t) * ntok * row), *vo = malloc(sizeof(uint16_t) * ntok * row);
    CHECK(vdo_gather(k, v, pt, sl, ko, vo, B, HKV, D, S, MAXP) == 0, "gather rc");
    for (int b = 0, t0 = 0; b < B; t0 += lens[b], ++b)
        for (int t = 0; t < lens[b]; ++t) {
            const size_t src = (size_t)pt[b * MAXP + t / S] * page + (size_t)(t % S) * row;
            CHECK(!memcmp(ko + (size_t)(t0 + t) * row, k + src, row * 2), "gather k %d %d", b, t);
            CHECK(!memcmp(vo + (size_t)(t0 + t) * row, v + src, row * 2), "gather v %d %d", b, t);
        }

    /* KV append: positions in range, negative and past the table */
    uint16_t *kn = malloc(sizeof(uint16_t) * B * row), *vn = malloc(sizeof(uint16_t) * B * row);
    for (size_t i = 0; i < (size_t)B * row; ++i) { kn[i] = (uint16_t)i; vn[i] = (uint16_t)(i ^ 0x5555u); }
    const int32_t pos[B] = {0, 17, -1, MAXP * S};
    uint16_t *k2 = malloc(sizeof(uint16_t) * pool * page), *v2 = malloc(sizeof(uint16_t) * pool * page);
    memcpy(k2, k, sizeof(uint16_t) * pool * page);
    memcpy(v2, v, sizeof(uint16_t) * pool * page);
    int32_t *posd = malloc(sizeof(pos));
    memcpy(posd, pos, sizeof(pos));
    CHECK(vdo_kv_append(kn, vn, k2, v2, pt, posd, B, HKV, D, S, MAXP) == 0, "append rc");
    for (int b = 0; b < B; ++b) {
        if (pos[b] < 0 || pos[b] >= MAXP * S)
            continue;
        const size_t dst = (size_t)pt[b * MAXP + pos[b] / S] * page + (size_t)(pos[b] % S) * row;
        CHECK(!memcmp(k2 + dst, kn + (size_t)b * row, row * 2), "append k %d", b);
        memcpy(k2 + dst, k + dst, row * 2);
        memcpy(v2 + dst, v + dst, row * 2);
    }
    CHECK(!memcmp(k2, k, sizeof(uint16_t) * pool * page) && !memcmp(v2, v, sizeof(uint16_t) * pool * page),
          "append touched other rows");

    /* GEMM: identity weight returns x */
    enum { M = 3, K = 40 };
    uint16_t *x = malloc(sizeof(uint16_t) * M * K), *w = calloc((size_t)K * K, sizeof(uint16_t));
    for (int i = 0; i < M * K; ++i) x[i] = bf16_of(small_value());
    for (int i = 0; i < K; ++i) w[i * K + i] = bf16_of(1.0f);
    double *y = malloc(sizeof(double) * M * K);
    CHECK(vdo_gemm_f64(x, w, y, M, K, K, 1) == 0, "gemm rc");
    for (int i = 0; i < M * K; ++i) CHECK(y[i] == f_of(x[i]), "gemm %d", i);

    /* softmax sums to one */
    double s[5] = {1.0, -3.0, 700.0, 699.5, -1e300}, wsm[5], z = 0.0;
    vdo_softmax_f64(s, 5, wsm);
    for (int i = 0; i < 5; ++i) z += wsm[i];
    CHECK(fabs(z - 1.0) < 1e-15, "softmax sum %g", z);

    free(pt); free(sl); free(q); free(k); free(v); free(out); free(rows); free(ko); free(vo);
    free(kn); free(vn); free(k2); free(v2); free(posd); free(x); free(w); free(y);
    if (failures)
        fprintf(stderr, "%d check(s) failed\n", failures);
    else
        printf("oracle under sanitizers: all checks passed\n");
    return failures ? 1 : 0;
}
