/* The library's host code under AddressSanitizer / UndefinedBehaviorSanitizer
 * (CPU test infrastructure): workspace queries over many shapes and every
 * argument-error path, all of which return before any GPU work; on a machine
 * without a GPU, valid calls that do reach the runtime must fail cleanly. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "vdecode.h"

static int failures = 0;
#define CHECK(c, ...) do { if (!(c)) { fprintf(stderr, __VA_ARGS__); fputc('\n', stderr); ++failures; } } while (0)

int main(void)
{
    void *F = (void *)(uintptr_t)0x10000;        /* 16-byte aligned, never dereferenced */
    void *MIS = (void *)(uintptr_t)0x10004;      /* misaligned */
    const int32_t *FI = (const int32_t *)F;

    for (int s = -1; s <= 5; ++s)
        CHECK(vd_status_string(s) && strlen(vd_status_string(s)) > 0, "status string %d", s);

    const size_t base = vd_decode_workspace_size(256, 32, 8, 128, 16, 1024, 0);
    CHECK(base > 0 && base == vd_decode_workspace_size(256, 32, 8, 128, 16, 1024, 0), "ws base");
    const int gs[5] = {1, 2, 4, 8, 16}, hkvs[4] = {1, 2, 4, 8};
    for (int gi = 0; gi < 5; ++gi)
        for (int hi = 0; hi < 4; ++hi)
            for (int B = 0; B <= 8192; B = B ? B * 8 : 1) {
                const size_t n = vd_decode_workspace_size(B, gs[gi] * hkvs[hi], hkvs[hi], 128, 16, 63, 0);
                CHECK(n > 0, "ws G %d Hkv %d B %d", gs[gi], hkvs[hi], B);
                CHECK(vd_decode_workspace_size(B, gs[gi] * hkvs[hi], hkvs[hi], 128, 16, 63,
                                               VD_FLAG_RANGE_TILES(1)) > 0, "forced ws");
            }
    CHECK(vd_decode_workspace_size(4, 32, 8, 64, 16, 63, 0) == 0, "head_dim 64");
    CHECK(vd_decode_workspace_size(4, 30, 8, 128, 16, 63, 0) == 0, "Hq 30");
    CHECK(vd_decode_workspace_size(9000, 32, 8, 128, 16, 63, 0) == 0, "B 9000");
    CHECK(vd_decode_workspace_size(8192, 262144, 16384, 128, 16, 1, 0) == 0, "32-bit limit");

    const size_t need = vd_decode_workspace_size(4, 32, 8, 128, 16, 63, 0);
#define ATTN(fn, q, k, v, pt, sl, out, B, hq, hkv, d, s, sc, mp, ws, wsb, fl) \
    fn(q, k, v, pt, sl, out, B, hq, hkv, d, s, sc, mp, ws, wsb, fl, NULL)
    for (int e = 0; e < 2; ++e) {
        int (*fn)(const void *, const void *, const void *, const int32_t *, const int32_t *, void *,
                  int, int, int, int, int, float, int, void *, size_t, unsigned, hipStream_t) =
            e ? vd_decode_partial : vd_decode_attn;
        CHECK(ATTN(fn, NULL, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.088f, 63, F, need, 0) == VD_ERROR_INVALID_VALUE, "null q");
        CHECK(ATTN(fn, MIS, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.088f, 63, F, need, 0) == VD_ERROR_INVALID_VALUE, "mis q");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.0f / 0.0f, 63, F, need, 0) == VD_ERROR_INVALID_VALUE, "nan scale");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.088f, 63, F, need, 1u << 7) == VD_ERROR_INVALID_VALUE, "flag");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, -1, 32, 8, 128, 16, 0.088f, 63, F, need, 0) == VD_ERROR_INVALID_VALUE, "B -1");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 4, 24, 8, 128, 16, 0.088f, 63, F, need, 0) == VD_ERROR_NOT_SUPPORTED, "G 3");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 4, 32, 8, 128, 32, 0.088f, 63, F, need, 0) == VD_ERROR_NOT_SUPPORTED, "S 32");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.088f, 63, F, need - 1, 0) == VD_ERROR_WORKSPACE_TOO_SMALL, "ws small");
        CHECK(ATTN(fn, F, F, F, FI, FI, F, 0, 32, 8, 128, 16, 0.088f, 63, F, need, 0) == VD_SUCCESS, "B 0");
    }
    CHECK(vd_decode_plan(NULL, 4, 32, 8, 128, 16, 63, F, need, 0, NULL) == VD_ERROR_INVALID_VALUE, "plan null");
    CHECK(vd_decode_combine(NULL, 4, 32, 8, 128, 16, 63, F, need, 0, NULL) == VD_ERROR_INVALID_VALUE, "combine null");
    CHECK(vd_decode_gather(F, F, FI, FI, NULL, F, 4, 8, 128, 16, 63, F, need, NULL) == VD_ERROR_INVALID_VALUE, "gather null");
    CHECK(vd_kv_append(F, F, F, F, FI, NULL, 4, 8, 128, 16, 63, NULL) == VD_ERROR_INVALID_VALUE, "append null");
    CHECK(vd_kv_append(F, F, F, F, FI, FI, 4, 8, 64, 16, 63, NULL) == VD_ERROR_NOT_SUPPORTED, "append D 64");
    CHECK(vd_gemm_bf16(F, F, F, 99, 64, 500, F, 1 << 20, 0, NULL) == VD_ERROR_NOT_SUPPORTED, "gemm K 500");
    CHECK(vd_gemm_bf16(F, F, F, 4, 64, 512, F, 1 << 20, VD_GEMM_FLAG_TILE(4), NULL) == VD_ERROR_NOT_SUPPORTED,
          "gemm 128-column tile on 64 columns");
    CHECK(vd_gemm_bf16(NULL, F, F, 1, 64, 512, F, 1 << 20, 0, NULL) == VD_ERROR_INVALID_VALUE, "gemm null");
    CHECK(vd_stream_read(NULL, 1024, F, 8, NULL) == VD_ERROR_INVALID_VALUE, "stream null");

    /* the GEMM plan over sizes and every forced tile and slice count
     * (including ones past the table): a workspace is 0 or S fp32 partials
     * of M x N with S a power of two up to 16 */
    {
        const int Ms[] = {1, 7, 16, 17, 63, 64, 65, 255, 256, 257, 513, 640, 1024, 4096, 1 << 16};
        const int Ns[] = {64, 128, 192, 256, 4096, 6144, 28672, 1 << 20};
        const int Ks[] = {512, 1024, 4096, 14336, 1 << 20};
        for (size_t a = 0; a < sizeof(Ms) / sizeof(Ms[0]); ++a)
            for (size_t b = 0; b < sizeof(Ns) / sizeof(Ns[0]); ++b)
                for (size_t c = 0; c < sizeof(Ks) / sizeof(Ks[0]); ++c)
                    for (int t = -1; t < 16; ++t)
                        for (int l = -1; l < 16; l += 3) {
                            const unsigned fl = (t >= 0 ? VD_GEMM_FLAG_TILE(t) : 0u) |
                                                (l >= 0 ? VD_GEMM_FLAG_SLICES_LOG2(l) : 0u);
                            const size_t n = vd_gemm_workspace_size(Ms[a], Ns[b], Ks[c], fl);
                            const size_t unit = (size_t)Ms[a] * Ns[b] * 4;
                            int ok = n == 0;
                            for (int S = 2; S <= 16 && !ok; S *= 2)
                                ok = n == unit * S;
                            CHECK(ok, "gemm ws M %d N %d K %d flags %#x: %zu", Ms[a], Ns[b], Ks[c], fl, n);
                        }
    }

    /* valid calls reach the runtime: without a device they must fail cleanly */
    const int rc = ATTN(vd_decode_attn, F, F, F, FI, FI, F, 4, 32, 8, 128, 16, 0.088f, 63, F, need, 0);
    CHECK(rc == VD_SUCCESS || rc == VD_ERROR_LAUNCH, "valid attn rc %d", rc);

    if (failures)
        fprintf(stderr, "%d check(s) failed\n", failures);
    else
        printf("host ABI under sanitizers: all checks passed\n");
    return failures ? 1 : 0;
}
