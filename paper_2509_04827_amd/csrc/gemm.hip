// Decode-step projection GEMM for MI355X (gfx950): y = x . w^T with few rows.
//
// A decode iteration multiplies the N_req current tokens by every weight
// matrix of the model; the paper charges this GEMM work to N_req in its
// decode latency model (Sec. 5.4, Eq. pred-itl) and traces the latency steps
// it sees at batch 256 -> 257 to GEMM tile quantisation (Sec. 3.3).  For
// decode batches up to 64 rows the GEMM reads far more weight bytes than it
// does arithmetic (2*M flop per weight element, against ~312 flop/B of MFMA
// to HBM balance), so this kernel streams the weights once at HBM speed:
//
//   * a workgroup owns 16 * NB output columns (NB 16-column MFMA blocks: 1
//     for batches up to 8 rows, 4 above, where the x rows are re-read less
//     often) and a slice of K; its four waves (eight when 16-column tiles
//     number at most one per CU) split the slice and merge their
//     accumulators in LDS in a fixed order;
//   * a wave loads the weight rows in whole 128-byte pieces (8 rows per
//     instruction, 8 lanes per row) and moves them through its own LDS tile
//     into the B operand of v_mfma_f32_16x16x32_bf16 (lane = output column):
//     the operand layout itself would read 64 bytes per row per instruction,
//     which streams 20-35% slower.  x rows go straight into the A operand
//     (lane = batch row).  Four K steps per batch, two batches in flight;
//   * when there are too few column tiles to fill the device, K is split
//     over workgroups as well; each slice writes an fp32 partial and a second
//     kernel adds the slices in order (deterministic, no atomics).
//
// x bf16 [M][K], w bf16 [N][K] (a linear layer's weight), y bf16 (RNE) or
// fp32 [M][N]; fp32 accumulation.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <stdint.h>

#include "vdecode.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kTileN = 64;                    // column granularity of N (the widest tile)
constexpr int kKStep = 32;                    // K per MFMA
constexpr int kUnroll = 4;                    // K steps per load batch (the LDS tile assumes 4)
constexpr int kBatchK = kKStep * kUnroll;     // 128
constexpr int kSliceAlign = 4 * kBatchK;      // K slice granularity: 512 (four waves x one batch)
constexpr int kMaxM = 64;
constexpr int kReduceThreads = 256;
constexpr int kGemmGroupsPerCU = 1;           // split K until this many workgroups exist

struct GemmArgs {
    const uint16_t *x, *w;
    void *y;
    float *part;
    int M, N, K, kslice;
};

template <int NB, int MB>
struct Batch {
    u32x4 w[NB][kUnroll];
    u32x4 x[MB][kUnroll];
};

__device__ inline unsigned short bf16_rne(float f)
{
    return __builtin_bit_cast(unsigned short, (__bf16)f);
}

// MODE 0: bf16 y, 1: fp32 y, 2: fp32 partial per K slice.  WAVES waves split
// the K slice (4, or 8 when there are few column tiles).
template <int NB, int MB, int MODE, int WAVES>
__global__ void __launch_bounds__(64 * WAVES)
gemm_kernel(const GemmArgs a)
{
    constexpr int kNB = NB;
    __shared__ f32x4 red[WAVES - 1][kNB * MB][64];
    // per wave: the batch's weight rows, 16 rows x 256 B (+16 B against bank
    // conflicts on the column reads) per block
    static_assert(kUnroll == 4, "two row halves x two K halves per block");
    __shared__ u32x4 wst[WAVES][kNB][16][4 * kUnroll + 1];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, grp = lane >> 4;
    const int n0 = blockIdx.x * 16 * kNB;
    const int slice = blockIdx.y;
    const int kw = a.kslice / WAVES;
    const int kb = slice * a.kslice + wave * kw;
    const int K = a.K, M = a.M;

    // loads: instruction (h, c) of a block reads rows 8h .. 8h+7, 128 B each
    // (k 64c .. 64c+63 of the batch), lane l: row 8h + l/8, k 64c + 8 (l % 8)
    const uint16_t *wp[kNB][2];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int h = 0; h < 2; ++h)
            wp[nb][h] = a.w + (size_t)(n0 + 16 * nb + 8 * h + (lane >> 3)) * K + kb + 8 * (lane & 7);
    const uint16_t *xp[MB];
    bool xv[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        xv[mb] = 16 * mb + r < M;
        xp[mb] = a.x + (size_t)(xv[mb] ? 16 * mb + r : 0) * K + kb + 8 * grp;
    }

    auto load = [&](Batch<kNB, MB> &B, int koff) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb)
                B.w[nb][u] = __builtin_nontemporal_load(
                    (const u32x4 *)(wp[nb][u & 1] + koff + 64 * (u >> 1)));
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                B.x[mb][u] = xv[mb] ? *(const u32x4 *)(xp[mb] + koff + kKStep * u)
                                    : u32x4{0u, 0u, 0u, 0u};
    };

    f32x4 acc[kNB][MB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](const Batch<kNB, MB> &B) {
        // through LDS into the B-operand layout: lane (r, grp) of K step u
        // takes row r, 16-byte chunk 4u + grp
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                wst[wave][nb][8 * (u & 1) + (lane >> 3)][8 * (u >> 1) + (lane & 7)] = B.w[nb][u];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) {
                const u32x4 wf = wst[wave][nb][r][4 * u + grp];
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, B.x[mb][u]), __builtin_bit_cast(bf16x8, wf),
                        acc[nb][mb], 0, 0, 0);
            }
    };

    // two batches in flight; past the end the prefetch re-reads the wave's
    // last batch (a cache hit) so every path issues the same loads
    const int nbatch = kw / kBatchK;
    Batch<kNB, MB> b0, b1;
    load(b0, 0);
    int i = 0;
    for (; i + 1 < nbatch; i += 2) {
        load(b1, (i + 1) * kBatchK);
        __builtin_amdgcn_sched_barrier(0);
        compute(b0);
        load(b0, min(i + 2, nbatch - 1) * kBatchK);
        __builtin_amdgcn_sched_barrier(0);
        compute(b1);
    }
    if (nbatch & 1)
        compute(b0);

    // merge the waves in order 0, 1, ..., WAVES - 1
    if (wave > 0) {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                red[wave - 1][nb * MB + mb][lane] = acc[nb][mb];
    }
    __syncthreads();
    if (wave != 0)
        return;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            f32x4 v = acc[nb][mb];
#pragma unroll
            for (int x = 0; x < WAVES - 1; ++x)
                v += red[x][nb * MB + mb][lane];
            // v[i]: row 16mb + 4grp + i, column n0 + 16nb + r
            const int n = n0 + 16 * nb + r;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = 16 * mb + 4 * grp + i;
                if (m < M) {
                    if constexpr (MODE == 2)
                        a.part[((size_t)slice * M + m) * a.N + n] = v[i];
                    else if constexpr (MODE == 1)
                        ((float *)a.y)[(size_t)m * a.N + n] = v[i];
                    else
                        ((uint16_t *)a.y)[(size_t)m * a.N + n] = bf16_rne(v[i]);
                }
            }
        }
    }
}

// y[e] = sum over slices s = 0 .. S-1 (in order) of part[s][e], four per thread.
template <int MODE>
__global__ void __launch_bounds__(kReduceThreads)
gemm_reduce_kernel(const float *__restrict__ part, void *__restrict__ y, size_t elems, int S)
{
    const size_t e4 = ((size_t)blockIdx.x * kReduceThreads + threadIdx.x) * 4;
    if (e4 >= elems)
        return;
    f32x4 v = *(const f32x4 *)(part + e4);
    for (int s = 1; s < S; ++s)
        v += *(const f32x4 *)(part + (size_t)s * elems + e4);
    if constexpr (MODE == 1) {
        *(f32x4 *)((float *)y + e4) = v;
    } else {
        uint16_t *o = (uint16_t *)y + e4;
        *(unsigned *)o = (unsigned)bf16_rne(v[0]) | ((unsigned)bf16_rne(v[1]) << 16);
        *(unsigned *)(o + 2) = (unsigned)bf16_rne(v[2]) | ((unsigned)bf16_rne(v[3]) << 16);
    }
}

bool aligned(const void *p, size_t al) { return ((uintptr_t)p & (al - 1)) == 0; }

// Compute units of the current device, queried once per device (0 = not yet).
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

int device_cus(int *cus)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VD_ERROR_LAUNCH;
    if (dev >= 0 && dev < kMaxDevices) {
        const int v = g_cus[dev].load(std::memory_order_relaxed);
        if (v > 0) {
            *cus = v;
            return VD_SUCCESS;
        }
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return VD_ERROR_LAUNCH;
    if (dev >= 0 && dev < kMaxDevices)
        g_cus[dev].store(n, std::memory_order_relaxed);
    *cus = n;
    return VD_SUCCESS;
}

int gemm_check(int M, int N, int K, unsigned flags)
{
    if (M <= 0 || N <= 0 || K <= 0)
        return VD_ERROR_INVALID_VALUE;
    if (flags & ~VD_FLAG_OUT_F32)
        return VD_ERROR_INVALID_VALUE;
    if (M > kMaxM || N % kTileN != 0 || K % kSliceAlign != 0)
        return VD_ERROR_NOT_SUPPORTED;
    if ((long long)N * K >= (1LL << 40) || (long long)M * N >= (1LL << 31))
        return VD_ERROR_NOT_SUPPORTED;
    return VD_SUCCESS;
}

// Columns per workgroup for a batch of M rows.
int gemm_nb(int M) { return M <= 8 ? 1 : 4; }

// K slices: the largest power of two dividing K / 512 that keeps the
// workgroup count within kGemmGroupsPerCU per CU.
int gemm_slices(int M, int N, int K, int cus)
{
    const int tiles = N / (16 * gemm_nb(M));
    const int units = K / kSliceAlign;
    int S = 1;
    while (units % (2 * S) == 0 && (long long)tiles * 2 * S <= (long long)kGemmGroupsPerCU * cus)
        S *= 2;
    return S;
}

// Waves per workgroup: 8 for 16-column tiles when they number at most one per
// CU (more K parallelism per tile: down and o_proj at small M), if the K
// slice is whole 8-wave batches; else 4.
int gemm_waves(int M, int N, int K, int S, int cus)
{
    return gemm_nb(M) == 1 && N / 16 <= cus && (K / S) % (8 * kBatchK) == 0 ? 8 : 4;
}

template <int NB, int MB, int WAVES>
void launch_gemm(const GemmArgs &g, int S, bool f32, hipStream_t stream)
{
    const dim3 grid(g.N / (16 * NB), S), block(64 * WAVES);
    if (S > 1)
        hipLaunchKernelGGL((gemm_kernel<NB, MB, 2, WAVES>), grid, block, 0, stream, g);
    else if (f32)
        hipLaunchKernelGGL((gemm_kernel<NB, MB, 1, WAVES>), grid, block, 0, stream, g);
    else
        hipLaunchKernelGGL((gemm_kernel<NB, MB, 0, WAVES>), grid, block, 0, stream, g);
}

}  // namespace

extern "C" {

size_t vd_gemm_workspace_size(int M, int N, int K, unsigned flags)
{
    if (gemm_check(M, N, K, flags))
        return 0;
    // any slice count the device may pick divides K / 512
    return (size_t)(K / kSliceAlign) * M * N * sizeof(float);
}

int vd_gemm_bf16(const void *x, const void *w, void *y, int M, int N, int K, void *workspace,
                 size_t workspace_bytes, unsigned flags, hipStream_t stream)
{
    int st = gemm_check(M, N, K, flags);
    if (st)
        return st;
    if (!x || !w || !y || !aligned(x, 16) || !aligned(w, 16) || !aligned(y, 16))
        return VD_ERROR_INVALID_VALUE;
    int cus = 0;
    if (device_cus(&cus) != VD_SUCCESS)
        return VD_ERROR_LAUNCH;
    const int S = gemm_slices(M, N, K, cus);
    if (S > 1) {
        if (!workspace || !aligned(workspace, 16))
            return VD_ERROR_INVALID_VALUE;
        if (workspace_bytes < (size_t)S * M * N * sizeof(float))
            return VD_ERROR_WORKSPACE_TOO_SMALL;
    }
    GemmArgs g;
    g.x = (const uint16_t *)x;
    g.w = (const uint16_t *)w;
    g.y = y;
    g.part = (float *)workspace;
    g.M = M;
    g.N = N;
    g.K = K;
    g.kslice = K / S;
    const bool f32 = flags & VD_FLAG_OUT_F32;
    if (gemm_nb(M) == 1) {
        if (gemm_waves(M, N, K, S, cus) == 8)
            launch_gemm<1, 1, 8>(g, S, f32, stream);
        else
            launch_gemm<1, 1, 4>(g, S, f32, stream);
    } else {
        switch ((M + 15) / 16) {
        case 1: launch_gemm<4, 1, 4>(g, S, f32, stream); break;
        case 2: launch_gemm<4, 2, 4>(g, S, f32, stream); break;
        case 3: launch_gemm<4, 3, 4>(g, S, f32, stream); break;
        default: launch_gemm<4, 4, 4>(g, S, f32, stream); break;
        }
    }
    if (S > 1) {
        const size_t elems = (size_t)M * N;   // N % 32 == 0, so elems % 4 == 0
        const dim3 grid((unsigned)((elems / 4 + kReduceThreads - 1) / kReduceThreads));
        if (f32)
            hipLaunchKernelGGL(gemm_reduce_kernel<1>, grid, dim3(kReduceThreads), 0, stream,
                               (const float *)workspace, y, elems, S);
        else
            hipLaunchKernelGGL(gemm_reduce_kernel<0>, grid, dim3(kReduceThreads), 0, stream,
                               (const float *)workspace, y, elems, S);
    }
    return hipGetLastError() == hipSuccess ? VD_SUCCESS : VD_ERROR_LAUNCH;
}

}  // extern "C"
