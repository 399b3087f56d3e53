// Decode-step projection GEMM for MI355X (gfx950): y = x . w^T for a decode
// batch of M rows.
//
// A decode iteration multiplies the N_req current tokens by every weight
// matrix of the model; the paper charges this GEMM work to N_req in its decode
// latency model (Sec. 5.4, Eq. pred-itl) and traces the latency steps it sees
// at batch 256 -> 257 to GEMM tile quantisation (Sec. 3.3).  Up to a few
// hundred rows the GEMM is bound by reading the weights (2*M flop per weight
// element against ~312 flop/B of MFMA-to-HBM balance); past that, by the
// matrix cores.  Two tiled kernels cover both, under one plan:
//
//   * a workgroup of four waves owns a BM x BN output tile and a K slice; the
//     x and w tiles of each K stage (BK columns) are loaded with 16-byte loads
//     (whole 128- or 256-byte row pieces) into registers, and from there into
//     one of two LDS buffers (rows padded by 16 bytes against bank
//     conflicts), P stages ahead of the one being multiplied; the tiles for
//     larger batches (128 x 128 and 256 x 128 with four waves; 192, 256 or
//     320 x 256 with eight) load their stages straight from memory into a
//     ring of LDS slots instead (gemm_dma_kernel), so the pipeline depth
//     costs no registers;
//   * each wave multiplies its (BN/WN) x (BM/WM) part of the tile with
//     v_mfma_f32_16x16x32_bf16, the w fragment as the A operand (lane = output
//     column) and the x fragment as B (lane = batch row), so the accumulator
//     holds four consecutive output columns of one row per lane and the
//     stores are 16 (fp32) or 8 (bf16) bytes wide;
//   * w is streamed past the caches when one row tile covers the batch (each
//     element is read once); x is re-read by every column tile and stays in
//     L2;
//   * the tiles that share a w tile (same columns, other rows) are given
//     workgroup indices that land on the same XCD at about the same time
//     (workgroups are dealt to the 8 XCDs round-robin), so w comes from HBM
//     once and from that XCD's L2 for the others;
//   * when the tiles cannot fill the device, K is split into S slices over
//     workgroups; each slice writes an fp32 partial and a second kernel adds
//     the slices in order (deterministic, no atomics).
//
// The tile shape and S follow from (M, N, K) alone (a cost model whose
// constants were fitted on MI355X), so the result and the workspace size do
// not depend on the device.
//
// x bf16 [M][K], w bf16 [N][K] (a linear layer's weight), y bf16 (RNE) or
// fp32 [M][N]; fp32 accumulation.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <stdint.h>

#include "vdecode.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;                 // four waves per workgroup (eight for the 256-column tiles)
constexpr int kNAlign = 64;                   // N granularity
constexpr int kKAlign = 512;                  // K granularity
constexpr int kReduceThreads = 256;
constexpr int kTargetCUs = 256;               // MI355X compute units: the tile table's target
constexpr int kMaxSlicesLog2 = 4;             // at most 16 K slices

enum { OUT_BF16 = 0, OUT_F32 = 1, OUT_PART = 2 };

struct GemmArgs {
    const uint16_t *x, *w;
    void *y;
    float *part;          // [S][M][N] fp32 partials when S > 1
    int M, N, K;
    int kslice;           // K columns per slice
    int S;                // slices
    int tiles_m;          // row tiles
    int groups;           // column tiles * S
};

__device__ inline unsigned short bf16_rne(float f)
{
    return __builtin_bit_cast(unsigned short, (__bf16)f);
}

// One tile configuration: BM x BN output tile, BK columns of K per stage,
// waves WM (rows) x WN (columns), P stages of loads in flight.  NT: w is
// loaded past the caches (one row tile reads each w tile once); without it,
// the row tiles that share a w tile find it in L2.
template <int BM, int BN, int BK, int WM, int WN, int P, int MODE, bool NT = true>
__global__ void __launch_bounds__(kThreads)
gemm_tile_kernel(const GemmArgs a)
{
    constexpr int CPR = BK / 8;                  // 16-byte chunks per row and stage
    constexpr int RS = BK + 8;                   // LDS row stride in bf16 (16-byte pad)
    constexpr int RPL = kThreads / CPR;          // rows one load instruction covers (all threads)
    constexpr int LX = BM / RPL, LW = BN / RPL;  // loads per thread and stage
    constexpr int TM = BM / WM, TN = BN / WN;    // a wave's rows and columns
    constexpr int FM = TM / 16, FN = TN / 16;    // its 16 x 16 blocks
    static_assert(WM * WN == kThreads / 64, "four waves");
    static_assert(BM % RPL == 0 && BN % RPL == 0 && LX >= 1 && LW >= 1, "whole loads");
    static_assert(TM % 16 == 0 && TN % 16 == 0 && BK % 32 == 0, "whole MFMA blocks");
    __shared__ __attribute__((aligned(16))) uint16_t lds[2][(BM + BN) * RS];

    // tile of this workgroup: the tiles_m row tiles of one group (column
    // tile, slice) sit 8 indices apart, within one window of 8 * tiles_m
    const int i = blockIdx.x, TMc = a.tiles_m, G = a.groups;
    const int full = G / 8 * 8;
    int tm, g;
    if (i < full * TMc) {
        const int sg = i / (8 * TMc), rem = i - sg * 8 * TMc;
        tm = rem >> 3;
        g = sg * 8 + (rem & 7);
    } else {
        const int j = i - full * TMc, r8 = G - full;
        tm = j / r8;
        g = full + (j - tm * r8);
    }
    const int tn = g / a.S, s = g - tn * a.S;
    const int m0 = tm * BM, n0 = tn * BN;
    const int M = a.M, N = a.N, K = a.K;
    const int nk = a.kslice / BK;

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int lrow = t / CPR, lc = (t % CPR) * 8;   // this thread's load row and column
    const uint16_t *xp = a.x + (size_t)min(m0 + lrow, M - 1) * K + (size_t)s * a.kslice + lc;
    const uint16_t *wp = a.w + (size_t)(n0 + lrow) * K + (size_t)s * a.kslice + lc;
    const size_t xstep = (size_t)RPL * K;           // next load's rows
    // rows past M repeat row M - 1 (loaded, never stored)
    int xrow_ok[LX];
#pragma unroll
    for (int l = 0; l < LX; ++l)
        xrow_ok[l] = m0 + lrow + l * RPL < M;

    u32x4 rx[P][LX], rw[P][LW];
    auto load = [&](u32x4 (&ox)[LX], u32x4 (&ow)[LW], int kt) {
        const size_t off = (size_t)min(kt, nk - 1) * BK;   // past the end: the last stage again
#pragma unroll
        for (int l = 0; l < LX; ++l)
            ox[l] = *(const u32x4 *)(xrow_ok[l] ? xp + l * xstep + off : xp + off);
#pragma unroll
        for (int l = 0; l < LW; ++l) {
            if constexpr (NT)
                ow[l] = __builtin_nontemporal_load((const u32x4 *)(wp + l * xstep + off));
            else
                ow[l] = *(const u32x4 *)(wp + l * xstep + off);
        }
    };
    auto store = [&](const u32x4 (&ox)[LX], const u32x4 (&ow)[LW], int buf) {
#pragma unroll
        for (int l = 0; l < LX; ++l)
            *(u32x4 *)&lds[buf][(lrow + l * RPL) * RS + lc] = ox[l];
#pragma unroll
        for (int l = 0; l < LW; ++l)
            *(u32x4 *)&lds[buf][(BM + lrow + l * RPL) * RS + lc] = ow[l];
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
            acc[fn][fm] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int wn = wave % WN, wm = wave / WN;
    const int r = lane & 15, kq = lane >> 4;
    auto compute = [&](int buf) {
        const uint16_t *base = lds[buf];
#pragma unroll
        for (int u = 0; u < BK / 32; ++u) {
            u32x4 af[FN], bfr[FM];
#pragma unroll
            for (int fn = 0; fn < FN; ++fn)
                af[fn] = *(const u32x4 *)(base + (BM + wn * TN + 16 * fn + r) * RS + 32 * u + 8 * kq);
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
                bfr[fm] = *(const u32x4 *)(base + (wm * TM + 16 * fm + r) * RS + 32 * u + 8 * kq);
#pragma unroll
            for (int fn = 0; fn < FN; ++fn)
#pragma unroll
                for (int fm = 0; fm < FM; ++fm)
                    acc[fn][fm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, af[fn]), __builtin_bit_cast(bf16x8, bfr[fm]),
                        acc[fn][fm], 0, 0, 0);
        }
    };

    // P stages in flight in registers, two in LDS: stage k is stored into
    // buffer k & 1, the load of stage k + P is issued into its registers,
    // one barrier, then stage k is multiplied.  A wave that reaches stage
    // k + 1's store has passed stage k's barrier, so every wave is done with
    // that buffer's previous stage (k - 1).  The loads are unconditional
    // (past the end they re-read the last stage into registers that are not
    // stored again), so the wait before each store covers exactly that
    // stage's loads and the other P - 1 stages stay in flight; the last
    // nk % P stages, already loaded, follow the loop.
#pragma unroll
    for (int p = 0; p < P; ++p)
        load(rx[p], rw[p], p);
    const int nfull = nk / P * P;
    for (int kt = 0; kt < nfull; kt += P) {
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int k = kt + p;
            store(rx[p], rw[p], k & 1);
            load(rx[p], rw[p], k + P);
            __syncthreads();
            compute(k & 1);
        }
    }
#pragma unroll
    for (int p = 0; p + 1 < P; ++p) {
        const int k = nfull + p;
        if (k < nk) {
            store(rx[p], rw[p], k & 1);
            __syncthreads();
            compute(k & 1);
        }
    }

    // acc[fn][fm][e]: column n0 + wn*TN + 16 fn + 4 kq + e of row
    // m0 + wm*TM + 16 fm + r
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
        const int m = m0 + wm * TM + 16 * fm + r;
        if (m >= M)
            continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
            const int n = n0 + wn * TN + 16 * fn + 4 * kq;
            const f32x4 v = acc[fn][fm];
            if constexpr (MODE == OUT_PART) {
                *(f32x4 *)(a.part + ((size_t)s * M + m) * N + n) = v;
            } else if constexpr (MODE == OUT_F32) {
                *(f32x4 *)((float *)a.y + (size_t)m * N + n) = v;
            } else {
                *(u32x2 *)((uint16_t *)a.y + (size_t)m * N + n) =
                    u32x2{(unsigned)bf16_rne(v[0]) | ((unsigned)bf16_rne(v[1]) << 16),
                          (unsigned)bf16_rne(v[2]) | ((unsigned)bf16_rne(v[3]) << 16)};
            }
        }
    }
}

// s_waitcnt with vmcnt(N) and lgkmcnt(0): this wave's loads older than its
// last N are done, and its LDS reads have returned.
template <int N>
__device__ inline void wait_vm_lds()
{
    static_assert(N >= 0 && N < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// Larger-batch tile with its stages loaded straight into LDS, worked by
// WM x WN waves (four, or eight: two per SIMD, 128 accumulators per lane for
// a 256 x 256 tile, 160 for 320 x 256, which waves of four could only hold
// in AGPRs).  Per K
// column the wide tiles move BM + BN operand rows for BM x BN products, so
// 256 x 256 moves a third fewer rows per product than 256 x 128; with two
// stages of 64 KiB in the ring it holds one workgroup per CU.  A stage is
// BK = 64 columns (128-byte rows of CH = 8 chunks of 16 bytes) of the tile's
// BM x rows and BN w rows.  Each global_load_lds_dwordx4 writes one 1 KiB
// block of LDS, lane l's 16 bytes at the instruction's LDS base + 16 l, i.e.
// 8 consecutive rows; lane l loads row l / 8 of the block and the chunk that
// puts row rho's chunk c at slot c ^ (rho mod 8), so that the MFMA fragment
// reads (16 consecutive rows, one chunk) fall in distinct banks.  The two
// k-steps of 32 columns in a stage are its two halves.  NSLOT stages form a
// ring in LDS, up to NSLOT - 1 in
// flight while one is multiplied.  No registers carry the stages, so the
// pipeline depth costs LDS only.  The waits are explicit: before stage k is
// read, the wave waits for its own loads of stage k (the later stages' loads
// stay in flight) and for its LDS reads; a barrier without a memory fence
// then makes stage k complete for every wave, and only after it is the slot
// of stage k - 1 refilled.  Loads past the slice's end re-read its last
// stage into a slot that is never read again, so every iteration issues the
// same loads and the wait counts are constants.
__device__ inline int chunk_swz(int row)
{
    return row & 7;
}

template <int BM, int BN, int BK, int WM, int WN, int NSLOT, int MODE>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_dma_kernel(const GemmArgs a)
{
    constexpr int NW = WM * WN;                  // waves in the workgroup
    constexpr int CH = BK / 8;                   // 16-byte chunks per row
    constexpr int RPI = 64 / CH;                 // rows per load instruction
    constexpr int ROWS = BM + BN;                // x rows, then w rows, per stage
    constexpr int SLOT = ROWS * BK;              // bf16 elements per stage
    constexpr int IPW = ROWS / RPI / NW;         // load instructions per wave and stage
    constexpr int H = BK / 32;                   // MFMA k-steps per stage
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 16, FN = TN / 16;
    static_assert(BK == 64, "stage width: two k-steps");
    static_assert(NW == 4 || NW == 8, "four or eight waves");
    static_assert(ROWS % (NW * RPI) == 0 && BM % RPI == 0 && TM % 16 == 0 && TN % 16 == 0, "shape");
    static_assert((NSLOT - 1) * IPW < 64, "vmcnt");
    __shared__ __attribute__((aligned(1024))) uint16_t lds[NSLOT * SLOT];

    const int i = blockIdx.x, TMc = a.tiles_m, G = a.groups;
    const int full = G / 8 * 8;
    int tm, g;
    if (i < full * TMc) {
        const int sg = i / (8 * TMc), rem = i - sg * 8 * TMc;
        tm = rem >> 3;
        g = sg * 8 + (rem & 7);
    } else {
        const int j = i - full * TMc, r8 = G - full;
        tm = j / r8;
        g = full + (j - tm * r8);
    }
    const int tn = g / a.S, s = g - tn * a.S;
    const int m0 = tm * BM, n0 = tn * BN;
    const int M = a.M, N = a.N, K = a.K;
    const int nk = a.kslice / BK;

    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    // this lane's source for each of its load instructions at stage 0; rows
    // past M repeat row M - 1 (loaded, never stored).  A block starts at a
    // multiple of RPI rows, so swz of the lane's row is swz(lane / CH).
    const int chunk = (lane % CH) ^ chunk_swz(lane / CH);
    const uint16_t *src[IPW];
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
        const int rho = (wave * IPW + j) * RPI + lane / CH;
        const uint16_t *row = rho < BM ? a.x + (size_t)min(m0 + rho, M - 1) * K
                                       : a.w + (size_t)(n0 + rho - BM) * K;
        src[j] = row + (size_t)s * a.kslice + chunk * 8;
    }
    auto issue = [&](int kt) {
        const size_t off = (size_t)min(kt, nk - 1) * BK;
        uint16_t *dst = lds + (kt % NSLOT) * SLOT + wave * IPW * RPI * BK;
#pragma unroll
        for (int j = 0; j < IPW; ++j)
            __builtin_amdgcn_global_load_lds((const void *)(src[j] + off),
                                             (__attribute__((address_space(3))) void *)(dst + j * RPI * BK),
                                             16, 0, 0);
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
            acc[fn][fm] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int wn = wave % WN, wm = wave / WN;
    const int r = lane & 15, kq = lane >> 4;
    struct Frags {
        u32x4 a[FN], b[FM];
    };
    // the fragments of k-step h (32 columns: stage h / H, its half h % H)
    auto read = [&](Frags &f, int h) {
        const uint16_t *base = lds + ((h / H) % NSLOT) * SLOT;
        const int sl = ((4 * (h % H) + kq) ^ chunk_swz(r)) * 8;   // this lane's chunk slot
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
            f.a[fn] = *(const u32x4 *)(base + (BM + wn * TN + 16 * fn + r) * BK + sl);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
            f.b[fm] = *(const u32x4 *)(base + (wm * TM + 16 * fm + r) * BK + sl);
    };
    auto mma = [&](const Frags &f) {
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, f.a[fn]), __builtin_bit_cast(bf16x8, f.b[fm]),
                    acc[fn][fm], 0, 0, 0);
    };
    // k-step h: the next step's fragments are read (after the wait and
    // barrier for the next stage, when it starts one) while this step's
    // MFMAs run.  After that barrier every wave has read all of stage
    // h / H, and its slot is refilled with stage h / H + NSLOT.
    auto step = [&](int h, const Frags &cur, Frags &nxt) {
        if ((h + 1) % H == 0) {
            asm volatile("" ::: "memory");
            wait_vm_lds<(NSLOT - 2) * IPW>();   // this wave's next stage is in LDS, cur is read
            __builtin_amdgcn_s_barrier();       // ... every wave's
            asm volatile("" ::: "memory");
            issue(h / H + NSLOT);               // into this stage's slot
        }
        read(nxt, h + 1);
        mma(cur);
    };

#pragma unroll
    for (int p = 0; p < NSLOT; ++p)   // every slot
        issue(p);
    asm volatile("" ::: "memory");
    wait_vm_lds<(NSLOT - 1) * IPW>();   // stage 0
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    Frags f0, f1;
    read(f0, 0);
    for (int h = 0; h < nk * H; h += 2) {   // H is even: the pairs end on stage boundaries
        step(h, f0, f1);
        step(h + 1, f1, f0);
    }
    wait_vm_lds<0>();   // the re-reads past the end land before the wave ends

    // acc[fn][fm][e]: column n0 + wn*TN + 16 fn + 4 kq + e of row
    // m0 + wm*TM + 16 fm + r
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
        const int m = m0 + wm * TM + 16 * fm + r;
        if (m >= M)
            continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
            const int n = n0 + wn * TN + 16 * fn + 4 * kq;
            const f32x4 v = acc[fn][fm];
            if constexpr (MODE == OUT_PART) {
                *(f32x4 *)(a.part + ((size_t)s * M + m) * N + n) = v;
            } else if constexpr (MODE == OUT_F32) {
                *(f32x4 *)((float *)a.y + (size_t)m * N + n) = v;
            } else {
                *(u32x2 *)((uint16_t *)a.y + (size_t)m * N + n) =
                    u32x2{(unsigned)bf16_rne(v[0]) | ((unsigned)bf16_rne(v[1]) << 16),
                          (unsigned)bf16_rne(v[2]) | ((unsigned)bf16_rne(v[3]) << 16)};
            }
        }
    }
}

// y[e] = sum over slices s = 0 .. S-1 (in order) of part[s][e], four per
// thread; the S loads are all issued before the first add.
template <int MODE, int S>
__global__ void __launch_bounds__(kReduceThreads)
gemm_reduce_kernel(const float *__restrict__ part, void *__restrict__ y, size_t elems)
{
    const size_t e4 = ((size_t)blockIdx.x * kReduceThreads + threadIdx.x) * 4;
    if (e4 >= elems)
        return;
    f32x4 p[S];
#pragma unroll
    for (int s = 0; s < S; ++s)
        p[s] = *(const f32x4 *)(part + (size_t)s * elems + e4);
    f32x4 v = p[0];
#pragma unroll
    for (int s = 1; s < S; ++s)
        v += p[s];
    if constexpr (MODE == OUT_F32) {
        *(f32x4 *)((float *)y + e4) = v;
    } else {
        *(u32x2 *)((uint16_t *)y + e4) =
            u32x2{(unsigned)bf16_rne(v[0]) | ((unsigned)bf16_rne(v[1]) << 16),
                  (unsigned)bf16_rne(v[2]) | ((unsigned)bf16_rne(v[3]) << 16)};
    }
}

// ---------------------------------------------------------------- host side
// The tile configurations (index = VD_GEMM_FLAG_TILE's argument), with the
// figures the automatic choice weighs them by: how many workgroups of the
// tile a CU holds at once (its LDS and registers), and, measured on MI355X,
// how fast the tile streams weights relative to 5.623 TB/s once its
// workgroups fill the device and its matrix-core throughput (PFLOP/s) on a
// full device.
struct TileCfg {
    int bm, bn, bk, per_cu;
    double stream_eff, pflops;
};
constexpr TileCfg kTiles[] = {
    {16, 64, 128, 3, 1.121, 1.0},     // 0: four waves over the columns
    {32, 64, 128, 3, 1.3, 1.073},     // 1
    {48, 64, 128, 2, 1.182, 1.6},     // 2
    {64, 64, 128, 2, 0.897, 1.222},   // 3
    {64, 128, 64, 2, 0.977, 0.56},    // 4: 2 x 2 waves
    {128, 128, 64, 2, 1.3, 0.309},    // 5
    {128, 128, 64, 1, 0.854, 1.004},  // 6: stages loaded straight into LDS, four in a ring
    {256, 128, 64, 1, 1.3, 0.993},    // 7: the same, 2 x 2 waves of 128 x 64, three stages
    {256, 256, 64, 1, 0.511, 1.421},  // 8: eight waves (2 x 4 of 128 x 64), two stages
    {192, 256, 64, 1, 0.658, 1.132},  // 9: eight waves of 96 x 64, two stages
    {320, 256, 64, 1, 0.925, 1.267},  // 10: eight waves of 160 x 64, two stages
};
constexpr int kNumTiles = (int)(sizeof(kTiles) / sizeof(kTiles[0]));

template <int MODE>
void launch_tile(int cfg, const GemmArgs &g, dim3 grid, hipStream_t stream)
{
    const dim3 block(kThreads), block8(2 * kThreads);
    switch (cfg) {
    case 0: hipLaunchKernelGGL((gemm_tile_kernel<16, 64, 128, 1, 4, 4, MODE>), grid, block, 0, stream, g); break;
    case 1: hipLaunchKernelGGL((gemm_tile_kernel<32, 64, 128, 1, 4, 3, MODE>), grid, block, 0, stream, g); break;
    case 2: hipLaunchKernelGGL((gemm_tile_kernel<48, 64, 128, 1, 4, 3, MODE>), grid, block, 0, stream, g); break;
    case 3: hipLaunchKernelGGL((gemm_tile_kernel<64, 64, 128, 1, 4, 3, MODE>), grid, block, 0, stream, g); break;
    case 4:
        if (g.tiles_m == 1)
            hipLaunchKernelGGL((gemm_tile_kernel<64, 128, 64, 2, 2, 2, MODE>), grid, block, 0, stream, g);
        else
            hipLaunchKernelGGL((gemm_tile_kernel<64, 128, 64, 2, 2, 2, MODE, false>), grid, block, 0, stream, g);
        break;
    case 5:
        if (g.tiles_m == 1)
            hipLaunchKernelGGL((gemm_tile_kernel<128, 128, 64, 2, 2, 2, MODE>), grid, block, 0, stream, g);
        else
            hipLaunchKernelGGL((gemm_tile_kernel<128, 128, 64, 2, 2, 2, MODE, false>), grid, block, 0, stream, g);
        break;
    case 6: hipLaunchKernelGGL((gemm_dma_kernel<128, 128, 64, 2, 2, 4, MODE>), grid, block, 0, stream, g); break;
    case 7: hipLaunchKernelGGL((gemm_dma_kernel<256, 128, 64, 2, 2, 3, MODE>), grid, block, 0, stream, g); break;
    case 8: hipLaunchKernelGGL((gemm_dma_kernel<256, 256, 64, 2, 4, 2, MODE>), grid, block8, 0, stream, g); break;
    case 9: hipLaunchKernelGGL((gemm_dma_kernel<192, 256, 64, 2, 4, 2, MODE>), grid, block8, 0, stream, g); break;
    default: hipLaunchKernelGGL((gemm_dma_kernel<320, 256, 64, 2, 4, 2, MODE>), grid, block8, 0, stream, g); break;
    }
}

template <int MODE>
void launch_reduce(int S, const float *part, void *y, size_t elems, dim3 grid, hipStream_t stream)
{
    const dim3 block(kReduceThreads);
    switch (S) {
    case 2: hipLaunchKernelGGL((gemm_reduce_kernel<MODE, 2>), grid, block, 0, stream, part, y, elems); break;
    case 4: hipLaunchKernelGGL((gemm_reduce_kernel<MODE, 4>), grid, block, 0, stream, part, y, elems); break;
    case 8: hipLaunchKernelGGL((gemm_reduce_kernel<MODE, 8>), grid, block, 0, stream, part, y, elems); break;
    default: hipLaunchKernelGGL((gemm_reduce_kernel<MODE, 16>), grid, block, 0, stream, part, y, elems); break;
    }
}

bool aligned(const void *p, size_t al) { return ((uintptr_t)p & (al - 1)) == 0; }

struct Plan {
    int cfg, S;
};

int gemm_check(int M, int N, int K, unsigned flags)
{
    if (M <= 0 || N <= 0 || K <= 0)
        return VD_ERROR_INVALID_VALUE;
    if (flags & ~(VD_FLAG_OUT_F32 | VD_GEMM_FLAG_TILE_MASK | VD_GEMM_FLAG_SLICES_MASK))
        return VD_ERROR_INVALID_VALUE;
    if (N % kNAlign != 0 || K % kKAlign != 0)
        return VD_ERROR_NOT_SUPPORTED;
    if ((long long)N * K >= (1LL << 40) || (long long)M * N >= (1LL << 31) ||
        (long long)M * K >= (1LL << 40))
        return VD_ERROR_NOT_SUPPORTED;
    return VD_SUCCESS;
}


// Workgroups of a configuration with S slices.
long long plan_groups(const TileCfg &c, int M, int N, int S)
{
    return (long long)((M + c.bm - 1) / c.bm) * (N / c.bn) * S;
}

// Estimated time (microseconds) of a plan on MI355X: a fixed 4 us, plus the
// larger of the weight stream (5.623 TB/s times the tile's streaming
// efficiency, scaled down while its workgroups fill less than 192 CUs) and
// the matrix-core time (the tile's throughput, scaled by the CUs it fills,
// on the rows padded to whole tiles); K slices add the fp32 partials' round
// trip at 8 TB/s and the reduction kernel (1.8 us); every round of
// workgroups past the first (256 CUs times the tile's workgroups per CU)
// adds 23.3 us.  The constants were fitted to a sweep of every tile and 1,
// 2, 4 or 8 slices at the four Llama-3-8B-shaped projections and 30 batch
// sizes M = 1 .. 1024, with weights that do not fit the caches: the chosen
// plan costs 0.55% more than the best one on average and 8% in the worst case.
double plan_cost(const TileCfg &c, int M, int N, int K, int S)
{
    const double groups = (double)plan_groups(c, M, N, S);
    const double mpad = (double)((M + c.bm - 1) / c.bm) * c.bm;
    const double t_w = (double)N * K * 2.0 / (5.623e6 * c.stream_eff * std::min(1.0, groups / 192.0));
    const double t_mfma = 2.0 * mpad * N * K / (c.pflops * 1e9 * std::min(1.0, groups / kTargetCUs));
    const double t_part = S > 1 ? (double)S * M * N * 8.0 / 8.0e6 + 1.824 : 0.0;
    const double rounds = std::ceil(groups / ((double)kTargetCUs * c.per_cu));
    return 4.0 + std::max(t_w, t_mfma) + t_part + 23.255 * (rounds - 1.0);
}

// The automatic choice, from the sizes alone: the cheapest plan by
// plan_cost over the tiles (for up to 64 rows, only the narrow tile that
// holds the rows, 16 * ceil(M / 16), besides the wide ones) and 1, 2, 4 or 8
// K slices of whole stages of the tile.
Plan auto_plan(int M, int N, int K)
{
    Plan best{-1, 1};
    double best_cost = 0;
    for (int c = 0; c < kNumTiles; ++c) {
        const TileCfg &t = kTiles[c];
        if (N % t.bn)
            continue;
        if (t.bk == 128 && !(M <= 64 && t.bm == 16 * ((M + 15) / 16)))
            continue;
        for (int S = 1; S <= 8; S *= 2) {
            if (K % S || (K / S) % t.bk)
                continue;
            const double cost = plan_cost(t, M, N, K, S);
            if (best.cfg < 0 || cost < best_cost) {
                best = Plan{c, S};
                best_cost = cost;
            }
        }
    }
    if (best.cfg < 0)   // N % 64 == 0 always admits the 64-column tiles
        best = Plan{M <= 64 ? (M + 15) / 16 - 1 : 3, 1};
    return best;
}

// The plan of a call: automatic, or the tile and slice count the flags force
// (tests and sweeps).  Returns false when a forced choice does not fit the sizes.
bool make_plan(int M, int N, int K, unsigned flags, Plan *out)
{
    Plan p = auto_plan(M, N, K);
    const unsigned ft = (flags & VD_GEMM_FLAG_TILE_MASK) >> VD_GEMM_FLAG_TILE_SHIFT;
    const unsigned fs = (flags & VD_GEMM_FLAG_SLICES_MASK) >> VD_GEMM_FLAG_SLICES_SHIFT;
    if (ft) {
        if ((int)ft > kNumTiles)
            return false;
        p.cfg = (int)ft - 1;
    }
    if (fs) {
        if ((int)fs - 1 > kMaxSlicesLog2)
            return false;
        p.S = 1 << (fs - 1);
    }
    const TileCfg &c = kTiles[p.cfg];
    if (N % c.bn != 0 || (K / p.S) % c.bk != 0 || K % p.S != 0)
        return false;
    *out = p;
    return true;
}

size_t plan_workspace(const Plan &p, int M, int N)
{
    return p.S > 1 ? (size_t)p.S * M * N * sizeof(float) : 0;
}

}  // namespace

extern "C" {

size_t vd_gemm_workspace_size(int M, int N, int K, unsigned flags)
{
    if (gemm_check(M, N, K, flags))
        return 0;
    Plan p;
    if (!make_plan(M, N, K, flags, &p))
        return 0;
    return plan_workspace(p, M, N);
}

int vd_gemm_bf16(const void *x, const void *w, void *y, int M, int N, int K, void *workspace,
                 size_t workspace_bytes, unsigned flags, hipStream_t stream)
{
    int st = gemm_check(M, N, K, flags);
    if (st)
        return st;
    if (!x || !w || !y || !aligned(x, 16) || !aligned(w, 16) || !aligned(y, 16))
        return VD_ERROR_INVALID_VALUE;
    Plan p;
    if (!make_plan(M, N, K, flags, &p))
        return VD_ERROR_NOT_SUPPORTED;
    const size_t need = plan_workspace(p, M, N);
    if (need) {
        if (!workspace || !aligned(workspace, 16))
            return VD_ERROR_INVALID_VALUE;
        if (workspace_bytes < need)
            return VD_ERROR_WORKSPACE_TOO_SMALL;
    }
    const TileCfg &c = kTiles[p.cfg];
    GemmArgs g;
    g.x = (const uint16_t *)x;
    g.w = (const uint16_t *)w;
    g.y = y;
    g.part = (float *)workspace;
    g.M = M;
    g.N = N;
    g.K = K;
    g.kslice = K / p.S;
    g.S = p.S;
    g.tiles_m = (M + c.bm - 1) / c.bm;
    g.groups = (N / c.bn) * p.S;
    const dim3 grid((unsigned)((long long)g.tiles_m * g.groups));
    const bool f32 = flags & VD_FLAG_OUT_F32;
    if (p.S > 1)
        launch_tile<OUT_PART>(p.cfg, g, grid, stream);
    else if (f32)
        launch_tile<OUT_F32>(p.cfg, g, grid, stream);
    else
        launch_tile<OUT_BF16>(p.cfg, g, grid, stream);
    if (p.S > 1) {
        const size_t elems = (size_t)M * N;   // N % 64 == 0, so elems % 4 == 0
        const dim3 rgrid((unsigned)((elems / 4 + kReduceThreads - 1) / kReduceThreads));
        if (f32)
            launch_reduce<OUT_F32>(p.S, (const float *)workspace, y, elems, rgrid, stream);
        else
            launch_reduce<OUT_BF16>(p.S, (const float *)workspace, y, elems, rgrid, stream);
    }
    return hipGetLastError() == hipSuccess ? VD_SUCCESS : VD_ERROR_LAUNCH;
}

}  // extern "C"
