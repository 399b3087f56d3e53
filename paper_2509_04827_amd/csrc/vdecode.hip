// libvdecode -- paged GQA decode attention for MI355X (gfx950, CDNA4).
//
// One decode step attends each request's newest query token to every token of
// its paged KV cache: the attention part of the decode iteration whose latency
// the paper models as growing with N_kv (Sec. 5.4, Eq. pred-itl), over a paged
// cache (Sec. 2.1).  The step is read-bound: every cached K and V byte is read
// once, so the kernels below are built around HBM traffic, not arithmetic.
//
// Three kernels on the caller's stream:
//   plan_kernel     one workgroup: per-request page counts, a split size that
//                   gives enough work items to fill all CUs, the split list
//                   and per-request split offsets (exclusive scans).
//   attn_kernel     persistent waves pull work items (request, KV head, page
//                   range) from a queue.  Per 16-token page:
//                     K rows are loaded straight into MFMA A operands (lane =
//                     token row), scores = K Q^T with v_mfma_f32_16x16x32_bf16
//                     against the group's G query heads (zero-padded to 16
//                     columns);
//                     online softmax in fp32 (exp2 domain, lazy rescaling);
//                     V rows are loaded coalesced (4 rows x 256 B per
//                     instruction) and transposed in registers with byte
//                     permutes into the A operand of
//                     v_mfma_f32_16x16x16_bf16, whose B operand is P exactly
//                     as the score MFMA left it (P split into bf16 hi + lo).
//                   Single-chunk requests write the output; the others write
//                   (max, normaliser, accumulator) partials.
//   combine_kernel  log-sum-exp merge of the partials per (request, q head).
//
// All arithmetic is fp32; bf16 is only the storage type of Q/K/V, the MFMA
// operand type, and the optional output type.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <stdint.h>

#include "vdecode.h"

namespace {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kMaxSplitPages = 64;     // one page-table window per wave
constexpr int kMaxSeqs = 8192;         // planner keeps split offsets in LDS
constexpr int kTargetItemsCap = 16384; // workspace is sized for this many items
constexpr int kItemsPerCU = 48;        // auto plan aims at this many items per CU
constexpr int kMinSplitPages = 4;
constexpr int kPlanThreads = 1024;
constexpr int kAttnThreads = 256;      // 4 independent waves per workgroup
constexpr int kAttnWGPerCU = 8;
constexpr int kCombineThreads = 64;
constexpr float kLog2e = 1.4426950408889634f;
// Lazy rescaling: the running max is only raised when a new score exceeds it
// by more than this (log2 units), so weights stay below 2^8 and acc/l never
// overflow, while most pages skip the accumulator rescale.
constexpr float kRescaleSlack = 8.0f;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

struct PlanHeader {
    int n_items;   // splits * n_kv_heads
    int n_splits;
    int split_pages;
    int queue;     // work-queue head
    int done;      // waves of the current attention launch that have finished
    int pad[3];
};
// The attention kernel leaves queue and done at 0 when its last wave exits,
// so one plan serves any number of attention launches.

// ---------------------------------------------------------------- workspace
struct WsLayout {
    size_t hdr, split_base, tok_base, splits, part_ml, part_acc, total;
    long long cap_splits;
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline long long ceil_div_ll(long long a, long long b) { return (a + b - 1) / b; }

// Capacity for the split list: automatic plans have at most
// max(targetcap / Hkv, B*maxp / 64) + B splits; a forced split size c at most
// B*maxp / c + B; never more than one per page.
inline WsLayout ws_layout(int B, int G, int Hkv, int maxp, int forced)
{
    const long long pages = (long long)B * maxp;
    long long cap;
    if (forced > 0)
        cap = ceil_div_ll(pages, forced) + B;
    else
        cap = std::max(ceil_div_ll(kTargetItemsCap, Hkv), ceil_div_ll(pages, kMaxSplitPages)) + B;
    cap = std::min(cap, pages);
    cap = std::max(cap, 1LL);
    const long long items = cap * Hkv;
    WsLayout l;
    size_t o = 0;
    l.hdr = o;        o = align_up(o + sizeof(PlanHeader), 256);
    l.split_base = o; o = align_up(o + sizeof(int) * (size_t)(B + 1), 256);
    l.tok_base = o;   o = align_up(o + sizeof(long long) * (size_t)(B + 1), 256);
    l.splits = o;     o = align_up(o + sizeof(int4) * (size_t)cap, 256);
    l.part_ml = o;    o = align_up(o + sizeof(float2) * (size_t)items * G, 256);
    l.part_acc = o;   o = align_up(o + sizeof(float) * (size_t)items * G * kHeadDim, 256);
    l.total = o;
    l.cap_splits = cap;
    return l;
}

// ---------------------------------------------------------------- planner
template <typename T>
__device__ T block_exclusive_scan(T v, T *sh, T &total)
{
    // Hillis-Steele inclusive scan over kPlanThreads values in LDS.
    const int t = threadIdx.x;
    sh[t] = v;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        T add = t >= off ? sh[t - off] : T(0);
        __syncthreads();
        sh[t] += add;
        __syncthreads();
    }
    const T incl = sh[t];
    total = sh[kPlanThreads - 1];
    __syncthreads();
    return incl - v;
}

__device__ inline int clamped_len(const int32_t *seq_lens, int b, int maxp)
{
    const int L = seq_lens[b];
    return L <= 0 ? 0 : min(L, maxp * kPage);
}

__global__ void __launch_bounds__(kPlanThreads)
plan_kernel(const int32_t *__restrict__ seq_lens, int B, int Hkv, int maxp, int forced,
            int target_items, char *__restrict__ ws, WsLayout lay)
{
    __shared__ int s_base[kMaxSeqs + 1];
    __shared__ long long s_scan[kPlanThreads];
    __shared__ int s_chunk;
    const int t = threadIdx.x;

    // total pages
    long long mine = 0;
    for (int b = t; b < B; b += kPlanThreads)
        mine += (clamped_len(seq_lens, b, maxp) + kPage - 1) / kPage;
    long long total_pages;
    block_exclusive_scan<long long>(mine, s_scan, total_pages);

    if (t == 0) {
        int c;
        if (forced > 0) {
            c = forced;
        } else {
            long long want = (total_pages * Hkv + target_items - 1) / target_items;
            c = (int)std::min<long long>(std::max<long long>(want, kMinSplitPages), kMaxSplitPages);
        }
        s_chunk = c;
    }
    __syncthreads();
    const int chunk = s_chunk;

    // per-request split offsets and token offsets
    int32_t *split_base = (int32_t *)(ws + lay.split_base);
    long long *tok_base = (long long *)(ws + lay.tok_base);
    int carry = 0;
    long long tcarry = 0;
    for (int b0 = 0; b0 < B; b0 += kPlanThreads) {
        const int b = b0 + t;
        const int L = b < B ? clamped_len(seq_lens, b, maxp) : 0;
        const int P = (L + kPage - 1) / kPage;
        const int ns = (P + chunk - 1) / chunk;
        long long tot_s, tot_t;
        const long long ex_s = block_exclusive_scan<long long>(ns, s_scan, tot_s);
        const long long ex_t = block_exclusive_scan<long long>(L, s_scan, tot_t);
        if (b < B) {
            s_base[b] = carry + (int)ex_s;
            split_base[b] = carry + (int)ex_s;
            tok_base[b] = tcarry + ex_t;
        }
        carry += (int)tot_s;
        tcarry += tot_t;
    }
    if (t == 0) {
        s_base[B] = carry;
        split_base[B] = carry;
        tok_base[B] = tcarry;
        PlanHeader *h = (PlanHeader *)(ws + lay.hdr);
        h->n_splits = carry;
        h->n_items = carry * Hkv;
        h->split_pages = chunk;
        h->queue = 0;
        h->done = 0;
    }
    __syncthreads();

    // split records {b, first page, end page, split index}
    int4 *splits = (int4 *)(ws + lay.splits);
    const int n_splits = s_base[B];
    for (int i = t; i < n_splits; i += kPlanThreads) {
        int lo = 0, hi = B;   // largest b with s_base[b] <= i
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (s_base[mid] <= i) lo = mid; else hi = mid;
        }
        const int b = lo;
        const int s = i - s_base[b];
        const int P = (clamped_len(seq_lens, b, maxp) + kPage - 1) / kPage;
        const int pb = s * chunk;
        splits[i] = make_int4(b, pb, min(pb + chunk, P), s);
    }
}

// ---------------------------------------------------------------- attention
struct AttnArgs {
    const uint16_t *q, *k, *v;
    const int32_t *pt, *seq_lens;
    void *out, *out2;               // attention: out; gather: k_out, v_out
    int *queue, *done;
    const PlanHeader *hdr;
    const int32_t *split_base;
    const int4 *splits;
    const long long *tok_base;
    float2 *part_ml;
    float *part_acc;
    int Hq, Hkv, pt_stride, maxp;
    float scale_log2;
};

enum { MODE_BF16 = 0, MODE_F32 = 1, MODE_GATHER = 2 };

struct Tile {
    u32x4 k[4];   // K[token r][d 8(4kk+grp) .. +8]          (score MFMA A operand)
    u32x4 v[4];   // V[token 4grp+j][d 8r .. 8r+8], j = 0..3  (raw rows)
};

__device__ inline u32x4 ldg16(const uint16_t *p) { return *(const u32x4 *)p; }

__device__ inline void load_tile(Tile &T, const uint16_t *kpage, const uint16_t *vpage,
                                 unsigned koff, unsigned voff, unsigned row)
{
    const uint16_t *kp = kpage + koff;
    const uint16_t *vp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        vp[j] = vpage + voff + j * row;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
        T.k[kk] = ldg16(kp + 32 * kk);
#pragma unroll
    for (int j = 0; j < 4; ++j)
        T.v[j] = ldg16(vp[j]);
}

__device__ inline float wave_max_groups(float x)
{
    // max over the 4 lane groups that share lane & 15
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    return x;
}

__device__ inline float sum_groups(float x)
{
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

__device__ inline unsigned short bf16_bits(float f)
{
    return __builtin_bit_cast(unsigned short, (__bf16)f);
}

__device__ inline float bf16_val(unsigned short h)
{
    return __builtin_bit_cast(float, (unsigned)h << 16);
}

// V^T operand of d-block `blk`: slots j = 0..3 hold V[token 4grp+j][d 8r+blk].
__device__ inline s16x4 v_operand(const Tile &T, int blk)
{
    const int w = blk >> 1;
    unsigned a, b;
    if ((blk & 1) == 0) {
        a = (T.v[0][w] & 0xFFFFu) | (T.v[1][w] << 16);
        b = (T.v[2][w] & 0xFFFFu) | (T.v[3][w] << 16);
    } else {
        a = (T.v[0][w] >> 16) | (T.v[1][w] & 0xFFFF0000u);
        b = (T.v[2][w] >> 16) | (T.v[3][w] & 0xFFFF0000u);
    }
    return __builtin_bit_cast(s16x4, u32x2{a, b});
}

template <int G, int MODE>
__global__ void __launch_bounds__(kAttnThreads)
attn_kernel(const AttnArgs a)
{
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;    // score MFMA: token row (A) / head column (B, D)
    const int grp = lane >> 4;  // lane group: k-slice of the operands, row block of D
    const int Hkv = a.Hkv;
    const unsigned row = (unsigned)Hkv * kHeadDim;        // elements per token row
    const size_t page_elems = (size_t)kPage * row;
    const int n_items = a.hdr->n_items;

    int item = 0;
    if (lane == 0)
        item = atomicAdd(a.queue, 1);
    item = __builtin_amdgcn_readfirstlane(item);

    while (item < n_items) {
        int next = 0;
        if (lane == 0)
            next = atomicAdd(a.queue, 1);

        const int split = item / Hkv;
        const int g = item - split * Hkv;
        const int4 rec = a.splits[split];
        const int b = rec.x, pb = rec.y, pe = rec.z;
        const int L = min(a.seq_lens[b], a.maxp * kPage);
        const int nsplit = a.split_base[b + 1] - a.split_base[b];
        const int np = pe - pb;

        // page ids of this item: lane l holds page_table[b][pb + l]
        int ptw = 0;
        if (lane < np)
            ptw = a.pt[(size_t)b * a.pt_stride + pb + lane];

        const unsigned koff = r * row + g * kHeadDim + 8 * grp;
        const unsigned voff = 4 * grp * row + g * kHeadDim + 8 * r;

        if constexpr (MODE == MODE_GATHER) {
            uint16_t *ko = (uint16_t *)a.out;
            uint16_t *vo = (uint16_t *)a.out2;
            const long long t0 = a.tok_base[b];
            for (int j = pb; j < pe; ++j) {
                const int pg = __builtin_amdgcn_readlane(ptw, j - pb);
                Tile T;
                load_tile(T, a.k + (size_t)pg * page_elems, a.v + (size_t)pg * page_elems,
                          koff, voff, row);
                const int valid = L - j * kPage;
                // K: the score operand as loaded, lane row r
                if (r < valid) {
                    uint16_t *dst = ko + (size_t)(t0 + j * kPage + r) * row + g * kHeadDim + 8 * grp;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk)
                        *(u32x4 *)(dst + 32 * kk) = T.k[kk];
                }
                // V: rebuild each token row chunk from the transposed operands
                s16x4 op[8];
#pragma unroll
                for (int blk = 0; blk < 8; ++blk)
                    op[blk] = v_operand(T, blk);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    if (4 * grp + jj < valid) {
                        u32x4 w;
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            w[e] = (unsigned)(unsigned short)op[2 * e][jj] |
                                   ((unsigned)(unsigned short)op[2 * e + 1][jj] << 16);
                        *(u32x4 *)(vo + (size_t)(t0 + j * kPage + 4 * grp + jj) * row +
                                   g * kHeadDim + 8 * r) = w;
                    }
                }
            }
        } else {
            // Q operand (B of the score MFMA): head column r, d slice 8(4kk+grp)
            u32x4 qreg[4];
            const uint16_t *qrow = a.q + ((size_t)b * a.Hq + g * G + r) * kHeadDim + 8 * grp;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                qreg[kk] = (r < G) ? ldg16(qrow + 32 * kk) : u32x4{0u, 0u, 0u, 0u};

            f32x4 acc[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            float m_run = -INFINITY;   // running max (log2 units) of head r
            float l_run = 0.f;         // this lane's share of the normaliser

            auto page_step = [&](const Tile &T, int j) {
                f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, T.k[kk]), __builtin_bit_cast(bf16x8, qreg[kk]),
                        s, 0, 0, 0);
                // s[i]: token 4grp+i, head r
                float sc[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    sc[i] = s[i] * a.scale_log2;
                Tile V = T;
                const int valid = L - j * kPage;
                if (valid < kPage) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (4 * grp + i >= valid) {
                            sc[i] = -INFINITY;
                            V.v[i] = u32x4{0u, 0u, 0u, 0u};
                        }
                    }
                }
                float tmax = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
                tmax = wave_max_groups(tmax);
                const bool need = tmax > m_run + kRescaleSlack;
                if (__builtin_amdgcn_ballot_w64(need)) {
                    const float m_new = need ? tmax : m_run;
                    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                    l_run *= alpha;
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        acc[i] *= alpha;
                    m_run = m_new;
                }
                s16x4 phi, plo;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p = __builtin_amdgcn_exp2f(sc[i] - m_run);
                    const unsigned short h = bf16_bits(p);
                    const float hf = bf16_val(h);
                    const unsigned short lo = bf16_bits(p - hf);
                    l_run += hf + bf16_val(lo);
                    phi[i] = (short)h;
                    plo[i] = (short)lo;
                }
#pragma unroll
                for (int blk = 0; blk < 8; ++blk) {
                    const s16x4 vop = v_operand(V, blk);
                    acc[blk] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, phi, acc[blk], 0, 0, 0);
                    acc[blk] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, plo, acc[blk], 0, 0, 0);
                }
            };

            const uint16_t *kb = a.k, *vb = a.v;
            Tile A, B;
            {
                const int pg = __builtin_amdgcn_readlane(ptw, 0);
                load_tile(A, kb + (size_t)pg * page_elems, vb + (size_t)pg * page_elems, koff, voff, row);
            }
            // Double-buffered page loop with a fixed trip count: the next page's
            // loads are issued before the current page is consumed (the
            // scheduling barriers keep the compiler from sinking them).  The
            // last prefetch of an even page count re-reads the final page,
            // which the caches serve; every path issues the same loads, so the
            // wait counts stay exact.
            auto load_page = [&](Tile &T, int jn) {
                const int pg = __builtin_amdgcn_readlane(ptw, jn - pb);
                load_tile(T, kb + (size_t)pg * page_elems, vb + (size_t)pg * page_elems, koff, voff, row);
            };
            int j = pb;
            for (int it = np >> 1; it > 0; --it) {
                load_page(B, j + 1);
                __builtin_amdgcn_sched_barrier(0);
                page_step(A, j);
                load_page(A, min(j + 2, pe - 1));
                __builtin_amdgcn_sched_barrier(0);
                page_step(B, j + 1);
                j += 2;
            }
            if (np & 1)
                page_step(A, j);

            const float l_tot = sum_groups(l_run);
            // acc[blk][i] = O[head r][d 32grp + 8i + blk]
            if (r < G) {
                const int h = g * G + r;
                if (nsplit == 1) {
                    const float inv = 1.0f / l_tot;
                    if constexpr (MODE == MODE_F32) {
                        float *o = (float *)a.out + ((size_t)b * a.Hq + h) * kHeadDim + 32 * grp;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            f32x4 w0, w1;
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                w0[e] = acc[e][i] * inv;
                                w1[e] = acc[4 + e][i] * inv;
                            }
                            *(f32x4 *)(o + 8 * i) = w0;
                            *(f32x4 *)(o + 8 * i + 4) = w1;
                        }
                    } else {
                        uint16_t *o = (uint16_t *)a.out + ((size_t)b * a.Hq + h) * kHeadDim + 32 * grp;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            u32x4 w;
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                w[e] = (unsigned)bf16_bits(acc[2 * e][i] * inv) |
                                       ((unsigned)bf16_bits(acc[2 * e + 1][i] * inv) << 16);
                            *(u32x4 *)(o + 8 * i) = w;
                        }
                    }
                } else {
                    float *o = a.part_acc + ((size_t)item * G + r) * kHeadDim + 32 * grp;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        f32x4 w0, w1;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            w0[e] = acc[e][i];
                            w1[e] = acc[4 + e][i];
                        }
                        *(f32x4 *)(o + 8 * i) = w0;
                        *(f32x4 *)(o + 8 * i + 4) = w1;
                    }
                    if (grp == 0)
                        a.part_ml[(size_t)item * G + r] = make_float2(m_run, l_tot);
                }
            }
        }
        item = __builtin_amdgcn_readfirstlane(next);
    }
    // Every wave has taken its last queue ticket; the last one out resets the
    // queue for the next launch.
    if (lane == 0) {
        const int total = (int)(gridDim.x * (kAttnThreads / 64));
        if (atomicAdd(a.done, 1) == total - 1) {
            atomicExch(a.queue, 0);
            atomicExch(a.done, 0);
        }
    }
}

// ---------------------------------------------------------------- combine
struct CombineArgs {
    void *out;
    const int32_t *split_base;
    const float2 *part_ml;
    const float *part_acc;
    int Hq, Hkv, G;
};

template <int MODE>
__global__ void __launch_bounds__(kCombineThreads)
combine_kernel(const CombineArgs a)
{
    const int bh = blockIdx.x;
    const int b = bh / a.Hq, h = bh - (bh / a.Hq) * a.Hq;
    const int g = h / a.G, hh = h - g * a.G;
    const int base = a.split_base[b];
    const int n = a.split_base[b + 1] - base;
    if (n == 1)
        return;
    const int lane = threadIdx.x;
    float o0 = 0.f, o1 = 0.f;
    if (n > 1) {
        float M = -INFINITY;
        for (int s = lane; s < n; s += 64)
            M = fmaxf(M, a.part_ml[((size_t)(base + s) * a.Hkv + g) * a.G + hh].x);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            M = fmaxf(M, __shfl_xor(M, off));
        float den = 0.f;
        int s = 0;
        for (; s + 4 <= n; s += 4) {
            float2 ml[4];
            float2 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const size_t it = ((size_t)(base + s + u) * a.Hkv + g) * a.G + hh;
                ml[u] = a.part_ml[it];
                v[u] = *(const float2 *)(a.part_acc + it * kHeadDim + 2 * lane);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float w = __builtin_amdgcn_exp2f(ml[u].x - M);
                den += w * ml[u].y;
                o0 += w * v[u].x;
                o1 += w * v[u].y;
            }
        }
        for (; s < n; ++s) {
            const size_t it = ((size_t)(base + s) * a.Hkv + g) * a.G + hh;
            const float2 ml = a.part_ml[it];
            const float2 v = *(const float2 *)(a.part_acc + it * kHeadDim + 2 * lane);
            const float w = __builtin_amdgcn_exp2f(ml.x - M);
            den += w * ml.y;
            o0 += w * v.x;
            o1 += w * v.y;
        }
        const float inv = 1.0f / den;
        o0 *= inv;
        o1 *= inv;
    }
    if constexpr (MODE == MODE_F32) {
        float *o = (float *)a.out + ((size_t)b * a.Hq + h) * kHeadDim + 2 * lane;
        *(float2 *)o = make_float2(o0, o1);
    } else {
        uint16_t *o = (uint16_t *)a.out + ((size_t)b * a.Hq + h) * kHeadDim + 2 * lane;
        *(unsigned *)o = (unsigned)bf16_bits(o0) | ((unsigned)bf16_bits(o1) << 16);
    }
}

// ---------------------------------------------------------------- host side
bool aligned(const void *p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool supported_g(int G) { return G == 1 || G == 2 || G == 4 || G == 8 || G == 16; }

int forced_pages(unsigned flags) { return (int)((flags & VD_FLAG_SPLIT_MASK) >> VD_FLAG_SPLIT_SHIFT); }

// Shape checks shared by every entry point.
int check_shapes(int num_seqs, int n_q_heads, int n_kv_heads, int head_dim, int page_size,
                 int max_pages_per_seq, unsigned flags)
{
    if (num_seqs < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 || page_size <= 0 ||
        max_pages_per_seq <= 0)
        return VD_ERROR_INVALID_VALUE;
    if (n_q_heads % n_kv_heads != 0)
        return VD_ERROR_INVALID_VALUE;
    if (flags & ~(VD_FLAG_OUT_F32 | VD_FLAG_SPLIT_MASK))
        return VD_ERROR_INVALID_VALUE;
    if (forced_pages(flags) > kMaxSplitPages)
        return VD_ERROR_INVALID_VALUE;
    if (head_dim != kHeadDim || page_size != kPage || !supported_g(n_q_heads / n_kv_heads) ||
        num_seqs > kMaxSeqs)
        return VD_ERROR_NOT_SUPPORTED;
    // 32-bit in-page offsets and page-table indices
    if ((long long)n_kv_heads * kHeadDim * kPage >= (1LL << 30) ||
        (long long)num_seqs * max_pages_per_seq >= (1LL << 31))
        return VD_ERROR_NOT_SUPPORTED;
    return VD_SUCCESS;
}

int launch_status()
{
    return hipGetLastError() == hipSuccess ? VD_SUCCESS : VD_ERROR_LAUNCH;
}

int num_cus(int *out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VD_ERROR_LAUNCH;
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return VD_ERROR_LAUNCH;
    *out = n;
    return VD_SUCCESS;
}

int enqueue_plan(const int32_t *seq_lens, int num_seqs, int n_q_heads, int n_kv_heads,
                 int max_pages_per_seq, void *workspace, unsigned flags, hipStream_t stream)
{
    int cus = 0;
    int st = num_cus(&cus);
    if (st)
        return st;
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads,
                                   max_pages_per_seq, forced_pages(flags));
    const int target = std::min(kTargetItemsCap, kItemsPerCU * cus);
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, seq_lens, num_seqs,
                       n_kv_heads, max_pages_per_seq, forced_pages(flags), target,
                       (char *)workspace, lay);
    return launch_status();
}

template <int G>
void launch_attn_g(const AttnArgs &args, int mode, dim3 grid, hipStream_t stream)
{
    if (mode == MODE_F32)
        hipLaunchKernelGGL((attn_kernel<G, MODE_F32>), grid, dim3(kAttnThreads), 0, stream, args);
    else
        hipLaunchKernelGGL((attn_kernel<G, MODE_BF16>), grid, dim3(kAttnThreads), 0, stream, args);
}

int enqueue_attn(const AttnArgs &args, int G, int mode, hipStream_t stream)
{
    int cus = 0;
    int st = num_cus(&cus);
    if (st)
        return st;
    const dim3 grid(cus * kAttnWGPerCU);
    if (mode == MODE_GATHER) {
        hipLaunchKernelGGL((attn_kernel<1, MODE_GATHER>), grid, dim3(kAttnThreads), 0, stream, args);
        return launch_status();
    }
    switch (G) {
    case 1: launch_attn_g<1>(args, mode, grid, stream); break;
    case 2: launch_attn_g<2>(args, mode, grid, stream); break;
    case 4: launch_attn_g<4>(args, mode, grid, stream); break;
    case 8: launch_attn_g<8>(args, mode, grid, stream); break;
    case 16: launch_attn_g<16>(args, mode, grid, stream); break;
    default: return VD_ERROR_NOT_SUPPORTED;
    }
    return launch_status();
}

AttnArgs make_args(const WsLayout &lay, void *workspace, int n_q_heads, int n_kv_heads,
                   int max_pages_per_seq, float scale)
{
    char *ws = (char *)workspace;
    AttnArgs a{};
    a.queue = &((PlanHeader *)(ws + lay.hdr))->queue;
    a.done = &((PlanHeader *)(ws + lay.hdr))->done;
    a.hdr = (const PlanHeader *)(ws + lay.hdr);
    a.split_base = (const int32_t *)(ws + lay.split_base);
    a.splits = (const int4 *)(ws + lay.splits);
    a.tok_base = (const long long *)(ws + lay.tok_base);
    a.part_ml = (float2 *)(ws + lay.part_ml);
    a.part_acc = (float *)(ws + lay.part_acc);
    a.Hq = n_q_heads;
    a.Hkv = n_kv_heads;
    a.pt_stride = max_pages_per_seq;
    a.maxp = max_pages_per_seq;
    a.scale_log2 = scale * kLog2e;
    return a;
}

int check_attn_args(const void *q, const void *k_pages, const void *v_pages,
                    const int32_t *page_table, const int32_t *seq_lens, const void *out,
                    int num_seqs, int n_q_heads, int n_kv_heads, int head_dim, int page_size,
                    float scale, int max_pages_per_seq, const void *workspace,
                    size_t workspace_bytes, unsigned flags)
{
    int st = check_shapes(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, flags);
    if (st)
        return st;
    if (!q || !k_pages || !v_pages || !page_table || !seq_lens || !out || !workspace)
        return VD_ERROR_INVALID_VALUE;
    if (!aligned(q, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(out, 16) ||
        !aligned(workspace, 16) || !aligned(page_table, 4) || !aligned(seq_lens, 4))
        return VD_ERROR_INVALID_VALUE;
    if (!std::isfinite(scale))
        return VD_ERROR_INVALID_VALUE;
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads,
                                   max_pages_per_seq, forced_pages(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    return VD_SUCCESS;
}

}  // namespace

// ---------------------------------------------------------------- C ABI
extern "C" {

const char *vd_status_string(int status)
{
    switch (status) {
    case VD_SUCCESS: return "VD_SUCCESS";
    case VD_ERROR_INVALID_VALUE: return "VD_ERROR_INVALID_VALUE";
    case VD_ERROR_NOT_SUPPORTED: return "VD_ERROR_NOT_SUPPORTED";
    case VD_ERROR_WORKSPACE_TOO_SMALL: return "VD_ERROR_WORKSPACE_TOO_SMALL";
    case VD_ERROR_LAUNCH: return "VD_ERROR_LAUNCH";
    default: return "VD_UNKNOWN_STATUS";
    }
}

size_t vd_decode_workspace_size(int num_seqs, int n_q_heads, int n_kv_heads, int head_dim,
                                int page_size, int max_pages_per_seq, unsigned flags)
{
    if (check_shapes(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size, max_pages_per_seq,
                     flags))
        return 0;
    return ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads, max_pages_per_seq,
                     forced_pages(flags)).total;
}

int vd_decode_plan(const int32_t *seq_lens, int num_seqs, int n_q_heads, int n_kv_heads,
                   int head_dim, int page_size, int max_pages_per_seq, void *workspace,
                   size_t workspace_bytes, unsigned flags, hipStream_t stream)
{
    int st = check_shapes(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, flags);
    if (st)
        return st;
    if (!seq_lens || !workspace || !aligned(seq_lens, 4) || !aligned(workspace, 16))
        return VD_ERROR_INVALID_VALUE;
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads,
                                   max_pages_per_seq, forced_pages(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    if (num_seqs == 0)
        return VD_SUCCESS;
    return enqueue_plan(seq_lens, num_seqs, n_q_heads, n_kv_heads, max_pages_per_seq,
                        workspace, flags, stream);
}

int vd_decode_partial(const void *q, const void *k_pages, const void *v_pages,
                      const int32_t *page_table, const int32_t *seq_lens, void *out,
                      int num_seqs, int n_q_heads, int n_kv_heads, int head_dim,
                      int page_size, float scale, int max_pages_per_seq, void *workspace,
                      size_t workspace_bytes, unsigned flags, hipStream_t stream)
{
    int st = check_attn_args(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs,
                             n_q_heads, n_kv_heads, head_dim, page_size, scale,
                             max_pages_per_seq, workspace, workspace_bytes, flags);
    if (st)
        return st;
    if (num_seqs == 0)
        return VD_SUCCESS;
    const int G = n_q_heads / n_kv_heads;
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_pages(flags));
    AttnArgs a = make_args(lay, workspace, n_q_heads, n_kv_heads, max_pages_per_seq, scale);
    a.q = (const uint16_t *)q;
    a.k = (const uint16_t *)k_pages;
    a.v = (const uint16_t *)v_pages;
    a.pt = page_table;
    a.seq_lens = seq_lens;
    a.out = out;
    return enqueue_attn(a, G, (flags & VD_FLAG_OUT_F32) ? MODE_F32 : MODE_BF16, stream);
}

int vd_decode_combine(void *out, int num_seqs, int n_q_heads, int n_kv_heads, int head_dim,
                      int page_size, int max_pages_per_seq, void *workspace,
                      size_t workspace_bytes, unsigned flags, hipStream_t stream)
{
    int st = check_shapes(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, flags);
    if (st)
        return st;
    if (!out || !workspace || !aligned(out, 16) || !aligned(workspace, 16))
        return VD_ERROR_INVALID_VALUE;
    const int G = n_q_heads / n_kv_heads;
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_pages(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    if (num_seqs == 0)
        return VD_SUCCESS;
    char *ws = (char *)workspace;
    CombineArgs c;
    c.out = out;
    c.split_base = (const int32_t *)(ws + lay.split_base);
    c.part_ml = (const float2 *)(ws + lay.part_ml);
    c.part_acc = (const float *)(ws + lay.part_acc);
    c.Hq = n_q_heads;
    c.Hkv = n_kv_heads;
    c.G = G;
    const dim3 grid((unsigned)num_seqs * n_q_heads);
    if (flags & VD_FLAG_OUT_F32)
        hipLaunchKernelGGL(combine_kernel<MODE_F32>, grid, dim3(kCombineThreads), 0, stream, c);
    else
        hipLaunchKernelGGL(combine_kernel<MODE_BF16>, grid, dim3(kCombineThreads), 0, stream, c);
    return launch_status();
}

int vd_decode_attn(const void *q, const void *k_pages, const void *v_pages,
                   const int32_t *page_table, const int32_t *seq_lens, void *out, int num_seqs,
                   int n_q_heads, int n_kv_heads, int head_dim, int page_size, float scale,
                   int max_pages_per_seq, void *workspace, size_t workspace_bytes,
                   unsigned flags, hipStream_t stream)
{
    int st = check_attn_args(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs,
                             n_q_heads, n_kv_heads, head_dim, page_size, scale,
                             max_pages_per_seq, workspace, workspace_bytes, flags);
    if (st)
        return st;
    if (num_seqs == 0)
        return VD_SUCCESS;
    st = vd_decode_plan(seq_lens, num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                        max_pages_per_seq, workspace, workspace_bytes, flags, stream);
    if (st)
        return st;
    st = vd_decode_partial(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs, n_q_heads,
                           n_kv_heads, head_dim, page_size, scale, max_pages_per_seq, workspace,
                           workspace_bytes, flags, stream);
    if (st)
        return st;
    return vd_decode_combine(out, num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                             max_pages_per_seq, workspace, workspace_bytes, flags, stream);
}

int vd_decode_gather(const void *k_pages, const void *v_pages, const int32_t *page_table,
                     const int32_t *seq_lens, void *k_out, void *v_out, int num_seqs,
                     int n_kv_heads, int head_dim, int page_size, int max_pages_per_seq,
                     void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int st = check_shapes(num_seqs, n_kv_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, 0);
    if (st)
        return st;
    if (!k_pages || !v_pages || !page_table || !seq_lens || !k_out || !v_out || !workspace)
        return VD_ERROR_INVALID_VALUE;
    if (!aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(k_out, 16) ||
        !aligned(v_out, 16) || !aligned(workspace, 16) || !aligned(page_table, 4) ||
        !aligned(seq_lens, 4))
        return VD_ERROR_INVALID_VALUE;
    const WsLayout lay = ws_layout(num_seqs, 1, n_kv_heads, max_pages_per_seq, 0);
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    if (num_seqs == 0)
        return VD_SUCCESS;
    st = enqueue_plan(seq_lens, num_seqs, n_kv_heads, n_kv_heads, max_pages_per_seq, workspace,
                      0, stream);
    if (st)
        return st;
    AttnArgs a = make_args(lay, workspace, n_kv_heads, n_kv_heads, max_pages_per_seq, 1.0f);
    a.k = (const uint16_t *)k_pages;
    a.v = (const uint16_t *)v_pages;
    a.pt = page_table;
    a.seq_lens = seq_lens;
    a.out = k_out;
    a.out2 = v_out;
    return enqueue_attn(a, 1, MODE_GATHER, stream);
}

}  // extern "C"
