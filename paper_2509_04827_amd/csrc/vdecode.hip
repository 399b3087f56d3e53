// libvdecode -- paged GQA decode attention for MI355X (gfx950, CDNA4).
//
// One decode step attends each request's newest query token to every token of
// its paged KV cache: the attention part of the decode iteration whose latency
// the paper models as growing with N_kv (Sec. 5.4, Eq. pred-itl), over a paged
// cache (Sec. 2.1).  The step is read-bound: every cached K and V byte is read
// once, so the kernels below are built around HBM traffic, not arithmetic.
//
// Work decomposition.  The KV heads are taken in groups of HW (HW divides
// n_kv_heads; 4 when it can be): one workgroup of HW waves, one wave per head,
// walks the pages of a head group together, so the group reads each token's
// HW head rows (HW x 256 B, contiguous in the token-major page) at about the
// same time.  A "tile" is one 16-token page of one head group.  All tiles of
// the step are laid out in one sequence, ordered by (request b, head group
// q, page j); a "segment" is the run of tiles of one (b, q).  The plan
// cuts the sequence into W ranges of equal length (W a multiple of the
// number of resident workgroups, four waves per CU, or one range per tile
// when there are fewer tiles than workgroups), so every workgroup streams
// the same number of tiles whatever the length mix.  A range may end inside
// a segment and may span several; each (range, segment) overlap is a
// "piece".  A piece that
// covers its whole segment writes the final output, the others write a (max,
// normaliser, accumulator) partial per head that the combine kernel merges.
// Pieces form a monotone path in (range, segment), so range + segment numbers
// them without collisions; a head's partial slot is that times HW plus its
// index in the group.
//
// Kernels on the caller's stream.  The whole step (vd_decode_attn) is two:
// a self-planned attention kernel and the combine kernel (the attention
// kernel alone for tiny steps, whose short plan cuts no segment; see
// short_plan).  The staged API
// runs the planner first, once per step, and a planned attention kernel per
// layer.
//   plan_kernel     one workgroup: tile offsets per request, range starts,
//                   a boundary record per range (which segment a range
//                   boundary cuts: its first partial slot and piece count),
//                   and the list of requests without tokens.
//   attn_kernel     R resident workgroups, each taking consecutive ranges,
//                   one wave per KV head of the group.  Self-planned, each
//                   workgroup first scans the request lengths in LDS to find
//                   its ranges' start and boundary records (the planner's
//                   arithmetic, so both cut identical ranges).  Per page:
//                     scores = K Q^T against the group's G query heads,
//                     for G <= 8 on the vector ALU: K rows are loaded like V
//                     (lane r, row block grp: tokens 4grp+j, dimensions
//                     8r..8r+8), each lane forms bf16 pair dot products
//                     with every head, and DPP row exchanges sum a token's
//                     16 slices while scattering the heads so that lane r
//                     ends with head r (score_valu); for G = 16, or on
//                     request, on the matrix cores: K rows go straight into
//                     the A operands of v_mfma_f32_16x16x32_bf16 (lane =
//                     token row; columns past G repeat head G-1 and are
//                     never stored).  Both leave the scores in the same
//                     layout (lane r, row block grp: tokens 4grp+i of head r);
//                     online softmax in fp32 (exp2 domain, lazy rescaling);
//                     V rows are loaded coalesced (4 rows x 256 B per
//                     instruction) and transposed in registers with byte
//                     permutes into the A operand of
//                     v_mfma_f32_16x16x16_bf16, whose B operand is P exactly
//                     as the score left it (P split into bf16 hi + lo).
//                   A wave's K/V stream runs on across pieces: the next
//                   piece's bounds come from scalar loads of request
//                   lengths, its page ids
//                   and Q are loaded a piece ahead, and its first page while
//                   the current piece's last page is consumed.  Piece results
//                   wait in LDS (up to 64 / G per wave) and are written when
//                   the wave's work is done, so no stores interleave with the
//                   stream.
//   combine_kernel  log-sum-exp merge of the partials of each segment that
//                   a range boundary cuts (zeros for requests without
//                   tokens).
//
// All arithmetic is fp32; bf16 is only the storage type of Q/K/V, the
// operand type of the MFMAs and pair dot products, and the optional output
// type.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <stdint.h>

#include "vdecode.h"

namespace {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kMaxSeqs = 8192;         // every request's tile offset fits in LDS when planning
constexpr int kMaxRangeTiles = 512;    // eight 64-entry page-id windows per piece
constexpr int kMaxResidentGroups = 4096;
constexpr int kPlanThreads = 1024;
constexpr int kHeadsPerGroup = 4;      // preferred KV heads (waves) per attention workgroup
constexpr int kAttnWavesPerCU = 4;     // resident attention waves per CU (one per SIMD)
constexpr int kDeferEntries = 64;      // LDS result entries per wave, over G query heads
constexpr int kPrePad = 6;             // self-planned prefix in LDS: one pad word per 64 entries
constexpr int kAttnMaxThreads = 64 * kHeadsPerGroup;
constexpr int kCombineThreads = 512;
// Short plans (see short_plan): every request at most this many pages, and
// all requests' tiles together at most a quarter of the resident workgroups.
constexpr int kShortMaxPages = 4;
constexpr int kCombineGroupsPerCU = 2;
constexpr float kLog2e = 1.4426950408889634f;
// Lazy rescaling: the running max is only raised when a new score exceeds it
// by more than this (log2 units), so weights stay below 2^8 and acc/l never
// overflow, while most pages skip the accumulator rescale.
constexpr float kRescaleSlack = 8.0f;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// The workspace header is the step record of the C ABI (vd_step_info):
// planner or self-planned prologue fill its sizes, the attention kernel's
// first workgroup its clock stamps.
typedef vd_step_info PlanHeader;

// ---------------------------------------------------------------- workspace
struct WsLayout {
    size_t hdr, tok_base, bounds, empty, ranges, part_ml, part_acc, total;
    long long cap;   // most ranges any plan of these sizes can have
};

__host__ __device__ inline long long ceil_div_ll(long long a, long long b) { return (a + b - 1) / b; }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// KV heads per attention workgroup: the preferred count if it divides Hkv,
// else the largest power of two that does.
inline int heads_per_group(int Hkv)
{
    for (int hw = kHeadsPerGroup; hw > 1; hw >>= 1)
        if (Hkv % hw == 0)
            return hw;
    return 1;
}

// Range capacity.  Automatic plans: W = R * ceil(T / (kMaxRangeTiles * R))
// with R resident workgroups, so W < R + T / kMaxRangeTiles.  A forced range
// length c: W = ceil(T / c).  T <= B * maxp * Hkv / HW tiles; partial slots
// (W + B * Hkv / HW) * HW.  The caller-sized workspace takes R at its bound
// kMaxResidentGroups, so its size does not depend on the device; the
// no-allocation entry point sizes its fixed scratch with the device's own R.
inline WsLayout ws_layout(int B, int G, int Hkv, int maxp, int forced,
                          int resident = kMaxResidentGroups)
{
    const int HW = heads_per_group(Hkv);
    const long long tiles = (long long)B * maxp * (Hkv / HW);
    long long cap = forced > 0 ? ceil_div_ll(tiles, forced)
                               : resident + ceil_div_ll(tiles, kMaxRangeTiles);
    cap = std::max(cap, 1LL);
    const long long slots = cap * HW + (long long)B * Hkv;
    WsLayout l;
    l.cap = cap;
    size_t o = 0;
    l.hdr = o;       o = align_up(o + sizeof(PlanHeader), 256);
    l.tok_base = o;  o = align_up(o + sizeof(long long) * (size_t)(B + 1), 256);
    l.bounds = o;    o = align_up(o + sizeof(int4) * (size_t)cap, 256);
    l.empty = o;     o = align_up(o + sizeof(int) * (size_t)B, 256);
    l.ranges = o;    o = align_up(o + sizeof(int4) * (size_t)(cap + 1), 256);
    l.part_ml = o;   o = align_up(o + sizeof(float2) * (size_t)slots * G, 256);
    l.part_acc = o;  o = align_up(o + sizeof(float) * (size_t)slots * G * kHeadDim, 256);
    l.total = o;
    return l;
}

// ---------------------------------------------------------------- planning
// The same arithmetic serves the planner kernel (staged API) and the
// attention kernel's own prologue (whole step), so both cut identical ranges.
constexpr int kPlanPerThread = kMaxSeqs / kPlanThreads;   // requests per planner thread

__device__ inline int clamped_len(const int32_t *seq_lens, int b, int maxp)
{
    const int L = seq_lens[b];
    return L <= 0 ? 0 : min(L, maxp * kPage);
}

// Number of ranges W for T tiles.  A forced length c gives ceil(T / c).
// Otherwise a step of at most R tiles gets one range per tile (as many
// workgroups stream as there are tiles, and the combine merges the pieces in
// one round of loads, which costs less than a longer chain of pages per
// wave); past that W is a multiple of R with at most kMaxRangeTiles tiles per
// range.  W <= T, so no range is empty.
// (All sizes here are below 2^31, so the 32-bit quotients are exact; unsigned
// arithmetic keeps the divisions short.)
__device__ inline unsigned ceil_div_u(unsigned a, unsigned b) { return (a + b - 1) / b; }

__device__ inline int plan_ranges(int T, int forced, int R, bool shrt)
{
    if (T == 0)
        return 0;
    const unsigned t = (unsigned)T;
    if (forced > 0)
        return (int)ceil_div_u(t, (unsigned)forced);
    if (shrt)   // at most one range per workgroup
        return T < R ? T : R;
    return T < R ? T : (int)((unsigned)R * ceil_div_u(t, (unsigned)kMaxRangeTiles * R));
}

// A short plan cuts no (request, head group) segment: each range starts at
// the first segment that begins at or after its equal-length start, so every
// piece is a whole segment, writes the final output, and nothing is left to
// merge.  It is chosen from the sizes alone (every request at most
// max_pages_per_seq pages), so the host knows that no combine kernel is
// needed: for tiny steps, every request at most kShortMaxPages pages and at
// most R / 4 (page, head group) tiles in all.  There a wave's chain of at
// most four pages costs less than the combine launch it saves (interleaved
// A/B on MI355X: 8-21% faster steps at 1-32 requests of 16-64 tokens); on
// larger steps the split plan's balance wins (2-4% at 64-512 requests of
// 16-64 tokens, and more on ragged mixes of longer requests).
__host__ __device__ inline bool short_plan(int B, int Hg, int maxp, int R, int forced)
{
    return forced <= 0 && maxp <= kShortMaxPages &&
           4LL * B * Hg * maxp <= (long long)R;
}

// first tile of range w: floor(w * T / W)
__device__ inline int range_start(int w, int T, int W)
{
    return (int)((unsigned long long)(unsigned)w * (unsigned)T / (unsigned)W);
}

// range holding tile t
__device__ inline int range_of(long long t, long long T, long long W)
{
    return (int)(((unsigned long long)(t + 1) * (unsigned long long)W - 1) / (unsigned long long)T);
}

// Ranges [lo, hi) of workgroup g of n: consecutive, as equal in number as
// they can be.
__device__ inline int2 group_ranges(int g, int n, int W)
{
    const unsigned long long w = (unsigned)W, u = (unsigned)n;
    return make_int2((int)((unsigned)g * w / u), (int)((unsigned)(g + 1) * w / u));
}

// Boundary record of range w >= 1, whose first tile t is page j of segment
// s (P pages): {s, first partial slot of s, pieces of s, index of this
// boundary among those inside s}.  A range that starts a segment (j = 0)
// gets pieces = 0: nothing to merge there.  The combine kernel reads one
// record per boundary.
__device__ inline int4 boundary_record(int w, int t, int s, int j, int P, int T, int W)
{
    if (j == 0)
        return make_int4(s, 0, 0, 0);
    const int first = t - j;
    const int w0 = range_of(first, T, W), w1 = range_of(first + P - 1, T, W);
    return make_int4(s, w0 + s, w1 - w0 + 1, w - w0 - 1);
}

// Word of entry b of a prefix array in LDS: PAD = 6 skips one word every
// 64, so that threads walking contiguous runs of entries (one run each)
// fall in different banks; PAD = 0 is the plain layout.
template <int PAD>
__device__ inline int pidx(int b) { return PAD ? b + (b >> PAD) : b; }

// Largest b in [0, B) with pre[b] <= t (pre ascending, pre[B] = T > t): the
// request holding tile t.
template <int PAD>
__device__ inline int find_request(const int *pre, int B, int t)
{
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (pre[pidx<PAD>(mid)] <= t) lo = mid; else hi = mid;
    }
    return lo;
}

// First tile of range w of a short plan: the start of the first segment that
// begins at or after floor(w * T / W); T for w = W.  A range may be empty.
template <int PAD>
__device__ inline int short_start(const int *pre, int B, int Hg, int w, int T, int W)
{
    if (w >= W)
        return T;
    const int t = range_start(w, T, W);   // < T
    const int b = find_request<PAD>(pre, B, t);
    const int P = (pre[pidx<PAD>(b + 1)] - pre[pidx<PAD>(b)]) / Hg;   // > 0: tile t lies in b
    const int off = t - pre[pidx<PAD>(b)];
    return pre[pidx<PAD>(b)] + (off + P - 1) / P * P;
}

// First tile of range w under either plan.
template <int PAD>
__device__ inline int plan_start(const int *pre, int B, int Hg, int w, int T, int W, bool shrt)
{
    return shrt ? short_start<PAD>(pre, B, Hg, w, T, W) : range_start(w, T, W);
}

// Descriptor {b, q, j, t} of range w, whose first tile t lies in request b,
// and its boundary record.
template <int PAD>
__device__ inline void entry_at(const int *pre, int b, int Hg, int w, int t, int T, int W,
                                int4 &desc, int4 &rec)
{
    const int P = (pre[pidx<PAD>(b + 1)] - pre[pidx<PAD>(b)]) / Hg;
    const int off = t - pre[pidx<PAD>(b)];
    const int q = off / P, j = off - q * P;
    desc = make_int4(b, q, j, t);
    rec = boundary_record(w, t, b * Hg + q, j, P, T, W);
}

// The same for range w starting at tile t: the request found by binary
// search.  A range starting at T (an empty last range of a short plan) gets
// the end sentinel and an empty record.
template <int PAD>
__device__ inline void range_entry(const int *pre, int B, int Hg, int w, int t, int T, int W,
                                   int4 &desc, int4 &rec)
{
    if (t >= T) {
        desc = make_int4(B, 0, 0, T);
        rec = make_int4(0, 0, 0, 0);
        return;
    }
    entry_at<PAD>(pre, find_request<PAD>(pre, B, t), Hg, w, t, T, W, desc, rec);
}

// Inclusive prefix sum over the 64 lanes of a wave on DPP: Hillis-Steele
// within rows of 16 lanes (row_shr 1, 2, 4, 8; lanes shifted in from outside
// the row read 0), then lane 15 of rows 0 and 2 added into rows 1 and 3
// (row_bcast:15) and lane 31 into rows 2 and 3 (row_bcast:31).  Six VALU
// adds, no LDS round trip.
__device__ inline unsigned wave_scan_dpp(unsigned x)
{
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);
    x += (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);
    return x;
}

template <typename T>
__device__ inline T wave_inclusive_scan(T x, int lane)
{
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T y = __shfl_up(x, off);
        if (lane >= off)
            x += y;
    }
    return x;
}

// One workgroup.  Thread t owns requests [t * per, (t + 1) * per): a serial
// prefix over its own requests, a wave scan of the per-thread totals and one
// scan of the per-wave totals give every request's first tile and token.
__global__ void __launch_bounds__(kPlanThreads)
plan_kernel(const int32_t *__restrict__ seq_lens, int B, int Hg, int maxp, int forced,
            int resident_groups, int shrt, char *__restrict__ ws, WsLayout lay)
{
    __shared__ int s_pre[kMaxSeqs + 1];
    __shared__ int s_wtiles[kPlanThreads / 64];
    __shared__ long long s_wtok[kPlanThreads / 64];
    __shared__ int s_nempty;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int per = (B + kPlanThreads - 1) / kPlanThreads;
    const int b0 = t * per;

    int tiles[kPlanPerThread];
    int lens[kPlanPerThread];
    int my_tiles = 0;
    long long my_tok = 0;
#pragma unroll
    for (int k = 0; k < kPlanPerThread; ++k) {
        const int b = b0 + k;
        lens[k] = (k < per && b < B) ? clamped_len(seq_lens, b, maxp) : 0;
        tiles[k] = (lens[k] + kPage - 1) / kPage * Hg;
        my_tiles += tiles[k];
        my_tok += lens[k];
    }
    const int inc_tiles = wave_inclusive_scan(my_tiles, lane);
    const long long inc_tok = wave_inclusive_scan(my_tok, lane);
    if (lane == 63) {
        s_wtiles[wv] = inc_tiles;
        s_wtok[wv] = inc_tok;
    }
    if (t == 0)
        s_nempty = 0;
    __syncthreads();
    int base_tiles = 0;
    long long base_tok = 0;
    for (int x = 0; x < wv; ++x) {
        base_tiles += s_wtiles[x];
        base_tok += s_wtok[x];
    }
    int pre = base_tiles + inc_tiles - my_tiles;
    long long tpre = base_tok + inc_tok - my_tok;
    long long *tok_base = (long long *)(ws + lay.tok_base);
    int *empty = (int *)(ws + lay.empty);
#pragma unroll
    for (int k = 0; k < kPlanPerThread; ++k) {
        const int b = b0 + k;
        if (k < per && b < B) {
            s_pre[b] = pre;
            tok_base[b] = tpre;
            if (tiles[k] == 0)
                empty[atomicAdd(&s_nempty, 1)] = b;
        }
        pre += tiles[k];
        tpre += lens[k];
    }
    if (t == kPlanThreads - 1) {
        // the last thread's running sums are the totals
        s_pre[B] = pre;
        tok_base[B] = tpre;
    }
    __syncthreads();
    const int T = s_pre[B];
    const int W = plan_ranges(T, forced, resident_groups, shrt != 0);

    // range starts {b, q, j, t} (range W is the end sentinel) and the
    // boundary records of ranges 1 .. W-1
    int4 *ranges = (int4 *)(ws + lay.ranges);
    int4 *bounds = (int4 *)(ws + lay.bounds);
    for (int w = t; w <= W; w += kPlanThreads) {
        if (w == W) {
            ranges[w] = make_int4(B, 0, 0, T);
            continue;
        }
        int4 desc, rec;
        range_entry<0>(s_pre, B, Hg, w, plan_start<0>(s_pre, B, Hg, w, T, W, shrt != 0), T, W,
                       desc, rec);
        ranges[w] = desc;
        if (w > 0)
            bounds[w] = rec;
    }
    if (t == 0) {
        PlanHeader *h = (PlanHeader *)(ws + lay.hdr);
        h->n_ranges = W;
        h->n_tiles = T;
        h->n_empty = s_nempty;   // final: every append happened before the barrier
    }
}

// ---------------------------------------------------------------- attention
struct AttnArgs {
    const uint16_t *q, *k, *v;
    const int32_t *pt, *seq_lens;
    void *out, *out2;               // attention: out; gather: k_out, v_out
    PlanHeader *hdr;                // read (planned) or written (self-planned)
    const int4 *ranges;             // planned only
    int4 *bounds;                   // self-planned: boundary records written here
    int *empty;                     // self-planned: requests without tokens
    const long long *tok_base;
    float2 *part_ml;
    float *part_acc;
    int Hq, Hkv, HW, pt_stride, maxp;
    int B, forced, resident;        // requests, forced range length (self-planned); R = grid size
    int shrt;                       // short plan (short_plan): no segment is cut
    int zero_empty;                 // self-planned short plan with no combine kernel after it:
                                    // the attention kernel writes the empty requests' zeros
    float scale_log2;
};

enum { MODE_BF16 = 0, MODE_F32 = 1, MODE_GATHER = 2 };

struct Tile {
    u32x4 k[4];   // MFMA score: K[token r][d 8(4kk+grp) .. +8]  (A operand)
                  // vector-ALU score: K[token 4grp+j][d 8r .. 8r+8], as v
    u32x4 v[4];   // V[token 4grp+j][d 8r .. 8r+8], j = 0..3  (raw rows)
};

// K/V bytes are read exactly once per step: stream them past the caches.
__device__ inline u32x4 ldg16_stream(const uint16_t *p)
{
    return __builtin_nontemporal_load((const u32x4 *)p);
}

__device__ inline u32x4 ldg16(const uint16_t *p) { return *(const u32x4 *)p; }

// VS: the vector-ALU score layout of K (the rows of V's layout; koff must
// then equal voff).
template <bool VS = false>
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
        T.k[kk] = ldg16_stream(VS ? kp + kk * row : kp + 32 * kk);
#pragma unroll
    for (int j = 0; j < 4; ++j)
        T.v[j] = ldg16_stream(vp[j]);
}

// The lane-group exchanges use the gfx950 row swaps (VALU, no LDS): with
// both operands x, v_permlane16_swap leaves rows {0,0,2,2} and {1,1,3,3} of
// x in its two results, and v_permlane32_swap halves {lo,lo} and {hi,hi}.
__device__ inline void swap16(float x, float &a, float &b)
{
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    a = __builtin_bit_cast(float, (unsigned)r[0]);
    b = __builtin_bit_cast(float, (unsigned)r[1]);
}

__device__ inline void swap32(float x, float &a, float &b)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    a = __builtin_bit_cast(float, (unsigned)r[0]);
    b = __builtin_bit_cast(float, (unsigned)r[1]);
}

__device__ inline float wave_max_groups(float x)
{
    // max over the 4 lane groups that share lane & 15
    float a, b;
    swap16(x, a, b);
    x = fmaxf(a, b);
    swap32(x, a, b);
    return fmaxf(a, b);
}

__device__ inline float sum_groups(float x)
{
    // (g0 + g1) + (g2 + g3) in every lane of the four groups
    float a, b;
    swap16(x, a, b);
    x = a + b;
    swap32(x, a, b);
    return a + b;
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

// Page ids of pages [jb, je) of request b, 64 per register: lane l of win[x]
// holds page_table[b][jb + 64 x + l].
struct PageIds {
    int win[kMaxRangeTiles / 64];
    __device__ inline int get(int i) const   // i uniform, 0 <= i < je - jb
    {
        const int w = i >> 6, l = i & 63;
        int id = __builtin_amdgcn_readlane(win[0], l);
#pragma unroll
        for (int x = 1; x < kMaxRangeTiles / 64; ++x)
            if (w == x)
                id = __builtin_amdgcn_readlane(win[x], l);
        return id;
    }
};

// Clamped to the piece's last page, so every lane loads (no branches) and the
// loads are counted the same way on every path.
__device__ inline PageIds load_page_ids(const int32_t *pt_row, int jb, int je, int lane)
{
    PageIds p;
#pragma unroll
    for (int x = 0; x < kMaxRangeTiles / 64; ++x)
        p.win[x] = pt_row[min(jb + 64 * x + lane, je - 1)];
    return p;
}

// The planner's tables and the request lengths are not written while the
// attention kernel runs (a self-planned kernel writes only the header,
// boundary records and empty-request list, which it never reads): read them
// through the constant address space, which gives scalar loads that are
// counted apart from the K/V stream.
typedef const __attribute__((address_space(4))) int32_t *const_i32p;

// A piece: pages [jb, je) of KV-head group q of request b, cut from range w.
struct Piece {
    int b, q, jb, je, L, w;
};

// Walks the ranges [w, w_end) of one workgroup and the pieces each covers,
// in order.  The ranges are consecutive, so the walk runs on from one into
// the next: a piece cut by a range end resumes at the next page.
struct PieceWalk {
    int w, w_end, T, W;
    int b, q, j, t, t_end;   // next tile: page j of head group q of request b

    __device__ inline bool next(const AttnArgs &a, int Hg, Piece &p)
    {
        const const_i32p lens = (const_i32p)a.seq_lens;
        while (true) {
            if (t >= t_end) {
                if (++w >= w_end)
                    return false;
                t_end = range_start(w + 1, T, W);
                continue;
            }
            const int L = min(lens[b], a.maxp * kPage);
            const int P = L > 0 ? (L + kPage - 1) / kPage : 0;
            if (P == 0) {   // request without tokens: no tiles
                ++b;
                continue;
            }
            const int n = min(P - j, t_end - t);
            p = Piece{b, q, j, j + n, L, w};
            t += n;
            if (j + n < P) {
                j += n;
            } else {
                j = 0;
                if (++q == Hg) {
                    q = 0;
                    ++b;
                }
            }
            return true;
        }
    }
};

// Self-planned prologue of the attention kernel (whole step, no planner
// kernel): the workgroup reads every request length and forms the tile
// prefix in LDS (in the result-entry space, not yet in use); from it come its
// own ranges' first tile and their boundary records.  Workgroup 0 also writes
// the header and the list of requests without tokens for the combine kernel.
// Returns false when the workgroup has no range.
template <int MODE>
__device__ inline bool self_plan(const AttnArgs &a, int Hg, int *s_pre, PieceWalk &walk)
{
    __shared__ uint2 s_wsum[kHeadsPerGroup];
    __shared__ int4 s_desc;
    // the launch shape comes from the arguments: reading blockDim / gridDim
    // costs a load from the dispatch packet at kernel start
    const int nt = 64 * a.HW, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, nw = a.HW;
    const int B = a.B;
    // eight loads in flight per thread, not one latency per request
    constexpr int kLoadBatch = 8;
    for (int b0 = tid; b0 < B; b0 += kLoadBatch * nt) {
        int L[kLoadBatch];
#pragma unroll
        for (int u = 0; u < kLoadBatch; ++u)   // branch-free: indices clamped into the array
            L[u] = a.seq_lens[min(b0 + u * nt, B - 1)];
#pragma unroll
        for (int u = 0; u < kLoadBatch; ++u) {   // past the end: a 0 into slot B, set later
            const int b = b0 + u * nt;
            const int n = (L[u] <= 0 ? 0 : (min(L[u], a.maxp * kPage) + kPage - 1) / kPage) * Hg;
            s_pre[pidx<kPrePad>(min(b, B))] = b < B ? n : 0;
        }
    }
    __syncthreads();
    // exclusive prefix of tiles in place; thread tid owns requests [c0, c1).
    // Two scans at once: tiles and non-empty requests.
    const int per = (B + nt - 1) / nt;
    const int c0 = min(B, tid * per), c1 = min(B, c0 + per);
    unsigned my_t = 0, my_n = 0;
#pragma unroll 8
    for (int b = c0; b < c1; ++b) {
        const int n = s_pre[pidx<kPrePad>(b)];
        my_t += (unsigned)n;
        my_n += n > 0;
    }
    const unsigned inc_t = wave_scan_dpp(my_t), inc_n = wave_scan_dpp(my_n);
    if (lane == 63)
        s_wsum[wv] = make_uint2(inc_t, inc_n);
    __syncthreads();
    unsigned base_t = 0, base_n = 0, tot_t = 0, tot_n = 0;
    for (int x = 0; x < nw; ++x) {
        const uint2 v = s_wsum[x];
        base_t += x < wv ? v.x : 0u;
        base_n += x < wv ? v.y : 0u;
        tot_t += v.x;
        tot_n += v.y;
    }
    const int T = (int)tot_t, nonempty = (int)tot_n;
    const int excl_t = (int)(base_t + inc_t - my_t), excl_n = (int)(base_n + inc_n - my_n);
    int run = excl_t;
#pragma unroll 8
    for (int b = c0; b < c1; ++b) {
        const int n = s_pre[pidx<kPrePad>(b)];
        s_pre[pidx<kPrePad>(b)] = run;
        run += n;
    }
    if (tid == 0)
        s_pre[pidx<kPrePad>(B)] = T;
    __syncthreads();

    const bool shrt = a.shrt != 0;
    const int W = plan_ranges(T, a.forced, a.resident, shrt);
    const int2 wr = group_ranges(blockIdx.x, a.resident, W);
    __shared__ int s_tend;   // short plan: the end of this workgroup's one range
    if (shrt) {
        // at most one range per workgroup, found by binary search; its
        // boundary record is empty (no segment is cut)
        if (tid == 0 && wr.x < wr.y) {
            const int t0 = short_start<kPrePad>(s_pre, B, Hg, wr.x, T, W);
            const int t1 = short_start<kPrePad>(s_pre, B, Hg, wr.x + 1, T, W);
            int4 desc, rec;
            range_entry<kPrePad>(s_pre, B, Hg, wr.x, t0, T, W, desc, rec);
            s_desc = desc;
            s_tend = t1;
            if (wr.x > 0)
                a.bounds[wr.x] = make_int4(0, 0, 0, 0);
        }
        if (a.zero_empty) {
            // no combine kernel follows: this workgroup writes the zero rows
            // of the requests without tokens in its share of the requests
            const int bz0 = (int)((long long)blockIdx.x * B / a.resident);
            const int bz1 = (int)((long long)(blockIdx.x + 1) * B / a.resident);
            const int row = a.Hq * kHeadDim;
            for (int b = bz0; b < bz1; ++b) {
                if (s_pre[pidx<kPrePad>(b + 1)] != s_pre[pidx<kPrePad>(b)])
                    continue;
                if constexpr (MODE == MODE_F32) {
                    float *o = (float *)a.out + (size_t)b * row;
                    for (int i = tid; i < row / 4; i += nt)
                        *(f32x4 *)(o + 4 * i) = f32x4{0.f, 0.f, 0.f, 0.f};
                } else {
                    uint16_t *o = (uint16_t *)a.out + (size_t)b * row;
                    for (int i = tid; i < row / 8; i += nt)
                        *(u32x4 *)(o + 8 * i) = u32x4{0u, 0u, 0u, 0u};
                }
            }
        }
    } else {
        if (wr.x < wr.y) {
            // the first range: its first tile lies among the requests of one
            // thread, which walks them (no search)
            const int t0 = range_start(wr.x, T, W);
            const int my0 = excl_t, my1 = excl_t + (int)my_t;
            if (my0 <= t0 && t0 < my1) {
                int b = c0;
                while (s_pre[pidx<kPrePad>(b + 1)] <= t0)
                    ++b;
                int4 desc, rec;
                entry_at<kPrePad>(s_pre, b, Hg, wr.x, t0, T, W, desc, rec);
                s_desc = desc;
                if (wr.x > 0)
                    a.bounds[wr.x] = rec;
            }
        }
        for (int w = wr.x + 1 + tid; w < wr.y; w += nt) {
            int4 desc, rec;
            range_entry<kPrePad>(s_pre, B, Hg, w, range_start(w, T, W), T, W, desc, rec);
            a.bounds[w] = rec;
        }
    }
    if (blockIdx.x == 0) {
        // header, and the requests without tokens in order: those before c0
        // number c0 minus the non-empty ones
        int pos = c0 - excl_n;
        for (int b = c0; b < c1; ++b)
            if (s_pre[pidx<kPrePad>(b + 1)] == s_pre[pidx<kPrePad>(b)])
                a.empty[pos++] = b;
        if (tid == 0) {
            a.hdr->n_ranges = W;
            a.hdr->n_tiles = T;
            a.hdr->n_empty = B - nonempty;
        }
    }
    __syncthreads();   // s_desc is set; the prefix is no longer read
    if (wr.x >= wr.y)
        return false;
    const int4 d = s_desc;
    const int t_end = shrt ? s_tend : range_start(wr.x + 1, T, W);
    if (d.w >= t_end)   // an empty range (short plans only)
        return false;
    walk = PieceWalk{wr.x, wr.y, T, W, d.x, d.y, d.z, d.w, t_end};
    return true;
}

// Q operand (B of the score MFMA): head column r, d slice 8(4kk+grp).  Columns
// r >= G repeat head G-1; their results are never stored.
template <int G>
__device__ inline void load_q(const AttnArgs &a, int b, int g, int lane, u32x4 (&qreg)[4])
{
    const int r = min(lane & 15, G - 1), grp = lane >> 4;
    const uint16_t *qrow = a.q + ((size_t)b * a.Hq + g * G + r) * kHeadDim + 8 * grp;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
        qreg[kk] = ldg16(qrow + 32 * kk);
}

// Registers of a wave's Q operand: four 16-byte slices for the MFMA score,
// one per head for the vector-ALU score.
template <int G, bool VS>
constexpr int kQRegs = VS ? G : 4;

// Q for the vector-ALU score: slot s holds head s ^ (r & (G-1)) at d
// 8r .. 8r+8, every head in an order rotated by the lane's own head bits.
template <int G>
__device__ inline void load_q_valu(const AttnArgs &a, int b, int g, int lane, u32x4 (&qv)[G])
{
    const int r = lane & 15;
    const uint16_t *qrow = a.q + ((size_t)b * a.Hq + g * G) * kHeadDim + 8 * r;
#pragma unroll
    for (int s = 0; s < G; ++s)
        qv[s] = ldg16(qrow + (size_t)(s ^ (r & (G - 1))) * kHeadDim);
}

template <bool VS, int G>
__device__ inline void load_q_any(const AttnArgs &a, int b, int g, int lane,
                                  u32x4 (&qreg)[kQRegs<G, VS>])
{
    if constexpr (VS)
        load_q_valu<G>(a, b, g, lane, qreg);
    else
        load_q<G>(a, b, g, lane, qreg);
}

template <int CTRL>
__device__ inline float dpp_row(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                                 CTRL, 0xF, 0xF, false));
}

// One exchange of the row reduction over LIVE slots: with more than one, the
// lane keeps the even slots, each plus its partner lane's next odd slot
// (which holds the same head, the partner's rotation differing in this
// step's bit); with one, a plain sum.
template <int CTRL, int LIVE, int G>
__device__ inline void row_fold(float (&v)[4][G])
{
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if constexpr (LIVE > 1) {
#pragma unroll
            for (int t = 0; t < LIVE / 2; ++t)
                v[j][t] = v[j][2 * t] + dpp_row<CTRL>(v[j][2 * t + 1]);
        } else {
            v[j][0] += dpp_row<CTRL>(v[j][0]);
        }
    }
}

// Q.K^T of a page's 16 tokens against G <= 8 heads on the vector ALU (the
// default score path for those G): lane (r, grp) forms the dot products of
// tokens 4grp+j over its eight dimensions 8r .. 8r+8 with each head (bf16
// pairs, fp32 sums), and the 16 lanes of row grp add up their slices through
// DPP row exchanges (quad permutes for lane bits 0 and 1, row rotations by 4
// and 8 lanes): the first log2 G exchanges halve the live head slots, the rest
// sum.  Lane r ends with head r & (G-1), so s[j] is token 4grp+j of head r,
// the layout of the MFMA score.
template <int G>
__device__ inline f32x4 score_valu(const Tile &T, const u32x4 (&qv)[G])
{
    static_assert(G <= 8, "head bits must stay within three lane bits");
    float v[4][G];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int s = 0; s < G; ++s) {
            float acc = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // element copies first: a bit cast of a vector element
                // itself reads element 0 in this compiler
                const unsigned kw = T.k[j][e], qw = qv[s][e];
                acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, kw),
                                                      __builtin_bit_cast(bf16x2, qw), acc, false);
            }
            v[j][s] = acc;
        }
    }
    row_fold<0xB1, G, G>(v);                          // quad_perm [1,0,3,2]: lane ^ 1
    row_fold<0x4E, (G > 1 ? G / 2 : 1), G>(v);        // quad_perm [2,3,0,1]: lane ^ 2
    row_fold<0x124, (G > 2 ? G / 4 : 1), G>(v);       // row_ror:4
    row_fold<0x128, (G > 4 ? G / 8 : 1), G>(v);       // row_ror:8: lane ^ 8
    return f32x4{v[0][0], v[1][0], v[2][0], v[3][0]};
}

// Copy-through gather of one piece (je - jb <= kMaxRangeTiles) for KV head
// g = q * HW + hi; its page ids were loaded during the previous piece.
__device__ inline void gather_piece(const AttnArgs &a, const Piece &pc, const PageIds &ids, int hi,
                                    int lane)
{
    const int r = lane & 15;    // score MFMA: token row (A) / head column (B, D)
    const int grp = lane >> 4;  // lane group: k-slice of the operands, row block of D
    const int Hkv = a.Hkv;
    const int b = pc.b, g = pc.q * a.HW + hi, jb = pc.jb, je = pc.je, L = pc.L;
    const unsigned row = (unsigned)Hkv * kHeadDim;        // elements per token row
    const size_t page_elems = (size_t)kPage * row;
    const unsigned koff = r * row + g * kHeadDim + 8 * grp;
    const unsigned voff = 4 * grp * row + g * kHeadDim + 8 * r;
    const uint16_t *kb = a.k, *vb = a.v;

    uint16_t *ko = (uint16_t *)a.out;
    uint16_t *vo = (uint16_t *)a.out2;
    const long long t0 = a.tok_base[b];
    for (int j = jb; j < je; ++j) {
        const int pg = ids.get(j - jb);
        Tile T;
        load_tile(T, kb + (size_t)pg * page_elems, vb + (size_t)pg * page_elems, koff, voff, row);
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
                *(u32x4 *)(vo + (size_t)(t0 + j * kPage + 4 * grp + jj) * row + g * kHeadDim +
                           8 * r) = w;
            }
        }
    }
}

// Attention over one piece (je - jb <= kMaxRangeTiles) for KV head
// g = q * HW + hi.  Page tiles go through a two-slot ring: the load of page
// s + 1 is issued before page s is consumed, and the last page's step issues
// the load of the next piece's first page.  The piece's first page is in slot
// PH (loaded by the previous piece); the next piece's lands in slot
// PH ^ (np & 1), which the function returns as np & 1.  The first and last
// steps are written out apart from the loop, so every load is waited for with
// an exact count.  fetch_next() walks to the next piece and loads its page
// ids and Q operand (into nids / the caller's registers) before the first
// step.
template <int G, bool VS, int PH, typename Fetch>
__device__ inline int attn_piece(const AttnArgs &a, const Piece &pc, const PageIds &ids,
                                 const u32x4 (&qreg)[kQRegs<G, VS>], Tile (&ring)[2], Fetch &&fetch_next,
                                 const PageIds &nids, const Piece &nxt, int hi, int lane,
                                 float *entry, float2 *entry_ml)
{
    const int r = lane & 15;    // score MFMA: token row (A) / head column (B, D)
    const int grp = lane >> 4;  // lane group: k-slice of the operands, row block of D
    const int Hkv = a.Hkv;
    const int g = pc.q * a.HW + hi, jb = pc.jb, je = pc.je, L = pc.L;
    const unsigned row = (unsigned)Hkv * kHeadDim;        // elements per token row
    const size_t page_elems = (size_t)kPage * row;
    const unsigned voff = 4 * grp * row + g * kHeadDim + 8 * r;
    const unsigned koff = VS ? voff : r * row + g * kHeadDim + 8 * grp;
    const uint16_t *kb = a.k, *vb = a.v;
    const int np = je - jb;

    fetch_next();

    f32x4 acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;   // running max (log2 units) of head r
    float l_run = 0.f;         // this lane's share of the normaliser

    auto page_step = [&](const Tile &T, int j) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
        if constexpr (VS) {
            s = score_valu<G>(T, qreg);
        } else {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, T.k[kk]), __builtin_bit_cast(bf16x8, qreg[kk]),
                    s, 0, 0, 0);
        }
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

    auto load_in = [&](Tile &T, int jn) {   // page jn of this piece
        const int pg = ids.get(jn - jb);
        load_tile<VS>(T, kb + (size_t)pg * page_elems, vb + (size_t)pg * page_elems, koff, voff,
                      row);
    };
    auto load_next = [&](Tile &T) {         // first page of the next piece
        const int ng = nxt.q * a.HW + hi;
        const int pg = nids.get(0);
        const unsigned nv = 4 * grp * row + ng * kHeadDim + 8 * r;
        load_tile<VS>(T, kb + (size_t)pg * page_elems, vb + (size_t)pg * page_elems,
                      VS ? nv : r * row + ng * kHeadDim + 8 * grp, nv, row);
    };
    constexpr int A = PH, B = PH ^ 1;
    if (np >= 2) {
        load_in(ring[B], jb + 1);
        __builtin_amdgcn_sched_barrier(0);
        page_step(ring[A], jb);
        int s = jb + 1;
        for (int it = (np - 2) / 2; it > 0; --it) {
            load_in(ring[A], s + 1);
            __builtin_amdgcn_sched_barrier(0);
            page_step(ring[B], s);
            load_in(ring[B], s + 2);
            __builtin_amdgcn_sched_barrier(0);
            page_step(ring[A], s + 1);
            s += 2;
        }
    }
    if (np & 1) {
        if (np >= 3) {
            load_in(ring[A], je - 1);
            __builtin_amdgcn_sched_barrier(0);
            page_step(ring[B], je - 2);
        }
        load_next(ring[B]);
        __builtin_amdgcn_sched_barrier(0);
        page_step(ring[A], je - 1);
    } else {
        load_next(ring[A]);
        __builtin_amdgcn_sched_barrier(0);
        page_step(ring[B], je - 1);
    }

    const float l_tot = sum_groups(l_run);
    // acc[blk][i] = O[head r][d 32grp + 8i + blk].  The results go to this
    // wave's LDS entry (lanes r < G hold head r): normalised for a whole
    // segment, else raw with (max, normaliser).  They reach global memory
    // in a batch later, so the K/V stream carries no stores.
    const bool whole = jb == 0 && je == (L + kPage - 1) / kPage;
    const float sc = whole ? 1.0f / l_tot : 1.0f;
    if (r < G) {
        float *srow = entry + r * kHeadDim + 32 * grp;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f32x4 w0, w1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                w0[e] = acc[e][i] * sc;
                w1[e] = acc[4 + e][i] * sc;
            }
            *(f32x4 *)(srow + 8 * i) = w0;
            *(f32x4 *)(srow + 8 * i + 4) = w1;
        }
        entry_ml[r] = make_float2(m_run, l_tot);
    }
    return np & 1;
}

// Each workgroup walks its ranges piece by piece, HW waves per piece (one KV
// head each).  The next piece's bounds (a scalar load of its request's
// length), page ids and Q operand are fetched at the start of a piece, and
// its first page while the piece's last page is consumed, so the K/V stream
// of a wave runs on across piece boundaries.
template <int G, int MODE, bool SELF, bool VS>
__device__ inline void attn_body(const AttnArgs &a)
{
    const int lane = threadIdx.x & 63;
    const int hi = threadIdx.x >> 6;          // KV head within the group
    const int HW = a.HW, Hg = a.Hkv / a.HW;
    extern __shared__ __attribute__((aligned(16))) char s_dyn[];
    PieceWalk walk;
    if constexpr (SELF) {
        if (!self_plan<MODE>(a, Hg, (int *)s_dyn, walk))
            return;
    } else {
        const const_i32p hdr = (const const_i32p)a.hdr;
        const int W = hdr[0], T = hdr[1];
        const int2 wr = group_ranges(blockIdx.x, a.resident, W);
        if (wr.x >= wr.y)
            return;
        // the first range's descriptor from the plan; entry wr.x + 1 gives
        // the tile where that range ends (entry W is the end sentinel)
        const const_i32p rg = (const_i32p)(a.ranges + wr.x);
        if (rg[3] >= rg[7])   // an empty range (short plans only)
            return;
        walk = PieceWalk{wr.x, wr.y, T, W, rg[0], rg[1], rg[2], rg[3], rg[7]};
    }
    Piece cur;
    if (!walk.next(a, Hg, cur))
        return;
    PageIds ids = load_page_ids(a.pt + (size_t)cur.b * a.pt_stride, cur.jb, cur.je, lane);
    if constexpr (MODE == MODE_GATHER) {
        while (true) {
            Piece nxt;
            const bool more = walk.next(a, Hg, nxt);
            if (!more)
                nxt = cur;
            const PageIds nids =
                load_page_ids(a.pt + (size_t)nxt.b * a.pt_stride, nxt.jb, nxt.je, lane);
            gather_piece(a, cur, ids, hi, lane);
            if (!more)
                break;
            cur = nxt;
            ids = nids;
        }
    } else {
        // Per wave: up to kDefer piece results, written out when the wave's
        // work is done (or when all entries are taken).  Dynamic LDS, sized
        // for the workgroup's HW waves (attn_lds_bytes).
        constexpr int kDefer = kDeferEntries / G;
        float (*s_res)[kDefer][G * kHeadDim] = (float (*)[kDefer][G * kHeadDim])s_dyn;
        float2 (*s_ml)[kDefer][G] =
            (float2 (*)[kDefer][G])(s_dyn + (size_t)HW * kDefer * G * kHeadDim * sizeof(float));
        int2 (*s_meta)[kDefer] =    // {whole, out row or partial slot}
            (int2 (*)[kDefer])(s_dyn + (size_t)HW * kDefer * G * (kHeadDim * sizeof(float) + sizeof(float2)));
        int n_res = 0;
        auto flush = [&]() {
            constexpr int kF32Chunks = G * kHeadDim / 4, kBf16Chunks = G * kHeadDim / 8;
            static_assert(kDefer <= 64, "one entry's {whole, target} per lane");
            // every entry's {whole, target} in one LDS read (lane e: entry e),
            // so the loop below waits on LDS only for the entries' data
            const int2 meta = s_meta[hi][min(lane, kDefer - 1)];
            for (int e = 0; e < n_res; ++e) {
                const int whole = __builtin_amdgcn_readlane(meta.x, e);
                const int tgt = __builtin_amdgcn_readlane(meta.y, e);
                const float *st = s_res[hi][e];
                if (whole && MODE == MODE_BF16) {
                    uint16_t *o = (uint16_t *)a.out + (size_t)tgt * kHeadDim;
#pragma unroll
                    for (int c0 = 0; c0 < kBf16Chunks; c0 += 64) {
                        const int c = c0 + (kBf16Chunks >= 64 ? lane : (lane & (kBf16Chunks - 1)));
                        const f32x4 x0 = *(const f32x4 *)(st + 8 * c);
                        const f32x4 x1 = *(const f32x4 *)(st + 8 * c + 4);
                        u32x4 w;
                        w[0] = (unsigned)bf16_bits(x0[0]) | ((unsigned)bf16_bits(x0[1]) << 16);
                        w[1] = (unsigned)bf16_bits(x0[2]) | ((unsigned)bf16_bits(x0[3]) << 16);
                        w[2] = (unsigned)bf16_bits(x1[0]) | ((unsigned)bf16_bits(x1[1]) << 16);
                        w[3] = (unsigned)bf16_bits(x1[2]) | ((unsigned)bf16_bits(x1[3]) << 16);
                        *(u32x4 *)(o + 8 * c) = w;
                    }
                } else {
                    float *o = whole ? (float *)a.out + (size_t)tgt * kHeadDim
                                     : a.part_acc + (size_t)tgt * G * kHeadDim;
#pragma unroll
                    for (int c0 = 0; c0 < kF32Chunks; c0 += 64) {
                        const int c = c0 + (kF32Chunks >= 64 ? lane : (lane & (kF32Chunks - 1)));
                        *(f32x4 *)(o + 4 * c) = *(const f32x4 *)(st + 4 * c);
                    }
                    if (!whole) {
                        const int hh = lane & (G - 1);
                        a.part_ml[(size_t)tgt * G + hh] = s_ml[hi][e][hh];
                    }
                }
            }
            n_res = 0;
        };
        constexpr int NQ = kQRegs<G, VS>;
        u32x4 qreg[NQ];
        load_q_any<VS, G>(a, cur.b, cur.q * HW + hi, lane, qreg);
        Tile ring[2];
        {   // first page of the first piece
            const unsigned row = (unsigned)a.Hkv * kHeadDim;
            const int r = lane & 15, grp = lane >> 4, g = cur.q * HW + hi;
            const size_t pg = (size_t)ids.get(0) * kPage * row;
            const unsigned voff = 4 * grp * row + g * kHeadDim + 8 * r;
            load_tile<VS>(ring[0], a.k + pg, a.v + pg,
                          VS ? voff : r * row + g * kHeadDim + 8 * grp, voff, row);
        }
        int ph = 0;
        while (true) {
            Piece nxt;
            bool more = false;
            PageIds nids;
            u32x4 nq[NQ];
            auto fetch_next = [&]() {
                more = walk.next(a, Hg, nxt);
                if (!more) {   // last piece: the final prefetch re-reads its last page
                    nxt = cur;
                    nxt.jb = cur.je - 1;
                }
                nids = load_page_ids(a.pt + (size_t)nxt.b * a.pt_stride, nxt.jb, nxt.je, lane);
                load_q_any<VS, G>(a, nxt.b, nxt.q * HW + hi, lane, nq);
            };
            if (n_res == kDefer)
                flush();
            float *entry = s_res[hi][n_res];
            float2 *entry_ml = s_ml[hi][n_res];
            const int flip =
                ph == 0 ? attn_piece<G, VS, 0>(a, cur, ids, qreg, ring, fetch_next, nids, nxt, hi, lane, entry, entry_ml)
                        : attn_piece<G, VS, 1>(a, cur, ids, qreg, ring, fetch_next, nids, nxt, hi, lane, entry, entry_ml);
            {
                const int g = cur.q * HW + hi;
                const bool whole = cur.jb == 0 && cur.je == (cur.L + kPage - 1) / kPage;
                const long long slot = ((long long)cur.w + (long long)cur.b * Hg + cur.q) * HW + hi;
                s_meta[hi][n_res] = make_int2(whole ? 1 : 0,
                                              whole ? cur.b * a.Hq + g * G : (int)slot);
                ++n_res;
            }
            if (!more)
                break;
            ph ^= flip;
            cur = nxt;
            ids = nids;
#pragma unroll
            for (int i = 0; i < NQ; ++i)
                qreg[i] = nq[i];
        }
        flush();
    }
}

// The first workgroup stamps the step record with the real-time and
// shader-clock counters at its start and end.
template <int G, int MODE, bool SELF, bool VS = false>
__global__ void __launch_bounds__(kAttnMaxThreads)
attn_kernel(const AttnArgs a)
{
    const bool stamp = blockIdx.x == 0 && threadIdx.x == 0;
    if (stamp) {
        a.hdr->t_start = __builtin_amdgcn_s_memrealtime();
        a.hdr->clk_start = __builtin_amdgcn_s_memtime();
    }
    attn_body<G, MODE, SELF, VS>(a);
    if (stamp) {
        a.hdr->t_end = __builtin_amdgcn_s_memrealtime();
        a.hdr->clk_end = __builtin_amdgcn_s_memtime();
    }
}

// ---------------------------------------------------------------- combine
struct CombineArgs {
    void *out;
    const PlanHeader *hdr;
    const int4 *bounds;     // boundary record per range 1 .. W-1
    const int *empty;       // requests without tokens
    const float2 *part_ml;
    const float *part_acc;
    int Hq, Hkv, G, HW;
    int grid;               // workgroups launched (not read from the dispatch packet)
    int cap;                // entries of bounds
};

// Work items, strided over the workgroups: one per range boundary, then one
// per request without tokens (its output rows are zeros).  A boundary
// inside a segment names that segment's first partial slot and piece count n
// and its own index i among the segment's n - 1 inner boundaries.  Boundary
// i merges query-head rows i, i + n - 1, ... of the segment's HW * G rows,
// so the rows are spread over the workgroups of all its boundaries.  Each
// output chunk (row, 4 floats of head_dim) gets P lanes of one wave, P a
// power of two no larger than n or kCombineMaxLanes, as many as the threads
// allow; lane p merges pieces p, p + P, ... (the loads of four pieces issued
// before use), then the P lanes' (max, normaliser, accumulator) are merged
// by lane shuffles.  A small step's merge is then one round of loads.
// Merging is a running log-sum-exp in the exp2 domain.
constexpr int kChunks = kHeadDim / 4;     // float4 chunks of one query head's output
constexpr int kCombineMaxLanes = 16;
constexpr int kCombineUnroll = 4;

struct Lse {
    float m, l;
    f32x4 o;
};

// Merge pieces p0, p0 + step, ... (< n) of one (slot row, chunk) into r.
__device__ inline void lse_pieces(const CombineArgs &a, Lse &r, int first, int n, int p0, int step,
                                  int hi, int hh, int c4)
{
    for (; p0 < n; p0 += step * kCombineUnroll) {
        float2 ml[kCombineUnroll];
        f32x4 v[kCombineUnroll];
#pragma unroll
        for (int k = 0; k < kCombineUnroll; ++k) {
            const int p = min(p0 + k * step, n - 1);
            const size_t it = ((size_t)(first + p) * a.HW + hi) * a.G + hh;
            ml[k] = a.part_ml[it];
            v[k] = *(const f32x4 *)(a.part_acc + it * kHeadDim + 4 * c4);
        }
        float Mb = r.m;
#pragma unroll
        for (int k = 0; k < kCombineUnroll; ++k)
            if (p0 + k * step < n)
                Mb = fmaxf(Mb, ml[k].x);
        const float sc = __builtin_amdgcn_exp2f(r.m - Mb);
        r.l *= sc;
        r.o *= sc;
#pragma unroll
        for (int k = 0; k < kCombineUnroll; ++k) {
            if (p0 + k * step < n) {
                const float w = __builtin_amdgcn_exp2f(ml[k].x - Mb);
                r.l += w * ml[k].y;
                r.o += w * v[k];
            }
        }
        r.m = Mb;
    }
}

template <int MODE>
__device__ inline void store_out(const CombineArgs &a, size_t dst, f32x4 o)
{
    if constexpr (MODE == MODE_F32) {
        *(f32x4 *)((float *)a.out + dst) = o;
    } else {
        *(u32x2 *)((uint16_t *)a.out + dst) =
            u32x2{(unsigned)bf16_bits(o[0]) | ((unsigned)bf16_bits(o[1]) << 16),
                  (unsigned)bf16_bits(o[2]) | ((unsigned)bf16_bits(o[3]) << 16)};
    }
}

// The rows of one segment that boundary record `rec` assigns to this
// workgroup.
template <int MODE>
__device__ inline void merge_boundary(const CombineArgs &a, int4 rec, int rows, int Hg)
{
    const int s = rec.x, first = rec.y, n = rec.z, i = rec.w;
    if (n == 0 || i >= rows)   // a range that starts its segment, or no row left here
        return;
    const int b = s / Hg, q = s - b * Hg;
    const int nb = n - 1;                     // inner boundaries of the segment, n >= 2
    const int outs = ((rows - 1 - i) / nb + 1) * kChunks;
    int lg = 0;   // P = 2^lg lanes per chunk
    while ((1 << lg) < kCombineMaxLanes && (2 << lg) <= n && (2 << lg) * outs <= kCombineThreads)
        ++lg;
    const int P = 1 << lg, G = a.G;
    for (int u = threadIdx.x; u - (int)threadIdx.x < outs * P; u += kCombineThreads) {
        // lane u: chunk bits 0-1 from u's bits 0-1 and the rest from its bits
        // above lg + 2, piece lane from the lg bits between, so that four
        // lanes in a row read 64 contiguous bytes of one piece and the P
        // lanes of a chunk sit 4 apart in the same wave.  Every lane takes
        // part in the shuffles; lanes past the end redo the last chunk and
        // store nothing.
        const int o = ((u >> (lg + 2)) << 2) | (u & 3), p = (u >> 2) & (P - 1);
        const int oc = min(o, outs - 1);
        const int row = i + (oc / kChunks) * nb, c4 = oc % kChunks;
        const int hi = row / G, hh = row - hi * G;
        Lse r = {-INFINITY, 0.f, {0.f, 0.f, 0.f, 0.f}};
        lse_pieces(a, r, first, n, p, P, hi, hh, c4);   // lane p < P <= n holds a piece
        for (int x = 4; x < 4 * P; x <<= 1) {
            const float m2 = __shfl_xor(r.m, x), l2 = __shfl_xor(r.l, x);
            f32x4 o2;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                o2[k] = __shfl_xor(r.o[k], x);
            const float M = fmaxf(r.m, m2);
            const float s1 = __builtin_amdgcn_exp2f(r.m - M), s2 = __builtin_amdgcn_exp2f(m2 - M);
            r.l = r.l * s1 + l2 * s2;
            r.o = r.o * s1 + o2 * s2;
            r.m = M;
        }
        if (o < outs && p == 0)
            store_out<MODE>(a, ((size_t)b * a.Hq + (q * a.HW + hi) * G + hh) * kHeadDim + 4 * c4,
                            r.o * (1.0f / r.l));
    }
}

template <int MODE>
__global__ void __launch_bounds__(kCombineThreads)
combine_kernel(const CombineArgs a)
{
    // the first item's boundary record is requested with the header, not
    // after it; entries past the plan's ranges (clamped into the array) are
    // read but not used
    const int last = a.cap - 1;
    int4 rec = a.bounds[min((int)blockIdx.x + 1, last)];
    const int W = a.hdr->n_ranges, n_empty = a.hdr->n_empty;
    // both loads in flight together: an empty use of all values here keeps
    // the record's load from being moved past the branch on the header
    asm volatile("" ::"s"(rec.x), "s"(rec.y), "s"(rec.z), "s"(rec.w), "s"(W), "s"(n_empty));
    const int rows = a.HW * a.G, Hg = a.Hkv / a.HW;
    const int n_bounds = W > 1 ? W - 1 : 0;
    for (int item = blockIdx.x; item < n_bounds + n_empty; item += a.grid) {
        // the next item's record is in flight while this one is merged
        const int4 rec_next = a.bounds[min(item + a.grid + 1, last)];
        if (item >= n_bounds) {
            const int b = a.empty[item - n_bounds];
            for (int u = threadIdx.x; u < a.Hq * kChunks; u += kCombineThreads)
                store_out<MODE>(a, (size_t)b * a.Hq * kHeadDim + 4 * u, f32x4{0.f, 0.f, 0.f, 0.f});
        } else {
            merge_boundary<MODE>(a, rec, rows, Hg);
        }
        rec = rec_next;
    }
}

// ---------------------------------------------------------------- KV append
// The step before attention in a decode iteration: each request's new K and
// V rows (n_kv_heads * head_dim bf16, contiguous in the token-major page) go
// to slot pos mod 16 of page page_table[b][pos / 16].  One wave per request,
// 16-byte loads and stores.
constexpr int kAppendThreads = 64;

__global__ void __launch_bounds__(kAppendThreads)
kv_append_kernel(const u32x4 *__restrict__ k_new, const u32x4 *__restrict__ v_new,
                 u32x4 *__restrict__ k_pages, u32x4 *__restrict__ v_pages,
                 const int32_t *__restrict__ page_table, const int32_t *__restrict__ positions,
                 int Hkv, int maxp)
{
    const int b = blockIdx.x;
    const int pos = positions[b];
    if (pos < 0 || pos >= maxp * kPage)
        return;
    const int pg = page_table[(size_t)b * maxp + pos / kPage];
    const int chunks = Hkv * kHeadDim / 8;          // 16-byte chunks per token row
    const size_t dst = ((size_t)pg * kPage + pos % kPage) * chunks;
    const size_t src = (size_t)b * chunks;
    for (int c = threadIdx.x; c < chunks; c += kAppendThreads) {
        k_pages[dst + c] = k_new[src + c];
        v_pages[dst + c] = v_new[src + c];
    }
}

// ---------------------------------------------------------------- HBM read ceiling
// Measurement aid: each workgroup streams its own contiguous chunk of the
// buffer with 16-byte non-temporal loads, 16 per thread in flight, and folds
// them into one word that is stored only if it equals a value no real data
// produces in practice (so the loads cannot be dropped).  Gives the read rate
// the attention kernel is measured against.  Contiguous chunks per workgroup
// read faster here (7.2 TB/s) than a stride over the whole grid (6.8 TB/s).
constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 16;

__global__ void __launch_bounds__(kStreamThreads)
stream_read_kernel(const u32x4 *__restrict__ p, size_t n16, size_t chunk, unsigned *__restrict__ sink)
{
    const size_t end = min((size_t)(blockIdx.x + 1) * chunk, n16);
    size_t i = (size_t)blockIdx.x * chunk + threadIdx.x;
    unsigned acc = 0;
    for (; i + (kStreamUnroll - 1) * kStreamThreads < end; i += kStreamUnroll * kStreamThreads) {
        u32x4 v[kStreamUnroll];
#pragma unroll
        for (int u = 0; u < kStreamUnroll; ++u)
            v[u] = __builtin_nontemporal_load(p + i + u * kStreamThreads);
#pragma unroll
        for (int u = 0; u < kStreamUnroll; ++u)
            acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < end; i += kStreamThreads) {
        const u32x4 v = p[i];
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    if (acc == 0x9E3779B9u)
        *sink = acc;
}

// ---------------------------------------------------------------- host side
bool aligned(const void *p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool supported_g(int G) { return G == 1 || G == 2 || G == 4 || G == 8 || G == 16; }

int forced_tiles(unsigned flags) { return (int)((flags & VD_FLAG_RANGE_MASK) >> VD_FLAG_RANGE_SHIFT); }

// Score path: the vector ALU for G <= 8 unless VD_FLAG_SCORE_MFMA, else the
// matrix cores.
bool valu_score(int G, unsigned flags) { return G <= 8 && !(flags & VD_FLAG_SCORE_MFMA); }

// Shape checks shared by every entry point.
int check_shapes(int num_seqs, int n_q_heads, int n_kv_heads, int head_dim, int page_size,
                 int max_pages_per_seq, unsigned flags)
{
    if (num_seqs < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 || page_size <= 0 ||
        max_pages_per_seq <= 0)
        return VD_ERROR_INVALID_VALUE;
    if (n_q_heads % n_kv_heads != 0)
        return VD_ERROR_INVALID_VALUE;
    if (flags & ~(VD_FLAG_OUT_F32 | VD_FLAG_SELF_PLAN | VD_FLAG_SCORE_MFMA | VD_FLAG_RANGE_MASK))
        return VD_ERROR_INVALID_VALUE;
    if (head_dim != kHeadDim || page_size != kPage || !supported_g(n_q_heads / n_kv_heads) ||
        num_seqs > kMaxSeqs)
        return VD_ERROR_NOT_SUPPORTED;
    // 32-bit in-page offsets, tile counts, token counts, output rows and
    // partial slots (fewer than (maxp + 1) * B * Hkv)
    if ((long long)n_kv_heads * kHeadDim * kPage >= (1LL << 30) ||
        (long long)num_seqs * (max_pages_per_seq + 1) * n_kv_heads >= (1LL << 31) ||
        (long long)num_seqs * max_pages_per_seq >= (1LL << 31) / kPage ||
        (long long)num_seqs * n_q_heads >= (1LL << 31))
        return VD_ERROR_NOT_SUPPORTED;
    return VD_SUCCESS;
}

int launch_status()
{
    return hipGetLastError() == hipSuccess ? VD_SUCCESS : VD_ERROR_LAUNCH;
}

// Compute units of the current device, queried once per device (0 = not yet).
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

int num_cus(int *out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VD_ERROR_LAUNCH;
    if (dev >= 0 && dev < kMaxDevices) {
        const int v = g_cus[dev].load(std::memory_order_relaxed);
        if (v > 0) {
            *out = v;
            return VD_SUCCESS;
        }
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return VD_ERROR_LAUNCH;
    if (dev >= 0 && dev < kMaxDevices)
        g_cus[dev].store(n, std::memory_order_relaxed);
    *out = n;
    return VD_SUCCESS;
}

// The attention kernel for G, output mode, planning (planned: tables from
// the planner kernel; self-planned: the whole step) and score path (`valu`:
// the vector-ALU score, G <= 8).
const void *attn_kernel_ptr(int G, int mode, bool self, bool valu)
{
    if (mode == MODE_GATHER)
        return self || valu ? nullptr : (const void *)attn_kernel<1, MODE_GATHER, false>;
    if (valu) {
#define VD_KV(g)                                                                               \
    (self ? (mode == MODE_F32 ? (const void *)attn_kernel<g, MODE_F32, true, true>              \
                              : (const void *)attn_kernel<g, MODE_BF16, true, true>)            \
          : (mode == MODE_F32 ? (const void *)attn_kernel<g, MODE_F32, false, true>             \
                              : (const void *)attn_kernel<g, MODE_BF16, false, true>))
        switch (G) {
        case 1: return VD_KV(1);
        case 2: return VD_KV(2);
        case 4: return VD_KV(4);
        case 8: return VD_KV(8);
        default: return nullptr;
        }
#undef VD_KV
    }
#define VD_K(g)                                                                                \
    (self ? (mode == MODE_F32 ? (const void *)attn_kernel<g, MODE_F32, true>                  \
                              : (const void *)attn_kernel<g, MODE_BF16, true>)                \
          : (mode == MODE_F32 ? (const void *)attn_kernel<g, MODE_F32, false>                 \
                              : (const void *)attn_kernel<g, MODE_BF16, false>))
    switch (G) {
    case 1: return VD_K(1);
    case 2: return VD_K(2);
    case 4: return VD_K(4);
    case 8: return VD_K(8);
    case 16: return VD_K(16);
    default: return nullptr;
    }
#undef VD_K
}

int log2_pow2(int x)
{
    int l = 0;
    while ((1 << l) < x)
        ++l;
    return l;
}

// Resident attention workgroups per (device, G, mode, HW), queried once: the
// occupancy query costs more host time than a small step's kernels.  0 means
// not queried yet; concurrent first calls store the same value.
std::atomic<int> g_resident[kMaxDevices][5][3][3];

// The self-planned prologue keeps the tile prefix of up to kMaxSeqs requests
// (padded) in the result-entry space of one wave (the smallest case: G = 16).
static_assert((kDeferEntries / 16) * (16 * kHeadDim * 4 + 16 * 8 + 2 * 4) >=
                  4 * (kMaxSeqs + 1 + ((kMaxSeqs + 1) >> kPrePad) + 1),
              "request prefix does not fit the attention kernel's LDS");

// Dynamic LDS of an attention workgroup: per wave, kDeferEntries / G piece
// results of G x head_dim floats, their (max, normaliser) pairs and a
// {whole, target} pair each.  The gather keeps nothing in LDS.
size_t attn_lds_bytes(int G, int mode, int HW)
{
    if (mode == MODE_GATHER)
        return 0;
    const size_t entries = (size_t)HW * (kDeferEntries / G);
    return entries * ((size_t)G * kHeadDim * sizeof(float) + G * sizeof(float2) + 2 * sizeof(int));
}

// Workgroups of the attention kernel (HW waves each) that fit on the device
// at once, at most kAttnWavesPerCU waves per CU.
int resident_attn_groups(int G, int mode, int HW, int *groups)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VD_ERROR_LAUNCH;
    const int gi = log2_pow2(G), hwi = log2_pow2(HW);
    std::atomic<int> *slot = (dev >= 0 && dev < kMaxDevices && gi < 5 && mode < 3 && hwi < 3)
                                 ? &g_resident[dev][gi][mode][hwi]
                                 : nullptr;
    if (slot) {
        const int v = slot->load(std::memory_order_relaxed);
        if (v > 0) {
            *groups = v;
            return VD_SUCCESS;
        }
    }
    int cus = 0;
    int st = num_cus(&cus);
    if (st)
        return st;
    // planned and self-planned kernels of both score paths must agree on R
    // (it sets the ranges)
    int per_cu = kAttnWavesPerCU;
    for (int v = 0; v < 4; ++v) {
        const bool self = v & 1, valu = v & 2;
        if ((mode == MODE_GATHER && (self || valu)) || (valu && !valu_score(G, 0)))
            continue;
        const void *k = attn_kernel_ptr(G, mode, self, valu);
        if (!k)
            return VD_ERROR_NOT_SUPPORTED;
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, 64 * HW,
                                                         attn_lds_bytes(G, mode, HW)) != hipSuccess ||
            n <= 0)
            return VD_ERROR_LAUNCH;
        per_cu = std::min(per_cu, n);
    }
    *groups = std::min(cus * std::min(per_cu, std::max(1, kAttnWavesPerCU / HW)), kMaxResidentGroups);
    if (slot)
        slot->store(*groups, std::memory_order_relaxed);
    return VD_SUCCESS;
}

int enqueue_plan(const int32_t *seq_lens, int num_seqs, int G, int n_kv_heads,
                 int max_pages_per_seq, void *workspace, unsigned flags, int mode,
                 hipStream_t stream)
{
    const int HW = heads_per_group(n_kv_heads);
    int groups = 0;
    int st = resident_attn_groups(G, mode, HW, &groups);
    if (st)
        return st;
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_tiles(flags));
    const int shrt = short_plan(num_seqs, n_kv_heads / HW, max_pages_per_seq, groups,
                                forced_tiles(flags)) ? 1 : 0;
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, seq_lens, num_seqs,
                       n_kv_heads / HW, max_pages_per_seq, forced_tiles(flags), groups, shrt,
                       (char *)workspace, lay);
    return launch_status();
}

int enqueue_attn(const AttnArgs &args, int G, int mode, bool self, bool valu, hipStream_t stream)
{
    int groups = 0;
    int st = resident_attn_groups(G, mode, args.HW, &groups);
    if (st)
        return st;
    const void *k = attn_kernel_ptr(G, mode, self, valu);
    if (!k)
        return VD_ERROR_NOT_SUPPORTED;
    AttnArgs copy = args;
    copy.resident = groups;
    copy.shrt = short_plan(args.B, args.Hkv / args.HW, args.maxp, groups, args.forced) ? 1 : 0;
    copy.zero_empty = copy.shrt && args.zero_empty;
    void *params[] = {(void *)&copy};
    if (hipLaunchKernel(k, dim3(groups), dim3(64 * args.HW), params,
                        attn_lds_bytes(G, mode, args.HW), stream) != hipSuccess)
        return VD_ERROR_LAUNCH;
    return launch_status();
}

AttnArgs make_args(const WsLayout &lay, void *workspace, int num_seqs, int n_q_heads,
                   int n_kv_heads, int max_pages_per_seq, float scale, unsigned flags)
{
    char *ws = (char *)workspace;
    AttnArgs a{};
    a.hdr = (PlanHeader *)(ws + lay.hdr);
    a.ranges = (const int4 *)(ws + lay.ranges);
    a.bounds = (int4 *)(ws + lay.bounds);
    a.empty = (int *)(ws + lay.empty);
    a.tok_base = (const long long *)(ws + lay.tok_base);
    a.part_ml = (float2 *)(ws + lay.part_ml);
    a.part_acc = (float *)(ws + lay.part_acc);
    a.Hq = n_q_heads;
    a.Hkv = n_kv_heads;
    a.HW = heads_per_group(n_kv_heads);
    a.pt_stride = max_pages_per_seq;
    a.maxp = max_pages_per_seq;
    a.B = num_seqs;
    a.forced = forced_tiles(flags);
    a.scale_log2 = scale * kLog2e;
    return a;
}

// Combine kernel over the workspace's header, boundary records and list of
// requests without tokens.
int enqueue_combine(void *out, int num_seqs, int n_q_heads, int n_kv_heads, const WsLayout &lay,
                    void *workspace, unsigned flags, hipStream_t stream)
{
    char *ws = (char *)workspace;
    CombineArgs c;
    c.out = out;
    c.hdr = (const PlanHeader *)(ws + lay.hdr);
    c.bounds = (const int4 *)(ws + lay.bounds);
    c.empty = (const int *)(ws + lay.empty);
    c.part_ml = (const float2 *)(ws + lay.part_ml);
    c.part_acc = (const float *)(ws + lay.part_acc);
    c.Hq = n_q_heads;
    c.Hkv = n_kv_heads;
    c.G = n_q_heads / n_kv_heads;
    c.HW = heads_per_group(n_kv_heads);
    c.cap = (int)lay.cap;
    int cus = 0;
    const int st = num_cus(&cus);
    if (st)
        return st;
    // work items: fewer than one per range plus one per request
    const long long items = lay.cap + (long long)num_seqs;
    const dim3 grid((unsigned)std::min<long long>((long long)cus * kCombineGroupsPerCU, items));
    c.grid = (int)grid.x;
    if (flags & VD_FLAG_OUT_F32)
        hipLaunchKernelGGL(combine_kernel<MODE_F32>, grid, dim3(kCombineThreads), 0, stream, c);
    else
        hipLaunchKernelGGL(combine_kernel<MODE_BF16>, grid, dim3(kCombineThreads), 0, stream, c);
    return launch_status();
}

// Sizes, flags, data pointers and scale of an attention call.
int check_attn_inputs(const void *q, const void *k_pages, const void *v_pages,
                      const int32_t *page_table, const int32_t *seq_lens, const void *out,
                      int num_seqs, int n_q_heads, int n_kv_heads, int head_dim, int page_size,
                      float scale, int max_pages_per_seq, unsigned flags)
{
    int st = check_shapes(num_seqs, n_q_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, flags);
    if (st)
        return st;
    if (!q || !k_pages || !v_pages || !page_table || !seq_lens || !out)
        return VD_ERROR_INVALID_VALUE;
    if (!aligned(q, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(out, 16) ||
        !aligned(page_table, 4) || !aligned(seq_lens, 4))
        return VD_ERROR_INVALID_VALUE;
    if (!std::isfinite(scale))
        return VD_ERROR_INVALID_VALUE;
    return VD_SUCCESS;
}

// The same and the caller's workspace.
int check_attn_args(const void *q, const void *k_pages, const void *v_pages,
                    const int32_t *page_table, const int32_t *seq_lens, const void *out,
                    int num_seqs, int n_q_heads, int n_kv_heads, int head_dim, int page_size,
                    float scale, int max_pages_per_seq, const void *workspace,
                    size_t workspace_bytes, unsigned flags)
{
    int st = check_attn_inputs(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs,
                               n_q_heads, n_kv_heads, head_dim, page_size, scale,
                               max_pages_per_seq, flags);
    if (st)
        return st;
    if (!workspace || !aligned(workspace, 16))
        return VD_ERROR_INVALID_VALUE;
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads,
                                   max_pages_per_seq, forced_tiles(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    return VD_SUCCESS;
}

int out_mode(unsigned flags) { return (flags & VD_FLAG_OUT_F32) ? MODE_F32 : MODE_BF16; }

// The attention kernel on checked arguments: planned (after the planner
// kernel) or self-planned.
int enqueue_partial(const void *q, const void *k_pages, const void *v_pages,
                    const int32_t *page_table, const int32_t *seq_lens, void *out, int num_seqs,
                    int n_q_heads, int n_kv_heads, float scale, int max_pages_per_seq,
                    const WsLayout &lay, void *workspace, unsigned flags, bool self,
                    bool zero_empty, hipStream_t stream)
{
    const int G = n_q_heads / n_kv_heads;
    AttnArgs a = make_args(lay, workspace, num_seqs, n_q_heads, n_kv_heads, max_pages_per_seq,
                           scale, flags);
    a.q = (const uint16_t *)q;
    a.k = (const uint16_t *)k_pages;
    a.v = (const uint16_t *)v_pages;
    a.pt = page_table;
    a.seq_lens = seq_lens;
    a.out = out;
    a.zero_empty = zero_empty ? 1 : 0;
    return enqueue_attn(a, G, out_mode(flags), self, valu_score(G, flags), stream);
}

// The whole step: the self-planned attention kernel, then the combine kernel
// unless the plan is short (no segment cut, so nothing to merge; the
// attention kernel then writes the empty requests' zeros itself).
int enqueue_step(const void *q, const void *k_pages, const void *v_pages,
                 const int32_t *page_table, const int32_t *seq_lens, void *out, int num_seqs,
                 int n_q_heads, int n_kv_heads, float scale, int max_pages_per_seq,
                 const WsLayout &lay, void *workspace, unsigned flags, hipStream_t stream)
{
    const int G = n_q_heads / n_kv_heads, HW = heads_per_group(n_kv_heads);
    int groups = 0;
    int st = resident_attn_groups(G, out_mode(flags), HW, &groups);
    if (st)
        return st;
    const bool shrt = short_plan(num_seqs, n_kv_heads / HW, max_pages_per_seq, groups,
                                 forced_tiles(flags));
    st = enqueue_partial(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs, n_q_heads,
                         n_kv_heads, scale, max_pages_per_seq, lay, workspace, flags, true, shrt,
                         stream);
    if (st || shrt)
        return st;
    return enqueue_combine(out, num_seqs, n_q_heads, n_kv_heads, lay, workspace, flags, stream);
}

// ---------------------------------------------------------------- fixed scratch
// The workspace of vd_decode_attn_noalloc: one array per device, part of the
// library's code object, so that entry point allocates nothing.  Host code
// never uses the array's name as an address (on the host it is a stand-in
// symbol): its device address is looked up once per device, with that device
// current, and every kernel argument is taken from there.
constexpr size_t kNoAllocScratchBytes = (size_t)VD_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

std::atomic<char *> g_scratch[kMaxDevices];

int noalloc_scratch(char **out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VD_ERROR_LAUNCH;
    if (dev >= 0 && dev < kMaxDevices) {
        char *p = g_scratch[dev].load(std::memory_order_acquire);
        if (p) {
            *out = p;
            return VD_SUCCESS;
        }
    }
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
        (void)hipGetLastError();   // leave no sticky error for the caller's next call
        return VD_ERROR_LAUNCH;
    }
    if (dev >= 0 && dev < kMaxDevices)   // concurrent first calls store the same address
        g_scratch[dev].store((char *)p, std::memory_order_release);
    *out = (char *)p;
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
    case VD_ERROR_SCRATCH_LIMIT: return "VD_ERROR_SCRATCH_LIMIT";
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
                     forced_tiles(flags)).total;
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
    const int G = n_q_heads / n_kv_heads;
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_tiles(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    if (num_seqs == 0)
        return VD_SUCCESS;
    return enqueue_plan(seq_lens, num_seqs, G, n_kv_heads, max_pages_per_seq, workspace, flags,
                        out_mode(flags), stream);
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
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads, max_pages_per_seq,
                                   forced_tiles(flags));
    return enqueue_partial(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs, n_q_heads,
                           n_kv_heads, scale, max_pages_per_seq, lay, workspace, flags,
                           (flags & VD_FLAG_SELF_PLAN) != 0, false, stream);
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
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_tiles(flags));
    if (workspace_bytes < lay.total)
        return VD_ERROR_WORKSPACE_TOO_SMALL;
    if (num_seqs == 0)
        return VD_SUCCESS;
    return enqueue_combine(out, num_seqs, n_q_heads, n_kv_heads, lay, workspace, flags, stream);
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
    const WsLayout lay = ws_layout(num_seqs, n_q_heads / n_kv_heads, n_kv_heads, max_pages_per_seq,
                                   forced_tiles(flags));
    return enqueue_step(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs, n_q_heads,
                        n_kv_heads, scale, max_pages_per_seq, lay, workspace, flags, stream);
}

int vd_decode_attn_noalloc(const void *q, const void *k_pages, const void *v_pages,
                           const int32_t *page_table, const int32_t *seq_lens, void *out,
                           int num_seqs, int n_q_heads, int n_kv_heads, int head_dim,
                           int page_size, float scale, int max_pages_per_seq, unsigned flags,
                           hipStream_t stream)
{
    // the checks of vd_decode_attn but the workspace's: the fixed scratch
    // replaces it, sized below
    int st = check_attn_inputs(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs,
                               n_q_heads, n_kv_heads, head_dim, page_size, scale,
                               max_pages_per_seq, flags);
    if (st)
        return st;
    if (num_seqs == 0)
        return VD_SUCCESS;
    const int G = n_q_heads / n_kv_heads;
    int groups = 0;
    st = resident_attn_groups(G, out_mode(flags), heads_per_group(n_kv_heads), &groups);
    if (st)
        return st;
    const WsLayout lay = ws_layout(num_seqs, G, n_kv_heads, max_pages_per_seq, forced_tiles(flags),
                                   groups);
    if (lay.total > kNoAllocScratchBytes)
        return VD_ERROR_SCRATCH_LIMIT;
    char *ws = nullptr;
    st = noalloc_scratch(&ws);
    if (st)
        return st;
    return enqueue_step(q, k_pages, v_pages, page_table, seq_lens, out, num_seqs, n_q_heads,
                        n_kv_heads, scale, max_pages_per_seq, lay, ws, flags, stream);
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
    st = enqueue_plan(seq_lens, num_seqs, 1, n_kv_heads, max_pages_per_seq, workspace, 0,
                      MODE_GATHER, stream);
    if (st)
        return st;
    AttnArgs a = make_args(lay, workspace, num_seqs, n_kv_heads, n_kv_heads, max_pages_per_seq,
                           1.0f, 0);
    a.k = (const uint16_t *)k_pages;
    a.v = (const uint16_t *)v_pages;
    a.pt = page_table;
    a.seq_lens = seq_lens;
    a.out = k_out;
    a.out2 = v_out;
    return enqueue_attn(a, 1, MODE_GATHER, false, false, stream);
}

int vd_kv_append(const void *k_new, const void *v_new, void *k_pages, void *v_pages,
                 const int32_t *page_table, const int32_t *positions, int num_seqs,
                 int n_kv_heads, int head_dim, int page_size, int max_pages_per_seq,
                 hipStream_t stream)
{
    int st = check_shapes(num_seqs, n_kv_heads, n_kv_heads, head_dim, page_size,
                          max_pages_per_seq, 0);
    if (st)
        return st;
    if (!k_new || !v_new || !k_pages || !v_pages || !page_table || !positions)
        return VD_ERROR_INVALID_VALUE;
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_pages, 16) ||
        !aligned(v_pages, 16) || !aligned(page_table, 4) || !aligned(positions, 4))
        return VD_ERROR_INVALID_VALUE;
    if (num_seqs == 0)
        return VD_SUCCESS;
    hipLaunchKernelGGL(kv_append_kernel, dim3(num_seqs), dim3(kAppendThreads), 0, stream,
                       (const u32x4 *)k_new, (const u32x4 *)v_new, (u32x4 *)k_pages,
                       (u32x4 *)v_pages, page_table, positions, n_kv_heads, max_pages_per_seq);
    return launch_status();
}

int vd_stream_read(const void *buf, size_t bytes, void *sink, int blocks, hipStream_t stream)
{
    if (!buf || !sink || blocks <= 0 || !aligned(buf, 16) || !aligned(sink, 4) || bytes % 16 != 0)
        return VD_ERROR_INVALID_VALUE;
    if (bytes == 0)
        return VD_SUCCESS;
    // contiguous chunks of whole 16-load batches; no workgroup without data
    const size_t n16 = bytes / 16, batch = (size_t)kStreamUnroll * kStreamThreads;
    const size_t chunk = (n16 + (size_t)blocks - 1) / (size_t)blocks;
    const size_t chunk_b = (chunk + batch - 1) / batch * batch;
    const size_t groups = (n16 + chunk_b - 1) / chunk_b;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)groups), dim3(kStreamThreads), 0, stream,
                       (const u32x4 *)buf, n16, chunk_b, (unsigned *)sink);
    return launch_status();
}

}  // extern "C"
