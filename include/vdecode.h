/*
 * vdecode.h -- libvdecode: batched single-token GQA decode attention over a
 * paged KV cache, for AMD Instinct MI355X (gfx950).
 *
 * The operation.  A decode iteration of a served model attends the newest
 * query token of each of N_req running requests to the N_kv tokens cached for
 * it; the paper models the iteration's attention work and KV-cache reads as
 * growing with N_kv (EcoPred, Sec. 5.4, Eq. pred-itl), with the cache held in
 * fixed-size pages (PagedAttention, Sec. 2.1).  For request b holding L_b
 * cached tokens and query head h (G = n_q_heads / n_kv_heads, g = h / G):
 *     s_t    = scale * <q[b][h], k_t>              for t = 0 .. L_b - 1
 *     out[b][h] = sum_t softmax(s)_t * v_t
 * with k_t, v_t = row (t mod page_size) of physical page
 * page_table[b][t / page_size], KV head g.  L_b = 0 gives out = 0.
 * The result is plain softmax attention: no causal mask (every cached token,
 * the current one included, is attended), no window, no soft-cap.
 *
 * Layouts (row-major, element sizes in brackets):
 *   q          bf16  [num_seqs][n_q_heads][head_dim]
 *   k_pages    bf16  [num_pages][page_size][n_kv_heads][head_dim]
 *   v_pages    bf16  same as k_pages
 *   page_table int32 [num_seqs][max_pages_per_seq]   entries >= ceil(L_b/page_size) unused
 *   seq_lens   int32 [num_seqs]   L_b, cached tokens including the current one
 *   out        bf16 (default) or fp32 (VD_FLAG_OUT_F32) [num_seqs][n_q_heads][head_dim]
 *
 * Supported shapes: head_dim = 128, page_size = 16,
 * G in {1, 2, 4, 8, 16}, 0 <= num_seqs <= 8192, and sizes whose indices fit
 * 32 bits: n_kv_heads * 2048 < 2^30, num_seqs * (max_pages_per_seq + 1) *
 * n_kv_heads < 2^31, num_seqs * max_pages_per_seq * 16 < 2^31 and
 * num_seqs * n_q_heads < 2^31.
 *
 * Conventions for every call:
 *   - Pointers are device pointers owned by the caller; the library never
 *     allocates, frees or synchronises.  Its only global state is a per-device
 *     cache of the compute-unit count and the kernels' occupancy, filled on
 *     first use (atomics), so calls from several threads are safe.
 *     Concurrent calls need distinct workspaces.  out must not alias an
 *     input.  A call enqueues kernel launches only, so it can be captured
 *     into a HIP graph (after one call on the device outside capture).
 *   - q, k_pages, v_pages, out, k_out, v_out and workspace must be 16-byte
 *     aligned; page_table and seq_lens 4-byte aligned.
 *   - Work is enqueued on `stream` and the call returns at once.
 *   - Argument errors are found on the host before anything is enqueued and
 *     return a nonzero vd_status; VD_ERROR_LAUNCH reports a failed launch.
 *   - num_seqs = 0 is valid: the arguments are checked as usual, then the
 *     call returns VD_SUCCESS with nothing enqueued.
 *   - Device-resident data is not validated: 0 <= L_b and every page id a
 *     request uses is a valid page of the pools are preconditions.  L_b larger
 *     than max_pages_per_seq * page_size is clamped to it.
 *   - bf16 inputs are read as stored; arithmetic is fp32; bf16 outputs are
 *     rounded to nearest even.
 */
#ifndef VDECODE_H
#define VDECODE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vd_status {
    VD_SUCCESS = 0,
    VD_ERROR_INVALID_VALUE = 1,       /* NULL pointer, bad size, misalignment, bad flag, non-finite scale */
    VD_ERROR_NOT_SUPPORTED = 2,       /* head_dim, page_size, G, num_seqs or a 32-bit size limit outside the supported set */
    VD_ERROR_WORKSPACE_TOO_SMALL = 3, /* workspace_bytes below vd_decode_workspace_size() */
    VD_ERROR_LAUNCH = 4,              /* a kernel launch failed (hipGetLastError) */
    VD_ERROR_SCRATCH_LIMIT = 5        /* vd_decode_attn_noalloc: the sizes need more than its fixed scratch */
} vd_status;

/* flags */
#define VD_FLAG_OUT_F32 (1u << 0)     /* out is fp32 instead of bf16 */
/* vd_decode_partial plans the step itself, inside the attention kernel, and
 * needs no vd_decode_plan before it; ignored by the other calls
 * (vd_decode_attn always plans this way). */
#define VD_FLAG_SELF_PLAN (1u << 1)
/* Score path.  For G = n_q_heads / n_kv_heads <= 8 the scores Q.K^T are
 * computed on the vector ALU (bf16 pair dot products, then DPP sums across
 * the lanes that hold one token's dimensions); for G = 16, and for any G with
 * this flag, on the matrix cores (an MFMA tile of 16 tokens by the G heads).
 * The rest of the step is the same.  The workspace, the plan and the
 * ranges do not depend on the path.  For measuring the two paths against
 * each other. */
#define VD_FLAG_SCORE_MFMA (1u << 2)
/* bits 8..15: cut the step's (page, KV head) tiles into ranges of this many
 * tiles (1..255) instead of the automatic partition (0).  Changes where the
 * split-K boundaries fall, not the result beyond rounding; for tests.  The
 * workspace must be sized with the same flags. */
#define VD_FLAG_RANGE_SHIFT 8u
#define VD_FLAG_RANGE_MASK (0xFFu << VD_FLAG_RANGE_SHIFT)
#define VD_FLAG_RANGE_TILES(n) (((unsigned)(n) & 0xFFu) << VD_FLAG_RANGE_SHIFT)

/* Human-readable name of a vd_status value; never NULL. */
const char *vd_status_string(int status);

/*
 * Step record.  Every attention launch (vd_decode_attn, vd_decode_partial,
 * vd_decode_gather) leaves one at offset 0 of its workspace: the plan's
 * sizes (from the planner, or from the self-planning kernel's first
 * workgroup), and two device counters that the kernel's first workgroup
 * reads when it starts and when it ends.  The counters
 * give the shader clock the step ran at, the quantity the paper's
 * frequency-latency relation is stated in (Sec. 3.2, Eq. t-alpha-beta):
 *   t_start, t_end      the constant-rate real-time counter (100 MHz on
 *                       MI355X)
 *   clk_start, clk_end  the shader-clock cycle counter
 * Mean shader clock in MHz = (clk_end - clk_start) * 100 / (t_end - t_start).
 * Read it after the call has completed (e.g. hipMemcpyAsync on the same
 * stream); the next call on the workspace overwrites it.
 */
typedef struct vd_step_info {
    int32_t n_ranges;    /* ranges the step's tiles were cut into */
    int32_t n_tiles;     /* (page, KV-head group) tiles */
    int32_t n_empty;     /* requests without tokens */
    int32_t reserved;
    uint64_t t_start, clk_start, t_end, clk_end;
} vd_step_info;

/*
 * Bytes of device workspace a call with these sizes needs: the plan and the
 * split-K partials (per partial and query head: running max, normaliser and
 * an fp32 head_dim accumulator).  Independent of the actual lengths and of
 * the device; grows with num_seqs * max_pages_per_seq * n_kv_heads / 256 for
 * very large caches.
 * `flags` as passed to the attention call: a forced range length
 * (VD_FLAG_RANGE_TILES) can need more room than the automatic plan.  (A size
 * query over the attention sizes alone could not say so; this one takes the
 * call's flags too.)  Returns 0 when the sizes or flags are invalid or
 * unsupported.
 */
size_t vd_decode_workspace_size(int num_seqs, int n_q_heads, int n_kv_heads,
                                int head_dim, int page_size,
                                int max_pages_per_seq, unsigned flags);

/*
 * The whole decode-attention step, enqueued on `stream`: the attention
 * kernel, planning the step itself (vd_decode_partial with
 * VD_FLAG_SELF_PLAN), then the combine kernel (vd_decode_combine).  Tiny
 * steps (every request at most 4 pages, and at most a quarter as many
 * (page, KV-head group) tiles as the device runs attention workgroups at
 * once) are cut into whole requests, leave nothing to merge, and run the
 * attention kernel alone.  The result equals that of the staged calls bit
 * for bit.
 * scale: the softmax scale applied to q.k (1/sqrt(head_dim) for standard
 * attention); must be finite.
 */
int vd_decode_attn(const void *q, const void *k_pages, const void *v_pages,
                   const int32_t *page_table, const int32_t *seq_lens,
                   void *out, int num_seqs, int n_q_heads, int n_kv_heads,
                   int head_dim, int page_size, float scale,
                   int max_pages_per_seq, void *workspace,
                   size_t workspace_bytes, unsigned flags, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid hipMalloc): the whole step
 * of vd_decode_attn, same arguments but no workspace.  Its workspace is a
 * fixed scratch array of VD_NOALLOC_SCRATCH_BYTES inside the library, one per
 * device (held from the device's first call until the process ends), so the
 * call allocates nothing, by any route.  The plan is cut for the device's own
 * number of resident workgroups, as vd_decode_attn's is, so the output equals
 * vd_decode_attn's bit for bit.
 * Limit: sizes whose plan and partials need more than the scratch return
 * VD_ERROR_SCRATCH_LIMIT with nothing enqueued.  The need is about
 * num_seqs * n_q_heads * 512 B plus ~2 KB per range; on MI355X, 256 requests
 * of up to 16384 tokens at 32:8 heads take 14 MB and 1024 of them 51 MB,
 * while 4000 requests at 32 query heads exceed the scratch.
 * Every call on one device shares that device's scratch and leaves its step
 * record (vd_step_info) at the scratch's start: calls that overlap on one
 * device (concurrent streams, host threads) race and must be serialised by
 * the caller, e.g. kept on one stream.  Nothing in the scratch needs to start
 * at zero; each call writes what it reads.  Errors as vd_decode_attn, plus
 * VD_ERROR_SCRATCH_LIMIT; VD_ERROR_LAUNCH also when the scratch's device
 * address cannot be found.
 */
#define VD_NOALLOC_SCRATCH_BYTES (64u << 20)
int vd_decode_attn_noalloc(const void *q, const void *k_pages, const void *v_pages,
                           const int32_t *page_table, const int32_t *seq_lens, void *out,
                           int num_seqs, int n_q_heads, int n_kv_heads, int head_dim,
                           int page_size, float scale, int max_pages_per_seq, unsigned flags,
                           hipStream_t stream);

/*
 * Stage 1 of 3: lay every (page, KV head) tile of the step out in one sequence
 * (request, KV head, page order) and cut it into equal ranges, as many as
 * (or a multiple of) the attention workgroups the device runs at once (one
 * per tile when the step has fewer tiles), so every wave streams the same number of tiles whatever
 * the length mix; write that plan into the workspace.  Depends only
 * on seq_lens and the sizes, so one plan serves every layer of a decode step.
 * Not needed before a vd_decode_partial with VD_FLAG_SELF_PLAN, which cuts
 * the same ranges itself.
 */
int vd_decode_plan(const int32_t *seq_lens, int num_seqs, int n_q_heads,
                   int n_kv_heads, int head_dim, int page_size,
                   int max_pages_per_seq, void *workspace,
                   size_t workspace_bytes, unsigned flags, hipStream_t stream);

/*
 * Stage 2 of 3: attention over every range of the plan in `workspace`.  A
 * (request, KV head) whose tiles fall in one range gets its final output
 * here; the others leave one partial per range they touch in the workspace.
 * Arguments as vd_decode_attn; seq_lens, the sizes and flags must match the
 * plan's.  Several calls may follow one plan (one per layer), each finished
 * by vd_decode_combine before the next reuses the workspace.  With
 * VD_FLAG_SELF_PLAN the kernel plans from seq_lens itself and writes what
 * vd_decode_combine reads; the plan in the workspace is then neither read
 * nor needed.
 */
int vd_decode_partial(const void *q, const void *k_pages, const void *v_pages,
                      const int32_t *page_table, const int32_t *seq_lens,
                      void *out, int num_seqs, int n_q_heads, int n_kv_heads,
                      int head_dim, int page_size, float scale,
                      int max_pages_per_seq, void *workspace,
                      size_t workspace_bytes, unsigned flags,
                      hipStream_t stream);

/*
 * Stage 3 of 3: log-sum-exp merge of the partials of every request that was
 * split, and zeros for requests with L_b = 0.  Sizes and flags as the
 * preceding vd_decode_partial's.
 */
int vd_decode_combine(void *out, int num_seqs, int n_q_heads, int n_kv_heads,
                      int head_dim, int page_size, int max_pages_per_seq,
                      void *workspace, size_t workspace_bytes, unsigned flags,
                      hipStream_t stream);

/*
 * Copy-through check of the gather: plans with the planner kernel, runs the
 * attention kernel's own page-table walk, K/V loads, tail masking and
 * matrix-operand assembly, and writes every cached K and V row it assembled
 * to k_out / v_out (bf16 [sum_b L_b][n_kv_heads][head_dim], requests in order,
 * tokens in logical order) instead of computing attention.  The result must
 * equal a host gather through page_table bit for bit.  Unlike a plain copy
 * it takes a workspace: the planner kernel writes the plan there and the
 * kernel walks it as the attention kernel does.  Workspace as for
 * vd_decode_attn with n_q_heads = n_kv_heads.
 */
int vd_decode_gather(const void *k_pages, const void *v_pages,
                     const int32_t *page_table, const int32_t *seq_lens,
                     void *k_out, void *v_out, int num_seqs, int n_kv_heads,
                     int head_dim, int page_size, int max_pages_per_seq,
                     void *workspace, size_t workspace_bytes,
                     hipStream_t stream);

/*
 * Append the current token of every request to the paged KV cache, the step
 * that precedes attention in a decode iteration (the newest token's K/V are
 * cached before the step attends to all L_b tokens; Sec. 5.4 counts them in
 * N_kv).  For each request b with 0 <= positions[b] < max_pages_per_seq *
 * page_size, copies k_new[b] and v_new[b] (bf16 [num_seqs][n_kv_heads]
 * [head_dim], 16-byte aligned) into row positions[b] mod page_size of page
 * page_table[b][positions[b] / page_size] of k_pages / v_pages (layouts as
 * above); other requests are skipped.  Bit-exact copies.  The page table
 * entry for that position must name a valid page (precondition).  Sizes as
 * vd_decode_gather (head_dim 128, page_size 16).
 */
int vd_kv_append(const void *k_new, const void *v_new, void *k_pages,
                 void *v_pages, const int32_t *page_table,
                 const int32_t *positions, int num_seqs, int n_kv_heads,
                 int head_dim, int page_size, int max_pages_per_seq,
                 hipStream_t stream);

/*
 * Decode-step projection: y[m][n] = sum_k x[m][k] * w[n][k] for the N_req
 * rows of a decode iteration (the GEMM work the paper's decode latency model
 * charges to N_req, Sec. 5.4, Eq. pred-itl; its batch steps, Sec. 3.3).
 *   x  bf16 [M][K], row-major           w  bf16 [N][K] (a linear layer's weight)
 *   y  bf16 (RNE) or fp32 with VD_FLAG_OUT_F32, [M][N]
 * fp32 accumulation.  The tile shape and the number of K slices follow from
 * (M, N, K) alone, so the result is the same on every device and run (fixed
 * reduction order).  Supported: M >= 1, N a multiple of 64, K a multiple of
 * 512, M * N < 2^31.  x, w, y, workspace 16-byte aligned.  The workspace
 * (vd_gemm_workspace_size, same flags) holds fp32 partials when K is split
 * across workgroups; it may be NULL when that size is 0.  Errors as above;
 * VD_ERROR_NOT_SUPPORTED also for a forced tile or slice count that does not
 * fit the sizes.
 * Flags for tests and sweeps (0 = the automatic choice): VD_GEMM_FLAG_TILE(c)
 * forces tile configuration c (0..10: BM x BN = 16x64, 32x64, 48x64, 64x64,
 * 64x128, 128x128, and five tiles whose K stages go straight from memory into
 * LDS, 128x128, 256x128, 256x256, 192x256 and 320x256; BM rows of x, BN of w;
 * BN = 128 needs N % 128 == 0, BN = 256 needs N % 256 == 0),
 * VD_GEMM_FLAG_SLICES_LOG2(l) forces 2^l K slices (l <= 4).
 * These bits mean something else for the attention calls.
 */
#define VD_GEMM_FLAG_TILE_SHIFT 8u
#define VD_GEMM_FLAG_TILE_MASK (0xFu << VD_GEMM_FLAG_TILE_SHIFT)
#define VD_GEMM_FLAG_TILE(c) ((((unsigned)(c) + 1u) & 0xFu) << VD_GEMM_FLAG_TILE_SHIFT)
#define VD_GEMM_FLAG_SLICES_SHIFT 12u
#define VD_GEMM_FLAG_SLICES_MASK (0xFu << VD_GEMM_FLAG_SLICES_SHIFT)
#define VD_GEMM_FLAG_SLICES_LOG2(l) ((((unsigned)(l) + 1u) & 0xFu) << VD_GEMM_FLAG_SLICES_SHIFT)
size_t vd_gemm_workspace_size(int M, int N, int K, unsigned flags);
int vd_gemm_bf16(const void *x, const void *w, void *y, int M, int N, int K,
                 void *workspace, size_t workspace_bytes, unsigned flags,
                 hipStream_t stream);

/*
 * Measurement aid, not part of the attention path: reads `bytes` (a multiple
 * of 16) from device buffer `buf` with 16-byte non-temporal loads, each of at
 * most `blocks` workgroups of 256 threads streaming one contiguous chunk,
 * and may write 4 bytes to device pointer `sink` (so the reads cannot be
 * optimised away).  Timing it gives the HBM read rate this device sustains,
 * the practical ceiling for vd_decode_attn.  buf 16-byte aligned, sink
 * 4-byte aligned, blocks > 0.
 */
int vd_stream_read(const void *buf, size_t bytes, void *sink, int blocks,
                   hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* VDECODE_H */
