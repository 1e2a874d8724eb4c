/*
 * xdit.h -- C ABI of the MI355X (gfx950) DiT attention hot path of xDiT
 * (arXiv 2411.01738): the PipeFusion patch step, the sequence-parallel chunk
 * step and the log-sum-exp merge of chunk partials, as one GPU executes them.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers: every tensor pointer is a DEVICE pointer, owned by the caller, at
 *   least 16-byte aligned, to dense row-major storage.  The library allocates
 *   nothing and keeps no state except a per-thread stream and error message,
 *   the GEMM plans of xdit_stage_step (hipBLASLt's own memory) and the static
 *   scratch array of xdit_chunk_attn_split_noalloc.  The one exception is
 *   xdit_lse_merge's `outs` / `lses`, which are HOST arrays holding `n`
 *   device pointers.
 * Layouts (the paper fixes none; this is the layout a QKV projection emits):
 *   activations  [B, N, H, d]  sequence-major, d contiguous (q, k, v, out,
 *                              fresh_k, fresh_v, merge partials)
 *   K/V buffer   [2, B, N, H, d]  plane 0 = K, plane 1 = V
 *   LSE          [B, H, Nq]    float32, natural log of sum_j exp(s_j) where
 *                              s_j = (q . k_j) / sqrt(d)
 * dtype: XDIT_BF16 or XDIT_F32, the element type of every activation tensor
 *   of a call (LSE is always float32).  bf16 calls compute QK^T and PV on the
 *   matrix cores with float32 accumulation and round the output to nearest
 *   even; f32 calls use float32 products throughout.
 * head_dim: 64, 72 or 128.
 * Softmax scale: always 1/sqrt(head_dim).  Attention is full (no mask).
 * Streams: every call is asynchronous on the stream set by xdit_set_stream
 *   for the calling thread (NULL = the default stream).  Device faults surface
 *   at the caller's next synchronisation.
 * Errors: 0 on success, a negative xdit_status otherwise.  Every argument is
 *   checked before anything is launched, so a rejected call has no side
 *   effects (the K/V buffer is untouched); xdit_last_error() then describes
 *   the problem.  NaN / Inf inputs are not checked and propagate.
 * A pointer may be NULL only where the tensor it stands for has no elements.
 * Tuning (environment, read at every call; results stay within the same
 *   tolerance, only the work decomposition changes): XDIT_ATTN_KERNEL = o2 |
 *   w32 | pp | w64 selects the bf16 attention decomposition, XDIT_ATTN_TILE =
 *   wide | narrow | quad its workgroup shape at head_dim <= 72, and
 *   XDIT_PARTITION = none | balanced the partition of *_split calls made with
 *   splits <= 0.  Unset, the library chooses.
 */
#ifndef XDIT_H
#define XDIT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { XDIT_BF16 = 0, XDIT_F32 = 1 };

/* Upper bound on the number of partials one xdit_lse_merge call accepts. */
#define XDIT_MAX_PARTIALS 64

/* Upper bound on the fresh row ranges of one xdit_patch_attn_ranges call. */
#define XDIT_MAX_RANGES 2

/* Upper bound on the key splits of one *_split call. */
#define XDIT_MAX_SPLITS 16

typedef enum {
    XDIT_OK = 0,
    XDIT_ERR_NULL = -1,        /* a required pointer is NULL                  */
    XDIT_ERR_DTYPE = -2,       /* unknown dtype                               */
    XDIT_ERR_SHAPE = -3,       /* negative or oversized dimension             */
    XDIT_ERR_RANGE = -4,       /* patch slice outside the buffer; bad n       */
    XDIT_ERR_LAYOUT = -5,      /* pointer not 16-byte aligned                 */
    XDIT_ERR_ALIAS = -6,       /* an output overlaps an input it must not     */
    XDIT_ERR_UNSUPPORTED = -7, /* head_dim not in {64, 72, 128}               */
    XDIT_ERR_HIP = -8          /* the HIP runtime refused a launch            */
} xdit_status;

/*
 * PipeFusion patch step (Section 4.1.2; buffer contents per Section 4.1.4).
 *
 * One layer's full-sequence K/V buffer holds, for every row, either fresh K/V
 * of the current diffusion step or stale K/V left by the previous step.  The
 * patch step first overwrites rows [patch_off, patch_off + patch_len) of both
 * planes with this patch's fresh K/V, then computes attention of the patch's
 * queries over all seq_len rows of the updated buffer, so the fresh slice is
 * seen by this call's own attention and by every later call.  Within one
 * diffusion step, calling this for patches 0..M-1 in order leaves patches
 * <= p fresh when patch p runs.
 *
 *   q        [B, patch_len, H, d]   queries of the patch's rows
 *   kv_buf   [2, B, seq_len, H, d]  the layer's K/V buffer; MUTATED in place:
 *                                   afterwards rows [off, off+len) equal
 *                                   fresh_k / fresh_v bit for bit and every
 *                                   other row is unchanged
 *   fresh_k, fresh_v [B, patch_len, H, d]
 *   out      [B, patch_len, H, d]   attention output
 * Requires 0 <= patch_off, 0 <= patch_len, patch_off + patch_len <= seq_len.
 * patch_len = 0 is a no-op.  out must not overlap any input; q, fresh_k and
 * fresh_v must not overlap kv_buf (the buffer is written while they are read).
 */
int xdit_patch_attn(const void* q, void* kv_buf, int64_t patch_off, int64_t patch_len,
                    const void* fresh_k, const void* fresh_v, void* out,
                    int64_t batch, int64_t seq_len, int64_t heads, int64_t head_dim,
                    int32_t dtype);

/*
 * The patch step in its general form (Sections 4.1.2 and 4.1.4): the fresh
 * K/V rows cover up to XDIT_MAX_RANGES disjoint row ranges of the buffer and
 * the queries are rows of their own.  Two uses come from the paper:
 *   - in-context conditioning (Section 4.1.2): the text tokens travel with
 *     patch 0, so that micro-step refreshes the patch's image rows and the
 *     text rows, and its queries are the rows of both;
 *   - hybrid parallelism (Section 4.1.4): a PipeFusion stage stores the K/V
 *     gathered over its sequence-parallel group while its queries are only
 *     the local shard, so every rank's buffer stays identical.
 * First rows [range_off[r], range_off[r] + range_len[r]) of both planes are
 * overwritten with the fresh rows (range 0's rows first, then range 1's),
 * then out = attention(q, updated K, updated V) and, if lse is not NULL, its
 * log-sum-exp.  xdit_patch_attn is the case of one range with q_len equal to
 * its length and no LSE.
 *
 *   q          [B, q_len, H, d]
 *   kv_buf     [2, B, seq_len, H, d]  MUTATED as above
 *   n_ranges   0 .. XDIT_MAX_RANGES; range_off / range_len are HOST arrays of
 *              n_ranges entries, each range inside [0, seq_len), pairwise
 *              disjoint (empty ranges allowed)
 *   fresh_k, fresh_v [B, F, H, d], F = sum of range_len
 *   out        [B, q_len, H, d]
 *   lse        [B, H, q_len] float32, or NULL
 * q_len = 0 performs only the update; F = 0 is plain attention over the
 * buffer.  out and lse must not overlap any input or each other; q and the
 * fresh rows must not overlap kv_buf.
 */
int xdit_patch_attn_ranges(const void* q, int64_t q_len, void* kv_buf, int32_t n_ranges,
                           const int64_t* range_off, const int64_t* range_len, const void* fresh_k,
                           const void* fresh_v, void* out, float* lse, int64_t batch,
                           int64_t seq_len, int64_t heads, int64_t head_dim, int32_t dtype);

/*
 * Sequence-parallel chunk step (Section 4.1.1: SP-Ring computes attention as
 * a parallel FlashAttention over K/V sub-blocks exchanged peer to peer).
 * Attention of q over one K/V chunk, returning the normalised partial output
 * and its log-sum-exp, which xdit_lse_merge combines across chunks.  With the
 * whole sequence as the chunk this is plain full attention.
 *
 *   q    [B, q_len, H, d]
 *   k, v [B, kv_len, H, d]
 *   out  [B, q_len, H, d]
 *   lse  [B, H, q_len] float32, or NULL to skip it
 * kv_len = 0 gives out = 0 and lse = -inf.  q_len = 0 is a no-op.
 * out and lse must not overlap q, k or v (or each other).
 */
int xdit_chunk_attn(const void* q, const void* k, const void* v, void* out, float* lse,
                    int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                    int64_t head_dim, int32_t dtype);

/*
 * Ring step with the merge fused in (Section 4.1.1: SP-Ring accumulates the
 * partial attention of each K/V sub-block it receives).  Attention of q over
 * one K/V chunk is merged into the running output and log-sum-exp of the
 * chunks before it:
 *   L = ln(e^{lse} + e^{lse_c}),  out = e^{lse - L} * out + e^{lse_c - L} * o_c
 * with (o_c, lse_c) this chunk's attention; out and lse are read, then
 * overwritten with the merged state.  A running lse of -inf marks an empty
 * state: its out is ignored (it may hold anything, NaN included), so a ring
 * starts from lse = -inf or from xdit_chunk_attn's result.  After every chunk
 * of the sequence, out and lse equal attention over the whole sequence.
 * Arguments and requirements as for xdit_chunk_attn, except that lse is
 * required.  The running out is stored in the I/O dtype after every step.
 */
int xdit_chunk_attn_accum(const void* q, const void* k, const void* v, void* out, float* lse,
                          int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                          int64_t head_dim, int32_t dtype);

/*
 * Log-sum-exp merge of n chunk partials into attention over the union of the
 * chunks (Section 4.1.1: the sharded computation gives the serial result):
 *   M = max_r lse_r,  L = M + ln sum_r exp(lse_r - M),
 *   out = sum_r exp(lse_r - L) * outs[r]      (float32 arithmetic)
 * A partial with lse = -inf (an empty chunk) has weight 0; if all are -inf,
 * out = 0 and L = -inf.
 *
 *   outs    HOST array of n device pointers, each [B, q_len, H, d] (dtype)
 *   lses    HOST array of n device pointers, each [B, H, q_len] float32
 *   n       1 <= n <= XDIT_MAX_PARTIALS
 *   out     [B, q_len, H, d]; may be exactly outs[r] (in-place), must not
 *           otherwise overlap a partial
 *   lse_out [B, H, q_len] float32 merged L, or NULL; must not overlap lses
 */
int xdit_lse_merge(const void* const* outs, const float* const* lses, int32_t n, void* out,
                   float* lse_out, int64_t batch, int64_t q_len, int64_t heads,
                   int64_t head_dim, int32_t dtype);

/*
 * Key-split forms of xdit_chunk_attn and xdit_patch_attn_ranges, for launches
 * whose query tiles (128 rows each, per batch and head) leave CUs of the 256
 * idle: too few query tiles, or a last round of workgroups that is nearly
 * empty.  The K/V sweep of a query tile is cut into consecutive parts that
 * run as separate workgroups; each part writes its partial output and
 * log-sum-exp (float32) into the workspace, and a fix-up launch combines the
 * parts of each cut sweep by the log-sum-exp merge of Section 4.1.1 (the
 * same arithmetic as xdit_lse_merge) into out and lse.  The results equal
 * the unsplit call's up to float32 rounding of the merge.
 *
 *   splits     1 .. XDIT_MAX_SPLITS, or <= 0 to let the library choose
 *              splits > 1: every sweep is cut into `splits` even parts;
 *              1: the unsplit call;
 *              <= 0: the library's choice from a time model of the launch:
 *              no cut, every sweep cut into s even parts (few query tiles),
 *              or the query tiles of the full rounds of workgroups swept
 *              whole and each of the r left over cut into min(16, 256 / r)
 *              parts (a nearly empty last round); a cut is taken only when
 *              the model saves at least 10 %
 *   workspace  device memory of at least xdit_split_workspace_bytes(...)
 *              bytes for the same sizes and splits, 256-byte aligned, not
 *              overlapping any argument; unused (may be NULL) when no cut
 *              happens.  Its contents on entry do not matter.
 * xdit_split_workspace_bytes returns 0 when the sizes lead to no cut, -1 for
 * sizes or splits the calls reject.  float32 calls, and calls whose sweeps
 * hold one K/V tile or less (128 keys at d <= 72, 64 at d = 128), run
 * unsplit.  Other arguments as for the unsplit calls.  The sweep and the
 * fix-up are two launches on the calling thread's stream.
 * xdit_chunk_attn_accum_split is the same for the ring step
 * xdit_chunk_attn_accum: the fix-up merges each cut sweep's result into the
 * running (out, lse) as the unsplit call does.
 */
int64_t xdit_split_workspace_bytes(int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                                   int64_t head_dim, int32_t dtype, int32_t splits);
int xdit_chunk_attn_split(const void* q, const void* k, const void* v, void* out, float* lse,
                          int32_t splits, void* workspace, int64_t workspace_bytes, int64_t batch,
                          int64_t q_len, int64_t kv_len, int64_t heads, int64_t head_dim,
                          int32_t dtype);
int xdit_chunk_attn_accum_split(const void* q, const void* k, const void* v, void* out, float* lse,
                                int32_t splits, void* workspace, int64_t workspace_bytes,
                                int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                                int64_t head_dim, int32_t dtype);
int xdit_patch_attn_split(const void* q, int64_t q_len, void* kv_buf, int32_t n_ranges,
                          const int64_t* range_off, const int64_t* range_len, const void* fresh_k,
                          const void* fresh_v, void* out, float* lse, int32_t splits,
                          void* workspace, int64_t workspace_bytes, int64_t batch, int64_t seq_len,
                          int64_t heads, int64_t head_dim, int32_t dtype);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation as xdit_chunk_attn_split, with the partial slots of cut sweeps
 * kept in a fixed device array inside the library instead of a caller
 * workspace.  Arguments and results as for xdit_chunk_attn_split without
 * the workspace.
 *   Limit: the partition's slots (xdit_split_workspace_bytes for the same
 *   sizes and splits) must fit in xdit_noalloc_scratch_bytes() bytes
 *   (16 MiB: the Flux 2048px share, 4224 queries over a 4224-key chunk with
 *   24 heads of 128, needs 15.9 MB); larger partitions are rejected with
 *   XDIT_ERR_RANGE before anything is launched.
 *   The array is one per GPU, allocated when the library is loaded onto it
 *   and held until the process ends; its device address is looked up on the
 *   first call on each device.  Every call on a GPU uses that GPU's array:
 *   calls that overlap on one GPU (other streams, other threads) race on it
 *   and must be ordered by the caller.  No call allocates or frees memory.
 */
int xdit_chunk_attn_split_noalloc(const void* q, const void* k, const void* v, void* out, float* lse,
                                  int32_t splits, int64_t batch, int64_t q_len, int64_t kv_len,
                                  int64_t heads, int64_t head_dim, int32_t dtype);
int64_t xdit_noalloc_scratch_bytes(void);

/*
 * The update half of the patch step on its own (Section 4.1.2): copy the
 * fresh K/V rows into rows [patch_off, patch_off + patch_len) of kv_buf,
 * bit for bit, leaving every other row unchanged.  xdit_patch_attn performs
 * the same update itself; this entry point serves callers that fill the
 * buffer without attending (e.g. storing K/V received by SP, Section 4.1.4).
 * Arguments and requirements as for xdit_patch_attn.
 */
int xdit_kv_update(void* kv_buf, int64_t patch_off, int64_t patch_len, const void* fresh_k,
                   const void* fresh_v, int64_t batch, int64_t seq_len, int64_t heads,
                   int64_t head_dim, int32_t dtype);

/*
 * One PipeFusion stage micro-step at one attention layer (Section 4.1.2: a
 * device runs each patch through its stage's layers; Section 3: QKV
 * projections come before self-attention, whose output is projected back):
 *
 *   q = x wq,  k = x wk,  v = x wv      (projections of the patch's rows)
 *   the patch step of xdit_patch_attn with fresh K/V = (k, v), output o
 *   y = o wo
 *
 *   x          [B, patch_len, C]        the patch's hidden states, C = hidden
 *   wq, wk, wv [C, H*d]                 row-major, so q[b, i] = x[b, i] wq
 *   wo         [H*d, C]
 *   kv_buf     [2, B, seq_len, H, d]    MUTATED as by xdit_patch_attn: rows
 *                                       [patch_off, patch_off + patch_len)
 *                                       take k and v bit for bit
 *   q, k, v, o [B, patch_len, H, d]     caller-owned intermediates, written
 *   y          [B, patch_len, C]        output
 * bf16 only (XDIT_ERR_UNSUPPORTED otherwise); the GEMMs (hipBLASLt) and the
 * attention accumulate in float32 and round each result to bf16.  No
 * biases, norms or gates.  No output may overlap another buffer or any
 * input; other requirements as for xdit_patch_attn; 1 <= hidden <= 65536.
 * The library allocates nothing itself; hipBLASLt keeps one handle per
 * device and per-shape plans from the first call on (its own host and
 * device memory).  The first call of each shape times hipBLASLt's candidate
 * algorithms on its own operands and synchronises the calling stream (so it
 * must not run under graph capture); later calls only launch.
 * XDIT_ERR_HIP if hipBLASLt refuses a GEMM.  Five launches on the calling
 * thread's stream.
 */
int xdit_stage_step(const void* x, const void* wq, const void* wk, const void* wv, const void* wo,
                    void* kv_buf, int64_t patch_off, int64_t patch_len, void* q, void* k, void* v,
                    void* o, void* y, int64_t batch, int64_t seq_len, int64_t heads,
                    int64_t head_dim, int64_t hidden, int32_t dtype);

/* Stream for the calling thread's later launches (a hipStream_t; NULL = the
 * default stream).  Always returns XDIT_OK. */
int xdit_set_stream(void* stream);
void* xdit_get_stream(void);

/* Message describing the calling thread's most recent failure ("" if none).
 * Valid until that thread's next call into the library. */
const char* xdit_last_error(void);

/* Library version string. */
const char* xdit_version(void);

#ifdef __cplusplus
}
#endif

#endif /* XDIT_H */
