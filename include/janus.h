/*
 * janus.h - C ABI of the MI355X (gfx950) library for the sparse-selection hot
 * path of append prefill in top-k sparse-attention LLMs.
 *
 * One append prefill of a layer, for a batch of sessions, is
 *
 *   janus_index_scores  indexer relevance of every candidate token   (Eq. 1)
 *   janus_index_scores_mxfp4  the same with MXFP4 (FP4) indexer keys
 *   janus_topk          the k best candidates per appended token     (Eq. 1)
 *   janus_topk_sharded  per-shard top-(k/G) over G history shards    (Eq. 3)
 *   janus_page_demand   union of the selections as a page set, plus
 *                       address-ordered runs of adjacent pages       (union after Eq. 1;
 *                                                                     Sec. 4.3 read packing)
 *   janus_predict_diff  corrective-read set: actual minus predicted  (Eq. 2 and after)
 *   janus_sparse_attn   attention over the selected tokens only      (after Eq. 1)
 *   janus_sparse_attn_split  the same with each row's selection split over
 *                       several blocks, for few rows (decode, Sec. 2.2)
 *   janus_sparse_attn_fp8kv  MLA attention over an FP8 KV cache (Sec. 5.1)
 *
 * Running index_scores + topk + page_demand on a predicted indexer query
 * (an earlier layer's hidden state through this layer's indexer) gives the
 * predicted union of Eq. (2).
 *
 * Conventions shared by every call
 *   - Pointers named "device" are HIP device pointers the caller allocated;
 *     the library never allocates, frees or keeps a pointer after returning.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Every call only enqueues work on it and returns; no call synchronises.
 *   - Outputs are overwritten in full (bitmaps are cleared by the call).
 *   - Host-detectable argument errors return a status and enqueue nothing:
 *     JANUS_ERR_INVALID_ARG for NULL required pointers and out-of-range sizes,
 *     JANUS_ERR_UNSUPPORTED for shapes/dtypes with no kernel,
 *     JANUS_ERR_WORKSPACE for a workspace smaller than required.
 *     A failed launch returns JANUS_ERR_DEVICE; device faults surface at the
 *     caller's next synchronisation.
 *   - Workspace: when a call takes (workspace, workspace_bytes), passing
 *     workspace == NULL stores the required byte count in *workspace_bytes and
 *     returns JANUS_OK without enqueuing anything, also when that count is 0:
 *     to run, pass a non-NULL workspace (any pointer when 0 bytes are needed;
 *     it is then never dereferenced).  The workspace needs no
 *     initialisation.  Calls that share a workspace must not overlap.
 *   - Token ids are session-local: ids 0..M_b-1 are the cached history and
 *     M_b..M_b+N_b-1 the appended tokens.  In id arrays, values outside
 *     [0, M_b+N_b) are padding, like -1.
 *   - Page tables map a session's logical page (id / page_size) to a physical
 *     page of one shared pool; entries must lie in [0, num_phys_pages).  A
 *     table [B, pt_ld] must cover the longest session: pt_ld * page_size >=
 *     max_ctx, else JANUS_ERR_INVALID_ARG (every call that takes one).
 *   - The library is stateless and reentrant.
 */
#ifndef JANUS_H
#define JANUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    JANUS_OK = 0,
    JANUS_ERR_INVALID_ARG = 1,
    JANUS_ERR_UNSUPPORTED = 2,
    JANUS_ERR_WORKSPACE = 3,
    JANUS_ERR_DEVICE = 4
} janus_status;

typedef enum {
    JANUS_F32 = 0,
    JANUS_BF16 = 1,
    JANUS_FP8_E4M3 = 2 /* OCP e4m3fn: bias 7, max 448, no infinities */
} janus_dtype;

/*
 * A ragged batch of B sessions (B = 1 for a single append prefill).  Session b
 * has a cached history of M_b tokens and appends N_b tokens (the P and L of
 * the paper's notation table).  Host fields size grids; device arrays locate
 * rows.  All device arrays are int32 except score_start.
 *
 * Entry granularity (the selection unit of DeepSeek-V4, Sec. 2.2 footnote;
 * the notation table applies to entries unchanged).  With entry_shift = e > 0
 * every candidate is an entry: one cached row (indexer key, KV) standing for
 * the E = 2^e consecutive tokens [E*j, E*j + E - 1], which exists once its
 * last token does.  Then, everywhere below, ids are entry ids and
 *   - session b holds C_b = (M_b + N_b) >> e entries (key rows, score row
 *     length), of which the (M_b >> e) below the append are history (M_b
 *     in the history ranges of topk_sharded and page_demand reads M_b >> e);
 *   - appended token i (position M_b + i) has the candidates
 *     0 .. ((M_b + i + 1) >> e) - 1, the entries complete at its position;
 *   - ctx_start and score_start are prefix sums of C_b and N_b * C_b, and
 *     max_ctx / total_ctx the max / sum of C_b;
 *   - pages hold page_size entries.
 * entry_shift = 0 is token granularity: C_b = M_b + N_b, candidates
 * 0 .. M_b + i.  entry_shift must lie in [0, 16].
 */
typedef struct {
    int32_t num_seqs;            /* B >= 1                                        */
    int32_t total_q;             /* host: sum_b N_b                               */
    int32_t max_q;               /* host: max_b N_b                               */
    int32_t max_ctx;             /* host: max_b C_b (tokens: M_b + N_b)           */
    int64_t total_ctx;           /* host: sum_b C_b                               */
    const int32_t *q_start;      /* device [B+1]: prefix sums of N_b -> rows of
                                    q, w, topk_idx and attention q/out            */
    const int32_t *ctx_start;    /* device [B+1]: prefix sums of C_b -> rows
                                    of the indexer keys and their scales          */
    const int32_t *hist_len;     /* device [B]: M_b                               */
    const int64_t *score_start;  /* device [B+1]: prefix sums of N_b*C_b          */
    int32_t entry_shift;         /* log2 tokens per entry; 0 = token granularity */
} janus_batch;

/*
 * Indexer scores (Eq. 1; the indexer form is the multi-head ReLU-weighted
 * dot product of the lightning indexer, which the paper leaves to the
 * model's report).  For appended token i of session b (absolute position
 * M_b+i) and candidate s in [0, M_b+i]:
 *
 *   S[i,s] = q_scale[i] * k_scale[s] * sum_{h<H} w[i,h] * max(0, sum_{j<d} q[i,h,j] * kI[s,j])
 *
 * Candidates s > M_b+i (later appended tokens) are written as -inf.
 *   q       device [total_q, H, d], dtype q_dt (row-major)
 *   q_scale device [total_q] fp32 (> 0), or NULL for 1
 *   kI      device [total_ctx, d], dtype k_dt; session b's keys start at row
 *           ctx_start[b] (history first, then the appended tokens)
 *   k_scale device [total_ctx] fp32 (> 0), or NULL for 1
 *   w       device [total_q, H] fp32, w >= 0
 *   scores  device fp32; row i of session b starts at
 *           scores + score_start[b] + i*(M_b+N_b) and holds M_b+N_b entries.
 * q_dt must equal k_dt.  fp8 with H = 64 and d = 128 runs on fp8 MFMA (the
 * head weights are applied in bf16: relative error <= 2^-8 per term); every
 * other dtype and shape runs on a plain vector kernel.  Accumulation is fp32.
 */
int janus_index_scores(const janus_batch *b,
                       const void *q, janus_dtype q_dt, const float *q_scale,
                       const void *kI, janus_dtype k_dt, const float *k_scale,
                       const float *w, int H, int d,
                       float *scores, void *stream);

/*
 * The same scores with MXFP4 indexer keys (DeepSeek-V4 keeps its indexer
 * keys in FP4; Sec. 5.1, models), read as OCP MXFP4: each key is d/2 bytes of
 * e2m1 elements (element j in the low nibble of byte j/2 when j is even, the
 * high nibble when odd) and d/32 E8M0 scale bytes, one per 32 elements,
 * element value = e2m1 * 2^(E - 127).
 *   q              device [total_q, H, d] fp8 e4m3fn, q_scale [total_q] or NULL
 *   kI             device [total_ctx, d/2] bytes
 *   k_block_scale  device [total_ctx, d/32] E8M0 bytes
 *   k_scale        device [total_ctx] fp32 or NULL (a per-token factor on top)
 *   w, scores      as for janus_index_scores
 * Products run on the fp8 x fp4 block-scaled MFMA; each head's product is
 * rounded to bf16 and the head weights are applied in bf16 (relative error
 * <= 2^-8 per term).  For batches with more than 4 appended tokens in a
 * session, each key's block scales are taken relative to the largest of its
 * d/32 (exact), except that a block more than 2^127 below that largest one
 * counts as exactly 2^-127 of it.  The E8M0 code 255 (NaN) is not a
 * supported input: such a key's scores are unspecified.  Requires H = 64,
 * d = 128 and contexts up to 2^24 tokens (else JANUS_ERR_UNSUPPORTED; d not a
 * multiple of 32: JANUS_ERR_INVALID_ARG).
 */
int janus_index_scores_mxfp4(const janus_batch *b,
                             const void *q, const float *q_scale,
                             const void *kI, const uint8_t *k_block_scale,
                             const float *k_scale, const float *w, int H, int d,
                             float *scores, void *stream);

/*
 * Top-k per appended token (the selection of Eq. 1): the k largest scores of
 * row i over candidates [0, M_b+i] under the strict order (score descending,
 * id ascending), so ties go to the lower id and -0.0 equals +0.0.  Rows with
 * fewer than k candidates select all of them.
 *   scores    device, laid out as written by janus_index_scores
 *   topk_idx  device [total_q, k] int32: the selected ids in ascending id
 *             order, then -1 padding.
 * Requires 1 <= k <= 6144 and max_ctx <= 2^19 (else JANUS_ERR_UNSUPPORTED).
 * No workspace is needed: pass workspace = NULL with *workspace_bytes set to
 * anything, or query it (always 0).
 */
int janus_topk(const janus_batch *b, const float *scores, int k,
               int32_t *topk_idx, void *workspace, size_t *workspace_bytes,
               void *stream);

/*
 * Synchronization-free sharded prediction (Eq. 3, Sec. 4.2): the history of
 * each session is split into num_shards contiguous shards of
 *   L_b = align * ceil(ceil(M_b / align) / num_shards)
 * tokens (shard n covers [n L_b, min(M_b, (n+1) L_b)); align = the page size
 * keeps every page in one shard), and every shard selects its own top
 * (k / num_shards) history tokens for each appended token, under the same
 * strict order as janus_topk and with no exchange between shards.  Only
 * history tokens are candidates.  One shard is Eq. 2's selection over the
 * history; the union of all shards' selections is what the shards prefetch
 * together (feed topk_idx to janus_page_demand).
 *   scores    device, laid out as written by janus_index_scores
 *   topk_idx  device [total_q, k] int32: slots n*(k/num_shards) ..
 *             (n+1)*(k/num_shards)-1 hold shard n's ids in ascending order,
 *             then -1 padding.
 * Requires num_shards >= 1, k % num_shards == 0 and align >= 1 (else
 * JANUS_ERR_INVALID_ARG), k / num_shards <= 6144 and max_ctx <= 2^19 (else
 * JANUS_ERR_UNSUPPORTED).  No workspace, as for janus_topk.
 */
int janus_topk_sharded(const janus_batch *b, const float *scores, int k,
                       int num_shards, int align, int32_t *topk_idx,
                       void *workspace, size_t *workspace_bytes, void *stream);

/*
 * Page demand (the union of the per-token selections that must be loaded
 * before attention, mapped to pages) and read packing (Sec. 4.3: one read per
 * maximal run of selected, physically adjacent pages; never an unselected
 * page), with runs split from their low end into pieces of at most max_run.
 *
 *   A = { page_table[b, s / page_size] : s in topk_idx rows of session b,
 *                                        0 <= s < min(limit_b, M_b+N_b) }
 *
 *   topk_idx   device [total_q, k] int32 session-local ids (others: padding)
 *   page_table device [B, pt_ld] int32, pt_ld * page_size >= max_ctx
 *   page_size  power of two >= 1
 *   limit      device [B] int32, or NULL for M_b (history pages only: the
 *              appended tokens' KV is produced in HBM and never loaded)
 *   bitmap     device [ceil(num_phys_pages/32)] uint32; page p is bit p%32 of
 *              word p/32
 *   page_list  device [num_phys_pages] int32: the set pages, ascending
 *   runs       device [2*num_phys_pages] int32: (start, length) pairs,
 *              ascending by start
 *   counts     device [2] int32: {number of pages, number of runs}
 * Requires num_phys_pages <= 2^19 (else JANUS_ERR_UNSUPPORTED) and
 * max_run >= 1.
 */
int janus_page_demand(const janus_batch *b, const int32_t *topk_idx, int k,
                      const int32_t *page_table, int pt_ld, int page_size,
                      const int32_t *limit, int num_phys_pages, int max_run,
                      uint32_t *bitmap, int32_t *page_list, int32_t *runs,
                      int32_t *counts, void *workspace, size_t *workspace_bytes,
                      void *stream);

/*
 * Corrective reads (Eq. 2 and the paragraph after it): pages of the actual
 * set A absent from the predicted set P, as a bitmap and as packed runs, with
 * the counts behind recall |A&P|/|A| and precision |A&P|/|P|.
 *   actual, predicted  device [ceil(num_phys_pages/32)] uint32 bitmaps
 *   miss               device [ceil(num_phys_pages/32)] uint32: A & ~P
 *   miss_runs          device [2*num_phys_pages] int32 (start, length) pairs
 *   counts             device [5] int32: {|A|, |P|, |A&P|, |A&~P|, #miss runs}
 * Requires num_phys_pages <= 2^19 (else JANUS_ERR_UNSUPPORTED) and
 * max_run >= 1.
 */
int janus_predict_diff(const uint32_t *actual, const uint32_t *predicted,
                       int num_phys_pages, int max_run,
                       uint32_t *miss, int32_t *miss_runs, int32_t *counts,
                       void *stream);

/*
 * Sparse attention over the selected tokens (the KV of S_t feeds core
 * attention; the paragraph after Eq. 1).  All Hq query heads share one KV
 * head (MQA; MLA in its absorbed form is the case dqk = 576, dv = 512 with V
 * the first 512 elements of each cached 576-element latent+rope row).
 *
 *   out[i,h,:] = sum_{s in S_i} p_s V_s,  p = softmax_s(scale * q[i,h,:] . K_s)
 *   lse[i,h]   = log sum_{s in S_i} exp(scale * q[i,h,:] . K_s)
 *
 * S_i = the ids of row i of topk_idx that lie in [0, M_b+i] (others are
 * padding).  K_s is the first dqk elements of pool row
 * (page_table[b, s/page_size]*page_size + s%page_size) of k_pool, V_s the
 * first dv elements of the same row of v_pool.  page_table is [B, pt_ld]
 * with pt_ld * page_size >= max_ctx.
 *   q       device [total_q, Hq, dqk] bf16
 *   k_pool  device bf16 rows of k_row_stride elements (>= dqk)
 *   v_pool  device bf16 rows of v_row_stride elements (>= dv); may equal k_pool
 *   out     device [total_q, Hq, dv], out_dt JANUS_BF16 or JANUS_F32
 *   lse     device [total_q, Hq] fp32, or NULL
 * A row with no valid id gets out = 0 and lse = -inf.  Softmax and
 * accumulation are fp32; products run on bf16 MFMA for
 *   - MLA: Hq in {16, 32, 64, 128}, dqk = 576, dv = 512, v_pool == k_pool,
 *     k <= 4096;
 *   - MQA: 1 <= Hq <= 16, dqk = dv = 128, k <= 1024 (separate or shared
 *     pools);
 * each with row strides that are multiples of 8 and at most 2^30, and
 * 16-byte aligned q and pools; otherwise on a plain vector kernel
 * (dqk <= 1024, dv <= 1024), else JANUS_ERR_UNSUPPORTED.
 */
int janus_sparse_attn(const janus_batch *b,
                      const void *q, int Hq, int dqk, int dv,
                      const void *k_pool, const void *v_pool,
                      int64_t k_row_stride, int64_t v_row_stride,
                      const int32_t *page_table, int pt_ld, int page_size,
                      const int32_t *topk_idx, int k, float scale,
                      void *out, janus_dtype out_dt, float *lse,
                      void *stream);

/*
 * The same attention with each row's selection split into slices that run
 * as separate blocks, merged afterwards (flash-decoding: every slice keeps
 * its own max and sum, the merge rescales them to the common max).  Meant
 * for few rows - the decode phase (Sec. 2.2: an append prefill with one
 * appended token per session) - where one block per row would leave most of
 * the GPU idle.  Same arguments and result as janus_sparse_attn, up to the
 * order of the fp32 sums, plus:
 *   num_splits       slices per row, 1 .. 16; 0 = one block per compute
 *                    unit of the current device, ceil(CUs / total_q) (at
 *                    most one slice per 32 selected ids either way)
 *   workspace        device scratch of *workspace_bytes bytes, or NULL to
 *                    query the size (written to *workspace_bytes, nothing
 *                    launched): total_q * splits * Hq * 514 * 4 bytes, or 0
 *                    when one slice results (then pass any non-NULL pointer
 *                    to run).  Too small: JANUS_ERR_WORKSPACE.
 * Only the MFMA shape of janus_sparse_attn is supported, and with more than
 * one slice the workspace and out must be 16-byte aligned (else
 * JANUS_ERR_UNSUPPORTED).  Calls on one stream may share a workspace; calls
 * that overlap in time need their own.
 */
int janus_sparse_attn_split(const janus_batch *b,
                            const void *q, int Hq, int dqk, int dv,
                            const void *k_pool, const void *v_pool,
                            int64_t k_row_stride, int64_t v_row_stride,
                            const int32_t *page_table, int pt_ld, int page_size,
                            const int32_t *topk_idx, int k, float softmax_scale,
                            void *out, janus_dtype out_dt, float *lse,
                            int num_splits, void *workspace, size_t *workspace_bytes,
                            void *stream);

/*
 * janus_sparse_attn_split without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same arguments (minus workspace
 * and workspace_bytes), same kernels and the same result as
 * janus_sparse_attn_split with the same num_splits.  The slices' partial
 * results go to a scratch array inside the library instead: one array of
 * JANUS_NOALLOC_SCRATCH_BYTES per GPU the call runs on, held until the
 * process ends, its address looked up on the first call on each device (the
 * call allocates nothing and needs no initialisation).
 *   - A launch needing more than JANUS_NOALLOC_SCRATCH_BYTES
 *     (total_q * splits * Hq * 514 * 4 bytes, 0 for one slice) returns
 *     JANUS_ERR_WORKSPACE and enqueues nothing.  With num_splits = 0 on a GPU
 *     of 256 compute units and Hq <= 128 it always fits.
 *   - Every call on one GPU shares that GPU's array: calls that may overlap
 *     in time on one GPU (different streams, different host threads) race
 *     and must be serialised by the caller.  Calls on one stream are fine.
 *   - With more than one slice, out must be 16-byte aligned.
 */
#define JANUS_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

int janus_sparse_attn_split_noalloc(const janus_batch *b,
                                    const void *q, int Hq, int dqk, int dv,
                                    const void *k_pool, const void *v_pool,
                                    int64_t k_row_stride, int64_t v_row_stride,
                                    const int32_t *page_table, int pt_ld, int page_size,
                                    const int32_t *topk_idx, int k, float softmax_scale,
                                    void *out, janus_dtype out_dt, float *lse,
                                    int num_splits, void *stream);

/*
 * Sparse MLA attention over a KV cache stored in FP8 (Sec. 5.1 keeps KV
 * states in FP8).  The same attention as janus_sparse_attn with dqk = 576
 * and dv = 512, where every cached row is
 *
 *   bytes 0..575    the 576 latent+rope elements, OCP fp8 e4m3fn
 *   bytes 576..579  the row's fp32 scale (> 0, finite)
 *   bytes 580..     unused, up to row_bytes
 *
 * and stands for the values scale * e4m3(byte): K_s is the whole row, V_s its
 * first 512 elements.  The row of id s is pool row
 * page_table[b, s/page_size]*page_size + s%page_size, at kv_pool + that * row_bytes.
 *   q        device [total_q, Hq, 576] bf16, 16-byte aligned; Hq in {16, 32, 64, 128}
 *   kv_pool  device, 16-byte aligned; row_bytes >= 592, a multiple of 16 and
 *            below 2^31
 *   k        <= 4096
 *   out, lse, num_splits, workspace, workspace_bytes: as janus_sparse_attn_split
 *            (num_splits = 1 runs unsplit and needs 0 bytes of workspace, but
 *            workspace == NULL is still a size query that launches nothing:
 *            pass any non-NULL pointer to run)
 * The stored values are exact in bf16: products run on bf16 MFMA, softmax and
 * accumulation in fp32.  Each key's scale multiplies its logit and, before the
 * bf16 rounding of the probabilities, its probability.  Shapes outside the
 * above return JANUS_ERR_UNSUPPORTED (alignment, row_bytes, Hq, k) or
 * JANUS_ERR_INVALID_ARG (row_bytes < 592, NULL pointers).
 */
int janus_sparse_attn_fp8kv(const janus_batch *b,
                            const void *q, int Hq,
                            const uint8_t *kv_pool, int64_t row_bytes,
                            const int32_t *page_table, int pt_ld, int page_size,
                            const int32_t *topk_idx, int k, float softmax_scale,
                            void *out, janus_dtype out_dt, float *lse,
                            int num_splits, void *workspace, size_t *workspace_bytes,
                            void *stream);

/* Static description of a status code. */
const char *janus_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* JANUS_H */
