/*
 * Plain CPU oracle for the sparse-selection hot path of append prefill.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this file's library.  It shares no
 * code, header, table or helper with the HIP library: every value here is
 * computed from the definitions, in double precision for floating point, with
 * scalar loops and no blocking.  OpenMP splits independent query rows only.
 *
 * Sources (section / equation of the paper):
 *   - selection of k history tokens per appended token by an indexer: Eq. (1),
 *     Sec. "Sparse Attention", prefill phase; appended tokens' own indexer keys
 *     are candidates too (same passage).  The indexer's formula is not printed
 *     in the paper (it defers to the model's technical report); the reading used
 *     is the lightning-indexer form: per query token t, heads h with weights
 *     w[t,h] >= 0, one indexer key per token shared by all heads,
 *         S[t,s] = sq[t] * sk[s] * sum_h w[t,h] * max(0, q[t,h,:] . kI[s,:]),
 *     over candidates s in [0, M+t] (self included); later positions are -inf.
 *   - union of the per-token selections loaded before attention: same
 *     section, the paragraph after Eq. (1).
 *   - predicted union and corrective reads S \ S_hat: Eq. (2) and the
 *     paragraph after it, Sec. "KV Selection Prediction"; recall and precision
 *     as defined under "Model-aligned prediction distance".
 *   - synchronization-free parallel prediction over history shards: Eq. (3),
 *     same section.
 *   - FP4 indexer keys (Sec. "Experiments", models: DeepSeek-V4 keeps its
 *     indexer keys in FP4), read as OCP MXFP4: e2m1 elements with one E8M0
 *     scale per 32 elements.
 *   - the decode phase as an append prefill with one appended token
 *     (Sec. "Decode phase"): the same functions with one row per session.
 *   - read packing: maximal runs of selected, physically adjacent blocks,
 *     address-ordered, never including unselected blocks: Sec. "Best-effort
 *     read packing".  Runs are additionally split from their low end into
 *     pieces of at most max_run pages.
 *   - sparse attention over the selected tokens only: the paragraph after
 *     Eq. (1) (KV of the selected tokens feed core attention); KV states kept
 *     in FP8 (Sec. "Experiments", models), read as e4m3 with one fp32 scale
 *     per cached row.
 *   - entry granularity (Sec. "Sparse Attention", footnote on DeepSeek-V4;
 *     the notation table applies unchanged): a candidate is an entry, one
 *     cached row standing for E consecutive tokens, E*j .. E*j + E - 1, which
 *     a token can select once the entry's last token precedes or is itself.
 *     Every function takes E (tokens per entry; 1 = token granularity) and
 *     counts ids, key rows and score columns in entries.
 *
 * Every function returns 0 on success and a negative value on bad arguments.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define JO_F32 0
#define JO_BF16 1
#define JO_FP8 2

/* OCP fp8 e4m3fn: 1 sign, 4 exponent bits (bias 7), 3 mantissa bits.
 * Exponent field 0 is subnormal (m * 2^-9); S.1111.111 is NaN; no infinities. */
double jo_fp8_e4m3fn_value(uint8_t b)
{
    int sign = (b >> 7) & 1;
    int e = (b >> 3) & 15;
    int m = b & 7;
    double v;
    if (e == 15 && m == 7)
        return NAN;
    if (e == 0)
        v = ldexp((double)m, -9);
    else
        v = ldexp(1.0 + m / 8.0, e - 7);
    return sign ? -v : v;
}

/* bf16: the upper 16 bits of an IEEE binary32 value. */
double jo_bf16_value(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double elem(const void *base, int dt, int64_t i)
{
    switch (dt) {
    case JO_F32: return (double)((const float *)base)[i];
    case JO_BF16: return jo_bf16_value(((const uint16_t *)base)[i]);
    default: return jo_fp8_e4m3fn_value(((const uint8_t *)base)[i]);
    }
}

/* Session of a global query row: q_start is the prefix sum of new lengths. */
static int session_of(int nseq, const int32_t *q_start, int row)
{
    int b = 0;
    while (b + 1 < nseq && q_start[b + 1] <= row)
        b++;
    return b;
}

/* Entry j (tokens E*j .. E*j+E-1) is a candidate at position p when its
 * last token is at or before p. */
static int entry_complete(int64_t j, int E, int64_t p)
{
    return (int64_t)E * j + (E - 1) <= p;
}

/* Entries whose whole region lies within the first n tokens. */
static int64_t whole_entries(int64_t n, int E)
{
    return n / E;
}

/* First key row of session b: the entries of the sessions before it. */
static int64_t key_base(const int32_t *q_start, const int32_t *hist_len, int b, int E)
{
    int64_t base = 0;
    for (int j = 0; j < b; j++)
        base += whole_entries((int64_t)hist_len[j] + (q_start[j + 1] - q_start[j]), E);
    return base;
}

/*
 * Indexer scores for a subset of query rows.
 * q [total_q, H, d] (dtype q_dt), q_scale [total_q] or NULL (= 1);
 * kI [total_ctx, d] (dtype k_dt), one row per token or entry; rows of session
 * b start after the earlier sessions' rows; k_scale [total_ctx] or NULL;
 * w [total_q, H].  out[r * out_ld + s] for s < out_ld: the score of candidate
 * s, -inf for ids the token cannot select yet (tokens: beyond M_b + i) and
 * beyond the session's rows.
 */
/*
 * OCP MX FP4 (e2m1): sign, two exponent bits (bias 1), one mantissa bit; an
 * exponent field of 0 is the subnormal m * 2^-1.  No infinities or NaN.
 */
double jo_e2m1_value(uint8_t code)
{
    const int s = (code >> 3) & 1, e = (code >> 1) & 3, m = code & 1;
    const double v = e == 0 ? 0.5 * m : (1.0 + 0.5 * m) * ldexp(1.0, e - 1);
    return s ? -v : v;
}

/* OCP MX E8M0 shared scale: 2^(e - 127); 255 is NaN. */
double jo_e8m0_value(uint8_t e)
{
    return e == 255 ? NAN : ldexp(1.0, (int)e - 127);
}

/*
 * Element j of key row `row` in MXFP4 (DeepSeek-V4 stores indexer keys in
 * FP4; read as OCP MXFP4): d/2 bytes per key, element j in the low nibble of
 * byte j/2 when j is even and the high nibble when odd, times the E8M0 scale
 * of its 32-element block (d/32 scale bytes per key).
 */
static double mxfp4_elem(const uint8_t *k, const uint8_t *bscale, int64_t row, int d, int j)
{
    const uint8_t byte = k[row * (d / 2) + j / 2];
    const uint8_t code = (j & 1) ? (uint8_t)(byte >> 4) : (uint8_t)(byte & 15);
    return jo_e2m1_value(code) * jo_e8m0_value(bscale[row * (d / 32) + j / 32]);
}

static int index_scores_impl(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                             const void *q, int q_dt, const float *q_scale,
                             const void *kI, int k_dt, const uint8_t *k_bscale, const float *k_scale,
                             const float *w, int H, int d,
                             int nrows, const int32_t *rows, double *out, int64_t out_ld);

int jo_index_scores(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                    const void *q, int q_dt, const float *q_scale,
                    const void *kI, int k_dt, const float *k_scale,
                    const float *w, int H, int d,
                    int nrows, const int32_t *rows, double *out, int64_t out_ld)
{
    return index_scores_impl(nseq, q_start, hist_len, E, q, q_dt, q_scale, kI, k_dt, NULL, k_scale, w, H, d,
                             nrows, rows, out, out_ld);
}

/* Eq. 1's scores with MXFP4 indexer keys (kI: [ctx rows][d/2] bytes, k_bscale: [ctx rows][d/32] E8M0). */
int jo_index_scores_mxfp4(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                          const void *q, int q_dt, const float *q_scale,
                          const uint8_t *kI, const uint8_t *k_bscale, const float *k_scale,
                          const float *w, int H, int d,
                          int nrows, const int32_t *rows, double *out, int64_t out_ld)
{
    if (!k_bscale || d % 32 != 0)
        return -1;
    return index_scores_impl(nseq, q_start, hist_len, E, q, q_dt, q_scale, kI, -1, k_bscale, k_scale, w, H, d,
                             nrows, rows, out, out_ld);
}

static int index_scores_impl(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                             const void *q, int q_dt, const float *q_scale,
                             const void *kI, int k_dt, const uint8_t *k_bscale, const float *k_scale,
                             const float *w, int H, int d,
                             int nrows, const int32_t *rows, double *out, int64_t out_ld)
{
    if (nseq < 1 || H < 1 || d < 1 || nrows < 0 || E < 1)
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
        int g = rows[r];
        if (g < 0 || g >= q_start[nseq]) {
            bad = 1;
            continue;
        }
        int b = session_of(nseq, q_start, g);
        int i = g - q_start[b];
        int64_t M = hist_len[b];
        int64_t ctx = whole_entries(M + (q_start[b + 1] - q_start[b]), E);
        int64_t kb = key_base(q_start, hist_len, b, E);
        double sq = q_scale ? (double)q_scale[g] : 1.0;
        double *qd = (double *)malloc(sizeof(double) * (size_t)H * d);
        for (int64_t e = 0; e < (int64_t)H * d; e++)
            qd[e] = elem(q, q_dt, (int64_t)g * H * d + e);
        double *kd = (double *)malloc(sizeof(double) * (size_t)d);
        for (int64_t s = 0; s < out_ld; s++) {
            if (!entry_complete(s, E, M + i) || s >= ctx) {
                out[(int64_t)r * out_ld + s] = -INFINITY;
                continue;
            }
            for (int j = 0; j < d; j++)
                kd[j] = k_bscale ? mxfp4_elem((const uint8_t *)kI, k_bscale, kb + s, d, j)
                                 : elem(kI, k_dt, (kb + s) * d + j);
            double acc = 0.0;
            for (int h = 0; h < H; h++) {
                double x = 0.0;
                for (int j = 0; j < d; j++)
                    x += qd[(int64_t)h * d + j] * kd[j];
                double relu = x > 0.0 ? x : 0.0;
                acc += (double)w[(int64_t)g * H + h] * relu;
            }
            double sk = k_scale ? (double)k_scale[kb + s] : 1.0;
            out[(int64_t)r * out_ld + s] = sq * sk * acc;
        }
        free(kd);
        free(qd);
    }
    return bad ? -2 : 0;
}

typedef struct {
    double v;
    int32_t idx;
} jo_cand;

/* Strict total order: larger score first, then smaller index. */
static int cand_cmp(const void *a, const void *b)
{
    const jo_cand *x = (const jo_cand *)a, *y = (const jo_cand *)b;
    if (x->v > y->v) return -1;
    if (x->v < y->v) return 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

/*
 * Top-k per query row (Eq. 1 selection).  scores[r * ld + s] holds row r's
 * fp32 scores (r indexes the given rows); candidates are the ids s the token
 * at position M_b + i can select (tokens: s in [0, M_b + i]).
 * out[r * k + j]: the selected ids in (score desc, id asc) order, then -1.
 */
int jo_topk(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
            int nrows, const int32_t *rows, const float *scores, int64_t ld,
            int k, int32_t *out)
{
    if (nseq < 1 || k < 1 || nrows < 0 || E < 1)
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
        int g = rows[r];
        if (g < 0 || g >= q_start[nseq]) {
            bad = 1;
            continue;
        }
        int b = session_of(nseq, q_start, g);
        int64_t pos = (int64_t)hist_len[b] + (g - q_start[b]);
        int64_t n = 0; /* candidates form a prefix of the ids */
        while (n < ld && entry_complete(n, E, pos))
            n++;
        jo_cand *c = (jo_cand *)malloc(sizeof(jo_cand) * (size_t)(n > 0 ? n : 1));
        for (int64_t s = 0; s < n; s++) {
            double v = (double)scores[(int64_t)r * ld + s];
            c[s].v = (v == 0.0) ? 0.0 : v; /* -0.0 compares equal to +0.0 */
            c[s].idx = (int32_t)s;
        }
        qsort(c, (size_t)n, sizeof(jo_cand), cand_cmp);
        for (int j = 0; j < k; j++)
            out[(int64_t)r * k + j] = (j < n) ? c[j].idx : -1;
        free(c);
    }
    return bad ? -2 : 0;
}

/*
 * Synchronization-free sharded prediction (Eq. 3, Sec. "KV Selection
 * Prediction", parallel prediction): the history [0, M_b) is split into G
 * contiguous shards C_n of L_b = align * ceil(ceil(M_b / align) / G) tokens
 * (shard n: [n L_b, min(M_b, (n+1) L_b)); align = page size keeps every page
 * in one shard), and each shard selects its own top-(k/G) history tokens per
 * query row, with no exchange between shards.  Only history tokens are
 * candidates (the equation ranges over the shard's history keys).
 * out[r * k + n * (k/G) + j]: shard n's selected ids in (score desc, id asc)
 * order, then -1.  Requires k % G == 0.
 */
int jo_topk_sharded(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                    int nrows, const int32_t *rows, const float *scores, int64_t ld,
                    int k, int G, int align, int32_t *out)
{
    if (nseq < 1 || k < 1 || G < 1 || k % G != 0 || align < 1 || nrows < 0 || E < 1)
        return -1;
    const int kg = k / G;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
        int g = rows[r];
        if (g < 0 || g >= q_start[nseq]) {
            bad = 1;
            continue;
        }
        int b = session_of(nseq, q_start, g);
        int64_t M = 0; /* history ids: entries complete before the append */
        while (M < ld && entry_complete(M, E, (int64_t)hist_len[b] - 1))
            M++;
        int64_t units = (M + align - 1) / align;
        int64_t L = (int64_t)align * ((units + G - 1) / G);
        jo_cand *c = (jo_cand *)malloc(sizeof(jo_cand) * (size_t)(L > 0 ? L : 1));
        for (int n = 0; n < G; n++) {
            int64_t lo = (int64_t)n * L, hi = lo + L;
            if (hi > M)
                hi = M;
            int64_t cnt = hi > lo ? hi - lo : 0;
            for (int64_t s = 0; s < cnt; s++) {
                double v = (double)scores[(int64_t)r * ld + lo + s];
                c[s].v = (v == 0.0) ? 0.0 : v; /* -0.0 compares equal to +0.0 */
                c[s].idx = (int32_t)(lo + s);
            }
            qsort(c, (size_t)cnt, sizeof(jo_cand), cand_cmp);
            for (int j = 0; j < kg; j++)
                out[(int64_t)r * k + (int64_t)n * kg + j] = (j < cnt) ? c[j].idx : -1;
        }
        free(c);
    }
    return bad ? -2 : 0;
}

/*
 * Page-demand set: A = { pt_b[s / page_size] : s selected by any row of
 * session b, 0 <= s < min(limit_b, C_b) }, over a shared physical pool, with
 * C_b the session's ids (tokens: M_b + N_b).
 * topk_idx [total_q, k] session-local ids (others are padding);
 * page_table [nseq, pt_ld]; limit [nseq] or NULL (= the history ids, the
 * entries wholly within the first M_b tokens).
 * bitmap [ceil(P/32)] (bit p%32 of word p/32); list ascending; *count.
 */
int jo_page_demand(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                   const int32_t *topk_idx, int k,
                   const int32_t *page_table, int pt_ld, int page_size,
                   const int32_t *limit, int num_phys_pages,
                   uint32_t *bitmap, int32_t *page_list, int32_t *count)
{
    if (nseq < 1 || k < 1 || page_size < 1 || num_phys_pages < 0 || E < 1)
        return -1;
    int nwords = (num_phys_pages + 31) / 32;
    unsigned char *sel = (unsigned char *)calloc((size_t)num_phys_pages + 1, 1);
    int bad = 0;
    for (int b = 0; b < nseq; b++) {
        int64_t ctx = whole_entries((int64_t)hist_len[b] + (q_start[b + 1] - q_start[b]), E);
        int64_t lim = limit ? limit[b] : whole_entries(hist_len[b], E);
        if (lim > ctx)
            lim = ctx;
        for (int g = q_start[b]; g < q_start[b + 1]; g++) {
            for (int j = 0; j < k; j++) {
                int64_t s = topk_idx[(int64_t)g * k + j];
                if (s < 0 || s >= lim)
                    continue;
                int64_t lp = s / page_size;
                if (lp >= pt_ld) {
                    bad = 1;
                    continue;
                }
                int p = page_table[(int64_t)b * pt_ld + lp];
                if (p < 0 || p >= num_phys_pages) {
                    bad = 1;
                    continue;
                }
                sel[p] = 1;
            }
        }
    }
    int c = 0;
    for (int w = 0; w < nwords; w++)
        bitmap[w] = 0;
    for (int p = 0; p < num_phys_pages; p++) {
        if (sel[p]) {
            bitmap[p / 32] |= 1u << (p % 32);
            page_list[c++] = p;
        }
    }
    *count = c;
    free(sel);
    return bad ? -2 : 0;
}

static int bit_at(const uint32_t *bm, int p)
{
    return (int)((bm[p / 32] >> (p % 32)) & 1u);
}

/*
 * Read packing over a page bitmap: walk pages in ascending address order; a
 * run starts at a set page whose predecessor is unset, or when the current run
 * already has max_run pages; it extends while the next page is set.
 * runs[2j] = start, runs[2j+1] = length.  Returns the number of runs in *n_runs.
 */
int jo_runs(const uint32_t *bitmap, int num_phys_pages, int max_run,
            int32_t *runs, int32_t *n_runs)
{
    if (num_phys_pages < 0 || max_run < 1)
        return -1;
    int n = 0;
    int p = 0;
    while (p < num_phys_pages) {
        if (!bit_at(bitmap, p)) {
            p++;
            continue;
        }
        int start = p;
        int len = 0;
        while (p < num_phys_pages && bit_at(bitmap, p) && len < max_run) {
            len++;
            p++;
        }
        runs[2 * n] = start;
        runs[2 * n + 1] = len;
        n++;
    }
    *n_runs = n;
    return 0;
}

/*
 * Corrective-read set (Eq. 2 and the following paragraph): miss = A minus the
 * predicted set, per page.  counts = {|A|, |P|, |A and P|, |miss|, #miss runs}.
 */
int jo_predict_diff(const uint32_t *actual, const uint32_t *predicted, int num_phys_pages,
                    int max_run, uint32_t *miss, int32_t *miss_runs, int32_t *counts)
{
    if (num_phys_pages < 0 || max_run < 1)
        return -1;
    int nwords = (num_phys_pages + 31) / 32;
    int ca = 0, cp = 0, cap = 0, cm = 0;
    for (int w = 0; w < nwords; w++)
        miss[w] = 0;
    for (int p = 0; p < num_phys_pages; p++) {
        int a = bit_at(actual, p), q = bit_at(predicted, p);
        ca += a;
        cp += q;
        cap += a && q;
        if (a && !q) {
            cm++;
            miss[p / 32] |= 1u << (p % 32);
        }
    }
    int32_t nr = 0;
    jo_runs(miss, num_phys_pages, max_run, miss_runs, &nr);
    counts[0] = ca;
    counts[1] = cp;
    counts[2] = cap;
    counts[3] = cm;
    counts[4] = nr;
    return 0;
}

/*
 * Sparse attention over the selected tokens of each query row.
 * q [nrows, Hq, dqk] bf16: the queries of the given rows, in the given order;
 * K row of session-local token s of session b:
 *   k_pool + ((pt_b[s / page_size] * page_size) + s % page_size) * k_row_stride,
 * its first dqk elements; V row likewise from v_pool, first dv elements (for
 * the latent-KV layout v_pool == k_pool and V is the head of the K row).
 * sel [nrows, k]: row r's selected ids; ids the token cannot select (tokens:
 * outside [0, M_b + i]) are padding.
 * out [nrows, Hq, dv]: softmax_s(scale * q.K_s) weighted sum of V_s;
 * lse [nrows, Hq] (may be NULL): log-sum-exp of the scaled logits.
 * A row with no valid id gives out = 0 and lse = -inf.
 */
static int sparse_attn_impl(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                            int nrows, const int32_t *rows,
                            const uint16_t *q, int Hq, int dqk, int dv,
                            const void *k_pool, const void *v_pool,
                            int64_t k_row_stride, int64_t v_row_stride, int kv_fp8,
                            const int32_t *page_table, int pt_ld, int page_size,
                            const int32_t *sel, int k, double scale,
                            double *out, double *lse);

int jo_sparse_attn(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                   int nrows, const int32_t *rows,
                   const uint16_t *q, int Hq, int dqk, int dv,
                   const uint16_t *k_pool, const uint16_t *v_pool,
                   int64_t k_row_stride, int64_t v_row_stride,
                   const int32_t *page_table, int pt_ld, int page_size,
                   const int32_t *sel, int k, double scale,
                   double *out, double *lse)
{
    return sparse_attn_impl(nseq, q_start, hist_len, E, nrows, rows, q, Hq, dqk, dv, k_pool, v_pool, k_row_stride,
                            v_row_stride, 0, page_table, pt_ld, page_size, sel, k, scale, out, lse);
}

/*
 * The same attention over a KV cache kept in FP8 (Sec. "Experiments",
 * models: KV states are stored in FP8).  MLA layout: a pool row of row_bytes
 * bytes holds 576 e4m3 elements, then the row's fp32 scale at byte 576; it
 * stands for scale * e4m3(byte).  K_s is the whole row, V_s its first 512
 * elements; q [nrows, Hq, 576] bf16, out [nrows, Hq, 512].
 */
int jo_sparse_attn_fp8kv(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                         int nrows, const int32_t *rows,
                         const uint16_t *q, int Hq,
                         const uint8_t *kv_pool, int64_t row_bytes,
                         const int32_t *page_table, int pt_ld, int page_size,
                         const int32_t *sel, int k, double scale,
                         double *out, double *lse)
{
    if (row_bytes < 580)
        return -1;
    return sparse_attn_impl(nseq, q_start, hist_len, E, nrows, rows, q, Hq, 576, 512, kv_pool, kv_pool, row_bytes,
                            row_bytes, 1, page_table, pt_ld, page_size, sel, k, scale, out, lse);
}

/* Element e of pool row `row`: bf16 (row stride in elements), or fp8 e4m3
 * times the fp32 scale stored after the row's 576 elements (stride in bytes). */
static double kv_elem(const void *pool, int64_t row, int64_t stride, int kv_fp8, int e)
{
    if (!kv_fp8)
        return jo_bf16_value(((const uint16_t *)pool)[row * stride + e]);
    const uint8_t *rp = (const uint8_t *)pool + row * stride;
    float sc;
    memcpy(&sc, rp + 576, sizeof sc);
    return jo_fp8_e4m3fn_value(rp[e]) * (double)sc;
}

static int sparse_attn_impl(int nseq, const int32_t *q_start, const int32_t *hist_len, int E,
                            int nrows, const int32_t *rows,
                            const uint16_t *q, int Hq, int dqk, int dv,
                            const void *k_pool, const void *v_pool,
                            int64_t k_row_stride, int64_t v_row_stride, int kv_fp8,
                            const int32_t *page_table, int pt_ld, int page_size,
                            const int32_t *sel, int k, double scale,
                            double *out, double *lse)
{
    if (nseq < 1 || Hq < 1 || dqk < 1 || dv < 1 || k < 1 || page_size < 1 || nrows < 0 || E < 1)
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
        int g = rows[r];
        if (g < 0 || g >= q_start[nseq]) {
            bad = 1;
            continue;
        }
        int b = session_of(nseq, q_start, g);
        int64_t pos = (int64_t)hist_len[b] + (g - q_start[b]); /* the token's position */
        double *logit = (double *)malloc(sizeof(double) * (size_t)k);
        int64_t *krow = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
        int64_t *vrow = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
        int nv = 0;
        for (int j = 0; j < k; j++) {
            int64_t s = sel[(int64_t)r * k + j];
            if (s < 0 || !entry_complete(s, E, pos))
                continue;
            int64_t lp = s / page_size;
            if (lp >= pt_ld) {
                bad = 1;
                continue;
            }
            int64_t phys = page_table[(int64_t)b * pt_ld + lp];
            int64_t slot = phys * page_size + s % page_size;
            krow[nv] = slot;
            vrow[nv] = slot;
            nv++;
        }
        for (int h = 0; h < Hq; h++) {
            const uint16_t *qh = q + ((int64_t)r * Hq + h) * dqk;
            double *o = out + ((int64_t)r * Hq + h) * dv;
            for (int e = 0; e < dv; e++)
                o[e] = 0.0;
            if (nv == 0) {
                if (lse)
                    lse[(int64_t)r * Hq + h] = -INFINITY;
                continue;
            }
            double m = -INFINITY;
            for (int j = 0; j < nv; j++) {
                double x = 0.0;
                for (int e = 0; e < dqk; e++)
                    x += jo_bf16_value(qh[e]) * kv_elem(k_pool, krow[j], k_row_stride, kv_fp8, e);
                logit[j] = scale * x;
                if (logit[j] > m)
                    m = logit[j];
            }
            double denom = 0.0;
            for (int j = 0; j < nv; j++) {
                double p = exp(logit[j] - m);
                denom += p;
                for (int e = 0; e < dv; e++)
                    o[e] += p * kv_elem(v_pool, vrow[j], v_row_stride, kv_fp8, e);
            }
            for (int e = 0; e < dv; e++)
                o[e] /= denom;
            if (lse)
                lse[(int64_t)r * Hq + h] = m + log(denom);
        }
        free(vrow);
        free(krow);
        free(logit);
    }
    return bad ? -2 : 0;
}
