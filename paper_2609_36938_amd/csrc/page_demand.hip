// Page demand (the union of the per-token selections, mapped through the page
// table to physical pages), read packing (Sec. 4.3: one read per maximal run
// of selected, physically adjacent pages, split from the low end at max_run)
// and the corrective-read set of Eq. (2) (actual minus predicted pages).
//
// Union: each block takes a contiguous range of query rows, maps every valid
// id to its physical page and sets it in an LDS bitmap (read-before-set, so
// the hot pages that every row selects cost one LDS read, not an atomic);
// the block then ORs its non-empty words into the global bitmap.
// Runs and lists: one 1024-thread block stages the bitmap in LDS (at most
// 64 KB) and walks it there; each thread owns a
// contiguous word range, and block-wide scans give it the page-list offset,
// the run offset, the last unset page before its range (where the run it
// starts in began) and the first unset page after it (where a run ends).
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <algorithm>

namespace janus {

constexpr int PD_THREADS = 256;
constexpr int PD_MAX_BLOCKS = 1024;
constexpr int RUN_THREADS = 1024;
constexpr int RUN_WAVES = RUN_THREADS / kWave;
constexpr int PD_MAX_PAGES = 1 << 19;  // 64 KB LDS bitmap

__global__ void bitmap_zero(uint32_t *__restrict__ bm, int nwords)
{
    int w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w < nwords)
        bm[w] = 0u;
}

__global__ __launch_bounds__(PD_THREADS) void page_union(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs, int es, int total_q,
    const int32_t *__restrict__ topk_idx, int k, const int32_t *__restrict__ page_table, int pt_ld,
    int page_shift, const int32_t *__restrict__ limit, int nwords, uint32_t *__restrict__ bitmap)
{
    extern __shared__ uint32_t sbm[];
    for (int w = threadIdx.x; w < nwords; w += PD_THREADS)
        sbm[w] = 0u;
    __syncthreads();
    const int rows_per = (total_q + gridDim.x - 1) / gridDim.x;
    const int r0 = blockIdx.x * rows_per;
    const int r1 = min(total_q, r0 + rows_per);
    int b = r0 < total_q ? session_of_row(q_start, num_seqs, r0) : 0;
    for (int r = r0; r < r1; ++r) {
        while (r >= q_start[b + 1])
            ++b;
        const int ctx = entries_of(hist_len[b] + (q_start[b + 1] - q_start[b]), es);
        const int lim = min(ctx, limit ? limit[b] : entries_of(hist_len[b], es));
        const int32_t *row = topk_idx + (int64_t)r * k;
        const int32_t *pt = page_table + (int64_t)b * pt_ld;
        for (int j = threadIdx.x; j < k; j += PD_THREADS) {
            const int s = row[j];
            if (s < 0 || s >= lim)
                continue;
            const int p = pt[s >> page_shift];
            const uint32_t bit = 1u << (p & 31);
            if (!(sbm[p >> 5] & bit))
                atomicOr(&sbm[p >> 5], bit);
        }
    }
    __syncthreads();
    for (int w = threadIdx.x; w < nwords; w += PD_THREADS) {
        const uint32_t v = sbm[w];
        if (v && (__atomic_load_n(&bitmap[w], __ATOMIC_RELAXED) & v) != v)
            atomicOr(&bitmap[w], v);
    }
}

struct RunShared {
    int32_t wi[RUN_WAVES];
    int32_t wx[RUN_WAVES];
    int32_t wn[RUN_WAVES];
};

// Block-wide exclusive scans over RUN_THREADS threads: sum, max, and a min
// over the threads after this one.
JANUS_DEV void run_scans(RunShared &sh, int cnt, int lastzero, int firstzero, int &cnt_excl, int &tot,
                         int &lz_before, int &fz_after)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int s = cnt, mx = lastzero, mn = firstzero;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_up(s, o, 64);
        int u = __shfl_up(mx, o, 64);
        int v = __shfl_down(mn, o, 64);
        if (lane >= o) {
            s += t;
            mx = max(mx, u);
        }
        if (lane + o < 64)
            mn = min(mn, v);
    }
    if (lane == 63) {
        sh.wi[wave] = s;
        sh.wx[wave] = mx;
    }
    if (lane == 0)
        sh.wn[wave] = mn;
    __syncthreads();
    int off = 0, mxo = -1, mno = 0x7fffffff, t = 0;
    for (int w = 0; w < RUN_WAVES; ++w) {
        t += sh.wi[w];
        if (w < wave) {
            off += sh.wi[w];
            mxo = max(mxo, sh.wx[w]);
        }
        if (w > wave)
            mno = min(mno, sh.wn[w]);
    }
    __syncthreads();
    // exclusive versions: remove this thread's own contribution
    const int incl_s = s + off;
    cnt_excl = incl_s - cnt;
    tot = t;
    int mx_excl = __shfl_up(mx, 1, 64);
    if (lane == 0)
        mx_excl = -1;
    lz_before = max(mx_excl, mxo);
    int mn_excl = __shfl_down(mn, 1, 64);
    if (lane == 63)
        mn_excl = 0x7fffffff;
    fz_after = min(mn_excl, mno);
}

// Walks the pages of `words` (nbits valid bits): writes the ascending page
// list (if list != NULL), the packed runs, and the two counts.
template <class Words>
JANUS_DEV void emit_list_runs(RunShared &sh, Words words, int nbits, int max_run, int32_t *list,
                              int32_t *runs, int32_t *n_pages_out, int32_t *n_runs_out)
{
    const int nwords = (nbits + 31) >> 5;
    const int wpt = (nwords + RUN_THREADS - 1) / RUN_THREADS;
    const int w0 = min(nwords, threadIdx.x * wpt), w1 = min(nwords, w0 + wpt);
    auto word = [&](int w) -> uint32_t {
        uint32_t v = words(w);
        const int hi = nbits - (w << 5);
        if (hi < 32)
            v &= (1u << hi) - 1u;
        return v;
    };
    // this range: set pages, last and first unset page
    int npages = 0, lastzero = -1, firstzero = 0x7fffffff;
    for (int w = w0; w < w1; ++w) {
        const uint32_t v = word(w);
        npages += __popc(v);
        if (v != 0xffffffffu) {
            if (firstzero == 0x7fffffff)
                firstzero = (w << 5) + __ffs(~v) - 1;
            lastzero = (w << 5) + 31 - __clz(~v);
        }
    }
    int page_off, total_pages, lz_before, fz_after;
    run_scans(sh, npages, lastzero, firstzero, page_off, total_pages, lz_before, fz_after);
    const int end_zero = min(fz_after, nbits);  // first unset page after this range (or nbits)
    // first walk: count run starts
    auto walk = [&](bool emit, int run_pos) -> int {
        int nstart = 0;
        int prev = (w0 << 5) - 1;
        // (p - start of p's run) mod max_run, carried from page to page; the
        // first page of this range may continue a run that began before it
        int rem = -1;
        int pos = page_off;
        for (int w = w0; w < w1; ++w) {
            uint32_t v = word(w);
            while (v) {
                const int p = (w << 5) + __ffs(v) - 1;
                v &= v - 1u;
                if (p != prev + 1)
                    rem = 0;
                else if (rem < 0)
                    rem = (p - (lz_before + 1)) % max_run;
                else
                    rem = rem + 1 == max_run ? 0 : rem + 1;
                prev = p;
                if (emit && list)
                    list[pos++] = p;
                if (rem == 0) {
                    if (emit) {
                        // run ends at the first unset page after p
                        int ez = end_zero;
                        for (int w2 = p >> 5; w2 < w1; ++w2) {
                            uint32_t z = ~word(w2);
                            if (w2 == (p >> 5))  // only pages above p
                                z &= ~((2u << (p & 31)) - 1u);
                            if (z) {
                                ez = (w2 << 5) + __ffs(z) - 1;
                                break;
                            }
                        }
                        if (ez > nbits)
                            ez = nbits;
                        runs[2 * (run_pos + nstart)] = p;
                        runs[2 * (run_pos + nstart) + 1] = min(max_run, ez - p);
                    }
                    ++nstart;
                }
            }
        }
        return nstart;
    };
    const int nstart = walk(false, 0);
    int run_off, total_runs, d0, d1;
    run_scans(sh, nstart, -1, 0x7fffffff, run_off, total_runs, d0, d1);
    walk(true, run_off);
    if (threadIdx.x == 0) {
        if (n_pages_out)
            *n_pages_out = total_pages;
        *n_runs_out = total_runs;
    }
}

__global__ __launch_bounds__(RUN_THREADS) void page_list_runs(const uint32_t *__restrict__ bitmap, int nbits,
                                                              int max_run, int32_t *__restrict__ list,
                                                              int32_t *__restrict__ runs, int32_t *__restrict__ counts)
{
    __shared__ RunShared sh;
    extern __shared__ uint32_t sw[];  // the bitmap's words
    const int nwords = (nbits + 31) >> 5;
    for (int w = threadIdx.x; w < nwords; w += RUN_THREADS)
        sw[w] = bitmap[w];
    __syncthreads();
    emit_list_runs(sh, [&](int w) { return sw[w]; }, nbits, max_run, list, runs, counts, counts + 1);
}

__global__ __launch_bounds__(RUN_THREADS) void predict_diff_kernel(
    const uint32_t *__restrict__ actual, const uint32_t *__restrict__ predicted, int nbits, int max_run,
    uint32_t *__restrict__ miss, int32_t *__restrict__ miss_runs, int32_t *__restrict__ counts)
{
    __shared__ RunShared sh;
    __shared__ int32_t red[3][RUN_WAVES];
    extern __shared__ uint32_t sw[];  // the miss set's words
    const int nwords = (nbits + 31) >> 5;
    int ca = 0, cp = 0, cap = 0;
    for (int w = threadIdx.x; w < nwords; w += RUN_THREADS) {
        uint32_t a = actual[w], p = predicted[w];
        const int hi = nbits - (w << 5);
        if (hi < 32) {
            a &= (1u << hi) - 1u;
            p &= (1u << hi) - 1u;
        }
        ca += __popc(a);
        cp += __popc(p);
        cap += __popc(a & p);
        miss[w] = a & ~p;
        sw[w] = a & ~p;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        ca += __shfl_xor(ca, o, 64);
        cp += __shfl_xor(cp, o, 64);
        cap += __shfl_xor(cap, o, 64);
    }
    if (lane == 0) {
        red[0][wave] = ca;
        red[1][wave] = cp;
        red[2][wave] = cap;
    }
    __syncthreads();  // also orders the staged miss words before the run walk reads them
    if (threadIdx.x == 0) {
        int a = 0, p = 0, ap = 0;
        for (int w = 0; w < RUN_WAVES; ++w) {
            a += red[0][w];
            p += red[1][w];
            ap += red[2][w];
        }
        counts[0] = a;
        counts[1] = p;
        counts[2] = ap;
        counts[3] = a - ap;
    }
    emit_list_runs(sh, [&](int w) { return sw[w]; }, nbits, max_run, nullptr, miss_runs, nullptr, counts + 4);
}

} // namespace janus

using namespace janus;

extern "C" int janus_page_demand(const janus_batch *bt, const int32_t *topk_idx, int k,
                                 const int32_t *page_table, int pt_ld, int page_size, const int32_t *limit,
                                 int num_phys_pages, int max_run, uint32_t *bitmap, int32_t *page_list,
                                 int32_t *runs, int32_t *counts, void *workspace, size_t *workspace_bytes,
                                 void *stream)
{
    (void)workspace;
    if (workspace_bytes)
        *workspace_bytes = 0;
    if (!batch_ok(bt) || !topk_idx || !page_table || !bitmap || !page_list || !runs || !counts || k < 1 ||
        pt_ld < 1 || !pow2(page_size) || !table_covers(bt, pt_ld, page_size) || num_phys_pages < 0 || max_run < 1)
        return JANUS_ERR_INVALID_ARG;
    if (num_phys_pages > PD_MAX_PAGES)
        return JANUS_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    const int nwords = (num_phys_pages + 31) >> 5;
    if (nwords > 0)
        hipLaunchKernelGGL(bitmap_zero, dim3(ceil_div(nwords, 256)), dim3(256), 0, st, bitmap, nwords);
    if (bt->total_q > 0 && nwords > 0) {
        const int64_t entries = (int64_t)bt->total_q * k;
        const int nblk = (int)std::min<int64_t>(std::min<int64_t>(PD_MAX_BLOCKS, bt->total_q),
                                                std::max<int64_t>(1, entries / (PD_THREADS * 16)));
        const int shift = __builtin_ctz((unsigned)page_size);
        hipLaunchKernelGGL(page_union, dim3(nblk), dim3(PD_THREADS), nwords * sizeof(uint32_t), st, bt->q_start,
                           bt->hist_len, bt->num_seqs, bt->entry_shift, bt->total_q, topk_idx, k, page_table, pt_ld,
                           shift, limit,
                           nwords, bitmap);
    }
    hipLaunchKernelGGL(page_list_runs, dim3(1), dim3(RUN_THREADS), std::max(nwords, 1) * sizeof(uint32_t), st, bitmap,
                       num_phys_pages, max_run, page_list, runs, counts);
    return launch_status();
}

extern "C" int janus_predict_diff(const uint32_t *actual, const uint32_t *predicted, int num_phys_pages,
                                  int max_run, uint32_t *miss, int32_t *miss_runs, int32_t *counts, void *stream)
{
    if (!actual || !predicted || !miss || !miss_runs || !counts || num_phys_pages < 0 || max_run < 1)
        return JANUS_ERR_INVALID_ARG;
    if (num_phys_pages > PD_MAX_PAGES)
        return JANUS_ERR_UNSUPPORTED;
    const int nwords = (num_phys_pages + 31) >> 5;
    hipLaunchKernelGGL(predict_diff_kernel, dim3(1), dim3(RUN_THREADS), std::max(nwords, 1) * sizeof(uint32_t),
                       as_stream(stream), actual, predicted, num_phys_pages, max_run, miss, miss_runs, counts);
    return launch_status();
}
