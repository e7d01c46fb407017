// Top-k per appended token (the selection half of Eq. 1's Idx) over the
// causal candidates [0, M+i] of each score row, exact under the strict order
// (score descending, id ascending).
//
// One 512-thread block per row, two blocks per CU.  A row (up to 557 KB at a
// 128K history) does not fit in LDS, so the block streams it from HBM once,
// keeping only candidates that beat a running threshold in an LDS buffer of
// 8192 (key, id) pairs:
//   1. threshold seed: a strided sample of whole 128-byte lines (1/32 of the
//      row) is radix-selected for a rank a little above k * (sample share), so
//      that in expectation ~1.3k elements pass - one extra read of 3% of the
//      row instead of a second full pass;
//   2. streaming filter: 16 KB per thread-block step in flight, ballot +
//      popcount compaction into the LDS buffer;  whenever the buffer could
//      overflow it is cut to exactly the k best and the threshold is raised to
//      the k-th best (key, id), so the buffer never loses a member of the
//      answer;  if the seed was too high (fewer than k passed), the row is
//      streamed again with no threshold;
//   3. exact selection: 8-bit-digit radix select on the order-preserving
//      score key finds the k-th key; ties on it are resolved by a second radix
//      select on ids (smallest first);
//   4. ordered output: the winners are set in an LDS bitmap over [0, n) and
//      written in ascending id order after a block scan of popcounts.
#include "janus_device.hpp"
#include "janus_host.hpp"

namespace janus {

constexpr int TK_THREADS = 512;
constexpr int TK_WAVES = TK_THREADS / kWave;
constexpr int TK_CAP = 8192;                  // LDS candidate buffer entries
constexpr int TK_STEP = TK_THREADS * 4;       // elements filtered per sub-step
constexpr int TK_UNROLL = 8;                  // float4 loads in flight per thread
constexpr int TK_ITER = TK_STEP * TK_UNROLL;  // elements per streaming iteration
constexpr int TK_MAX_K = TK_CAP - TK_STEP;    // 6144
constexpr int TK_MAX_N = TK_CAP * 64;         // bitmap of the output step: 2^19 ids
constexpr int TK_SAMPLE_LINES = 128;          // ~1/32 of a 128K row, in 32-element lines

struct TopkShared {
    uint32_t key[TK_CAP];
    int32_t id[TK_CAP];
    uint32_t hist[256];
    int32_t wsum[TK_WAVES];
    int32_t count;
    uint32_t sel_v;
    int32_t sel_rem;
    uint32_t thr_key;
    int32_t thr_id;
};

JANUS_DEV uint64_t lanemask_lt() { return (1ull << (threadIdx.x & 63)) - 1ull; }

// Inclusive prefix sum over the block (TK_THREADS values); also returns the total.
JANUS_DEV int block_inclusive_scan(TopkShared &sm, int v, int &total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_up(v, o, 64);
        if (lane >= o)
            v += t;
    }
    if (lane == 63)
        sm.wsum[wave] = v;
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < TK_WAVES; ++w) {
        int s = sm.wsum[w];
        off += (w < wave) ? s : 0;
        tot += s;
    }
    __syncthreads();
    total = tot;
    return v + off;
}

// LDS histogram increment with a fast path when the whole wave hits one bin.
JANUS_DEV void hist_add(uint32_t *hist, bool on, uint32_t bin)
{
    uint64_t act = __ballot(on);
    if (act == 0)
        return;
    uint32_t first = __shfl(bin, __ffsll((unsigned long long)act) - 1, 64);
    uint64_t same = __ballot(on && bin == first);
    if (same == act) {
        if ((threadIdx.x & 63) == (uint32_t)(__ffsll((unsigned long long)act) - 1))
            atomicAdd(&hist[first], (uint32_t)__popcll(act));
        return;
    }
    if (on)
        atomicAdd(&hist[bin], 1u);
}

// Radix select over buffer entries [0, cnt) that satisfy pred(e): returns in
// sm.sel_v the value V (of val(e)) such that fewer than `want` entries have a
// larger value and at least `want` have a value >= V; sm.sel_rem is how many
// entries equal to V are needed to make up `want`.
template <class Val, class Pred>
JANUS_DEV void radix_select(TopkShared &sm, int cnt, int want, Val val, Pred pred)
{
    uint32_t prefix = 0, mask = 0;
    int rem = want;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int t = threadIdx.x; t < 256; t += TK_THREADS)
            sm.hist[t] = 0;
        __syncthreads();
        for (int e0 = 0; e0 < cnt; e0 += TK_THREADS) {
            int e = e0 + threadIdx.x;
            bool on = false;
            uint32_t v = 0;
            if (e < cnt && pred(e)) {
                v = val(e);
                on = (v & mask) == prefix;
            }
            hist_add(sm.hist, on, (v >> shift) & 255u);
        }
        __syncthreads();
        // suffix sums from bin 255 down, on the first 256 threads
        int h = threadIdx.x < 256 ? (int)sm.hist[255 - threadIdx.x] : 0;
        int tot;
        int incl = block_inclusive_scan(sm, h, tot);
        if (threadIdx.x < 256 && incl >= rem && incl - h < rem) {
            sm.sel_v = 255u - threadIdx.x;
            sm.sel_rem = rem - (incl - h);
        }
        __syncthreads();
        prefix |= sm.sel_v << shift;
        mask |= 255u << shift;
        rem = sm.sel_rem;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        sm.sel_v = prefix;
        sm.sel_rem = rem;
    }
    __syncthreads();
}

// Finds the k-th best (key, id) among the cnt buffered candidates:
// returns T (key) and I (the largest id among the winners with key T).
// Winners are exactly: key > T, or key == T and id <= I.
JANUS_DEV void kth_best(TopkShared &sm, int cnt, int k, uint32_t &T, int32_t &I)
{
    radix_select(sm, cnt, k, [&](int e) { return sm.key[e]; }, [&](int) { return true; });
    T = sm.sel_v;
    const int need = sm.sel_rem;  // winners among key == T
    // Ties on T: the `need` smallest ids win; select the largest of ~id.
    const uint32_t Tl = T;
    radix_select(sm, cnt, need, [&](int e) { return ~(uint32_t)sm.id[e]; },
                 [&](int e) { return sm.key[e] == Tl; });
    I = (int32_t)~sm.sel_v;
}

// Keep exactly the k winners in the buffer and raise the threshold to them.
JANUS_DEV void compact(TopkShared &sm, int k)
{
    const int cnt = sm.count;
    uint32_t T;
    int32_t I;
    kth_best(sm, cnt, k, T, I);
    constexpr int PER = TK_CAP / TK_THREADS;
    uint32_t kk[PER];
    int32_t ii[PER];
    uint32_t keep = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int e = threadIdx.x + j * TK_THREADS;
        kk[j] = 0u;
        ii[j] = 0;
        if (e < cnt) {
            kk[j] = sm.key[e];
            ii[j] = sm.id[e];
            if (kk[j] > T || (kk[j] == T && ii[j] <= I))
                keep |= 1u << j;
        }
    }
    const int nk = __popc(keep);
    int tot;
    int pos = block_inclusive_scan(sm, nk, tot) - nk;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (keep & (1u << j)) {
            sm.key[pos] = kk[j];
            sm.id[pos] = ii[j];
            ++pos;
        }
    if (threadIdx.x == 0) {
        sm.count = tot;  // == k
        sm.thr_key = T;
        sm.thr_id = I;
    }
    __syncthreads();
}

// Appends the accepted (key, id) pairs of this thread's up-to-4 elements.
JANUS_DEV void append4(TopkShared &sm, const float v[4], int id0, int nvalid, uint32_t tk, int32_t ti)
{
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int id = id0 + j;
        const uint32_t key = score_key(v[j]);
        const bool acc = j < nvalid && (key > tk || (key == tk && id < ti));
        const uint64_t m = __ballot(acc);
        if (m == 0)
            continue;
        int base = 0;
        if ((threadIdx.x & 63) == 0)
            base = atomicAdd(&sm.count, __popcll(m));
        base = __shfl(base, 0, 64);
        if (acc) {
            const int pos = base + __popcll(m & lanemask_lt());
            sm.key[pos] = key;
            sm.id[pos] = id;
        }
    }
}

// One pass over [0, n) of the row, filtering against the running threshold.
JANUS_DEV void stream_row(TopkShared &sm, const float *__restrict__ row, int n, int k)
{
    // scalar head up to 16-byte alignment, then float4 body, then scalar tail
    const int head = min(n, (int)(((16 - (reinterpret_cast<uintptr_t>(row) & 15)) & 15) >> 2));
    const int nbody4 = (n - head) >> 2;
    const int tail0 = head + (nbody4 << 2);
    {
        if (sm.count + TK_STEP > TK_CAP)
            compact(sm, k);
        float v[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        int nv = 0, id0 = 0;
        if (threadIdx.x == 0) {
            for (int j = 0; j < head; ++j)
                v[j] = row[j];
            nv = head;
            id0 = 0;
        } else if (threadIdx.x == 1) {
            for (int j = 0; j < n - tail0; ++j)
                v[j] = row[tail0 + j];
            nv = n - tail0;
            id0 = tail0;
        }
        append4(sm, v, id0, nv, sm.thr_key, sm.thr_id);
        __syncthreads();
    }
    const v4f *body = reinterpret_cast<const v4f *>(row + head);
    const int niter = (nbody4 * 4 + TK_ITER - 1) / TK_ITER;
    v4f cur[TK_UNROLL];
#pragma unroll
    for (int u = 0; u < TK_UNROLL; ++u) {
        const int v4 = u * TK_THREADS + threadIdx.x;
        cur[u] = v4 < nbody4 ? body[v4] : v4f{0.f, 0.f, 0.f, 0.f};
    }
    for (int it = 0; it < niter; ++it) {
        v4f nxt[TK_UNROLL];
        const int nb = (it + 1) * (TK_ITER / 4);
#pragma unroll
        for (int u = 0; u < TK_UNROLL; ++u) {
            const int v4 = nb + u * TK_THREADS + threadIdx.x;
            nxt[u] = (it + 1 < niter && v4 < nbody4) ? body[v4] : v4f{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < TK_UNROLL; ++u) {
            if (sm.count + TK_STEP > TK_CAP)
                compact(sm, k);
            const int v4 = it * (TK_ITER / 4) + u * TK_THREADS + threadIdx.x;
            const int nv = v4 < nbody4 ? 4 : 0;
            float v[4] = {cur[u][0], cur[u][1], cur[u][2], cur[u][3]};
            append4(sm, v, head + 4 * v4, nv, sm.thr_key, sm.thr_id);
            __syncthreads();
        }
#pragma unroll
        for (int u = 0; u < TK_UNROLL; ++u)
            cur[u] = nxt[u];
    }
}

__global__ __launch_bounds__(TK_THREADS, 2) void topk_rows(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len,
    const int64_t *__restrict__ score_start, int num_seqs,
    const float *__restrict__ scores, int k, int32_t *__restrict__ topk_idx)
{
    __shared__ TopkShared sm;
    const int g = blockIdx.x;
    const int b = session_of_row(q_start, num_seqs, g);
    const int i = g - q_start[b];
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = M + N;
    const int n = M + i + 1;
    const float *row = scores + score_start[b] + (int64_t)i * ctx;
    int32_t *out = topk_idx + (int64_t)g * k;

    if (n <= k) {
        for (int j = threadIdx.x; j < k; j += TK_THREADS)
            out[j] = j < n ? j : -1;
        return;
    }
    if (threadIdx.x == 0) {
        sm.count = 0;
        sm.thr_key = 0u;  // accept everything: key > 0, or key == 0 and id < INT_MAX
        sm.thr_id = 0x7fffffff;
    }
    __syncthreads();

    if (n > TK_CAP) {
        // 1. threshold seed from a sample of whole lines
        const int nlines = n >> 5;
        const int stride = max(1, nlines / TK_SAMPLE_LINES);
        const int nsl = min(TK_SAMPLE_LINES, nlines);
        const int m = nsl * 32;
        for (int e = threadIdx.x; e < m; e += TK_THREADS) {
            const int line = (e >> 5) * stride;
            sm.key[e] = score_key(row[(line << 5) + (e & 31)]);
        }
        __syncthreads();
        // rank r of the sample ~ 1.3 * k * (m / n) + 8
        const int r = min(m, (int)(1.3f * (float)k * (float)m / (float)n) + 8);
        radix_select(sm, m, r, [&](int e) { return sm.key[e]; }, [&](int) { return true; });
        if (threadIdx.x == 0) {
            sm.thr_key = sm.sel_v;         // accept key >= seed
            sm.thr_id = 0x7fffffff;
            sm.count = 0;
        }
        __syncthreads();
    }
    // 2. one streaming pass (two if the seed was above the k-th key)
    stream_row(sm, row, n, k);
    if (sm.count < k) {
        __syncthreads();
        if (threadIdx.x == 0) {
            sm.count = 0;
            sm.thr_key = 0u;
            sm.thr_id = 0x7fffffff;
        }
        __syncthreads();
        stream_row(sm, row, n, k);
    }
    // 3. exact k-th best among the buffered candidates
    const int cnt = sm.count;
    uint32_t T;
    int32_t I;
    kth_best(sm, cnt, k, T, I);
    constexpr int PER = TK_CAP / TK_THREADS;
    int32_t win[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int e = threadIdx.x + j * TK_THREADS;
        win[j] = -1;
        if (e < cnt) {
            const uint32_t key = sm.key[e];
            const int32_t id = sm.id[e];
            if (key > T || (key == T && id <= I))
                win[j] = id;
        }
    }
    __syncthreads();
    // 4. ascending output through an LDS bitmap over [0, n)
    uint32_t *bm = sm.key;  // reuse: TK_CAP*2 words (the key and id arrays are contiguous)
    const int nwords = (n + 31) >> 5;
    for (int wd = threadIdx.x; wd < nwords; wd += TK_THREADS)
        bm[wd] = 0u;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (win[j] >= 0)
            atomicOr(&bm[win[j] >> 5], 1u << (win[j] & 31));
    __syncthreads();
    const int wpt = (nwords + TK_THREADS - 1) / TK_THREADS;
    const int w0 = threadIdx.x * wpt;
    int c = 0;
    for (int wd = w0; wd < min(nwords, w0 + wpt); ++wd)
        c += __popc(bm[wd]);
    int tot;
    int pos = block_inclusive_scan(sm, c, tot) - c;
    for (int wd = w0; wd < min(nwords, w0 + wpt); ++wd) {
        uint32_t bits = bm[wd];
        while (bits) {
            const int bit = __ffs(bits) - 1;
            bits &= bits - 1;
            out[pos++] = (wd << 5) + bit;
        }
    }
    for (int j = tot + threadIdx.x; j < k; j += TK_THREADS)
        out[j] = -1;
}

} // namespace janus

using namespace janus;

extern "C" int janus_topk(const janus_batch *bt, const float *scores, int k, int32_t *topk_idx,
                          void *workspace, size_t *workspace_bytes, void *stream)
{
    (void)workspace;
    if (workspace_bytes)
        *workspace_bytes = 0;
    if (!batch_ok(bt) || !bt->score_start || !scores || !topk_idx || k < 1)
        return JANUS_ERR_INVALID_ARG;
    if (k > TK_MAX_K || bt->max_ctx > TK_MAX_N)
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0)
        return JANUS_OK;
    hipLaunchKernelGGL(topk_rows, dim3(bt->total_q), dim3(TK_THREADS), 0, as_stream(stream), bt->q_start,
                       bt->hist_len, bt->score_start, bt->num_seqs, scores, k, topk_idx);
    return launch_status();
}
