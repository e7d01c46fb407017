// Top-k per appended token (the selection half of Eq. 1's Idx) over the
// causal candidates [0, M+i] of each score row, exact under the strict order
// (score descending, id ascending).
//
// One 512-thread block per row.  A row (up to 557 KB at a 128K history) does
// not fit in LDS, so the block streams it from HBM once, keeping only
// candidates that beat a running threshold in an LDS buffer of CAP (key, id)
// pairs (CAP = 4096 for k <= 2048, two blocks per CU; else 8192):
//   1. threshold seed: a strided sample of whole 128-byte lines (1/32 of a
//      128K row) is radix-selected on its top 16 key bits for a rank a little
//      above k * (sample share), so that in expectation ~1.3k elements pass;
//   2. streaming filter: the row moves in 8 KB stages, one float4 per thread,
//      through a ring of five registers per thread: four stages are in flight
//      while one is filtered, with one LDS-only barrier per stage.  Each wave
//      appends its accepted elements with one LDS atomic.  Slots past the
//      buffer's end are not written; at the next barrier the buffer is cut to
//      exactly the k best, the threshold rises to the k-th best (key, id), and
//      the dropped elements - still in their register - are filtered again,
//      so no member of the answer is ever lost.  If the seed was above the
//      k-th key (fewer than k passed), the row is streamed again with no
//      threshold;
//   3. exact selection: 8-bit-digit radix select on the order-preserving
//      score key finds the k-th key; ties on it are resolved by a second radix
//      select on ids (smallest first) when they exist;
//   4. ordered output: the winners are set in an LDS bitmap over [0, n),
//      turned into ascending ids by a block scan of popcounts and written out
//      through LDS, coalesced.
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <type_traits>

namespace janus {

constexpr int TK_THREADS = 512;
constexpr int TK_WAVES = TK_THREADS / kWave;
constexpr int TK_STAGE4 = TK_THREADS;     // float4 per stage: one per thread
constexpr int TK_RING = 5;                // register ring depth; TK_RING - 1 stages in flight
constexpr int TK_MAX_K = 6144;            // with CAP = 8192: >= 2048 free slots after a cut
constexpr int TK_SMALL_K = 2048;          // with CAP = 4096
constexpr int TK_SAMPLE_LINES = 128;      // ~1/32 of a 128K row, in 32-element lines
constexpr int TK_SAMPLE_PT = TK_SAMPLE_LINES * 32 / TK_THREADS;

// Output step: bitmap words per prefix group, and the group prefix plus the
// staged ids live in `aux` (CAP/4 + max k words).
constexpr int TK_GROUP = 8;
constexpr int tk_max_k(int cap) { return cap <= 4096 ? TK_SMALL_K : TK_MAX_K; }

template <int CAP>
struct TopkShared {
    uint32_t key[CAP];
    int32_t id[CAP];   // directly behind key: the output bitmap spans both
    int32_t aux[2 * CAP / TK_GROUP + tk_max_k(CAP)];
    uint32_t hist[2][256];
    int32_t wsum[TK_WAVES];
    int32_t count;
    uint32_t sel_v;
    int32_t sel_rem;
    int32_t sel_cnt;
    uint32_t thr_key;  // accept (key, id) > (thr_key, thr_id) in the strict order:
    int32_t thr_id;    //   key > thr_key, or key == thr_key and id < thr_id
    float thr_f;       // thr_key as a score (the same test on floats)
};

JANUS_DEV uint64_t lanemask_lt() { return (1ull << (threadIdx.x & 63)) - 1ull; }

// Workgroup barrier that orders LDS only.  __syncthreads() also waits for
// every outstanding global load.
JANUS_DEV void lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Score of an order-preserving key (inverse of score_key).  Keys below that of
// -inf are not scores; they map to -inf, which only makes a threshold looser.
JANUS_DEV float key_score(uint32_t key)
{
    if (key < 0x007fffffu)
        return -INFINITY;
    return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}

// Sets the running threshold (thread 0 only; the caller synchronises).
template <int CAP>
JANUS_DEV void set_threshold(TopkShared<CAP> &sm, uint32_t key, int32_t id)
{
    sm.thr_key = key;
    sm.thr_id = key < 0x007fffffu ? 0x7fffffff : id;
    sm.thr_f = key_score(key);
}

// Wave-uniform buffer resource over [base, base + bytes): loads past the end
// return zeros.
JANUS_DEV __amdgpu_buffer_rsrc_t row_rsrc(const void *base, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    void *p = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// Inclusive prefix sum over the block (TK_THREADS values); also returns the total.
template <int CAP>
JANUS_DEV int block_inclusive_scan(TopkShared<CAP> &sm, int v, int &total)
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
    lds_sync();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < TK_WAVES; ++w) {
        int s = sm.wsum[w];
        off += (w < wave) ? s : 0;
        tot += s;
    }
    lds_sync();
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

// Radix select over buffer entries [0, cnt) that satisfy pred(e), on the
// 8-bit digits of val(e) from the top down to the digit at lo_shift: returns
// in sm.sel_v the prefix V (the value with the lower lo_shift bits cleared)
// such that fewer than `want` entries have a larger prefix and at least `want`
// have a prefix >= V; sm.sel_rem is how many entries with prefix V are needed
// to make up `want`, and sm.sel_cnt how many entries have prefix V.
// Two barriers per digit: the histograms alternate between two buffers (the
// idle one is cleared during the other's pass) and one wave ranks the bins.
template <int CAP, class Val, class Pred>
JANUS_DEV void radix_select(TopkShared<CAP> &sm, int cnt, int want, Val val, Pred pred, int lo_shift = 0)
{
    if (threadIdx.x < 256) {
        sm.hist[0][threadIdx.x] = 0u;
        sm.hist[1][threadIdx.x] = 0u;
    }
    lds_sync();
    uint32_t prefix = 0, mask = 0;
    int rem = want;
    int buf = 0;
    for (int shift = 24; shift >= lo_shift; shift -= 8, buf ^= 1) {
        uint32_t *hist = sm.hist[buf];
        if (threadIdx.x < 256 && shift < 24)
            sm.hist[buf ^ 1][threadIdx.x] = 0u;  // read by the previous pass, used by the next
        for (int e0 = 0; e0 < cnt; e0 += TK_THREADS) {
            int e = e0 + threadIdx.x;
            bool on = false;
            uint32_t v = 0;
            if (e < cnt && pred(e)) {
                v = val(e);
                on = (v & mask) == prefix;
            }
            hist_add(hist, on, (v >> shift) & 255u);
        }
        lds_sync();
        if (threadIdx.x < 64) {
            // lane l holds bins 255-4l .. 252-4l; suffix sums from bin 255 down
            const int l = threadIdx.x;
            int h[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[j] = (int)hist[255 - 4 * l - j];
                sum += h[j];
            }
            int incl = sum;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int t = __shfl_up(incl, o, 64);
                if (l >= o)
                    incl += t;
            }
            int c = incl - sum;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (c < rem && c + h[j] >= rem) {
                    sm.sel_v = (uint32_t)(255 - 4 * l - j);
                    sm.sel_rem = rem - c;
                    sm.sel_cnt = h[j];
                }
                c += h[j];
            }
        }
        lds_sync();
        prefix |= sm.sel_v << shift;
        mask |= 255u << shift;
        rem = sm.sel_rem;
    }
    lds_sync();  // everyone has read sel_* before thread 0 rewrites them
    if (threadIdx.x == 0) {
        sm.sel_v = prefix;
        sm.sel_rem = rem;
    }
    lds_sync();
}

// Finds the k-th best (key, id) among the cnt buffered candidates:
// returns T (key) and I (the largest id among the winners with key T).
// Winners are exactly: key > T, or key == T and id <= I.
template <int CAP>
JANUS_DEV void kth_best(TopkShared<CAP> &sm, int cnt, int k, uint32_t &T, int32_t &I)
{
    radix_select(sm, cnt, k, [&](int e) { return sm.key[e]; }, [&](int) { return true; });
    T = sm.sel_v;
    const int need = sm.sel_rem;  // winners among key == T
    if (need == sm.sel_cnt) {     // all of them: no tie to break
        I = 0x7fffffff;
        lds_sync();
        return;
    }
    // Ties on T: the `need` smallest ids win; select the largest of ~id.
    const uint32_t Tl = T;
    radix_select(sm, cnt, need, [&](int e) { return ~(uint32_t)sm.id[e]; },
                 [&](int e) { return sm.key[e] == Tl; });
    I = (int32_t)~sm.sel_v;
}

// Cuts the buffer to exactly its k best entries, in place and in order, and
// raises the threshold to the k-th best.
template <int CAP>
__device__ __noinline__ void compact(TopkShared<CAP> &sm, int k)
{
    const int cnt = sm.count;
    uint32_t T;
    int32_t I;
    kth_best(sm, cnt, k, T, I);
    int out = 0;
    // chunks of 4 entries per thread: every chunk is read before any of it is
    // overwritten, and its destination ends before the next chunk begins
    for (int c0 = 0; c0 < cnt; c0 += 4 * TK_THREADS) {
        uint32_t kk[4];
        int32_t ii[4];
        uint32_t keep = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = c0 + 4 * threadIdx.x + j;
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
        int pos = out + block_inclusive_scan(sm, nk, tot) - nk;  // its barriers order reads before writes
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (keep & (1u << j)) {
                sm.key[pos] = kk[j];
                sm.id[pos] = ii[j];
                ++pos;
            }
        out += tot;
    }
    if (threadIdx.x == 0) {
        sm.count = out;  // == k
        set_threshold(sm, T, I);
    }
    lds_sync();
}

// Appends this thread's accepted elements among x[0..3] (ids id0..id0+3, those
// flagged in pend) and returns the flags of those that found no slot.
template <int CAP>
JANUS_DEV uint32_t append4(TopkShared<CAP> &sm, v4f x, uint32_t pend, int id0)
{
    const float tf = sm.thr_f;
    uint32_t acc = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        acc |= (x[j] >= tf ? 1u : 0u) << j;
    acc &= pend;
    if (__ballot(acc != 0) == 0)
        return 0u;
    // an element equal to the threshold passes only with a smaller id
    const int32_t ti = sm.thr_id;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (x[j] == tf && id0 + j >= ti)
            acc &= ~(1u << j);
    // wave exclusive prefix of the per-lane counts (<= 4), bit-sliced over ballots
    const int c = __popc(acc);
    int excl = 0, tot = 0;
#pragma unroll
    for (int bit = 0; bit < 3; ++bit) {
        const uint64_t m = __ballot((c >> bit) & 1);
        excl += __popcll(m & lanemask_lt()) << bit;
        tot += __popcll(m) << bit;
    }
    int base = 0;
    if ((threadIdx.x & 63) == 0 && tot > 0)
        base = atomicAdd(&sm.count, tot);
    base = __shfl(base, 0, 64);
    int slot = base + excl;
    uint32_t dropped = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (acc & (1u << j)) {
            if (slot < CAP) {
                sm.key[slot] = score_key(x[j]);
                sm.id[slot] = id0 + j;
            } else {
                dropped |= 1u << j;
            }
            ++slot;
        }
    return dropped;
}

// After a barrier: if some elements of the previous stage found no slot, cut
// the buffer and filter them again (block-uniform loop; rare).
template <int CAP>
JANUS_DEV void recover(TopkShared<CAP> &sm, v4f x, uint32_t pend, int id0, int k)
{
    while (sm.count > CAP) {
        lds_sync();
        if (threadIdx.x == 0)
            sm.count = CAP;  // every slot below the cap was written
        lds_sync();
        compact(sm, k);
        pend = append4(sm, x, pend, id0);
        lds_sync();
    }
}

// One pass over [0, n) of the row, filtering against the running threshold;
// with `seed`, the threshold is first set from a sample of the row.
template <int CAP>
JANUS_DEV void stream_row(TopkShared<CAP> &sm, const float *__restrict__ row, int n, int k, bool seed)
{
    static_assert(TK_RING == 5, "the ring is unrolled by hand");
    // unaligned head (< 4 elements), 16-byte aligned body of float4s, tail (< 4)
    const int head = min(n, (int)(((16 - (reinterpret_cast<uintptr_t>(row) & 15)) & 15) >> 2));
    const int nbody4 = (n - head) >> 2;
    const int tail0 = head + (nbody4 << 2);
    const __amdgpu_buffer_rsrc_t body = row_rsrc(row + head, 16u * (uint32_t)nbody4);
    const int nst = (nbody4 + TK_STAGE4 - 1) / TK_STAGE4;
    // this thread's float4 of stage j (zeros past the body)
    auto load = [&](int j) {
        return __builtin_bit_cast(
            v4f, __builtin_amdgcn_raw_buffer_load_b128(body, 16 * (j * TK_STAGE4 + (int)threadIdx.x), 0, 0));
    };

    // seed sample and the head/tail elements go to registers first, then the
    // first stages are put in flight, then the sample is ranked under them
    const int nlines = n >> 5;
    const int stride = max(1, nlines / TK_SAMPLE_LINES);
    const int m = seed ? min(TK_SAMPLE_LINES, nlines) * 32 : 0;
    float smp[TK_SAMPLE_PT];
#pragma unroll
    for (int j = 0; j < TK_SAMPLE_PT; ++j) {
        const int e = (int)threadIdx.x + j * TK_THREADS;
        smp[j] = e < m ? row[(((e >> 5) * stride) << 5) + (e & 31)] : 0.f;
    }
    // thread 0 takes the head, thread 1 the tail
    const int ht0 = threadIdx.x == 1 ? tail0 : 0;
    const int htn = threadIdx.x == 0 ? head : (threadIdx.x == 1 ? n - tail0 : 0);
    v4f ht;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        ht[j] = j < htn ? row[ht0 + j] : 0.f;

    v4f x0 = load(0), x1 = load(1), x2 = load(2), x3 = load(3), x4;

    if (seed) {
#pragma unroll
        for (int j = 0; j < TK_SAMPLE_PT; ++j) {
            const int e = (int)threadIdx.x + j * TK_THREADS;
            if (e < m)
                sm.key[e] = score_key(smp[j]);
        }
        lds_sync();
        // rank ~ 1.3 * k * (m / n) + 8; two digits suffice, since the seed only
        // has to be at or below the k-th key
        const int r = min(m, (int)(1.3f * (float)k * (float)m / (float)n) + 8);
        radix_select(sm, m, r, [&](int e) { return sm.key[e]; }, [&](int) { return true; }, 16);
        if (threadIdx.x == 0) {
            set_threshold(sm, sm.sel_v, 0x7fffffff);  // accept key >= seed
            sm.count = 0;
        }
        lds_sync();
    }
    append4(sm, ht, (1u << htn) - 1u, ht0);  // at most 8 entries: room is certain

    uint32_t drop = 0;  // previous stage's elements that found no slot
    int drop_id0 = 0;
    // stage j is filtered from ring register cur; prev held stage j-1 and
    // receives stage j+4 once j-1's overflow (if any) is settled
    auto step = [&](v4f &cur, v4f &prev, int j) {
        lds_sync();
        if (sm.count > CAP)
            recover(sm, prev, drop, drop_id0, k);
        prev = load(j + TK_RING - 1);
        const int v4 = j * TK_STAGE4 + (int)threadIdx.x;
        drop_id0 = head + 4 * v4;
        drop = append4(sm, cur, v4 < nbody4 ? 0xfu : 0u, drop_id0);
    };
    // whole turns of the ring (stages past the body are zeros and masked
    // off), so that the loop has one exit and the ring needs no copies
    for (int j = 0; j < nst; j += TK_RING) {
        step(x0, x4, j);
        step(x1, x0, j + 1);
        step(x2, x1, j + 2);
        step(x3, x2, j + 3);
        step(x4, x3, j + 4);
    }
    // the last stage's overflow
    lds_sync();
    if (sm.count > CAP)
        recover(sm, x4, drop, drop_id0, k);
}

template <int CAP>
__global__ __launch_bounds__(TK_THREADS, CAP <= 4096 ? 4 : 2) void topk_rows(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len,
    const int64_t *__restrict__ score_start, int num_seqs, int es,
    const float *__restrict__ scores, int k_row, int32_t *__restrict__ topk_idx, int shards, int align)
{
    __shared__ TopkShared<CAP> sm;
    // causal rows (shards == 0): block g selects k_row of its candidates
    // (tokens: [0, M+i]);
    // sharded rows: block g*shards + n selects k_row/shards of history shard n
    const int g = shards ? blockIdx.x / shards : blockIdx.x;
    const int b = session_of_row(q_start, num_seqs, g);
    const int i = g - q_start[b];
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = entries_of(M + N, es);
    const int Mh = entries_of(M, es);  // history candidates
    int base = 0, n = last_cand(M, i, es) + 1, k = k_row;
    int32_t *out = topk_idx + (int64_t)g * k_row;
    if (shards) {
        const int sh = blockIdx.x - g * shards;
        const int units = (Mh + align - 1) / align;        // pages of the history
        const int L = align * ((units + shards - 1) / shards);  // candidates per shard
        base = min(Mh, sh * L);
        n = min(Mh, base + L) - base;
        k = k_row / shards;
        out += sh * k;
    }
    const float *row = scores + score_start[b] + (int64_t)i * ctx + base;

    if (n <= k) {
        for (int j = threadIdx.x; j < k; j += TK_THREADS)
            out[j] = j < n ? base + j : -1;
        return;
    }
    if (threadIdx.x == 0) {
        sm.count = 0;
        set_threshold(sm, 0u, 0x7fffffff);  // accept everything
    }
    lds_sync();

    // 2. one streaming pass (two if the seed was above the k-th key)
    stream_row(sm, row, n, k, n > CAP);
    if (sm.count < k) {
        lds_sync();
        if (threadIdx.x == 0) {
            sm.count = 0;
            set_threshold(sm, 0u, 0x7fffffff);
        }
        lds_sync();
        stream_row(sm, row, n, k, false);
    }
    // 3. exact k-th best among the buffered candidates
    const int cnt = sm.count;
    uint32_t T;
    int32_t I;
    kth_best(sm, cnt, k, T, I);
    constexpr int PER = CAP / TK_THREADS;
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
    lds_sync();
    // 4. ascending output: the winners are set in an LDS bitmap over [0, n)
    //    (in the key and id arrays); prefix counts per group of TK_GROUP
    //    words give each winner its rank, and the ids are staged by rank in
    //    aux and written out coalesced
    uint32_t *bm = sm.key;
    const int nwords = (n + 31) >> 5;  // <= 2 * CAP (checked by the launcher)
    for (int wd = threadIdx.x; wd < nwords; wd += TK_THREADS)
        bm[wd] = 0u;
    lds_sync();
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (win[j] >= 0)
            atomicOr(&bm[win[j] >> 5], 1u << (win[j] & 31));
    lds_sync();
    constexpr int MAXG = 2 * CAP / TK_GROUP;          // groups of the largest bitmap
    constexpr int GPT = (MAXG + TK_THREADS - 1) / TK_THREADS;
    int32_t *grp = sm.aux;                            // exclusive prefix per group
    int32_t *stage = sm.aux + MAXG;                   // ids by rank
    const int ngroups = (nwords + TK_GROUP - 1) / TK_GROUP;
    int gc[GPT], c = 0;
#pragma unroll
    for (int u = 0; u < GPT; ++u) {
        const int g = threadIdx.x * GPT + u;
        gc[u] = 0;
        if (g < ngroups)
#pragma unroll
            for (int w = 0; w < TK_GROUP; ++w)
                gc[u] += g * TK_GROUP + w < nwords ? __popc(bm[g * TK_GROUP + w]) : 0;
        c += gc[u];
    }
    int tot;
    int pos = block_inclusive_scan(sm, c, tot) - c;
#pragma unroll
    for (int u = 0; u < GPT; ++u) {
        const int g = threadIdx.x * GPT + u;
        if (g < ngroups)
            grp[g] = pos;
        pos += gc[u];
    }
    lds_sync();
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (win[j] >= 0) {
            const int id = win[j], w = id >> 5, g = w / TK_GROUP;
            int r = grp[g] + __popc(bm[w] & ((1u << (id & 31)) - 1u));
            for (int w2 = g * TK_GROUP; w2 < w; ++w2)
                r += __popc(bm[w2]);
            stage[r] = id;
        }
    lds_sync();
    for (int j = threadIdx.x; j < k; j += TK_THREADS)
        out[j] = j < tot ? base + stage[j] : -1;
}

} // namespace janus

using namespace janus;

// Launch over total_q rows (shards == 0) or total_q * shards (row, shard) pairs.
static int launch_topk(const janus_batch *bt, const float *scores, int k, int32_t *topk_idx, int shards,
                       int align, void *stream)
{
    const int kk = shards ? k / shards : k;
    // the output bitmap spans the key and id arrays: max_ctx <= 2 * CAP * 32
    if (kk > TK_MAX_K || bt->max_ctx > 2 * 8192 * 32)
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0)
        return JANUS_OK;
    const dim3 grid((unsigned)bt->total_q * (unsigned)(shards ? shards : 1));
    if (kk <= TK_SMALL_K && bt->max_ctx <= 2 * 4096 * 32)
        hipLaunchKernelGGL(topk_rows<4096>, grid, dim3(TK_THREADS), 0, as_stream(stream), bt->q_start, bt->hist_len,
                           bt->score_start, bt->num_seqs, bt->entry_shift, scores, k, topk_idx, shards, align);
    else
        hipLaunchKernelGGL(topk_rows<8192>, grid, dim3(TK_THREADS), 0, as_stream(stream), bt->q_start, bt->hist_len,
                           bt->score_start, bt->num_seqs, bt->entry_shift, scores, k, topk_idx, shards, align);
    return launch_status();
}

extern "C" int janus_topk(const janus_batch *bt, const float *scores, int k, int32_t *topk_idx,
                          void *workspace, size_t *workspace_bytes, void *stream)
{
    (void)workspace;
    if (workspace_bytes)
        *workspace_bytes = 0;
    if (!batch_ok(bt) || !bt->score_start || !scores || !topk_idx || k < 1)
        return JANUS_ERR_INVALID_ARG;
    return launch_topk(bt, scores, k, topk_idx, 0, 1, stream);
}

extern "C" int janus_topk_sharded(const janus_batch *bt, const float *scores, int k, int num_shards, int align,
                                  int32_t *topk_idx, void *workspace, size_t *workspace_bytes, void *stream)
{
    (void)workspace;
    if (workspace_bytes)
        *workspace_bytes = 0;
    if (!batch_ok(bt) || !bt->score_start || !scores || !topk_idx || k < 1 || num_shards < 1 ||
        k % num_shards != 0 || align < 1)
        return JANUS_ERR_INVALID_ARG;
    return launch_topk(bt, scores, k, topk_idx, num_shards, align, stream);
}
