// Indexer relevance scores (Eq. 1's Idx, lightning-indexer form):
//   S[i,s] = sq[i] * sk[s] * sum_h w[i,h] * max(0, q[i,h,:] . kI[s,:]),  s <= M+i
//
// fp8 path (d = 128): one v_mfma_f32_16x16x128_f8f6f4 covers a whole 128-dim
// dot product, so each MFMA is a 16 (token,head) x 16 key tile and the only
// reduction left is the ReLU-weighted sum over heads, done in the epilogue.
// The 16 MFMA rows are 4 tokens x 4 heads, ordered so that output rows
// 4g..4g+3 of every tile belong to token g: each lane then owns one
// (token, key) score and sums all H heads in registers, with no cross-lane
// reduction.  A wave keeps its 4 tokens' queries (4 x H x 128 fp8) resident
// in VGPRs and streams 16-key operand blocks straight from L2; the column
// of block j is key s0 + 4c + j, so after 4 blocks a lane holds 4 adjacent
// keys and stores them as one 16-byte write (256 contiguous bytes per token).
// Key blocks wholly past every token's causal limit skip the MFMAs.
//
// Epilogue: the MFMA applies an E8M0 scale of 2^-25 to the query operand, so
// every product lands in (-1, 1): |q.k| <= 128 * 448 * 448 < 2^25 for any
// e4m3 inputs.  On that range the clamping form of v_cvt_pk_bf16_f32 (which
// clamps to [0, 1] after rounding to nearest even) is exactly ReLU followed
// by the bf16 rounding, so each pair of outputs costs one convert and one
// v_dot2_f32_bf16 against head weights pre-multiplied by 2^25: 4 VALU ops
// per 16x16x128 MFMA.  The fp8 MFMA and the VALU do not overlap on this
// chip, so VALU ops per MFMA bound the kernel.  Every term is non-negative,
// so the two bf16 roundings bound the relative error of a score by 2^-8.
//
// The clamp modifier cannot be requested from the compiler, so the convert
// is inline assembly; the compiler does not insert the wait states a VALU
// read of an MFMA result needs ahead of inline assembly, so the four MFMAs
// of a group are issued from one assembly block that ends with the wait
// states (12 for an 8-pass fp8 MFMA, what the compiler itself emits) and
// starts with the one a VALU write of an MFMA source needs.
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <algorithm>

namespace janus {

constexpr int IDX_TPW = 2;                          // tokens per wave
constexpr int IDX_WAVES = 4;                        // waves per block
constexpr int IDX_KEY_CHUNK = 2048;                 // keys per block
constexpr int GEN_TOK_TILE = 8;                     // vector kernel: tokens per block
constexpr int GEN_KEY_TILE = 32;                    // vector kernel: keys per block

// Block tile slot -> (session, first session-local token); false past the end.
JANUS_DEV bool tile_slot(const int32_t *q_start, int num_seqs, int slot, int tile, int &b, int &t0)
{
    int acc = 0;
    for (int s = 0; s < num_seqs; ++s) {
        int nt = (q_start[s + 1] - q_start[s] + tile - 1) / tile;
        if (slot < acc + nt) {
            b = s;
            t0 = (slot - acc) * tile;
            return true;
        }
        acc += nt;
    }
    return false;
}

// E8M0 scales of the query (byte 0: 2^-25) and key (byte 1: 2^0) operands,
// one register for both (op_sel picks the byte)
constexpr int IDX_MFMA_SCALES = 0x7f66;

// Four 16x16x128 fp8 MFMAs sharing the key operand, with the query scale
// 2^-25; the results may be read by any instruction after the block.
JANUS_DEV void mfma4_fp8_scaled(v4f &c0, v4f &c1, v4f &c2, v4f &c3, const v8i &a0, const v8i &a1,
                                const v8i &a2, const v8i &a3, const v8i &bk, int scales)
{
    asm("s_nop 1\n\t"
        "v_mfma_scale_f32_16x16x128_f8f6f4 %0, %4, %8, 0, %9, %9 op_sel:[0,1,0] op_sel_hi:[0,0,0]\n\t"
        "v_mfma_scale_f32_16x16x128_f8f6f4 %1, %5, %8, 0, %9, %9 op_sel:[0,1,0] op_sel_hi:[0,0,0]\n\t"
        "v_mfma_scale_f32_16x16x128_f8f6f4 %2, %6, %8, 0, %9, %9 op_sel:[0,1,0] op_sel_hi:[0,0,0]\n\t"
        "v_mfma_scale_f32_16x16x128_f8f6f4 %3, %7, %8, 0, %9, %9 op_sel:[0,1,0] op_sel_hi:[0,0,0]\n\t"
        "s_nop 11"
        : "=&v"(c0), "=&v"(c1), "=&v"(c2), "=&v"(c3)
        : "v"(a0), "v"(a1), "v"(a2), "v"(a3), "v"(bk), "v"(scales));
}

// (min(max(x,0),1), min(max(y,0),1)) rounded to a bf16 pair.
JANUS_DEV v2bf clamp01_bf16x2(float x, float y)
{
    v2bf r;
    asm("v_cvt_pk_bf16_f32 %0, %1, %2 clamp" : "=v"(r) : "v"(x), "v"(y));
    return r;
}

constexpr int IDX_STAGE = 128;                      // keys per LDS stage (16 KB)
constexpr int IDX_XCD = 8;                          // L2 domains (XCDs) of the chip

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt <= n only.
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Wave-uniform buffer resource over [base, base + bytes): stores past
// `bytes` are dropped by the hardware.
JANUS_DEV __amdgpu_buffer_rsrc_t make_buffer_rsrc(void *base, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    void *p = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// Workgroup barrier without a memory fence: LDS hand-offs here are ordered by
// explicit waitcnts, and a fence would also drain the pending score stores.
JANUS_DEV void lds_barrier() { __builtin_amdgcn_s_barrier(); }

// x from lane (lane ^ 16): a swizzle within each half-wave.
JANUS_DEV float xor_lanes16(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
}

// Block id -> (token tile slot, key chunk).  Workgroups are dispatched round
// robin over the XCDs, so block L runs on XCD L % 8; all blocks of key chunk
// c are given to XCD c % 8, which keeps each XCD's share of the keys (about
// 1/8 of them) resident in that XCD's L2.
JANUS_DEV bool xcd_tile_chunk(int L, int nchunks, int ntiles, int &tile, int &chunk)
{
    const int x = L % IDX_XCD, s = L / IDX_XCD;
    const int nc = (nchunks - x + IDX_XCD - 1) / IDX_XCD;  // chunks owned by this XCD
    if (nc <= 0 || s >= nc * ntiles)
        return false;
    tile = s / nc;
    chunk = x + IDX_XCD * (s % nc);
    return true;
}

// LDS stage layout: key row r (128 bytes) holds its 16-byte column c at slot
// c ^ ((r >> 1) & 7), so the 16 rows read by one 16-lane group land in 16
// different bank groups.
//
// TPW tokens per wave: an MFMA tile's 16 rows are TPW tokens x RPT = 16/TPW
// heads, ordered so that output rows 4g..4g+3 (lane group g) hold one token
// (g*TPW/4) and 4 consecutive heads.  A lane sums its heads in registers; the
// 4/TPW lane groups that share a token are then added across lanes.  Fewer
// tokens per wave means fewer registers and more waves per SIMD, whose VALU
// epilogues then run under the other waves' MFMAs.
template <int H, int TPW>
__global__ __launch_bounds__(256, (TPW == 4 ? 2 : 4)) void index_scores_fp8_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs,
    int nchunks, int key_chunk, int ntiles, const uint8_t *__restrict__ q, const float *__restrict__ q_scale,
    const uint8_t *__restrict__ kI, const float *__restrict__ k_scale, const float *__restrict__ w,
    float *__restrict__ scores)
{
    constexpr int RPT = 16 / TPW;   // heads of one token per MFMA tile
    constexpr int HB = H / RPT;     // MFMA tiles per 16-key block
    constexpr int TOK_TILE = 4 * TPW;
    // two separate stage buffers (not one 2-D array), so the compiler can tell
    // the DMA into one from the LDS reads of the other and keeps the prefetch
    // asynchronous
    __shared__ __attribute__((aligned(16))) uint8_t sKey0[IDX_STAGE * 128];
    __shared__ __attribute__((aligned(16))) uint8_t sKey1[IDX_STAGE * 128];
    __shared__ float sKs0[IDX_STAGE];
    __shared__ float sKs1[IDX_STAGE];
    int slot, chunk, b, tile0;
    if (!xcd_tile_chunk(blockIdx.x, nchunks, ntiles, slot, chunk))
        return;
    if (!tile_slot(q_start, num_seqs, slot, TOK_TILE, b, tile0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = M + N;
    const int key_lo = chunk * key_chunk;
    if (key_lo >= ctx)
        return;
    const int key_hi = min(ctx, key_lo + key_chunk);
    // wave index in a scalar register
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tw0 = tile0 + wave * TPW;
    const bool wave_on = tw0 < N;
    const int r16 = lane & 15, kg = lane >> 4;
    const int qrow0 = q_start[b];
    const int64_t kbase = ctx_start[b];
    // block-wide causal limit: stages past it need no keys
    const int block_lim = M + min(tile0 + TOK_TILE - 1, N - 1);
    const int key_end = min(key_hi, block_lim + 1);

    auto issue = [&](int k0, uint8_t *kdst, float *sdst) {
        // the lane index passes through an empty asm so that its per-lane
        // address terms are recomputed here each stage instead of being
        // hoisted out of the key loop and kept live (or spilled) across it
        int ln = lane;
        asm volatile("" : "+v"(ln));
        // 16 wave-instructions of 1 KB fill the 16 KB stage; lane L of
        // instruction i fills chunk 64i + L = (row, slot)
#pragma unroll
        for (int i = wave; i < IDX_STAGE * 8 / 64; i += 4) {
            const int qch = 64 * i + ln;
            const int r = qch >> 3, sl = qch & 7;
            const int c = sl ^ ((r >> 1) & 7);
            int key = k0 + r;
            if (key >= ctx)
                key = ctx - 1;
            const uint8_t *src = kI + ((kbase + key) << 7) + 16 * c;
            __builtin_amdgcn_global_load_lds((const void *)src, (lds_void_t *)(kdst + 1024 * i), 16, 0, 0);
        }
        // the stage's key scales, one dword per lane (two instructions, waves 0 and 1)
        if (k_scale && wave < 2) {
            const int key = min(k0 + 64 * wave + ln, ctx - 1);
            __builtin_amdgcn_global_load_lds((const void *)(k_scale + kbase + key),
                                             (lds_void_t *)(sdst + 64 * wave), 4, 0, 0);
        }
    };
    if (key_lo < key_end)
        issue(key_lo, sKey0, sKs0);

    // A operand: MFMA row r16 = (token r16/RPT, head RPT*hb + r16%RPT), bytes 32*kg..32*kg+31.
    const int a_tok = tw0 + r16 / RPT;
    const bool a_ok = a_tok < N;
    const int64_t a_row = (int64_t)qrow0 + (a_ok ? a_tok : 0);
    v8i a[HB];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        if (a_ok)
            a[hb] = *(const v8i *)(q + ((a_row * H + RPT * hb + (r16 % RPT)) << 7) + 32 * kg);
        else
            a[hb] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
    }
    // Output rows 4*kg..4*kg+3 of every tile: token tw0 + 4*kg/RPT, heads RPT*hb + (4*kg)%RPT + i.
    const int e_tok = tw0 + (4 * kg) / RPT;
    const bool e_ok = e_tok < N;
    const int64_t e_row = (int64_t)qrow0 + (e_ok ? e_tok : 0);
    const int hsub = (4 * kg) % RPT;
    // head weights times the token's query scale (a positive factor of every
    // term) and 2^25 (undoing the MFMA's query scale), rounded once to bf16 pairs
    const float sq = (q_scale ? q_scale[e_row] : 1.0f) * 0x1p25f;
    v2bf wv[HB][2];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        v4f t = *(const v4f *)(w + e_row * H + RPT * hb + hsub);
        wv[hb][0] = __builtin_convertvector((v2f){t[0] * sq, t[1] * sq}, v2bf);
        wv[hb][1] = __builtin_convertvector((v2f){t[2] * sq, t[3] * sq}, v2bf);
    }
    const int lim = M + e_tok;  // last causal candidate of this lane's token
    const int wave_lim = M + min(tw0 + TPW - 1, N - 1);
    int scales = IDX_MFMA_SCALES;
    // this lane's two 16-byte columns (2*kg, 2*kg+1) of LDS row 16*j + r16
    const int g8 = (r16 >> 1) & 7;
    const int off0 = r16 * 128 + 16 * ((2 * kg) ^ g8), off1 = r16 * 128 + 16 * ((2 * kg + 1) ^ g8);
    // lanes sharing a token split the stores: group-in-token index
    constexpr int GPT = 4 / TPW;            // lane groups per token
    const int gin = kg % GPT;
    // Scores leave through buffer stores over this block's rows: a lane with
    // nothing to write uses an offset past the range and the hardware drops
    // it, so every wave issues the same number of stores per full stage and
    // the stage can wait for its key prefetch with vmcnt(STAGE_STORES)
    // instead of draining the stores.
    const int nrows_blk = max(0, min(TOK_TILE, N - tile0));
    const int64_t blk_off = score_start[b] + (int64_t)tile0 * ctx;
    const __amdgpu_buffer_rsrc_t rsrc = make_buffer_rsrc(scores + blk_off, (uint32_t)((int64_t)nrows_blk * ctx * 4));
    const bool row_ok = e_ok && wave_on;
    const uint32_t lane_row_off = (uint32_t)((int64_t)(e_tok - tile0) * ctx * 4);
    constexpr int STORES_PER_GROUP = 4 / GPT;
    constexpr int STAGE_STORES = (IDX_STAGE / 64) * STORES_PER_GROUP;
    // every token of the block sees all keys below this bound
    const int interior_end = min(ctx, M + tile0 + 1);

    // one stage: compute the keys in (stg, ks) while the next stage streams in
    auto stage = [&](int k0, const uint8_t *stg, const float *ks) {
#pragma unroll
        for (int gsub = 0; gsub < IDX_STAGE / 64; ++gsub) {
            const int s0 = k0 + 64 * gsub;
            if (s0 >= key_hi)
                break;
            float res[4];
            const bool skip = !wave_on || s0 > wave_lim;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (skip) {
                    res[j] = -INFINITY;
                    continue;
                }
                const uint8_t *rowb = stg + (64 * gsub + 16 * j) * 128;
                v4i lo = *(const v4i *)(rowb + off0), hi = *(const v4i *)(rowb + off1);
                const v8i bk = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
                for (int h4 = 0; h4 < HB; h4 += 4) {
                    v4f c[4];
                    mfma4_fp8_scaled(c[0], c[1], c[2], c[3], a[h4], a[h4 + 1], a[h4 + 2], a[h4 + 3], bk, scales);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        acc0 = __builtin_amdgcn_fdot2_f32_bf16(clamp01_bf16x2(c[u][0], c[u][1]), wv[h4 + u][0], acc0, false);
                        acc1 = __builtin_amdgcn_fdot2_f32_bf16(clamp01_bf16x2(c[u][2], c[u][3]), wv[h4 + u][1], acc1, false);
                    }
                }
                float r = acc0 + acc1;
                if (GPT >= 2)
                    r += xor_lanes16(r);
                if (GPT >= 4)
                    r += __shfl_xor(r, 32, 64);
                res[j] = r;
            }
            // res[j] is token e_tok at key s0 + 16*j + r16 (before the key
            // scale); the GPT lane groups of a token hold the same values and
            // take turns, so each store instruction writes with every lane
#pragma unroll
            for (int js = 0; js < STORES_PER_GROUP; ++js) {
                float v = res[js * GPT];
#pragma unroll
                for (int u = 1; u < GPT; ++u)
                    v = gin == u ? res[js * GPT + u] : v;
                const int jj = js * GPT + gin;
                const int s = s0 + 16 * jj + r16;
                const float kscale = k_scale ? ks[64 * gsub + 16 * jj + r16] : 1.0f;
                uint32_t off;
                if (s0 + 64 <= interior_end) {  // block-uniform: no causal or range checks
                    v *= kscale;
                    off = row_ok ? lane_row_off + 4u * (uint32_t)s : 0x80000000u;
                } else {
                    v = s > lim ? -INFINITY : v * kscale;
                    off = (row_ok && s < ctx) ? lane_row_off + 4u * (uint32_t)s : 0x80000000u;
                }
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rsrc, off, 0, 0);
            }
        }
    };
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int k0 = key_lo; k0 < key_hi; k0 += 2 * IDX_STAGE) {
        // even stage: read buffer 0, fill buffer 1
        if (k0 + IDX_STAGE < key_end)
            issue(k0 + IDX_STAGE, sKey1, sKs1);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0, sKey0, sKs0);
        // the next stage's keys have landed once at most this stage's stores are pending
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
        if (k0 + IDX_STAGE >= key_hi)
            break;
        // odd stage: read buffer 1, fill buffer 0
        if (k0 + 2 * IDX_STAGE < key_end)
            issue(k0 + 2 * IDX_STAGE, sKey0, sKs0);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0 + IDX_STAGE, sKey1, sKs1);
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
    }
}

// Plain vector kernel for any dtype and shape: one (token, key) score per thread.
__global__ __launch_bounds__(256) void index_scores_vector(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs,
    const void *__restrict__ q, int q_dt, const float *__restrict__ q_scale,
    const void *__restrict__ kI, int k_dt, const float *__restrict__ k_scale,
    const float *__restrict__ w, int H, int d, float *__restrict__ scores)
{
    int b, t0;
    if (!tile_slot(q_start, num_seqs, blockIdx.y, GEN_TOK_TILE, b, t0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = M + N;
    const int i = t0 + threadIdx.x / GEN_KEY_TILE;
    const int s = blockIdx.x * GEN_KEY_TILE + threadIdx.x % GEN_KEY_TILE;
    if (i >= N || s >= ctx)
        return;
    float *dst = scores + score_start[b] + (int64_t)i * ctx + s;
    if (s > M + i) {
        *dst = -INFINITY;
        return;
    }
    const int64_t g = (int64_t)q_start[b] + i;
    const int64_t ks = (int64_t)ctx_start[b] + s;
    float acc = 0.f;
    for (int h = 0; h < H; ++h) {
        float x = 0.f;
        for (int j = 0; j < d; ++j)
            x = fmaf(load_elem(q, q_dt, (g * H + h) * d + j), load_elem(kI, k_dt, ks * d + j), x);
        acc = fmaf(w[g * H + h], fmaxf(x, 0.f), acc);
    }
    *dst = acc * (q_scale ? q_scale[g] : 1.f) * (k_scale ? k_scale[ks] : 1.f);
}

} // namespace janus

using namespace janus;

extern "C" int janus_index_scores(const janus_batch *bt, const void *q, janus_dtype q_dt,
                                  const float *q_scale, const void *kI, janus_dtype k_dt,
                                  const float *k_scale, const float *w, int H, int d,
                                  float *scores, void *stream)
{
    if (!batch_ok(bt) || !bt->ctx_start || !bt->score_start || !q || !kI || !w || !scores || H < 1 || d < 1)
        return JANUS_ERR_INVALID_ARG;
    if (!dtype_ok(q_dt) || !dtype_ok(k_dt))
        return JANUS_ERR_INVALID_ARG;
    if (q_dt != k_dt)
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0 || bt->max_ctx == 0)
        return JANUS_OK;
    hipStream_t st = as_stream(stream);
    const int nseq = bt->num_seqs;
    if (q_dt == JANUS_FP8_E4M3 && d == 128 && H == 64) {
        // key chunks: a multiple of the XCD count, each a whole number of
        // stages and about IDX_KEY_CHUNK keys long
        const int per_xcd_keys = ceil_div(bt->max_ctx, IDX_XCD);
        const int chunks_per_xcd = std::max(1, ceil_div(per_xcd_keys, IDX_KEY_CHUNK));
        const int key_chunk = ceil_div(ceil_div(per_xcd_keys, chunks_per_xcd), IDX_STAGE) * IDX_STAGE;
        const int nchunks = ceil_div(bt->max_ctx, key_chunk);
        constexpr int TPW = IDX_TPW;
        const int ntiles = ceil_div(bt->total_q, 4 * TPW) + nseq;
        const int per_xcd = ceil_div(nchunks, IDX_XCD) * ntiles;
        hipLaunchKernelGGL((index_scores_fp8_mfma<64, TPW>), dim3(IDX_XCD * per_xcd), dim3(256), 0, st, bt->q_start,
                           bt->ctx_start, bt->hist_len, bt->score_start, nseq, nchunks, key_chunk, ntiles,
                           (const uint8_t *)q, q_scale, (const uint8_t *)kI, k_scale, w, scores);
        return launch_status();
    }
    dim3 grid(ceil_div(bt->max_ctx, GEN_KEY_TILE), ceil_div(bt->total_q, GEN_TOK_TILE) + nseq);
    hipLaunchKernelGGL(index_scores_vector, grid, dim3(GEN_TOK_TILE * GEN_KEY_TILE), 0, st, bt->q_start,
                       bt->ctx_start, bt->hist_len, bt->score_start, nseq, q, (int)q_dt, q_scale, kI, (int)k_dt,
                       k_scale, w, H, d, scores);
    return launch_status();
}
