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
// Epilogue: the head weights are held as bf16 pairs and each MFMA's four
// fp32 outputs are rounded to bf16 pairs, clamped at zero with a packed
// 16-bit integer max (a negative bf16 is a negative int16), and accumulated
// with v_dot2_f32_bf16 into fp32: 6 VALU ops per 16x16x128 MFMA instead of 8,
// and half the weight registers.  Every term is non-negative, so the two
// roundings bound the relative error of a score by 2^-8.
#include "janus_device.hpp"
#include "janus_host.hpp"

namespace janus {

constexpr int IDX_TPW = 4;                          // tokens per wave
constexpr int IDX_WAVES = 4;                        // waves per block
constexpr int IDX_TOK_TILE = IDX_TPW * IDX_WAVES;   // tokens per block
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

template <int H>
__global__ __launch_bounds__(256, 2) void index_scores_fp8_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs,
    const uint8_t *__restrict__ q, const float *__restrict__ q_scale,
    const uint8_t *__restrict__ kI, const float *__restrict__ k_scale,
    const float *__restrict__ w, float *__restrict__ scores)
{
    constexpr int HB = H / 4;  // MFMA tiles per 16-key block (4 heads of 4 tokens each)
    int b, tile0;
    if (!tile_slot(q_start, num_seqs, blockIdx.y, IDX_TOK_TILE, b, tile0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = M + N;
    const int key_lo = blockIdx.x * IDX_KEY_CHUNK;
    if (key_lo >= ctx)
        return;
    const int key_hi = min(ctx, key_lo + IDX_KEY_CHUNK);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int tw0 = tile0 + wave * IDX_TPW;
    if (tw0 >= N)
        return;
    const int r16 = lane & 15, kg = lane >> 4;
    const int qrow0 = q_start[b];

    // A operand: MFMA row r16 = (token r16/4, head 4*hb + r16%4), bytes 32*kg..32*kg+31.
    const int a_tok = tw0 + (r16 >> 2);
    const bool a_ok = a_tok < N;
    const int64_t a_row = (int64_t)qrow0 + (a_ok ? a_tok : 0);
    v8i a[HB];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        if (a_ok)
            a[hb] = *(const v8i *)(q + ((a_row * H + 4 * hb + (r16 & 3)) << 7) + 32 * kg);
        else
            a[hb] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
    }
    // Output rows 4*kg..4*kg+3 of every tile: token tw0 + kg, heads 4*hb + i.
    const int e_tok = tw0 + kg;
    const bool e_ok = e_tok < N;
    const int64_t e_row = (int64_t)qrow0 + (e_ok ? e_tok : 0);
    v2bf wv[HB][2];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        v4f t = *(const v4f *)(w + e_row * H + 4 * hb);
        wv[hb][0] = __builtin_convertvector((v2f){t[0], t[1]}, v2bf);
        wv[hb][1] = __builtin_convertvector((v2f){t[2], t[3]}, v2bf);
    }
    const float sq = q_scale ? q_scale[e_row] : 1.0f;
    const int lim = M + e_tok;  // last causal candidate of this lane's token
    const int wave_lim = M + min(tw0 + IDX_TPW - 1, N - 1);
    float *out_row = scores + score_start[b] + (int64_t)e_tok * ctx;
    const int64_t kbase = ctx_start[b];
    const v4f zero = {0.f, 0.f, 0.f, 0.f};

    for (int s0 = key_lo; s0 < key_hi; s0 += 64) {
        float res[4];
        if (s0 > wave_lim) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                res[j] = -INFINITY;
        } else {
#pragma unroll 1
            for (int j = 0; j < 4; ++j) {
                const int s = s0 + 4 * r16 + j;
                v8i bk = v8i{0, 0, 0, 0, 0, 0, 0, 0};
                if (s < ctx)
                    bk = *(const v8i *)(kI + ((kbase + s) << 7) + 32 * kg);
                float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
                for (int hb = 0; hb < HB; ++hb) {
                    v4f c = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a[hb], bk, zero, 0, 0, 0, 0, 0, 0);
                    acc0 = __builtin_amdgcn_fdot2_f32_bf16(relu_bf16x2(c[0], c[1]), wv[hb][0], acc0, false);
                    acc1 = __builtin_amdgcn_fdot2_f32_bf16(relu_bf16x2(c[2], c[3]), wv[hb][1], acc1, false);
                }
                res[j] = acc0 + acc1;
            }
        }
        if (!e_ok)
            continue;
        const int sb = s0 + 4 * r16;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int s = sb + j;
            if (s > lim)
                res[j] = -INFINITY;
            else
                res[j] *= sq * (k_scale ? k_scale[kbase + s] : 1.0f);
        }
        float *dst = out_row + sb;
        if (sb + 3 < ctx && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
            *(v4f *)dst = v4f{res[0], res[1], res[2], res[3]};
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (sb + j < ctx)
                    dst[j] = res[j];
        }
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
        dim3 grid(ceil_div(bt->max_ctx, IDX_KEY_CHUNK), ceil_div(bt->total_q, IDX_TOK_TILE) + nseq);
        hipLaunchKernelGGL(index_scores_fp8_mfma<64>, grid, dim3(256), 0, st, bt->q_start, bt->ctx_start,
                           bt->hist_len, bt->score_start, nseq, (const uint8_t *)q, q_scale,
                           (const uint8_t *)kI, k_scale, w, scores);
        return launch_status();
    }
    dim3 grid(ceil_div(bt->max_ctx, GEN_KEY_TILE), ceil_div(bt->total_q, GEN_TOK_TILE) + nseq);
    hipLaunchKernelGGL(index_scores_vector, grid, dim3(GEN_TOK_TILE * GEN_KEY_TILE), 0, st, bt->q_start,
                       bt->ctx_start, bt->hist_len, bt->score_start, nseq, q, (int)q_dt, q_scale, kI, (int)k_dt,
                       k_scale, w, H, d, scores);
    return launch_status();
}
