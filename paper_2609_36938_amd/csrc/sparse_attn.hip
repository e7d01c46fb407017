// Sparse attention over the selected tokens (the KV of S_t feeds core
// attention; the paragraph after Eq. 1), with all query heads sharing one KV
// head.  MLA in its absorbed form is the case dqk = 576 (512 latent + 64
// rope), dv = 512, V = the first 512 elements of each cached row.
//
// MFMA kernel (MLA shape): one block per query token, one wave per 16*HB heads.
// The token's selected rows are gathered through the page table in tiles of
// 32 into LDS twice: row-major (the A operand of S^T = K Q^T, one 16-byte read
// per lane) and transposed as key pairs (the B operand of O = P V).  The
// queries stay in VGPRs for the whole token; S^T is formed so that each lane's
// outputs are 8 keys of one head, which is exactly an A operand of the P V
// product, so P never leaves registers.  Softmax is online in fp32 (exp2
// domain); O accumulates in fp32 MFMA accumulators.
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <algorithm>

namespace janus {

constexpr int MLA_DQK = 576;
constexpr int MLA_DV = 512;
constexpr int MLA_KT = 32;                  // keys per tile
constexpr int MLA_STEPS = MLA_DQK / 32;     // MFMA K-steps over the 576 dims
constexpr int MLA_NB = MLA_DV / 16;         // 16-wide dv blocks
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

JANUS_DEV v8bf as_v8bf(v4i x) { return __builtin_bit_cast(v8bf, x); }
typedef short v8s16 __attribute__((ext_vector_type(8)));

constexpr int MLA_CPR = MLA_DQK * 2 / 16;      // 16-byte chunks per cached row (72)
constexpr int MLA_PCH = MLA_CPR + 2;            // LDS row pitch in chunks: 1184 B reads the K operand conflict-free
constexpr int MLA_ROWB = MLA_PCH * 16;          // LDS bytes per tile row
constexpr int MLA_TILE_CH = MLA_KT * MLA_PCH;   // chunks per tile (2336)
constexpr int MLA_TILE_INS = (MLA_TILE_CH + 63) / 64;  // wave-instructions per tile (37)
constexpr int MLA_MAX_K = 4096;                 // selected ids per token held in LDS
constexpr float RESCALE_SLACK = 8.0f;           // log2 headroom before O is rescaled

typedef short v4s16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4s16 lds_v4s16;

// Transposing LDS read (ds_read_b64_tr_b16): within each 16-lane group,
// lane i's element j is element i%4 of the 8 bytes addressed by lane 4j+i/4.
JANUS_DEV v4s16 lds_read_tr16(const uint8_t *lds_base, int byte_off)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s16 *)((__attribute__((address_space(3))) uint8_t *)lds_base + byte_off));
}

template <int NW, int HB>
__global__ __launch_bounds__(64 * NW, 1) void sparse_mla_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ kv, int64_t row_stride,
    const int32_t *__restrict__ page_table, int pt_ld, int page_shift, const int32_t *__restrict__ topk,
    int k, float scale_log2, void *__restrict__ out, int out_f32, float *__restrict__ lse)
{
    constexpr int HW = 16 * HB;  // heads per wave: HB 16-head MFMA blocks
    constexpr int HQ = HW * NW;
    constexpr int NT = 64 * NW;
    __shared__ __attribute__((aligned(16))) uint8_t sKV[2][MLA_TILE_INS * 64 * 16];
    __shared__ int32_t sSlot[MLA_MAX_K];

    const int g = blockIdx.x;
    const int b = session_of_row(q_start, num_seqs, g);
    const int lim = hist_len[b] + (g - q_start[b]);  // last causal id
    const int32_t *pt = page_table + (int64_t)b * pt_ld;
    const int psz_mask = (1 << page_shift) - 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c16 = lane & 15, grp = lane >> 4;
    const int head0 = HW * wave;

    // physical row of every selected id (-1: padding)
    for (int j = tid; j < k; j += NT) {
        const int s = topk[(int64_t)g * k + j];
        sSlot[j] = (s >= 0 && s <= lim) ? ((pt[s >> page_shift] << page_shift) + (s & psz_mask)) : -1;
    }
    // queries of head head0 + 16*hb + c16, dims 32*step + 8*grp .. +7
    v8bf qf[HB][MLA_STEPS];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        const uint16_t *qr = q + ((int64_t)g * HQ + head0 + 16 * hb + c16) * MLA_DQK + 8 * grp;
#pragma unroll
        for (int st = 0; st < MLA_STEPS; ++st)
            qf[hb][st] = as_v8bf(*(const v4i *)(qr + 32 * st));
    }
    v4f o[HB][MLA_NB];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int nb = 0; nb < MLA_NB; ++nb)
            o[hb][nb] = v4f{0.f, 0.f, 0.f, 0.f};
    float m[HB], lsum[HB];  // per head head0 + 16*hb + c16
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        m[hb] = -INFINITY;
        lsum[hb] = 0.f;
    }
    __syncthreads();

    const int ntiles = (k + MLA_KT - 1) / MLA_KT;
    // gather of tile t into buffer: wave-instruction j fills LDS chunks 64j .. 64j+63
    // (chunks 72 and 73 of each row are padding and load a dummy; padding ids load row 0)
    auto issue = [&](int t, int buf) {
        for (int j = wave; j < MLA_TILE_INS; j += NW) {
            const int qch = 64 * j + lane;
            if (qch < MLA_TILE_CH) {
                const int r = qch / MLA_PCH;
                int c = qch - r * MLA_PCH;
                if (c >= MLA_CPR)
                    c = 0;
                const int key = MLA_KT * t + r;
                int slot = key < k ? sSlot[key] : -1;
                if (slot < 0)
                    slot = 0;  // padding rows read a real row; their logits are masked
                const uint16_t *src = kv + (int64_t)slot * row_stride + 8 * c;
                __builtin_amdgcn_global_load_lds((const void *)src, (lds_void *)(&sKV[buf][(64 * j) * 16]), 16,
                                                 0, 0);
            }
        }
    };
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int buf = t & 1;
        if (t + 1 < ntiles)
            issue(t + 1, buf ^ 1);
        const uint8_t *tile = sKV[buf];
        // S^T[key][head] = K Q^T for keys 16*kb + 4*grp + i
        v4f st[2][HB];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int hb = 0; hb < HB; ++hb)
                st[kb][hb] = v4f{0.f, 0.f, 0.f, 0.f};
            const int r = 16 * kb + c16;
            const uint8_t *row = tile + r * MLA_ROWB;
#pragma unroll
            for (int step = 0; step < MLA_STEPS; ++step) {
                const v8bf a = as_v8bf(*(const v4i *)(row + 16 * (4 * step + grp)));
#pragma unroll
                for (int hb = 0; hb < HB; ++hb)
                    st[kb][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[hb][step], st[kb][hb], 0, 0, 0);
            }
        }
        // online softmax (exp2 domain) with lazy rescaling of O
        bool okk[2][4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = MLA_KT * t + 16 * kb + 4 * grp + i;
                okk[kb][i] = key < k && sSlot[key] >= 0;
            }
        v8bf pa[HB];
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) {
            float x[2][4];
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    x[kb][i] = okk[kb][i] ? st[kb][hb][i] * scale_log2 : -INFINITY;
                    mx = fmaxf(mx, x[kb][i]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const bool grow = mx > m[hb] + RESCALE_SLACK || (m[hb] == -INFINITY && mx > -INFINITY);
            if (__ballot(grow)) {
                const float mnew = grow ? mx : m[hb];
                const float alpha = (m[hb] == -INFINITY) ? 0.f : exp2f(m[hb] - mnew);
                lsum[hb] *= alpha;
                m[hb] = mnew;
                float ai[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    ai[i] = __shfl(alpha, 4 * grp + i, 64);
#pragma unroll
                for (int nb = 0; nb < MLA_NB; ++nb)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        o[hb][nb][i] *= ai[i];
            }
            float pv[2][4];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[kb][i] = (m[hb] == -INFINITY) ? 0.f : exp2f(x[kb][i] - m[hb]);
                    lsum[hb] += pv[kb][i];
                }
            pa[hb] = v8bf{(__bf16)pv[0][0], (__bf16)pv[0][1], (__bf16)pv[0][2], (__bf16)pv[0][3],
                          (__bf16)pv[1][0], (__bf16)pv[1][1], (__bf16)pv[1][2], (__bf16)pv[1][3]};
        }
        // O += P V; V operand: keys 4*grp + r' (slots 0-3) and 16 + 4*grp + r' (slots 4-7),
        // lane (r' = c16/4, cc = c16%4) addresses dims 16*nb + 4*cc .. +3 of its key row
        const int rr0 = 4 * grp + (c16 >> 2), rr1 = 16 + rr0, cc = c16 & 3;
        const uint8_t *row0 = tile + rr0 * MLA_ROWB, *row1 = tile + rr1 * MLA_ROWB;
#pragma unroll
        for (int nb = 0; nb < MLA_NB; ++nb) {
            const int ch = 2 * nb + (cc >> 1), sub = (cc & 1) * 8;
            const v4s16 lo = lds_read_tr16(row0, 16 * ch + sub);
            const v4s16 hi = lds_read_tr16(row1, 16 * ch + sub);
            const v8bf bv = __builtin_bit_cast(v8bf, (v8s16){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
            for (int hb = 0; hb < HB; ++hb)
                o[hb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[hb], bv, o[hb][nb], 0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }
    // normalise and store: O rows are heads head0 + 16*hb + 4*grp + i, column dim 16*nb + c16
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        float l = lsum[hb];
        l += __shfl_xor(l, 16, 64);
        l += __shfl_xor(l, 32, 64);
        const float inv = l > 0.f ? 1.f / l : 0.f;
        if (lse && grp == 0)
            lse[(int64_t)g * HQ + head0 + 16 * hb + c16] = l > 0.f ? (m[hb] + log2f(l)) * LN2 : -INFINITY;
        float iv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            iv[i] = __shfl(inv, 4 * grp + i, 64);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t orow = ((int64_t)g * HQ + head0 + 16 * hb + 4 * grp + i) * MLA_DV;
#pragma unroll
            for (int nb = 0; nb < MLA_NB; ++nb) {
                const float v = o[hb][nb][i] * iv[i];
                if (out_f32)
                    ((float *)out)[orow + 16 * nb + c16] = v;
                else
                    ((uint16_t *)out)[orow + 16 * nb + c16] = f32_to_bf16_rne(v);
            }
        }
    }
}

// Plain vector kernel for any (Hq, dqk, dv) and separate K/V pools: one
// block per (token, head); 256 keys per chunk, one logit per thread.
constexpr int VEC_THREADS = 256;
constexpr int VEC_MAX_DQK = 1024;

__global__ __launch_bounds__(VEC_THREADS) void sparse_attn_vector(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs,
    const uint16_t *__restrict__ q, int Hq, int dqk, int dv, const uint16_t *__restrict__ k_pool,
    const uint16_t *__restrict__ v_pool, int64_t k_rs, int64_t v_rs, const int32_t *__restrict__ page_table,
    int pt_ld, int page_shift, const int32_t *__restrict__ topk, int k, float scale_log2,
    void *__restrict__ out, int out_f32, float *__restrict__ lse)
{
    __shared__ float sq[VEC_MAX_DQK];
    __shared__ float sp[VEC_THREADS];
    __shared__ int64_t sslot[VEC_THREADS];
    __shared__ float sred[VEC_THREADS / 64];
    const int g = blockIdx.x / Hq, h = blockIdx.x % Hq;
    const int b = session_of_row(q_start, num_seqs, g);
    const int lim = hist_len[b] + (g - q_start[b]);
    const int32_t *pt = page_table + (int64_t)b * pt_ld;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int e = tid; e < dqk; e += VEC_THREADS)
        sq[e] = bf16_to_f32(q[((int64_t)g * Hq + h) * dqk + e]);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};  // dims tid, tid+256, ... (dv <= 1024)
    float m = -INFINITY, l = 0.f;
    for (int c0 = 0; c0 < k; c0 += VEC_THREADS) {
        __syncthreads();
        float x = -INFINITY;
        int64_t slot = -1;
        if (c0 + tid < k) {
            const int s = topk[(int64_t)g * k + c0 + tid];
            if (s >= 0 && s <= lim) {
                slot = ((int64_t)pt[s >> page_shift] << page_shift) + (s & ((1 << page_shift) - 1));
                float d = 0.f;
                const uint16_t *kr = k_pool + slot * k_rs;
                for (int e = 0; e < dqk; ++e)
                    d = fmaf(sq[e], bf16_to_f32(kr[e]), d);
                x = d * scale_log2;
            }
        }
        sslot[tid] = slot;
        float mx = x;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1)
            mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        if (lane == 0)
            sred[wave] = mx;
        __syncthreads();
        mx = sred[0];
        for (int w = 1; w < VEC_THREADS / 64; ++w)
            mx = fmaxf(mx, sred[w]);
        const float mnew = fmaxf(m, mx);
        const bool none = mnew == -INFINITY;
        const float alpha = none ? 1.f : exp2f(m - mnew);
        const float p = (none || slot < 0) ? 0.f : exp2f(x - mnew);
        sp[tid] = p;
        float ps = p;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1)
            ps += __shfl_xor(ps, o, 64);
        __syncthreads();
        if (lane == 0)
            sred[wave] = ps;
        __syncthreads();
        ps = 0.f;
        for (int w = 0; w < VEC_THREADS / 64; ++w)
            ps += sred[w];
        l = l * alpha + ps;
        m = mnew;
        for (int j = 0; j < 4; ++j)
            acc[j] *= alpha;
        const int nk = min(VEC_THREADS, k - c0);
        for (int kk = 0; kk < nk; ++kk) {
            const int64_t sl = sslot[kk];
            if (sl < 0)
                continue;
            const float pk = sp[kk];
            const uint16_t *vr = v_pool + sl * v_rs;
            for (int j = 0; j < 4; ++j) {
                const int e = tid + j * VEC_THREADS;
                if (e < dv)
                    acc[j] = fmaf(pk, bf16_to_f32(vr[e]), acc[j]);
            }
        }
    }
    const float inv = l > 0.f ? 1.f / l : 0.f;
    for (int j = 0; j < 4; ++j) {
        const int e = tid + j * VEC_THREADS;
        if (e < dv) {
            const int64_t oi = ((int64_t)g * Hq + h) * dv + e;
            if (out_f32)
                ((float *)out)[oi] = acc[j] * inv;
            else
                ((uint16_t *)out)[oi] = f32_to_bf16_rne(acc[j] * inv);
        }
    }
    if (lse && tid == 0)
        lse[(int64_t)g * Hq + h] = l > 0.f ? (m + log2f(l)) * LN2 : -INFINITY;
}

} // namespace janus

using namespace janus;

extern "C" int janus_sparse_attn(const janus_batch *bt, const void *q, int Hq, int dqk, int dv,
                                 const void *k_pool, const void *v_pool, int64_t k_row_stride,
                                 int64_t v_row_stride, const int32_t *page_table, int pt_ld, int page_size,
                                 const int32_t *topk_idx, int k, float scale, void *out, janus_dtype out_dt,
                                 float *lse, void *stream)
{
    if (!batch_ok(bt) || !q || !k_pool || !v_pool || !page_table || !topk_idx || !out || Hq < 1 || dqk < 1 ||
        dv < 1 || k < 1 || pt_ld < 1 || !pow2(page_size) || k_row_stride < dqk || v_row_stride < dv)
        return JANUS_ERR_INVALID_ARG;
    if (out_dt != JANUS_BF16 && out_dt != JANUS_F32)
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0)
        return JANUS_OK;
    hipStream_t st = as_stream(stream);
    const int shift = __builtin_ctz((unsigned)page_size);
    const float sl2 = scale * LOG2E;
    const int of32 = out_dt == JANUS_F32;
    const bool mla = dqk == MLA_DQK && dv == MLA_DV && v_pool == k_pool && v_row_stride == k_row_stride &&
                     (k_row_stride % 8) == 0 && (reinterpret_cast<uintptr_t>(k_pool) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(q) & 15) == 0;
    if (mla && k <= MLA_MAX_K && (Hq == 128 || Hq == 64 || Hq == 32 || Hq == 16)) {
        const auto *qq = (const uint16_t *)q;
        const auto *kv = (const uint16_t *)k_pool;
        auto launch = [&](auto kern, int nw) {
            hipLaunchKernelGGL(kern, dim3(bt->total_q), dim3(64 * nw), 0, st, bt->q_start, bt->hist_len,
                               bt->num_seqs, qq, kv, k_row_stride, page_table, pt_ld, shift, topk_idx, k, sl2, out,
                               of32, lse);
        };
        if (Hq == 128)
            launch(sparse_mla_mfma<8, 1>, 8);
        else if (Hq == 64)
            launch(sparse_mla_mfma<4, 1>, 4);
        else if (Hq == 32)
            launch(sparse_mla_mfma<2, 1>, 2);
        else
            launch(sparse_mla_mfma<1, 1>, 1);
        return launch_status();
    }
    if (dqk > VEC_MAX_DQK || dv > 4 * VEC_THREADS)
        return JANUS_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(sparse_attn_vector, dim3((int64_t)bt->total_q * Hq), dim3(VEC_THREADS), 0, st, bt->q_start,
                       bt->hist_len, bt->num_seqs, (const uint16_t *)q, Hq, dqk, dv, (const uint16_t *)k_pool,
                       (const uint16_t *)v_pool, k_row_stride, v_row_stride, page_table, pt_ld, shift, topk_idx, k,
                       sl2, out, of32, lse);
    return launch_status();
}
