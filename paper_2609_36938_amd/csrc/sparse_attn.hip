// Sparse attention over the selected tokens (the KV of S_t feeds core
// attention; the paragraph after Eq. 1), with all query heads sharing one KV
// head.  MLA in its absorbed form is the case dqk = 576 (512 latent + 64
// rope), dv = 512, V = the first 512 elements of each cached row.
//
// MFMA kernel (MLA shape): one block of NW waves per query token.
//   * The token's selected rows are gathered through the page table, 32 at a
//     time, straight into LDS (global_load_lds), into a ring of three tile
//     buffers: while tile t is computed, tiles t+1 and t+2 are in flight.
//     Waits are counted (vmcnt) and barriers order LDS only, so the gathers
//     are never drained early.
//   * Wave w holds the queries of heads 16w..16w+15 in registers and forms
//     S^T = K Q^T for them from the row-major tile (one 16-byte read per
//     lane, loaded one K-step ahead), so that each lane's outputs are 8 keys
//     of one head: exactly an A operand of the P V product.  Softmax is
//     online in the exp2 domain; the running max moves only when a logit
//     exceeds it by a slack, and the cross-lane max reduction runs only then.
//   * The waves exchange their P fragments (1 KB each) and rescale factors
//     through LDS, and wave w then computes O for all heads over its own
//     slice of 512/NW output dims, reading V through the transposing LDS
//     read (ds_read_b64_tr_b16): each wave reads 1/NW of the tile's V.
//   * O accumulates in fp32 MFMA accumulators and is normalised at the end.
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <algorithm>
#include <mutex>
#include <type_traits>

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
constexpr int MLA_TILE_CH = MLA_KT * MLA_PCH;   // chunks per tile (2368)
constexpr int MLA_MAX_K = 4096;                 // selected ids per token held in LDS
constexpr float RESCALE_SLACK = 8.0f;           // log2 headroom before O is rescaled
// Running max before any valid logit: finite and below every logit, so that
// the rescale test needs no special case and exp2(x - m) of a padding key
// (x = -inf) is 0.
constexpr float M_INIT = -3.0e38f;

typedef short v4s16 __attribute__((ext_vector_type(4)));

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt <= n only.
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Workgroup barrier over LDS that leaves the tile gathers in flight: this
// wave's LDS operations are complete (lgkmcnt 0), the compiler may move no
// memory access across it, and no fence drains the outstanding loads.
JANUS_DEV void lds_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4s16 lds_v4s16;

// The lane id made inside the code that uses it: the compiler can neither
// hoist it out of a rarely taken branch nor keep it live (and spill it)
// across the tile loop.
JANUS_DEV int lane_here()
{
    int ln;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
    return ln;
}


// Largest of the 8 MFMA results in a (with b): v_max3 on the raw results.
// The compiler puts a canonicalizing max in front of each MFMA result it
// passes to fmaxf; written as assembly the reduction is four instructions,
// after the wait states a VALU read of an MFMA result needs (the compiler
// inserts none ahead of inline assembly).
JANUS_DEV float max8(const v4f &a, const v4f &b)
{
    float x, y;
    asm("s_nop 7\n\ts_nop 7\n\t"
        "v_max3_f32 %0, %2, %3, %4\n\t"
        "v_max3_f32 %1, %5, %6, %7"
        : "=&v"(x), "=&v"(y)
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(b[0]), "v"(b[1]));
    float z;
    asm("v_max3_f32 %0, %1, %2, %3\n\tv_max3_f32 %0, %0, %4, %5"
        : "=&v"(z)
        : "v"(x), "v"(y), "v"(a[3]), "v"(b[2]), "v"(b[3]));
    return z;
}

// Transposing LDS read (ds_read_b64_tr_b16): within each 16-lane group,
// lane i's element j is element i%4 of the 8 bytes addressed by lane 4j+i/4.
JANUS_DEV v4s16 lds_read_tr16(const uint8_t *lds_base, int byte_off)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s16 *)((__attribute__((address_space(3))) uint8_t *)lds_base + byte_off));
}

// One 16-byte-per-lane gather into LDS (global_load_lds_dwordx4: lane l's
// 16 bytes from src land at dst + 16 l), written as assembly so that the
// compiler does not wait for every outstanding LDS read at the next use of
// any of them, as it does after the builtin.  M0 holds the LDS address (one
// wait state before the load reads it) and is restored afterwards.
JANUS_DEV void gather16(const uint8_t *src, uint8_t *dst)
{
    const uint32_t m = (uint32_t)(uintptr_t)(lds_void *)dst;
    int saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, off\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "s"(m), "v"(src)
                 : "memory");
}

// Every wave issues the same number of gather instructions per tile, so a
// counted wait is exact; instruction slots past the tile's chunks load a
// dummy chunk into padding.
// fp8 KV rows: 576 e4m3 bytes, the row's fp32 scale at byte 576, padding to
// 592 bytes (37 chunks, all gathered).  A tile keeps that pitch in LDS, with
// keys 16..31 a further 128 bytes on: the K reads (keys c16 and c16+16, in
// separate instructions) and the transposing V reads (keys 4g+j and
// 16+4g+j, together) then each touch distinct 16-byte bank groups.
constexpr int KV8_ROWB = 592;
constexpr int KV8_CPR = KV8_ROWB / 16;                   // 37
constexpr int KV8_GAP = 8;                               // chunks between keys 15 and 16
constexpr int KV8_TILE_CH = MLA_KT * KV8_CPR + KV8_GAP;  // 1192
constexpr int KV8_SCALE = MLA_DQK;                       // byte of the scale in a row
JANUS_DEV int kv8_key_off(int r) { return r * KV8_ROWB + (r >= 16 ? KV8_GAP * 16 : 0); }
// fp8 rows: K-step at which a tile's key scales are read (their LDS latency
// passes under the remaining steps; at step 4, the last, 1.3% slower)
constexpr int KS_STEP = 3;
// fp8 rows: S^T = K Q^T on the fp8 MFMA (16x16x128), in five K-steps: dims
// 128c .. 128c+127 for c < 4 (lane group grp holds dims 128c + 32grp .. +31),
// then the 64 tail dims, whose MFMA takes the high parts of the queries in
// lane groups 0-1 and the low parts in groups 2-3 against the same key bytes
constexpr int KV8_STEPS = 5;

// bf16 rows in a tile buffer: dims 0..511 of key row r ("main", 1 KB) at
// r * MLA_ROWB, so that one gather instruction loads one row and its source
// row is wave-uniform; dims 512..575 of the 32 rows ("tail", 4 KB) after
// them, in four 1 KB blocks of eight rows, one gather instruction each.  In
// tail block m, row r (= 8m + i) and chunk cc (dims 512 + 8cc ..) sit at
// 16-byte slot 8*(cc ^ m) + (i ^ cc): the 16 rows of one K-operand read then
// fall in 16 different 16-byte bank groups.
constexpr int MLA_TAIL = MLA_KT * MLA_ROWB;      // 37888
constexpr int MLA_BUF16 = MLA_TAIL + 4 * 1024;   // 41984
JANUS_DEV int tail_off(int r, int cc)
{
    const int m = r >> 3;
    return MLA_TAIL + 1024 * m + 16 * (8 * (cc ^ m) + ((r & 7) ^ cc));
}

template <bool KV8>
constexpr int mla_tile_ch() { return KV8 ? KV8_TILE_CH : MLA_TILE_CH; }
template <int NW, bool KV8>
constexpr int mla_ipw() { return ((mla_tile_ch<KV8>() + 63) / 64 + NW - 1) / NW; }
template <int NW, bool KV8>
constexpr int mla_buf_bytes() { return KV8 ? NW * mla_ipw<NW, KV8>() * 64 * 16 : MLA_BUF16; }

// Tile chunk 64*j + lane (j wave-uniform) -> key row r and chunk c of that
// row.  Chunks that are not part of a row (bf16 row padding, the fp8 gap)
// load chunk 0 of key r: a dummy.  For bf16 rows the division by the row
// pitch is done once per wave, leaving each lane an add and a compare.
template <bool KV8>
JANUS_DEV void tile_chunk_j(int j, int lane, int &r, int &c)
{
    if constexpr (KV8) {
        const int qch = 64 * j + lane;
        const bool hi = qch >= 16 * KV8_CPR;
        const int q2 = hi ? qch - 16 * KV8_CPR - KV8_GAP : qch;
        const int rr = q2 < 0 ? 0 : q2 / KV8_CPR;
        r = rr + (hi ? 16 : 0);
        c = q2 < 0 ? 0 : q2 - rr * KV8_CPR;
    } else {
        const int base = 64 * j;
        const int r0 = base / MLA_PCH, rem = base - r0 * MLA_PCH;
        const int t = rem + lane;  // < 2 * MLA_PCH
        const bool wrap = t >= MLA_PCH;
        r = r0 + (wrap ? 1 : 0);
        c = wrap ? t - MLA_PCH : t;
        if (c >= MLA_CPR)
            c = 0;
    }
}

// 8 fp8 e4m3 values -> 8 bf16 (exact: e4m3 values are bf16 values)
JANUS_DEV v8bf fp8x8_to_bf16(v2i x);

// four fp32 values -> four fp8 e4m3 bytes (round to nearest even); the
// values are within the format's range
JANUS_DEV int fp8x4_of(float a, float b, float c, float d)
{
    v2s w = {0, 0};
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, a, b, 1.0f, false);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, c, d, 1.0f, true);
    return __builtin_bit_cast(int, w);
}

// 32 bf16 query values (four 16-byte words) times inv, split into two fp8
// parts, hi + lo == x * inv exactly for |x * inv| < 256 and |x * inv| >= 2^-2
// (hi keeps the 4 leading significant bits of the 8, lo the remaining 4);
// smaller values lose at most 2^-10 to the underflow of lo
JANUS_DEV void split_fp8x32(const v4i (&x)[4], float inv, v8i &hi, v8i &lo)
{
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int w0 = x[u][2 * h], w1 = x[u][2 * h + 1];
            const float f0 = __builtin_bit_cast(float, w0 << 16) * inv;
            const float f1 = __builtin_bit_cast(float, w0 & (int)0xffff0000) * inv;
            const float f2 = __builtin_bit_cast(float, w1 << 16) * inv;
            const float f3 = __builtin_bit_cast(float, w1 & (int)0xffff0000) * inv;
            const int hw = fp8x4_of(f0, f1, f2, f3);
            const v2f b01 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(hw, 1.0f, false);
            const v2f b23 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(hw, 1.0f, true);
            hi[2 * u + h] = hw;
            lo[2 * u + h] = fp8x4_of(f0 - b01[0], f1 - b01[1], f2 - b23[0], f3 - b23[1]);
        }
}

// S^T += K Q^T over 128 dims on fp8 operands (E8M0 scales 1)
JANUS_DEV v4f mfma_fp8x128(v8i a, v8i b, v4f c)
{
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

JANUS_DEV v8bf fp8x8_to_bf16(v2i x)
{
    const v2bf a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[0], 1.0f, false);
    const v2bf b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[0], 1.0f, true);
    const v2bf c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[1], 1.0f, false);
    const v2bf d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[1], 1.0f, true);
    return v8bf{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// Transposing LDS read of bytes (ds_read_b64_tr_b8): within each 16-lane
// group, lane i's byte j is byte i%8 of the 8 bytes addressed by lane 2j+i/8.
JANUS_DEV v2i lds_read_tr8(const uint8_t *lds_base, int byte_off)
{
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32(
        (__attribute__((address_space(3))) v2i *)((__attribute__((address_space(3))) uint8_t *)lds_base + byte_off));
}

template <int NW, bool SPLIT, bool KV8>
__global__ __launch_bounds__(64 * NW, 1) void sparse_mla_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs, int es,
    const uint16_t *__restrict__ q, const uint8_t *__restrict__ kv, int64_t row_bytes,
    const int32_t *__restrict__ page_table, int pt_ld, int page_shift, const int32_t *__restrict__ topk,
    int k, float scale_log2, void *__restrict__ out, int out_f32, float *__restrict__ lse, int num_splits,
    float *__restrict__ part)
{
    constexpr int HQ = 16 * NW;  // one 16-head MFMA block per wave for S and P
    constexpr int NT = 64 * NW;
    constexpr int IPW = mla_ipw<NW, KV8>();
    constexpr int BUF = mla_buf_bytes<NW, KV8>();
    constexpr int TILE_CH = mla_tile_ch<KV8>();
    // three tile buffers; tile_step's restrict-qualified pointers let the
    // compiler see that reading one never waits for the gather into another
    __shared__ __attribute__((aligned(16))) uint8_t sKV0[BUF];
    __shared__ __attribute__((aligned(16))) uint8_t sKV1[BUF];
    __shared__ __attribute__((aligned(16))) uint8_t sKV2[BUF];
    __shared__ int32_t sSlot[MLA_MAX_K];
    __shared__ v4i sP[NW * 64];      // P fragments: wave w's lane l at 64w + l
    __shared__ float sAlpha[HQ];     // O rescale factor per head this tile
    __shared__ int32_t sResc[NW];    // wave w's heads were rescaled this tile
    __shared__ float sInvL[HQ];      // 1 / softmax denominator per head
    __shared__ v8i sQT[KV8 ? NW * 64 : 1];  // fp8 rows: the tail K-step's query operand, wave w's lane l at 64w + l

    // SPLIT: block (g, sp) is token g, slice sp of its selection (whole
    // tiles); otherwise block g is token g over its whole selection
    const int g = SPLIT ? blockIdx.x / num_splits : blockIdx.x;
    int kl = k;  // ids in this block's slice (may be 0 when split)
    const int32_t *sel = topk + (int64_t)g * k;
    if constexpr (SPLIT) {
        const int sp = blockIdx.x % num_splits;
        const int tps = ((k + MLA_KT - 1) / MLA_KT + num_splits - 1) / num_splits;
        const int j0 = min(k, sp * tps * MLA_KT);
        kl = min(k, j0 + tps * MLA_KT) - j0;
        sel += j0;
    }
    const int b = session_of_row(q_start, num_seqs, g);
    const int lim = last_cand(hist_len[b], g - q_start[b], es);  // last causal id
    const int32_t *pt = page_table + (int64_t)b * pt_ld;
    const int psz_mask = (1 << page_shift) - 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c16 = lane & 15, grp = lane >> 4;
    const int head0 = 16 * wave;

    // physical row of every selected id (-1: padding)
    for (int j = tid; j < kl; j += NT) {
        const int s = sel[j];
        sSlot[j] = (s >= 0 && s <= lim) ? ((pt[s >> page_shift] << page_shift) + (s & psz_mask)) : -1;
    }
    // queries of head head0 + c16.  bf16 rows: dims 32*step + 8*grp .. +7.
    // fp8 rows: q = s * (hi + lo) with hi and lo fp8 and s a power of two per
    // head (max |q| / s < 256), so that S^T runs on the fp8 MFMA straight
    // from the stored key bytes; qf[c] and qf[4 + c] hold hi and lo of dims
    // 128c + 32grp .. +31, and sQT the tail (dims 512 + 32(grp & 1) .. +31:
    // hi in lane groups 0-1, lo in 2-3), read back at each tile's tail step
    // (its registers are what the kernel lacks).  The split is exact for
    // every value above 2^-10 of its head's largest and loses at most
    // 2^-18 of that largest below, so a logit is within 576 * 2^-18 *
    // max|q| * max|k| (under 2^-8.8 of their product) of q.k, beside fp32
    // rounding
    using QReg = std::conditional_t<KV8, v8i, v8bf>;
    QReg qf[KV8 ? 8 : MLA_STEPS];
    float ksc = scale_log2;  // logit scale (fp8 rows: times s)
    if constexpr (KV8) {
        const uint16_t *qr = q + ((int64_t)g * HQ + head0 + c16) * MLA_DQK;
        auto qword = [&](int c, int u) {
            return *(const v4i *)(qr + (c < 4 ? 128 * c + 32 * grp : MLA_DV + 32 * (grp & 1)) + 8 * u);
        };
        // max |q| over the head: lanes c16 + 16 * grp (finite bf16
        // magnitudes order as integers);
        // the words are read again for the split, one step at a time, so
        // that they are never all held in registers
        int mlo = 0, mhi = 0;
#pragma unroll
        for (int c = 0; c < 5; ++c)
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const v4i w = qword(c, u);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    mlo = max(mlo, w[e] & 0x7fff);
                    mhi = max(mhi, (int)((uint32_t)w[e] >> 16) & 0x7fff);
                }
            }
        asm volatile("" ::: "memory");
        int mq = max(mlo, mhi);
#pragma unroll
        for (int off = 16; off <= 32; off <<= 1)
            mq = max(mq, __shfl_xor(mq, off));
        int ex;
        (void)frexpf(__builtin_bit_cast(float, mq << 16), &ex);  // max |q| < 2^ex
        ex = min(max(ex, -100), 120);
        const float inv = ldexpf(1.0f, 8 - ex);
        ksc = scale_log2 * ldexpf(1.0f, ex - 8);
#pragma unroll
        for (int c = 0; c < 5; ++c) {
            const v4i raw[4] = {qword(c, 0), qword(c, 1), qword(c, 2), qword(c, 3)};
            if (c < 4) {
                split_fp8x32(raw, inv, qf[c], qf[4 + c]);
            } else {
                v8i th, tl;
                split_fp8x32(raw, inv, th, tl);
                sQT[64 * wave + lane] = grp < 2 ? th : tl;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        const uint16_t *qr = q + ((int64_t)g * HQ + head0 + c16) * MLA_DQK + 8 * grp;
#pragma unroll
        for (int st = 0; st < MLA_STEPS; ++st)
            qf[st] = as_v8bf(*(const v4i *)(qr + 32 * st));
    }
    // O for all HQ heads (head block hb = rows 16*hb .. 16*hb+15) over this
    // wave's NBW blocks of 16 output dims, dims 16*(NBW*wave + nl) + c16
    constexpr int NBW = MLA_NB / NW;
    v4f o[NW][NBW];
#pragma unroll
    for (int hb = 0; hb < NW; ++hb)
#pragma unroll
        for (int nl = 0; nl < NBW; ++nl)
            o[hb][nl] = v4f{0.f, 0.f, 0.f, 0.f};
    float m = M_INIT, lsum = 0.f;  // head head0 + c16
    __syncthreads();

    const int ntiles = (kl + MLA_KT - 1) / MLA_KT;
    // ---- fp8 rows: gather of tile t: the wave's instruction i fills LDS
    // chunks 64j .. 64j+63, j = wave + NW*i (chunks of the gap load a dummy;
    // padding ids load row 0; slots past the tile load a dummy too)
    auto issue = [&](int t, int i0, int i1, uint8_t *__restrict__ dst) {
#pragma unroll 1
        for (int i = i0; i < i1; ++i) {
            const int j = wave + NW * i;
            const int qch = 64 * j + lane;
            int r, c;
            tile_chunk_j<KV8>(j, lane, r, c);
            const int key = MLA_KT * t + r;
            int slot = (qch < TILE_CH && key < kl) ? sSlot[key] : -1;
            if (slot < 0)
                slot = 0;  // padding rows read a real row; their logits are masked
            const uint8_t *src = kv + (uint64_t)(uint32_t)slot * (uint32_t)row_bytes + 16 * c;
            gather16(src, dst + (64 * j) * 16);
        }
    };

    // a fixed group of the wave's gather instructions [I0, I1): their slots
    // are read together, so the group waits for one LDS round trip
    auto issue_group = [&](auto I0c, auto I1c, int t, uint8_t *__restrict__ dst) {
        constexpr int I0 = decltype(I0c)::value, I1 = decltype(I1c)::value, NG = I1 - I0;
        int ln = lane;
        asm volatile("" : "+v"(ln));  // keep the chunk positions in this loop, not hoisted out of it
        int slot[NG], cc[NG];
#pragma unroll
        for (int u = 0; u < NG; ++u) {
            const int qch = 64 * (wave + NW * (I0 + u)) + ln;
            int r, c;
            tile_chunk_j<KV8>(wave + NW * (I0 + u), ln, r, c);
            const int key = MLA_KT * t + r;
            slot[u] = (qch < TILE_CH && key < kl) ? sSlot[key] : -1;
            cc[u] = c;
        }
#pragma unroll
        for (int u = 0; u < NG; ++u) {
            const int j = wave + NW * (I0 + u);
            const int sl = slot[u] < 0 ? 0 : slot[u];  // padding rows read a real row; their logits are masked
            const uint8_t *src = kv + (uint64_t)(uint32_t)sl * (uint32_t)row_bytes + 16 * cc[u];
            gather16(src, dst + (64 * j) * 16);
        }
    };
    constexpr bool SPREAD8 = KV8 && IPW >= 2;
    auto spread_part = [&](auto Qc, int t, uint8_t *__restrict__ dst) {
        constexpr int Q = decltype(Qc)::value;
        constexpr int I0 = IPW <= 5 ? Q : Q * IPW / 5;
        constexpr int I1 = IPW <= 5 ? (Q < IPW ? Q + 1 : Q) : (Q + 1) * IPW / 5;
        if constexpr (I1 > I0)
            issue_group(std::integral_constant<int, I0>{}, std::integral_constant<int, I1>{}, t, dst);
    };

    // ---- bf16 rows: wave w gathers main rows MROWS*w .. MROWS*w+MROWS-1
    // (one instruction each: a wave-uniform source row, its slot taken from
    // a register of prefetched slots) and tail blocks m = w + NW*u < 4
    constexpr int MROWS = MLA_KT / NW;
    constexpr int NTAIL = NW >= 4 ? 1 : 4 / NW;
    const bool has_tail = wave < 4;  // (every wave when NW <= 4)
    // the row and chunk tail block m's lane loads
    auto tail_rc = [&](int m, int ln, int &r, int &cc) {
        cc = (ln >> 3) ^ m;
        r = 8 * m + ((ln & 7) ^ cc);
    };
    // slots of tile tt: lane l < 32 (and l - 32) holds row l's, ts[u] the
    // one of the row this lane loads in tail block wave + NW*u
    auto read_slots = [&](int tt, int &vs, int (&ts)[NTAIL]) {
        int ln = lane;
        asm volatile("" : "+v"(ln));
        vs = sSlot[min(MLA_KT * tt + (ln & 31), kl - 1)];
#pragma unroll
        for (int u = 0; u < NTAIL; ++u) {
            int r, cc;
            tail_rc(min(wave + NW * u, 3), ln, r, cc);
            ts[u] = sSlot[min(MLA_KT * tt + r, kl - 1)];
        }
    };
    // main row i of this wave for tile tt
    auto fire_main = [&](int i, int tt, int vs, uint8_t *__restrict__ dst) {
        const int r = MROWS * wave + i;
        int sl = __builtin_amdgcn_readlane(vs, r);
        if (MLA_KT * tt + r >= kl || sl < 0)
            sl = 0;  // padding rows read a real row; their logits are masked
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const uint8_t *src = kv + (uint64_t)(uint32_t)sl * (uint32_t)row_bytes + 16 * ln;
        gather16(src, dst + r * MLA_ROWB);
    };
    auto fire_tails = [&](int tt, const int (&ts)[NTAIL], uint8_t *__restrict__ dst) {
        int ln = lane;
        asm volatile("" : "+v"(ln));
#pragma unroll
        for (int u = 0; u < NTAIL; ++u) {
            const int m = wave + NW * u;
            int r, cc;
            tail_rc(m, ln, r, cc);
            const int sl = (MLA_KT * tt + r < kl && ts[u] >= 0) ? ts[u] : 0;
            const uint8_t *src = kv + (uint64_t)(uint32_t)sl * (uint32_t)row_bytes + 16 * (64 + cc);
            gather16(src, dst + MLA_TAIL + 1024 * m);
        }
    };
    // all of tile tt's gathers at once (the first two tiles)
    auto issue_all = [&](int tt, uint8_t *__restrict__ dst) {
        if constexpr (KV8) {
            issue(tt, 0, IPW, dst);
        } else {
            int vs, ts[NTAIL];
            read_slots(tt, vs, ts);
#pragma unroll 1
            for (int i = 0; i < MROWS; ++i)
                fire_main(i, tt, vs, dst);
            if (has_tail)
                fire_tails(tt, ts, dst);
        }
    };
    // wait until this wave's gathers of the tile before the newest one
    // have landed (pending: the newest tile's are in flight)
    auto wait_gathers = [&](bool pending) {
        if (!pending)
            __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
        else if constexpr (KV8)
            __builtin_amdgcn_s_waitcnt(vmcnt_only(IPW));
        else if (has_tail)
            __builtin_amdgcn_s_waitcnt(vmcnt_only(MROWS + NTAIL));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_only(MROWS));
    };
    // issue point q (0..4) inside tile t's S loop, for the gathers of tile
    // t+2: bf16 main rows in four parts, then the tails; fp8 in five groups
    // (with eight waves one instruction each) or all at point 0
    auto issue_part = [&](int t, int part, int vs, const int (&ts)[NTAIL], uint8_t *__restrict__ dst) {
        if (t + 2 >= ntiles)
            return;
        if constexpr (KV8) {
            if constexpr (SPREAD8) {
                switch (part) {
                case 0: spread_part(std::integral_constant<int, 0>{}, t + 2, dst); break;
                case 1: spread_part(std::integral_constant<int, 1>{}, t + 2, dst); break;
                case 2: spread_part(std::integral_constant<int, 2>{}, t + 2, dst); break;
                case 3: spread_part(std::integral_constant<int, 3>{}, t + 2, dst); break;
                case 4: spread_part(std::integral_constant<int, 4>{}, t + 2, dst); break;
                default: break;
                }
            } else if (part == 0) {
                issue(t + 2, 0, IPW, dst);
            }
        } else if (part < 4) {
#pragma unroll
            for (int i = part * MROWS / 4; i < (part + 1) * MROWS / 4; ++i)
                fire_main(i, t + 2, vs, dst);
        } else if (has_tail) {
            fire_tails(t + 2, ts, dst);
        }
    };
    auto tile_step = [&](int t, const uint8_t *__restrict__ tile, uint8_t *__restrict__ next) {
        // slots of tile t+2's gathers (bf16), read now so that their LDS
        // latency passes under the first K-steps (rows past the selection
        // read a clamped slot and are redirected when their gather fires)
        int vs = 0, ts[NTAIL];
#pragma unroll
        for (int u = 0; u < NTAIL; ++u)
            ts[u] = 0;
        if constexpr (!KV8)
            read_slots(t + 2, vs, ts);
        int vslot;
        float ks[2][4];  // fp8 rows: scales of keys 16*kb + 4*grp + i
        // S^T[key][head] = K Q^T for keys 16*kb + 4*grp + i
        v4f st0 = v4f{0.f, 0.f, 0.f, 0.f}, st1 = st0;
        // K operands for keys c16 and c16 + 16: bf16 rows, 16 bytes per lane
        // and K-step; fp8 rows, 32 (the key bytes themselves).  Q and O fill
        // most of the registers, so the compiler alone keeps too few operand
        // reads in flight: each step loads the operands of a later step into
        // a ring (bf16 two steps ahead, fp8 one), and a scheduling fence per
        // step keeps it from hoisting more than that.  The ring keeps its
        // reads in flight only because the gathers are assembly (gather16):
        // after the builtin the compiler waits for every outstanding LDS read
        using KRaw = v4i;
        constexpr int SB = 64;  // bytes per K-step
        const uint8_t *row0 = tile + c16 * MLA_ROWB + 16 * grp;
        const uint8_t *row1 = row0 + 16 * MLA_ROWB;
        // fp8 rows: the waves raise their priority over the MFMA loops, so
        // that a wave still in them is issued ahead of one in the softmax
        // or P·V VALU work
        if constexpr (KV8)
            __builtin_amdgcn_s_setprio(1);
        // K operand of a step for keys c16 (h = 0) and c16 + 16 (h = 1): bf16
        // steps 16 and 17 (dims 512..575) come from the tail blocks
        // (tail addresses from an opaque copy of the lane index, so that the
        // compiler computes them here instead of keeping them for the whole loop)
        int lnk = lane;
        asm volatile("" : "+v"(lnk));
        auto kop = [&](int step, int h) -> KRaw {
            if (!KV8 && step >= 16)
                return *(const KRaw *)(tile + tail_off((lnk & 15) + 16 * h, 4 * (step - 16) + (lnk >> 4)));
            return *(const KRaw *)((h ? row1 : row0) + SB * step);
        };
        // two steps ahead: a three-entry ring (fp8 rows: a two-entry ring
        // of step pairs, each 16-byte read holding two steps' operands)
        constexpr int AHEAD = 2;
        KRaw ring[AHEAD + 1][2];
        // fp8 rows: key bytes of K-step c (tail: lane groups 2-3 repeat the
        // bytes of groups 0-1).  Operand j = 2c + h (keys c16 + 16h) lives in
        // kring[j % 3]: a step's first MFMAs find the next step's keys c16
        // loaded, and each operand's register is refilled after its last MFMA
        const uint8_t *arow0 = tile + kv8_key_off(c16) + 32 * grp, *arow1 = tile + kv8_key_off(c16 + 16) + 32 * grp;
        const int tail8 = MLA_DV + 32 * (grp & 1) - 32 * grp;
        auto kop8 = [&](int c, int h) -> v8i {
            // an opaque offset keeps each read in its step (the compiler
            // otherwise hoists them all to the top of the tile)
            int o = c < 4 ? 128 * c : tail8;
            asm volatile("" : "+v"(o));
            const uint8_t *p = (h ? arow1 : arow0) + o;
            const v4i a = *(const v4i *)p, b = *(const v4i *)(p + 16);
            return v8i{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        };
        v8i kring[3], qtail;
        constexpr int NSTEP = KV8 ? KV8_STEPS : MLA_STEPS;
        if constexpr (KV8) {
            kring[0] = kop8(0, 0);
            kring[1] = kop8(0, 1);
            kring[2] = kop8(1, 0);
        } else {
#pragma unroll
            for (int a = 0; a < AHEAD; ++a) {
                ring[a][0] = kop(a, 0);
                ring[a][1] = kop(a, 1);
            }
        }
#pragma unroll
        for (int step = 0; step < NSTEP; ++step) {
            if constexpr (KV8) {
                const int j0 = 2 * step;
                if (step == 3)
                    qtail = sQT[64 * wave + lnk];
                const v8i qa = step < 4 ? qf[step] : qtail;
                st0 = mfma_fp8x128(kring[j0 % 3], qa, st0);
                st1 = mfma_fp8x128(kring[(j0 + 1) % 3], qa, st1);
                if (step < 4) {
                    st0 = mfma_fp8x128(kring[j0 % 3], qf[4 + step], st0);
                    kring[j0 % 3] = kop8(step + 1, 1);
                    st1 = mfma_fp8x128(kring[(j0 + 1) % 3], qf[4 + step], st1);
                    if (step + 2 < NSTEP)
                        kring[(j0 + 1) % 3] = kop8(step + 2, 0);
                }
                // a use of the products here keeps the MFMAs in their step:
                // the compiler otherwise sinks them all past the branches of
                // the gather issue, holding every step's key operands at once
                asm volatile("" ::"v"(st0), "v"(st1));
            } else {
            if (step + AHEAD < MLA_STEPS) {
                ring[(step + AHEAD) % (AHEAD + 1)][0] = kop(step + AHEAD, 0);
                ring[(step + AHEAD) % (AHEAD + 1)][1] = kop(step + AHEAD, 1);
            }
            st0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(ring[step % (AHEAD + 1)][0]), qf[step], st0, 0, 0,
                                                          0);
            st1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(ring[step % (AHEAD + 1)][1]), qf[step], st1, 0, 0,
                                                          0);
            }
            // issue points: fp8 at every step; bf16 at 2, 6, 10, 14 and 17,
            // after the slots read at the top of the tile have landed
            if (KV8 || step % 4 == 2 || step == MLA_STEPS - 1)
                issue_part(t, KV8 ? step : (step == MLA_STEPS - 1 ? 4 : step / 4), vs, ts, next);
            // this tile's slots (for its valid keys), read under the last
            // MFMAs (bf16 rows: the last three steps, fp8 rows: two)
            if (step == (KV8 ? NSTEP - 2 : NSTEP - 3))
                vslot = sSlot[min(MLA_KT * t + (lane & 31), kl - 1)];
            if constexpr (KV8) {
                if (step == KS_STEP) {
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            ks[kb][i] = *(const float *)(tile + kv8_key_off(16 * kb + 4 * grp + i) + KV8_SCALE);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (KV8)
            __builtin_amdgcn_s_setprio(0);
        // online softmax (exp2 domain) with lazy rescaling of O.  Valid keys
        // of the tile come as a 32-bit mask (lanes 32-63 repeat 0-31); this
        // lane's keys are 16*kb + 4*grp + i
        const uint32_t vbits = (uint32_t)__ballot(MLA_KT * t + (lane & 31) < kl && vslot >= 0);
        const uint32_t vmask = vbits >> (4 * (KV8 ? grp : lane_here() >> 4));
        // the common case - every key of the tile valid, bf16 rows and a
        // positive scale - takes the max over the raw products and one fma
        // per probability, with no masks
        const bool fast = vbits == 0xFFFFFFFFu && scale_log2 > 0.f;
        // fp8 rows: each key's scale (ks, read from step KS_STEP on)
        // multiplies its logit and its probability
        float x[2][4];
        float mx = -INFINITY;
        if (fast) {
            if constexpr (KV8) {
                // fp8 rows: no masks, each logit times its key's scale
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    x[0][i] = st0[i] * (ksc * ks[0][i]);
                    x[1][i] = st1[i] * (ksc * ks[1][i]);
                }
                mx = fmaxf(fmaxf(fmaxf(x[0][0], x[0][1]), fmaxf(x[0][2], x[0][3])),
                           fmaxf(fmaxf(x[1][0], x[1][1]), fmaxf(x[1][2], x[1][3])));
            } else {
                mx = scale_log2 * max8(st0, st1);
            }
        } else {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool ok = (vmask >> (16 * kb + i)) & 1u;
                    const float sc = KV8 ? ksc * ks[kb][i] : scale_log2;
                    x[kb][i] = ok ? (kb ? st1[i] : st0[i]) * sc : -INFINITY;
                    mx = fmaxf(mx, x[kb][i]);
                }
        }
        // the running max m is common to a head's four lane groups; it only
        // moves when some key exceeds it by the slack, which is rare after
        // the first tiles, so the cross-lane reduction runs only then
        const bool over = mx > m + RESCALE_SLACK;
        const bool resc = __ballot(over) != 0;
        if (resc) {
            const int ln = lane_here();
            mx = fmaxf(mx, __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((ln ^ 16) << 2,
                                                                                  __builtin_bit_cast(int, mx))));
            mx = fmaxf(mx, __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((ln ^ 32) << 2,
                                                                                  __builtin_bit_cast(int, mx))));
            const bool grow = mx > m + RESCALE_SLACK;
            const float mnew = grow ? mx : m;
            const float alpha = __builtin_amdgcn_exp2f(m - mnew);
            lsum *= alpha;
            m = mnew;
            if (ln < 16)
                sAlpha[head0 + ln] = alpha;
        }
        if (lane == 0)
            sResc[wave] = resc;
        float pv[2][4];
        if (fast) {
            // m is finite here: a finite max has just been taken
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if constexpr (KV8) {
                        pv[kb][i] = __builtin_amdgcn_exp2f(x[kb][i] - m);
                        lsum += pv[kb][i];
                        pv[kb][i] *= ks[kb][i];  // V_s = scale_s * (stored row)
                    } else {
                        pv[kb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(kb ? st1[i] : st0[i], scale_log2, -m));
                        lsum += pv[kb][i];
                    }
                }
        } else {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[kb][i] = __builtin_amdgcn_exp2f(x[kb][i] - m);
                    lsum += pv[kb][i];
                    if constexpr (KV8)  // V_s = scale_s * (stored row); padding keys stay 0
                        pv[kb][i] = ((vmask >> (16 * kb + i)) & 1u) ? pv[kb][i] * ks[kb][i] : 0.f;
                }
        }
        const v8bf pa = v8bf{(__bf16)pv[0][0], (__bf16)pv[0][1], (__bf16)pv[0][2], (__bf16)pv[0][3],
                             (__bf16)pv[1][0], (__bf16)pv[1][1], (__bf16)pv[1][2], (__bf16)pv[1][3]};
        sP[64 * wave + lane] = __builtin_bit_cast(v4i, pa);
        lds_barrier();

        // O += P V over this wave's output dims for every head.  The P
        // fragment of head block hb is exactly an A operand (rows: heads
        // 16*hb + c16; slots: keys 4*grp + i and 16 + 4*grp + i).  V operand:
        // those keys, lane (r' = c16/4, cc = c16%4) addressing dims
        // 16*nb + 4*cc .. +3 of its key row
        // head blocks rescaled this tile (wave-uniform), read before the V
        // operands so that waiting for them does not wait for those
        uint32_t rmask = 0;
#pragma unroll
        for (int hb = 0; hb < NW; ++hb)
            rmask |= (sResc[hb] != 0 ? 1u : 0u) << hb;
        v8bf bv[NBW];
        if constexpr (KV8) {
            // fp8 rows: lane (c16, grp) addresses key j = c16/2 of the P
            // fragment's order (4*grp + j, then 16 + 4*grp + j - 4), bytes
            // 8*(c16&1) .. of a 16-dim block; the byte transpose hands it
            // those 8 keys at dim 16*nb + c16
            const int j = c16 >> 1;
            const int vkey8 = j < 4 ? 4 * grp + j : 12 + 4 * grp + j;
            const uint8_t *vrow = tile + kv8_key_off(vkey8) + 8 * (c16 & 1);
#pragma unroll
            for (int nl = 0; nl < NBW; ++nl)
                bv[nl] = fp8x8_to_bf16(lds_read_tr8(vrow, 16 * (NBW * wave + nl)));
        } else {
            const int rr0 = 4 * grp + (c16 >> 2), cc = c16 & 3;
            const uint8_t *vrow0 = tile + rr0 * MLA_ROWB, *vrow1 = vrow0 + 16 * MLA_ROWB;
            const int voff = 16 * (cc >> 1) + (cc & 1) * 8;
#pragma unroll
            for (int nl = 0; nl < NBW; ++nl) {
                const int nb = NBW * wave + nl;
                const v4s16 lo = lds_read_tr16(vrow0, voff + 32 * nb);
                const v4s16 hi = lds_read_tr16(vrow1, voff + 32 * nb);
                bv[nl] = __builtin_bit_cast(v8bf, (v8s16){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
            }
        }
        if constexpr (KV8)
            __builtin_amdgcn_s_setprio(1);
        // P fragments one head block ahead
        v4i pf[2];
        pf[0] = sP[lane];
#pragma unroll
        for (int hb = 0; hb < NW; ++hb) {
            if (hb + 1 < NW)
                pf[(hb + 1) & 1] = sP[64 * (hb + 1) + lane];
            if (rmask & (1u << hb)) {
                float ai[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    ai[i] = sAlpha[16 * hb + 4 * grp + i];
#pragma unroll
                for (int nl = 0; nl < NBW; ++nl)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        o[hb][nl][i] *= ai[i];
            }
            const v8bf ph = __builtin_bit_cast(v8bf, pf[hb & 1]);
#pragma unroll
            for (int nl = 0; nl < NBW; ++nl)
                o[hb][nl] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, bv[nl], o[hb][nl], 0, 0, 0);
        }
        if constexpr (KV8)
            __builtin_amdgcn_s_setprio(0);
        // tile t+1 has landed once at most tile t+2's gathers are pending; the
        // barrier also frees this tile's buffer for the gather of tile t+3
        wait_gathers(t + 2 < ntiles);
        lds_barrier();
    };

    // the queries have landed before any gather goes out: the compiler does
    // not count the gathers (assembly), so it must see nothing of its own
    // outstanding inside the tile loop
    __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
    if (ntiles > 0)
        issue_all(0, sKV0);
    if (ntiles > 1)
        issue_all(1, sKV1);
    wait_gathers(ntiles > 1);
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
        const int r3 = t % 3;
        uint8_t *cur = r3 == 0 ? sKV0 : r3 == 1 ? sKV1 : sKV2;
        uint8_t *nxt = r3 == 0 ? sKV2 : r3 == 1 ? sKV0 : sKV1;
        tile_step(t, cur, nxt);
    }
    if constexpr (SPLIT) {
        // one slice of a split selection: this slice's unnormalised O, and per
        // head the max it is relative to (exp2 domain) and its sum, for
        // attn_combine; layout [blocks][HQ][MLA_DV] then [blocks][HQ][2]
        float l = lsum;
        l += __shfl_xor(l, 16, 64);
        l += __shfl_xor(l, 32, 64);
        if (grp == 0) {
            float *ml = part + (int64_t)gridDim.x * HQ * MLA_DV + ((int64_t)blockIdx.x * HQ + head0 + c16) * 2;
            ml[0] = l > 0.f ? m : -INFINITY;  // an empty slice: -inf, as the merge expects
            ml[1] = l;
        }
#pragma unroll
        for (int hb = 0; hb < NW; ++hb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int h = 16 * hb + 4 * grp + i;
                float *orow = part + ((int64_t)blockIdx.x * HQ + h) * MLA_DV;
#pragma unroll
                for (int nl = 0; nl < NBW; ++nl)
                    orow[16 * (NBW * wave + nl) + c16] = o[hb][nl][i];
            }
        return;
    }
    // normalise and store: O rows of head block hb are heads 16*hb + 4*grp + i,
    // column dims 16*(NBW*wave + nl) + c16
    {
        float l = lsum;
        l += __shfl_xor(l, 16, 64);
        l += __shfl_xor(l, 32, 64);
        if (grp == 0) {
            sInvL[head0 + c16] = l > 0.f ? 1.f / l : 0.f;
            if (lse)
                lse[(int64_t)g * HQ + head0 + c16] = l > 0.f ? (m + log2f(l)) * LN2 : -INFINITY;
        }
    }
    __syncthreads();
#pragma unroll
    for (int hb = 0; hb < NW; ++hb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int h = 16 * hb + 4 * grp + i;
            const float inv = sInvL[h];
            const int64_t orow = ((int64_t)g * HQ + h) * MLA_DV;
#pragma unroll
            for (int nl = 0; nl < NBW; ++nl) {
                const int d = 16 * (NBW * wave + nl) + c16;
                const float v = o[hb][nl][i] * inv;
                if (out_f32)
                    ((float *)out)[orow + d] = v;
                else
                    ((uint16_t *)out)[orow + d] = f32_to_bf16_rne(v);
            }
        }
}

// MQA kernel for up to 16 query heads with dqk = dv = 128 and separate K and
// V pools (the attention of the small config: 8 heads sharing one KV head).
// One wave per query token, four independent waves per block (no block
// barriers).  A wave holds its token's queries as the B operand of
// S^T = K Q^T (heads past Hq are zero rows), gathers each 32-key tile's K
// and V rows straight into its own double-buffered LDS tiles, and needs no
// P exchange: its S^T lanes hold 8 keys of one head, the A operand of P V.
// K rows keep 16-byte chunk c at slot c ^ (row & 15), V rows at slot
// c ^ 2(row & 7), so that the K-operand reads and the transposing V reads
// touch distinct bank groups; the gather loads each lane's chunk from the
// pool so that it lands in its swizzled slot.
constexpr int MQA_D = 128;                     // dqk = dv
constexpr int MQA_ROWB = MQA_D * 2;            // bytes per K or V row
constexpr int MQA_TILEB = MLA_KT * MQA_ROWB;   // one 32-row tile (8 KB)
constexpr int MQA_MAX_K = 1024;                // selected ids per token held in LDS
constexpr int MQA_WAVES = 4;                   // tokens per block

__global__ __launch_bounds__(64 * MQA_WAVES, 1) void sparse_mqa_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs, int es, int total_q,
    const uint16_t *__restrict__ q, int Hq, const uint8_t *__restrict__ k_pool, const uint8_t *__restrict__ v_pool,
    int64_t k_row_bytes, int64_t v_row_bytes, const int32_t *__restrict__ page_table, int pt_ld, int page_shift,
    const int32_t *__restrict__ topk, int k, float scale_log2, void *__restrict__ out, int out_f32,
    float *__restrict__ lse)
{
    // per wave: K and V tiles, two of each (separate arrays, so that the
    // compiler tells the gathers into one from the reads of the other), and
    // the token's slots
    __shared__ __attribute__((aligned(16))) uint8_t sK0[MQA_WAVES][MQA_TILEB];
    __shared__ __attribute__((aligned(16))) uint8_t sV0[MQA_WAVES][MQA_TILEB];
    __shared__ __attribute__((aligned(16))) uint8_t sK1[MQA_WAVES][MQA_TILEB];
    __shared__ __attribute__((aligned(16))) uint8_t sV1[MQA_WAVES][MQA_TILEB];
    __shared__ int32_t sSlotW[MQA_WAVES][MQA_MAX_K];
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = blockIdx.x * MQA_WAVES + wave;
    if (g >= total_q)
        return;
    const int c16 = lane & 15, grp = lane >> 4;
    const int b = session_of_row(q_start, num_seqs, g);
    const int lim = last_cand(hist_len[b], g - q_start[b], es);
    const int32_t *pt = page_table + (int64_t)b * pt_ld;
    const int32_t *sel = topk + (int64_t)g * k;
    const int psz_mask = (1 << page_shift) - 1;
    int32_t *slots = sSlotW[wave];
    for (int j = lane; j < k; j += 64) {
        const int s = sel[j];
        slots[j] = (s >= 0 && s <= lim) ? ((pt[s >> page_shift] << page_shift) + (s & psz_mask)) : -1;
    }
    // B operand of S^T = K Q^T: head c16, dims 32*st + 8*grp .. +7
    v8bf qf[4];
    {
        const bool hv = c16 < Hq;
        const uint16_t *qr = q + ((int64_t)g * Hq + (hv ? c16 : 0)) * MQA_D + 8 * grp;
#pragma unroll
        for (int st = 0; st < 4; ++st)
            qf[st] = hv ? as_v8bf(*(const v4i *)(qr + 32 * st)) : as_v8bf(v4i{0, 0, 0, 0});
    }
    // O for heads 4*grp + i over dims 16*nb + c16
    v4f o[8];
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
        o[nb] = v4f{0.f, 0.f, 0.f, 0.f};
    float m = -INFINITY, lsum = 0.f;  // head c16
    __builtin_amdgcn_s_waitcnt(0);     // slots written (this wave reads only its own)

    const int ntiles = (k + MLA_KT - 1) / MLA_KT;
    // gathers of tile t: instruction i loads rows 4i .. 4i+3 (lane l: row
    // 4i + l/16, LDS slot l%16, which holds the row's chunk l%16 ^ swizzle)
    auto issue = [&](int t, uint8_t *__restrict__ kd, uint8_t *__restrict__ vd) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = 4 * i + grp;
            const int j = MLA_KT * t + r;
            int sl = j < k ? slots[j] : -1;
            if (sl < 0)
                sl = 0;  // padding rows read a real row; their logits are masked
            const int ck = c16 ^ (r & 15), cv = c16 ^ (2 * (r & 7));
            const uint8_t *ks = k_pool + (uint64_t)(uint32_t)sl * (uint64_t)k_row_bytes + 16 * ck;
            const uint8_t *vs = v_pool + (uint64_t)(uint32_t)sl * (uint64_t)v_row_bytes + 16 * cv;
            gather16(ks, kd + 1024 * i);
            gather16(vs, vd + 1024 * i);
        }
    };
    if (ntiles > 0)
        issue(0, sK0[wave], sV0[wave]);
    // one tile: its K and V tiles (kt, vt) and the buffers (kn, vn) that take
    // tile t+1's gathers first (they held tile t-1, read in full by now).
    // All four are restrict-qualified, so that the reads of this tile are not
    // made to wait for those gathers.
    auto tile_step = [&](int t, const uint8_t *__restrict__ kt, const uint8_t *__restrict__ vt,
                         uint8_t *__restrict__ kn, uint8_t *__restrict__ vn) {
        if (t + 1 < ntiles) {
            issue(t + 1, kn, vn);
            __builtin_amdgcn_s_waitcnt(vmcnt_only(16));  // tile t has landed
        } else {
            __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
        }
        // S^T for keys 16*kb + 4*grp + i of head c16
        v4f st0 = v4f{0.f, 0.f, 0.f, 0.f}, st1 = st0;
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const int c = 4 * st + grp;
            const v4i k0 = *(const v4i *)(kt + c16 * MQA_ROWB + 16 * (c ^ c16));
            const v4i k1 = *(const v4i *)(kt + (16 + c16) * MQA_ROWB + 16 * (c ^ c16));
            st0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(k0), qf[st], st0, 0, 0, 0);
            st1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(k1), qf[st], st1, 0, 0, 0);
        }
        const int jr = MLA_KT * t + (lane & 31);
        const int vslot = jr < k ? slots[jr] : -1;
        const uint32_t vbits = (uint32_t)__ballot(vslot >= 0);
        const uint32_t vmask = vbits >> (4 * grp);
        float x[2][4];
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool ok = (vmask >> (16 * kb + i)) & 1u;
                x[kb][i] = ok ? (kb ? st1[i] : st0[i]) * scale_log2 : -INFINITY;
                mx = fmaxf(mx, x[kb][i]);
            }
        const bool over = mx > m + RESCALE_SLACK || (m == -INFINITY && mx > -INFINITY);
        if (__ballot(over) != 0) {
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const bool grow = mx > m + RESCALE_SLACK || (m == -INFINITY && mx > -INFINITY);
            const float mnew = grow ? mx : m;
            const float alpha = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - mnew);
            lsum *= alpha;
            m = mnew;
            // O rows are heads 4*grp + i: their factors from lanes 4*grp + i
            float ai[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                ai[i] = __shfl(alpha, 4 * grp + i, 64);
#pragma unroll
            for (int nb = 0; nb < 8; ++nb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    o[nb][i] *= ai[i];
        }
        float pv[2][4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pv[kb][i] = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(x[kb][i] - m);
                lsum += pv[kb][i];
            }
        const v8bf pa = v8bf{(__bf16)pv[0][0], (__bf16)pv[0][1], (__bf16)pv[0][2], (__bf16)pv[0][3],
                             (__bf16)pv[1][0], (__bf16)pv[1][1], (__bf16)pv[1][2], (__bf16)pv[1][3]};
        // V operand: keys 4*grp + j and 16 + 4*grp + j (the P fragment's
        // order), lane (r' = c16/4, cc = c16%4) addressing dims 16*nb + 4*cc ..
        const int rr0 = 4 * grp + (c16 >> 2), cc = c16 & 3;
        const int sw = 2 * (rr0 & 7);  // rr0 + 16 has the same swizzle
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
            const int off = 16 * ((2 * nb + (cc >> 1)) ^ sw) + 8 * (cc & 1);
            const v4s16 lo = lds_read_tr16(vt, rr0 * MQA_ROWB + off);
            const v4s16 hi = lds_read_tr16(vt, (rr0 + 16) * MQA_ROWB + off);
            const v8bf bv = __builtin_bit_cast(v8bf, (v8s16){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
            o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, bv, o[nb], 0, 0, 0);
        }
    };
    // tile t in buffers t % 2 (the loop unrolled by two)
    for (int t = 0; t < ntiles; t += 2) {
        tile_step(t, sK0[wave], sV0[wave], sK1[wave], sV1[wave]);
        if (t + 1 < ntiles)
            tile_step(t + 1, sK1[wave], sV1[wave], sK0[wave], sV0[wave]);
    }
    float l = lsum;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const float inv = l > 0.f ? 1.f / l : 0.f;
    if (grp == 0 && c16 < Hq && lse)
        lse[(int64_t)g * Hq + c16] = l > 0.f ? (m + log2f(l)) * LN2 : -INFINITY;
    float iv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        iv[i] = __shfl(inv, 4 * grp + i, 64);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = 4 * grp + i;
        if (h >= Hq)
            continue;
        const int64_t orow = ((int64_t)g * Hq + h) * MQA_D;
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
            const int d = 16 * nb + c16;
            const float v = o[nb][i] * iv[i];
            if (out_f32)
                ((float *)out)[orow + d] = v;
            else
                ((uint16_t *)out)[orow + d] = f32_to_bf16_rne(v);
        }
    }
}

// Merge of a selection split into S slices (flash-decoding): per (token,
// head), with slice maxima m_s and sums l_s, M = max m_s, w_s = 2^(m_s - M),
// O = sum_s w_s O_s / sum_s w_s l_s and lse = (M + log2 sum_s w_s l_s) ln 2.
// One wave per (token, head), four heads per block; lane l handles dims
// 8l .. 8l+7 with 16-byte loads and stores (dv = 512).
constexpr int COMBINE_HEADS = 4;
constexpr int COMBINE_THREADS = 64 * COMBINE_HEADS;
constexpr int MAX_SPLITS = 16;

__global__ __launch_bounds__(COMBINE_THREADS) void attn_combine(const float *__restrict__ part, int splits, int Hq,
                                                                int dv, void *__restrict__ out, int out_f32,
                                                                float *__restrict__ lse)
{
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * COMBINE_HEADS + w;  // token * Hq + head
    const int64_t g = row / Hq, h = row % Hq;
    const int64_t ntok = (int64_t)gridDim.x * COMBINE_HEADS / Hq;
    const float *ml = part + ntok * splits * Hq * dv;
    float ms[MAX_SPLITS], M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < MAX_SPLITS; ++sp) {
        ms[sp] = sp < splits ? ml[((g * splits + sp) * Hq + h) * 2] : -INFINITY;
        M = fmaxf(M, ms[sp]);
    }
    float L = 0.f;
#pragma unroll
    for (int sp = 0; sp < MAX_SPLITS; ++sp) {
        ms[sp] = (ms[sp] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms[sp] - M);  // the weight w_s
        if (sp < splits)
            L += ms[sp] * ml[((g * splits + sp) * Hq + h) * 2 + 1];
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    v4f acc0 = v4f{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
    for (int sp = 0; sp < MAX_SPLITS; ++sp)
        if (sp < splits) {
            const v4f *src = (const v4f *)(part + ((g * splits + sp) * Hq + h) * dv) + 2 * lane;
            acc0 += ms[sp] * src[0];
            acc1 += ms[sp] * src[1];
        }
    acc0 *= inv;
    acc1 *= inv;
    if (out_f32) {
        v4f *dst = (v4f *)((float *)out + row * dv) + 2 * lane;
        dst[0] = acc0;
        dst[1] = acc1;
    } else {
        const uint32_t p0 = f32_to_bf16_rne(acc0[0]) | ((uint32_t)f32_to_bf16_rne(acc0[1]) << 16);
        const uint32_t p1 = f32_to_bf16_rne(acc0[2]) | ((uint32_t)f32_to_bf16_rne(acc0[3]) << 16);
        const uint32_t p2 = f32_to_bf16_rne(acc1[0]) | ((uint32_t)f32_to_bf16_rne(acc1[1]) << 16);
        const uint32_t p3 = f32_to_bf16_rne(acc1[2]) | ((uint32_t)f32_to_bf16_rne(acc1[3]) << 16);
        ((v4i *)((uint16_t *)out + row * dv))[lane] = v4i{(int)p0, (int)p1, (int)p2, (int)p3};
    }
    if (lse && lane == 0)
        lse[row] = L > 0.f ? (M + log2f(L)) * LN2 : -INFINITY;
}

// Plain vector kernel for any (Hq, dqk, dv) and separate K/V pools: one
// block per (token, head); 256 keys per chunk, one logit per thread.
constexpr int VEC_THREADS = 256;
constexpr int VEC_MAX_DQK = 1024;

__global__ __launch_bounds__(VEC_THREADS) void sparse_attn_vector(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ hist_len, int num_seqs, int es,
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
    const int lim = last_cand(hist_len[b], g - q_start[b], es);
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

namespace janus {

// the MLA MFMA kernels cover this shape (V inside the K rows, 16-byte aligned)
static bool mla_shape(const void *q, int Hq, int dqk, int dv, const void *k_pool, const void *v_pool,
                      int64_t k_row_stride, int64_t v_row_stride, int k)
{
    return dqk == MLA_DQK && dv == MLA_DV && v_pool == k_pool && v_row_stride == k_row_stride &&
           (k_row_stride % 8) == 0 && k_row_stride <= (1 << 30) && (reinterpret_cast<uintptr_t>(k_pool) & 15) == 0 &&
           (reinterpret_cast<uintptr_t>(q) & 15) == 0 && k <= MLA_MAX_K &&
           (Hq == 128 || Hq == 64 || Hq == 32 || Hq == 16);
}

// the MQA shape the MFMA kernel above takes: dqk = dv = 128, at most 16
// heads, k <= 1024, row strides a multiple of 8 elements, 16-byte aligned q
// and pools
static bool mqa_shape(const void *q, int Hq, int dqk, int dv, const void *k_pool, const void *v_pool,
                      int64_t k_row_stride, int64_t v_row_stride, int k)
{
    return dqk == MQA_D && dv == MQA_D && Hq >= 1 && Hq <= 16 && k <= MQA_MAX_K && (k_row_stride % 8) == 0 &&
           (v_row_stride % 8) == 0 && k_row_stride <= (1 << 30) && v_row_stride <= (1 << 30) &&
           (reinterpret_cast<uintptr_t>(k_pool) & 15) == 0 && (reinterpret_cast<uintptr_t>(v_pool) & 15) == 0 &&
           (reinterpret_cast<uintptr_t>(q) & 15) == 0;
}

// one launch of the MLA kernel: splits blocks per token, each over one slice
// of the selection (part = NULL: splits = 1, normalised output); pool rows
// of row_bytes bytes, bf16 or (kv8) fp8 with an inline scale
template <bool KV8>
static void launch_mla(const janus_batch *bt, const void *q, int Hq, const void *k_pool, int64_t row_bytes,
                       const int32_t *page_table, int pt_ld, int shift, const int32_t *topk_idx, int k, float sl2,
                       void *out, int of32, float *lse, int splits, float *part, hipStream_t st)
{
    const auto *qq = (const uint16_t *)q;
    const auto *kv = (const uint8_t *)k_pool;
    auto launch = [&](auto kern, int nw) {
        hipLaunchKernelGGL(kern, dim3(bt->total_q * splits), dim3(64 * nw), 0, st, bt->q_start, bt->hist_len,
                           bt->num_seqs, bt->entry_shift, qq, kv, row_bytes, page_table, pt_ld, shift, topk_idx, k,
                           sl2, out, of32, lse, splits, part);
    };
    if (part) {
        if (Hq == 128)
            launch(sparse_mla_mfma<8, true, KV8>, 8);
        else if (Hq == 64)
            launch(sparse_mla_mfma<4, true, KV8>, 4);
        else if (Hq == 32)
            launch(sparse_mla_mfma<2, true, KV8>, 2);
        else
            launch(sparse_mla_mfma<1, true, KV8>, 1);
    } else {
        if (Hq == 128)
            launch(sparse_mla_mfma<8, false, KV8>, 8);
        else if (Hq == 64)
            launch(sparse_mla_mfma<4, false, KV8>, 4);
        else if (Hq == 32)
            launch(sparse_mla_mfma<2, false, KV8>, 2);
        else
            launch(sparse_mla_mfma<1, false, KV8>, 1);
    }
}

// Slices per row: as given, or (0) enough for one block per compute unit (a
// block fills a CU's LDS, so more slices only queue a second round), at most
// one slice per 32-id tile and MAX_SPLITS.  Only the automatic count asks the
// device.
static int mla_split_count(const janus_batch *bt, int k, int num_splits, int *splits)
{
    int sp = num_splits;
    if (sp == 0) {
        int dev = 0, cus = 256;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return JANUS_ERR_DEVICE;
        const int tq = std::max(bt->total_q, 1);
        sp = std::min(MAX_SPLITS, std::max(1, (cus + tq - 1) / tq));
    }
    *splits = std::min(sp, (k + MLA_KT - 1) / MLA_KT);
    return JANUS_OK;
}

// Workspace bytes of a split launch: each slice's unnormalised O, max and sum.
static size_t mla_split_bytes(const janus_batch *bt, int Hq, int splits)
{
    return splits > 1 ? (size_t)bt->total_q * splits * Hq * (MLA_DV + 2) * sizeof(float) : (size_t)0;
}

// The MLA kernel over a whole or sliced selection (see janus_sparse_attn_split
// for the slice count and workspace rules).
template <bool KV8>
static int run_mla(const janus_batch *bt, const void *q, int Hq, const void *pool, int64_t row_bytes,
                   const int32_t *page_table, int pt_ld, int page_size, const int32_t *topk_idx, int k, float scale,
                   void *out, janus_dtype out_dt, float *lse, int num_splits, void *workspace,
                   size_t *workspace_bytes, void *stream)
{
    int splits = 1;
    if (const int rc = mla_split_count(bt, k, num_splits, &splits); rc != JANUS_OK)
        return rc;
    const size_t need = mla_split_bytes(bt, Hq, splits);
    if (!workspace) {
        *workspace_bytes = need;
        return JANUS_OK;
    }
    if (*workspace_bytes < need)
        return JANUS_ERR_WORKSPACE;
    // the slice merge moves 16 bytes per lane
    if (splits > 1 && (((reinterpret_cast<uintptr_t>(workspace) | reinterpret_cast<uintptr_t>(out)) & 15) != 0))
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0)
        return JANUS_OK;
    hipStream_t st = as_stream(stream);
    const int shift = __builtin_ctz((unsigned)page_size);
    const float sl2 = scale * LOG2E;
    const int of32 = out_dt == JANUS_F32;
    if (splits == 1) {
        launch_mla<KV8>(bt, q, Hq, pool, row_bytes, page_table, pt_ld, shift, topk_idx, k, sl2, out, of32, lse, 1,
                        nullptr, st);
        return launch_status();
    }
    float *part = static_cast<float *>(workspace);
    launch_mla<KV8>(bt, q, Hq, pool, row_bytes, page_table, pt_ld, shift, topk_idx, k, sl2, out, of32, lse, splits,
                    part, st);
    if (hipGetLastError() != hipSuccess)
        return JANUS_ERR_DEVICE;
    // Hq is a multiple of COMBINE_HEADS (16 .. 128) and dv = 512 = 64 lanes x 8
    hipLaunchKernelGGL(attn_combine, dim3((int64_t)bt->total_q * Hq / COMBINE_HEADS), dim3(COMBINE_THREADS), 0, st,
                       part, splits, Hq, MLA_DV, out, of32, lse);
    return launch_status();
}

static bool attn_args_ok(const janus_batch *bt, const void *q, int Hq, int dqk, int dv, const void *k_pool,
                         const void *v_pool, int64_t k_row_stride, int64_t v_row_stride, const int32_t *page_table,
                         int pt_ld, int page_size, const int32_t *topk_idx, int k, const void *out)
{
    return batch_ok(bt) && q && k_pool && v_pool && page_table && topk_idx && out && Hq >= 1 && dqk >= 1 &&
           dv >= 1 && k >= 1 && pt_ld >= 1 && pow2(page_size) && table_covers(bt, pt_ld, page_size) &&
           k_row_stride >= dqk && v_row_stride >= dv;
}

}  // namespace janus

extern "C" int janus_sparse_attn(const janus_batch *bt, const void *q, int Hq, int dqk, int dv,
                                 const void *k_pool, const void *v_pool, int64_t k_row_stride,
                                 int64_t v_row_stride, const int32_t *page_table, int pt_ld, int page_size,
                                 const int32_t *topk_idx, int k, float scale, void *out, janus_dtype out_dt,
                                 float *lse, void *stream)
{
    if (!attn_args_ok(bt, q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, page_table, pt_ld, page_size,
                      topk_idx, k, out))
        return JANUS_ERR_INVALID_ARG;
    if (out_dt != JANUS_BF16 && out_dt != JANUS_F32)
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0)
        return JANUS_OK;
    hipStream_t st = as_stream(stream);
    const int shift = __builtin_ctz((unsigned)page_size);
    const float sl2 = scale * LOG2E;
    const int of32 = out_dt == JANUS_F32;
    if (mla_shape(q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, k)) {
        launch_mla<false>(bt, q, Hq, k_pool, 2 * k_row_stride, page_table, pt_ld, shift, topk_idx, k, sl2, out, of32,
                          lse, 1, nullptr, st);
        return launch_status();
    }
    if (mqa_shape(q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, k)) {
        hipLaunchKernelGGL(sparse_mqa_mfma, dim3((bt->total_q + MQA_WAVES - 1) / MQA_WAVES), dim3(64 * MQA_WAVES), 0,
                           st, bt->q_start, bt->hist_len, bt->num_seqs, bt->entry_shift, (int)bt->total_q,
                           (const uint16_t *)q, Hq, (const uint8_t *)k_pool, (const uint8_t *)v_pool,
                           2 * k_row_stride, 2 * v_row_stride, page_table, pt_ld, shift, topk_idx, k, sl2, out, of32,
                           lse);
        return launch_status();
    }
    if (dqk > VEC_MAX_DQK || dv > 4 * VEC_THREADS)
        return JANUS_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(sparse_attn_vector, dim3((int64_t)bt->total_q * Hq), dim3(VEC_THREADS), 0, st, bt->q_start,
                       bt->hist_len, bt->num_seqs, bt->entry_shift, (const uint16_t *)q, Hq, dqk, dv,
                       (const uint16_t *)k_pool,
                       (const uint16_t *)v_pool, k_row_stride, v_row_stride, page_table, pt_ld, shift, topk_idx, k,
                       sl2, out, of32, lse);
    return launch_status();
}

extern "C" int janus_sparse_attn_split(const janus_batch *bt, const void *q, int Hq, int dqk, int dv,
                                       const void *k_pool, const void *v_pool, int64_t k_row_stride,
                                       int64_t v_row_stride, const int32_t *page_table, int pt_ld, int page_size,
                                       const int32_t *topk_idx, int k, float scale, void *out, janus_dtype out_dt,
                                       float *lse, int num_splits, void *workspace, size_t *workspace_bytes,
                                       void *stream)
{
    if (!attn_args_ok(bt, q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, page_table, pt_ld, page_size,
                      topk_idx, k, out) ||
        !workspace_bytes || num_splits < 0 || num_splits > MAX_SPLITS)
        return JANUS_ERR_INVALID_ARG;
    if (out_dt != JANUS_BF16 && out_dt != JANUS_F32)
        return JANUS_ERR_UNSUPPORTED;
    if (!mla_shape(q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, k))
        return JANUS_ERR_UNSUPPORTED;
    return run_mla<false>(bt, q, Hq, k_pool, 2 * k_row_stride, page_table, pt_ld, page_size, topk_idx, k, scale, out,
                          out_dt, lse, num_splits, workspace, workspace_bytes, stream);
}

extern "C" int janus_sparse_attn_fp8kv(const janus_batch *bt, const void *q, int Hq, const uint8_t *kv_pool,
                                       int64_t row_bytes, const int32_t *page_table, int pt_ld, int page_size,
                                       const int32_t *topk_idx, int k, float scale, void *out, janus_dtype out_dt,
                                       float *lse, int num_splits, void *workspace, size_t *workspace_bytes,
                                       void *stream)
{
    if (!batch_ok(bt) || !q || !kv_pool || !page_table || !topk_idx || !out || !workspace_bytes || Hq < 1 ||
        k < 1 || pt_ld < 1 || !pow2(page_size) || !table_covers(bt, pt_ld, page_size) || row_bytes < KV8_ROWB ||
        num_splits < 0 ||
        num_splits > MAX_SPLITS)
        return JANUS_ERR_INVALID_ARG;
    if (out_dt != JANUS_BF16 && out_dt != JANUS_F32)
        return JANUS_ERR_UNSUPPORTED;
    if ((row_bytes % 16) != 0 || row_bytes > INT32_MAX || (reinterpret_cast<uintptr_t>(kv_pool) & 15) != 0 ||
        (reinterpret_cast<uintptr_t>(q) & 15) != 0 || k > MLA_MAX_K ||
        !(Hq == 128 || Hq == 64 || Hq == 32 || Hq == 16))
        return JANUS_ERR_UNSUPPORTED;
    return run_mla<true>(bt, q, Hq, kv_pool, row_bytes, page_table, pt_ld, page_size, topk_idx, k, scale, out,
                         out_dt, lse, num_splits, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// Split attention without a caller workspace: the slices' partial results go
// to a static device array of this library (one per GPU, kept until the
// process ends).  Its address is taken once per device, with that device
// current, on the entry point's first call there; the array's own name is a
// host-side stand-in that must never reach a kernel.
namespace janus {

constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(128) << 20;  // JANUS_NOALLOC_SCRATCH_BYTES
constexpr int NOALLOC_MAX_DEVICES = 64;
static_assert(NOALLOC_SCRATCH_BYTES == JANUS_NOALLOC_SCRATCH_BYTES, "header and library disagree");

static __device__ __align__(256) uint8_t scratch[NOALLOC_SCRATCH_BYTES];

static std::mutex g_scratch_mu;
static void *g_scratch_dev[NOALLOC_MAX_DEVICES];  // device address of scratch, per device

// This device's copy of the scratch array (its device address), looked up
// on the first call on the device.
static int device_scratch(void **ptr)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= NOALLOC_MAX_DEVICES)
        return JANUS_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
            return JANUS_ERR_DEVICE;
        g_scratch_dev[dev] = p;
    }
    *ptr = g_scratch_dev[dev];
    return JANUS_OK;
}

}  // namespace janus

extern "C" int janus_sparse_attn_split_noalloc(const janus_batch *bt, const void *q, int Hq, int dqk, int dv,
                                               const void *k_pool, const void *v_pool, int64_t k_row_stride,
                                               int64_t v_row_stride, const int32_t *page_table, int pt_ld,
                                               int page_size, const int32_t *topk_idx, int k, float scale, void *out,
                                               janus_dtype out_dt, float *lse, int num_splits, void *stream)
{
    if (!attn_args_ok(bt, q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, page_table, pt_ld, page_size,
                      topk_idx, k, out) ||
        num_splits < 0 || num_splits > MAX_SPLITS)
        return JANUS_ERR_INVALID_ARG;
    if (out_dt != JANUS_BF16 && out_dt != JANUS_F32)
        return JANUS_ERR_UNSUPPORTED;
    if (!mla_shape(q, Hq, dqk, dv, k_pool, v_pool, k_row_stride, v_row_stride, k))
        return JANUS_ERR_UNSUPPORTED;
    int splits = 1;
    if (const int rc = mla_split_count(bt, k, num_splits, &splits); rc != JANUS_OK)
        return rc;
    size_t cap = NOALLOC_SCRATCH_BYTES;
    if (mla_split_bytes(bt, Hq, splits) > cap)
        return JANUS_ERR_WORKSPACE;
    void *ws = nullptr;
    if (const int rc = device_scratch(&ws); rc != JANUS_OK)
        return rc;
    return run_mla<false>(bt, q, Hq, k_pool, 2 * k_row_stride, page_table, pt_ld, page_size, topk_idx, k, scale, out,
                          out_dt, lse, num_splits, ws, &cap, stream);
}
