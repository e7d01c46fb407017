// Indexer relevance scores (Eq. 1's Idx, lightning-indexer form):
//   S[i,s] = sq[i] * sk[s] * sum_h w[i,h] * max(0, q[i,h,:] . kI[s,:]),  s <= M+i
//
// fp8 path (d = 128): one v_mfma_f32_16x16x128_f8f6f4 covers a whole 128-dim
// dot product, so each MFMA is a 16 (token, head) x 16 key tile and the only
// reduction left is the ReLU-weighted sum over heads, done in the epilogue.
// The prefill kernel keeps each wave's two tokens' queries (2 x H x 128 fp8)
// in VGPRs and streams the keys through LDS; the row-tile kernel (decode
// shapes, MXFP4 keys) reads its keys straight from global memory.
//
// Epilogue: the MFMA applies an E8M0 scale of 2^-25 to the query operand, so
// every product lands in (-1, 1): |q.k| <= 128 * 448 * 448 < 2^25 for any
// e4m3 inputs.  On that range the clamping form of v_cvt_pk_bf16_f32 (which
// clamps to [0, 1] after rounding to nearest even) is exactly ReLU followed
// by the bf16 rounding, with head weights pre-multiplied by 2^25.  The fp8
// MFMA and the VALU do not overlap on this chip, so VALU work per MFMA bounds
// the kernels.  The row-tile kernel dots each converted pair with its weights
// (v_dot2c_f32_bf16): 4 VALU ops per MFMA.  The prefill kernel feeds the
// converted pairs to a bf16 MFMA whose A operand holds the weights, which
// sums the heads of a token across lanes as well: 2 VALU ops per fp8 MFMA
// and one bf16 MFMA per two, which other waves' VALU work overlaps.  Every
// term is non-negative, so the two bf16 roundings bound the relative error
// of a score by 2^-8.
//
// The clamp modifier cannot be requested from the compiler, so the convert
// is inline assembly; the compiler does not insert the wait states a VALU
// read of an MFMA result needs ahead of inline assembly, so the MFMAs of a
// group are issued from one assembly block that carries its own wait states
// (12 for an 8-pass fp8 MFMA, what the compiler itself emits) and starts
// with the one a VALU write of an MFMA source needs.
#include "janus_device.hpp"
#include "janus_host.hpp"

#include <algorithm>
#include <cmath>

namespace janus {

constexpr int IDX_TPW = 2;                          // tokens per wave
constexpr int IDX_WAVES = 4;                        // waves per block
constexpr int IDX_KEY_CHUNK = 16384;                // target keys per block: long blocks spread each block's query and weight loads over more keys
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

// One group of four head tiles against one 16-key block: four 16x16x128
// fp8 MFMAs sharing the key operand (query scale 2^-25, so every product is
// below 1 in magnitude), then each pair of outputs clamped to [0, 1] and
// rounded to bf16 - ReLU - and the weighted head sum on a bf16 MFMA.  The
// converts pack the outputs so that v[112:115] holds tiles 0 and 1 and
// v[116:119] tiles 2 and 3: lane group g's eight bf16 are rows 4g..4g+3 of
// the first tile, then of the second, at the lane's key.  That is the B
// operand (32 slots x 16 keys) of v_mfma_f32_16x16x32_bf16, whose A operand
// (wp0, wp1) holds the head weights of each slot in the row of the slot's
// token and zeros elsewhere, so the MFMA adds up a token's weighted heads
// across the lane groups.  The converts cost one VALU instruction per two
// outputs, and a bf16 MFMA, unlike an fp8 one, leaves most of its cycles to
// the VALU work of the other waves.  The MFMA results live in v[112:127],
// declared clobbered, so the group is one block whose wait states are
// written out (the counts the compiler itself emits for these pairs of
// instructions): two ahead of the MFMAs (a VALU write of one of their
// sources); twelve between an 8-pass MFMA and a VALU read of its result,
// where each later 8-pass MFMA counts as four, so the converts read MFMA k's
// result 16, 14, 12 and 12 wait states after it; two or more between a
// convert and the head-sum MFMA that reads it; none between two dependent
// head-sum MFMAs; eight at the end, before anything reads hc.  FIRST starts
// the sum at zero.
#define IDX_MFMA(dst, a) \
    "v_mfma_scale_f32_16x16x128_f8f6f4 " dst ", %[" a "], %[bk], 0, %[sc], %[sc] op_sel:[0,1,0] op_sel_hi:[0,0,0]\n\t"
#define IDX_HEAD_GROUP_CLOBBERS                                                                       \
    "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", \
        "v125", "v126", "v127"
#define IDX_HEAD_SUM(C0)                                                                              \
    "s_nop 1\n\t" IDX_MFMA("v[112:115]", "a0") IDX_MFMA("v[116:119]", "a1") IDX_MFMA("v[120:123]", "a2")  \
        IDX_MFMA("v[124:127]", "a3")                                                                  \
    "s_nop 3\n\t"                                                                                     \
    "v_cvt_pk_bf16_f32 v112, v112, v113 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v113, v114, v115 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v114, v116, v117 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v115, v118, v119 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v116, v120, v121 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v117, v122, v123 clamp\n\t"                                                    \
    "s_nop 1\n\t"                                                                                     \
    "v_cvt_pk_bf16_f32 v118, v124, v125 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v119, v126, v127 clamp\n\t"                                                    \
    "s_nop 1\n\t"                                                                                     \
    "v_mfma_f32_16x16x32_bf16 %[hc], %[wp0], v[112:115], " C0 "\n\t"                                 \
    "v_mfma_f32_16x16x32_bf16 %[hc], %[wp1], v[116:119], %[hc]\n\t"                                  \
    "s_nop 7"
#define IDX_HEAD_SUM_INPUTS                                                                            \
    [a0] "v"(a0), [a1] "v"(a1), [a2] "v"(a2), [a3] "v"(a3), [bk] "v"(bk), [sc] "v"(scales), [wp0] "v"(wp0), \
        [wp1] "v"(wp1)

template <bool FIRST>
JANUS_DEV void head_sum_group(v4f &hc, const v8i &a0, const v8i &a1, const v8i &a2, const v8i &a3, const v8i &bk,
                              int scales, const v8bf &wp0, const v8bf &wp1)
{
    if (FIRST)
        asm(IDX_HEAD_SUM("0") : [hc] "=&v"(hc) : IDX_HEAD_SUM_INPUTS : IDX_HEAD_GROUP_CLOBBERS);
    else
        asm(IDX_HEAD_SUM("%[hc]") : [hc] "+v"(hc) : IDX_HEAD_SUM_INPUTS : IDX_HEAD_GROUP_CLOBBERS);
}

// The row-tile kernel's group with MXFP4 keys, after expand_e2m1 has widened
// them to fp8 (sa = 2^6 undoes its 2^-6, sb is the lane's E8M0 block scale).
// Block scales can make a product of any size, so ReLU is not folded into
// the convert here: each pair is rounded to bf16, its sign clamped with a
// packed int16 max (a negative bf16 is a negative int16), and dotted with
// its weights into acc (v_dot2c); the lane groups' sums are added afterwards.  Convert, max and dot of a pair are at least two instructions apart
// (one wait state after a VALU write read by a packed op).
#define IDX_MFMA_F4(dst, a) \
    "v_mfma_scale_f32_16x16x128_f8f6f4 " dst ", %[" a "], %[bk], 0, %[sa], %[sb] op_sel_hi:[0,0,0]\n\t"
#define F4_CVT(r, r1) "v_cvt_pk_bf16_f32 v" #r ", v" #r ", v" #r1 "\n\t"
#define F4_MAX(r) "v_pk_max_i16 v" #r ", v" #r ", 0\n\t"
#define F4_DOT(r, w) "v_dot2c_f32_bf16 %[acc], v" #r ", %[" w "]\n\t"
#define IDX_HEAD_GROUP_F4(INIT)                                                                          \
    INIT "s_nop 1\n\t" IDX_MFMA_F4("v[112:115]", "a0") IDX_MFMA_F4("v[116:119]", "a1")                    \
        IDX_MFMA_F4("v[120:123]", "a2") IDX_MFMA_F4("v[124:127]", "a3") "s_nop 0\n\t"                    \
        F4_CVT(112, 113)                                                                                   \
        F4_CVT(114, 115) F4_MAX(112)                                                                       \
        F4_CVT(116, 117) F4_MAX(114) F4_DOT(112, "w00")                                                    \
        F4_CVT(118, 119) F4_MAX(116) F4_DOT(114, "w01")                                                    \
        F4_CVT(120, 121) F4_MAX(118) F4_DOT(116, "w10")                                                    \
        F4_CVT(122, 123) F4_MAX(120) F4_DOT(118, "w11")                                                    \
        F4_CVT(124, 125) F4_MAX(122) F4_DOT(120, "w20")                                                    \
        F4_CVT(126, 127) F4_MAX(124) F4_DOT(122, "w21")                                                    \
        F4_MAX(126) F4_DOT(124, "w30")                                                                     \
        F4_DOT(126, "w31") "s_nop 2"
#define IDX_HEAD_GROUP_F4_INPUTS                                                                       \
    [a0] "v"(a0), [a1] "v"(a1), [a2] "v"(a2), [a3] "v"(a3), [bk] "v"(bk), [sa] "v"(sa), [sb] "v"(sb),   \
        [w00] "v"(w[0][0]), [w01] "v"(w[0][1]), [w10] "v"(w[1][0]), [w11] "v"(w[1][1]), [w20] "v"(w[2][0]), \
        [w21] "v"(w[2][1]), [w30] "v"(w[3][0]), [w31] "v"(w[3][1])

// The MXFP4 prefill group: the fp8 prefill group (head sums on a bf16 MFMA)
// with e2m1 keys as the B operand (blgp 4: 16 bytes per lane, lane group g
// holding the key's elements 32g .. 32g+31, MX block g) and separate scales:
// sa = 2^-25 for the queries, sb = the lane's block scale divided by the
// largest of its key's four (so at most 1).  Every product then stays below
// 128 * 448 * 6 * 2^-25 < 1 in magnitude and the clamping convert is ReLU,
// as in the fp8 group; the wait states are the fp8 group's (the same 8-pass
// MFMA), with one more after the fourth MFMA.
#define IDX_MFMA_F4C(dst, a) \
    "v_mfma_scale_f32_16x16x128_f8f6f4 " dst ", %[" a "], %[bk], 0, %[sa], %[sb] op_sel_hi:[0,0,0] blgp:4\n\t"
#define IDX_HEAD_SUM_F4C(C0)                                                                          \
    "s_nop 1\n\t" IDX_MFMA_F4C("v[112:115]", "a0") IDX_MFMA_F4C("v[116:119]", "a1")                  \
        IDX_MFMA_F4C("v[120:123]", "a2") IDX_MFMA_F4C("v[124:127]", "a3")                            \
    "s_nop 4\n\t"                                                                                     \
    "v_cvt_pk_bf16_f32 v112, v112, v113 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v113, v114, v115 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v114, v116, v117 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v115, v118, v119 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v116, v120, v121 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v117, v122, v123 clamp\n\t"                                                    \
    "s_nop 1\n\t"                                                                                     \
    "v_cvt_pk_bf16_f32 v118, v124, v125 clamp\n\t"                                                    \
    "v_cvt_pk_bf16_f32 v119, v126, v127 clamp\n\t"                                                    \
    "s_nop 1\n\t"                                                                                     \
    "v_mfma_f32_16x16x32_bf16 %[hc], %[wp0], v[112:115], " C0 "\n\t"                                 \
    "v_mfma_f32_16x16x32_bf16 %[hc], %[wp1], v[116:119], %[hc]\n\t"                                  \
    "s_nop 7"
#define IDX_HEAD_SUM_F4C_INPUTS                                                                        \
    [a0] "v"(a0), [a1] "v"(a1), [a2] "v"(a2), [a3] "v"(a3), [bk] "v"(bk), [sa] "v"(sa), [sb] "v"(sb),   \
        [wp0] "v"(wp0), [wp1] "v"(wp1)

template <bool FIRST>
JANUS_DEV void head_sum_group_f4c(v4f &hc, const v8i &a0, const v8i &a1, const v8i &a2, const v8i &a3,
                                  const v4i &bk, int sa, int sb, const v8bf &wp0, const v8bf &wp1)
{
    if (FIRST)
        asm(IDX_HEAD_SUM_F4C("0") : [hc] "=&v"(hc) : IDX_HEAD_SUM_F4C_INPUTS : IDX_HEAD_GROUP_CLOBBERS);
    else
        asm(IDX_HEAD_SUM_F4C("%[hc]") : [hc] "+v"(hc) : IDX_HEAD_SUM_F4C_INPUTS : IDX_HEAD_GROUP_CLOBBERS);
}
constexpr int IDX_SCALE_2M25 = 127 - 25;  // E8M0 2^-25

// MXFP4 keys as fp8: an e2m1 nibble (sign, 2-bit exponent, 1-bit mantissa,
// bias 1) placed at bits 7 and 4..2 of a byte is the e4m3 code (bias 7) of
// the same value times 2^-6; the e2m1 subnormal 0.5 lands on the e4m3
// subnormal 2^-7, and zero on zero.  Of 8 nibbles (element 2i in the low
// nibble of byte i) the low nibbles give elements 0, 2, 4, 6 and the high
// ones 1, 3, 5, 7: the query operand is put in the same order by evens_odds,
// which leaves every dot product as it was.
JANUS_DEV v8i expand_e2m1(const v4i &u)
{
    v8i r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t x = (uint32_t)u[i];
        r[2 * i] = (int)(((x << 4) & 0x80808080u) | ((x << 2) & 0x1C1C1C1Cu));
        r[2 * i + 1] = (int)((x & 0x80808080u) | ((x >> 2) & 0x1C1C1C1Cu));
    }
    return r;
}

// fp8 elements 8i .. 8i+7 (registers 2i, 2i+1) -> the even ones in register
// 2i, the odd ones in 2i+1
JANUS_DEV v8i evens_odds(const v8i &a)
{
    v8i r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[2 * i] = (int)__builtin_amdgcn_perm((uint32_t)a[2 * i + 1], (uint32_t)a[2 * i], 0x06040200u);
        r[2 * i + 1] = (int)__builtin_amdgcn_perm((uint32_t)a[2 * i + 1], (uint32_t)a[2 * i], 0x07050301u);
    }
    return r;
}
constexpr int F4_QUERY_SCALE = 127 + 6;  // E8M0 2^6

template <bool FIRST>
JANUS_DEV void head_group_f4(float &acc, const v8i &a0, const v8i &a1, const v8i &a2, const v8i &a3, const v8i &bk,
                             int sa, int sb, const v2bf (*w)[2])
{
    if (FIRST)
        asm(IDX_HEAD_GROUP_F4("v_mov_b32 %[acc], 0\n\t")
            : [acc] "=&v"(acc)
            : IDX_HEAD_GROUP_F4_INPUTS
            : IDX_HEAD_GROUP_CLOBBERS);
    else
        asm(IDX_HEAD_GROUP_F4("")
            : [acc] "+v"(acc)
            : IDX_HEAD_GROUP_F4_INPUTS
            : IDX_HEAD_GROUP_CLOBBERS);
}

constexpr int IDX_STAGE = 128;                      // keys per LDS stage (16 KB)
constexpr int IDX_XCD = 8;                          // L2 domains (XCDs) of the chip

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt <= n only.
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// s_waitcnt immediate that waits for lgkmcnt = 0 only.
constexpr int IDX_LGKM0 = 15 | (3 << 14) | (7 << 4);

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
// Two tokens per wave: an MFMA tile's 16 rows are 2 tokens x 8 heads,
// ordered so that output rows 4g..4g+3 (lane group g) hold token g/2 and 4
// consecutive heads.  The head-sum MFMA adds a token's heads over its two
// lane groups and over each pair of tiles, and returns token t's sums of the
// 16 keys in lane group t.  Two tokens per wave keep the registers at 128,
// for four waves per SIMD.
template <int H, int TPW>
__global__ __launch_bounds__(256, (TPW == 4 ? 2 : 4)) void index_scores_fp8_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs, int es,
    int nchunks, int key_chunk, int ntiles, const uint8_t *__restrict__ q, const float *__restrict__ q_scale,
    const uint8_t *__restrict__ kI, const float *__restrict__ k_scale, const float *__restrict__ w,
    float *__restrict__ scores)
{
    // the head sums come out in rows 0 and 4 of the head-sum MFMA: two tokens of 8 heads per tile
    static_assert(TPW == 2 && H % 16 == 0, "two tokens per wave");
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
    const int ctx = entries_of(M + N, es);
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
    const int block_lim = last_cand(M, min(tile0 + TOK_TILE - 1, N - 1), es);
    const int key_end = min(key_hi, block_lim + 1);

    // Key DMA: lane L of wave instruction i (i = wave + 4j, j < 4) fills
    // 16-byte chunk 64i + L of the stage, i.e. key row 8i + L/8 at slot L%8,
    // which holds column slot ^ ((row >> 1) & 7) = slot ^ ((4*wave + L/16) & 7).
    // The lane's byte offset into the stage's keys is therefore fixed, and
    // the four instructions differ by 4 KB.
    const uint32_t kvoff = 1024u * wave + 128u * (lane >> 3) + 16u * ((lane & 7) ^ ((4 * wave + (lane >> 4)) & 7));
    auto issue = [&](int k0, uint8_t *kdst, float *sdst) {
        // buffer over the keys from k0 on: rows past the context read as
        // zeros (their scores are never stored)
        const __amdgpu_buffer_rsrc_t krs =
            make_buffer_rsrc((void *)(kI + ((kbase + k0) << 7)), (uint32_t)(ctx - k0) << 7);
#pragma unroll
        for (int j = 0; j < IDX_STAGE * 8 / 64 / IDX_WAVES; ++j)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lds_void_t *)(kdst + 1024 * (wave + IDX_WAVES * j)), 16,
                                                     kvoff + 4096u * j, 0, 0, 0);
        // the stage's key scales, one dword per lane (waves 0 and 1)
        if (k_scale && wave < 2) {
            const __amdgpu_buffer_rsrc_t srs =
                make_buffer_rsrc((void *)(k_scale + kbase + k0), (uint32_t)(ctx - k0) << 2);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void_t *)(sdst + 64 * wave), 4, 4u * (64 * wave + lane),
                                                     0, 0, 0);
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
    // term) and 2^25 (undoing the MFMA's query scale), rounded once to bf16.
    // The head-sum MFMA's A operand of tile pair p (tiles 2p, 2p+1): row
    // 4*(kg/2) is token kg/2's, and lane (kg, r16 = 4*(kg/2)) holds the
    // weights of the heads in its slots (those of rows 4kg..4kg+3 of each
    // tile); every other lane holds zeros.
    const float sq = (q_scale ? q_scale[e_row] : 1.0f) * 0x1p25f;
    const bool hs_lane = r16 == 4 * (kg >> 1);
    v8bf wA[HB / 2];
#pragma unroll
    for (int p = 0; p < HB / 2; ++p) {
        const v4f t0 = *(const v4f *)(w + e_row * H + RPT * (2 * p) + hsub);
        const v4f t1 = *(const v4f *)(w + e_row * H + RPT * (2 * p + 1) + hsub);
        const float f = hs_lane ? sq : 0.0f;
        wA[p] = __builtin_convertvector((v8f){t0[0] * f, t0[1] * f, t0[2] * f, t0[3] * f, t1[0] * f, t1[1] * f,
                                              t1[2] * f, t1[3] * f},
                                        v8bf);
    }
    const int wave_lim = last_cand(M, min(tw0 + TPW - 1, N - 1), es);
    int scales = IDX_MFMA_SCALES;
    // this lane's two 16-byte columns (2*kg, 2*kg+1) of LDS row 16*j + r16
    const int g8 = (r16 >> 1) & 7;
    const int off0 = r16 * 128 + 16 * ((2 * kg) ^ g8), off1 = r16 * 128 + 16 * ((2 * kg + 1) ^ g8);
    // The head sums land in row 4t of the head-sum MFMA's output for token
    // tw0 + t: lane group t (lanes 16t .. 16t+15) holds token t's sums of the
    // block's 16 keys in element 0, and one store per 16-key block writes
    // them for both tokens.  Scores leave through buffer stores over this
    // block's rows: a lane with nothing to write (lane groups 2 and 3, or a
    // token past the tile) uses an offset past the range and the hardware
    // drops it, so every wave issues the same number of stores per full stage
    // and the stage can wait for its key prefetch with vmcnt(STAGE_STORES)
    // instead of draining the stores.
    const int s_tok = tw0 + kg;
    const int nrows_blk = max(0, min(TOK_TILE, N - tile0));
    const int64_t blk_off = score_start[b] + (int64_t)tile0 * ctx;
    const __amdgpu_buffer_rsrc_t rsrc = make_buffer_rsrc(scores + blk_off, (uint32_t)((int64_t)nrows_blk * ctx * 4));
    const bool row_ok = kg < TPW && s_tok < N && wave_on;
    const uint32_t lane_row_off = (uint32_t)((int64_t)(s_tok - tile0) * ctx * 4);
    const int lim = last_cand(M, s_tok, es);  // last causal candidate of this lane's token
    constexpr int STORES_PER_GROUP = 4;
    constexpr int STAGE_STORES = (IDX_STAGE / 64) * STORES_PER_GROUP;
    // every token of the block sees all keys below this bound
    const int interior_end = min(ctx, last_cand(M, tile0, es) + 1);

    // one stage: compute the keys in (stg, ks) while the next stage streams in
    auto stage = [&](int k0, const uint8_t *stg, const float *ks) {
#pragma unroll
        for (int gsub = 0; gsub < IDX_STAGE / 64; ++gsub) {
            const int s0 = k0 + 64 * gsub;
            if (s0 >= key_hi)
                break;
            const bool skip = !wave_on || s0 > wave_lim;
#pragma unroll
            for (int j = 0; j < STORES_PER_GROUP; ++j) {
                // token tw0 + kg at key s0 + 16*j + r16 (kg < 2), before the key scale
                float v = -INFINITY;
                if (!skip) {
                    const uint8_t *rowb = stg + (64 * gsub + 16 * j) * 128;
                    v4i lo = *(const v4i *)(rowb + off0), hi = *(const v4i *)(rowb + off1);
                    const v8i bk = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    v4f hc;
                    head_sum_group<true>(hc, a[0], a[1], a[2], a[3], bk, scales, wA[0], wA[1]);
#pragma unroll
                    for (int h4 = 4; h4 < HB; h4 += 4)
                        head_sum_group<false>(hc, a[h4], a[h4 + 1], a[h4 + 2], a[h4 + 3], bk, scales, wA[h4 / 2],
                                              wA[h4 / 2 + 1]);
                    v = hc[0];
                }
                const int s = s0 + 16 * j + r16;
                const float kscale = k_scale ? ks[64 * gsub + 16 * j + r16] : 1.0f;
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

// bf16 queries and keys (d = 128, H = 64) on bf16 MFMA.  The structure of
// the fp8 kernel above - 4 waves of 2 tokens, keys streamed through LDS in
// 128-key stages by buffer-to-LDS DMA, XCD-aware key chunks, counted
// buffer stores - with v_mfma_f32_16x16x32_bf16: a 16 (token, head) x 16
// key tile takes four K-steps of 32 dims, and each key operand read from LDS
// feeds the wave's 8 head tiles.  A key row is 256 bytes; its 16-byte chunk
// c sits at slot c ^ (row & 15), so the 16 rows of one operand read fall in
// 16 different bank groups.  The epilogue stays in fp32 (ReLU as a max, the
// weighted head sum as fmas against fp32 weights): bf16 scores are held to
// 1e-3 of the row maximum, which a bf16 rounding of each term would not
// leave room for.
constexpr int B16_ROW = 256;  // bytes per bf16 key row (128 dims)
JANUS_DEV v8bf as_v8bf(v4i x) { return __builtin_bit_cast(v8bf, x); }

__global__ __launch_bounds__(256, 2) void index_scores_bf16_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs, int es,
    int nchunks, int key_chunk, int ntiles, const uint16_t *__restrict__ q, const float *__restrict__ q_scale,
    const uint8_t *__restrict__ kI, const float *__restrict__ k_scale, const float *__restrict__ w,
    float *__restrict__ scores)
{
    constexpr int H = 64, TPW = 2, RPT = 16 / TPW, HB = H / RPT, TOK_TILE = 4 * TPW;
    __shared__ __attribute__((aligned(16))) uint8_t sKey0[IDX_STAGE * B16_ROW];
    __shared__ __attribute__((aligned(16))) uint8_t sKey1[IDX_STAGE * B16_ROW];
    __shared__ float sKs0[IDX_STAGE];
    __shared__ float sKs1[IDX_STAGE];
    int slot, chunk, b, tile0;
    if (!xcd_tile_chunk(blockIdx.x, nchunks, ntiles, slot, chunk))
        return;
    if (!tile_slot(q_start, num_seqs, slot, TOK_TILE, b, tile0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = entries_of(M + N, es);
    const int key_lo = chunk * key_chunk;
    if (key_lo >= ctx)
        return;
    const int key_hi = min(ctx, key_lo + key_chunk);
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tw0 = tile0 + wave * TPW;
    const bool wave_on = tw0 < N;
    const int r16 = lane & 15, kg = lane >> 4;
    const int qrow0 = q_start[b];
    const int64_t kbase = ctx_start[b];
    const int block_lim = last_cand(M, min(tile0 + TOK_TILE - 1, N - 1), es);
    const int key_end = min(key_hi, block_lim + 1);

    // Key DMA: instruction j of wave `wave` fills stage bytes 4096j + 1024wave
    // + 16lane = key row 16j + 4wave + lane/16, slot lane%16, which holds
    // chunk (lane%16) ^ (row & 15); the lane's source offset is therefore
    // fixed apart from 4096j.
    const int drow = 4 * wave + (lane >> 4);
    const uint32_t kvoff = (uint32_t)(B16_ROW * drow + 16 * ((lane & 15) ^ (drow & 15)));
    auto issue = [&](int k0, uint8_t *kdst, float *sdst) {
        const __amdgpu_buffer_rsrc_t krs =
            make_buffer_rsrc((void *)(kI + (kbase + k0) * B16_ROW), (uint32_t)(ctx - k0) * B16_ROW);
#pragma unroll
        for (int j = 0; j < IDX_STAGE * B16_ROW / 16 / 256; ++j)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lds_void_t *)(kdst + 4096 * j + 1024 * wave), 16,
                                                     kvoff + 4096u * j, 0, 0, 0);
        if (k_scale && wave < 2) {
            const __amdgpu_buffer_rsrc_t srs =
                make_buffer_rsrc((void *)(k_scale + kbase + k0), (uint32_t)(ctx - k0) << 2);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void_t *)(sdst + 64 * wave), 4, 4u * (64 * wave + lane),
                                                     0, 0, 0);
        }
    };
    if (key_lo < key_end)
        issue(key_lo, sKey0, sKs0);

    // A operand of head tile hb, K-step st: MFMA row r16 = (token r16/RPT,
    // head RPT*hb + r16%RPT), dims 32st + 8kg .. +7
    const int a_tok = tw0 + r16 / RPT;
    const bool a_ok = a_tok < N;
    const int64_t a_row = (int64_t)qrow0 + (a_ok ? a_tok : 0);
    v8bf a[HB][4];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int st = 0; st < 4; ++st)
            a[hb][st] = a_ok ? as_v8bf(*(const v4i *)(q + (a_row * H + RPT * hb + (r16 % RPT)) * 128 + 32 * st + 8 * kg))
                             : as_v8bf(v4i{0, 0, 0, 0});
    // output rows 4kg..4kg+3 of every tile: token tw0 + 4kg/RPT, heads
    // RPT*hb + (4kg)%RPT + i; their weights times the token's query scale
    const int e_tok = tw0 + (4 * kg) / RPT;
    const bool e_ok = e_tok < N;
    const int64_t e_row = (int64_t)qrow0 + (e_ok ? e_tok : 0);
    const int hsub = (4 * kg) % RPT;
    const float sq = q_scale ? q_scale[e_row] : 1.0f;
    float wv[HB][4];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        const v4f t = *(const v4f *)(w + e_row * H + RPT * hb + hsub);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            wv[hb][i] = t[i] * sq;
    }
    const int lim = last_cand(M, e_tok, es);
    const int wave_lim = last_cand(M, min(tw0 + TPW - 1, N - 1), es);
    constexpr int GPT = 4 / TPW;  // lane groups per token
    const int gin = kg % GPT;
    const int nrows_blk = max(0, min(TOK_TILE, N - tile0));
    const int64_t blk_off = score_start[b] + (int64_t)tile0 * ctx;
    const __amdgpu_buffer_rsrc_t rsrc = make_buffer_rsrc(scores + blk_off, (uint32_t)((int64_t)nrows_blk * ctx * 4));
    const bool row_ok = e_ok && wave_on;
    const uint32_t lane_row_off = (uint32_t)((int64_t)(e_tok - tile0) * ctx * 4);
    constexpr int STORES_PER_GROUP = 4 / GPT;
    constexpr int STAGE_STORES = (IDX_STAGE / 64) * STORES_PER_GROUP;
    const int interior_end = min(ctx, last_cand(M, tile0, es) + 1);

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
                // key operand of 16-key block (gsub, j): key row r = 64gsub +
                // 16j + r16, chunk 4st + kg at slot (4st + kg) ^ r16
                const uint8_t *rowb = stg + (64 * gsub + 16 * j + r16) * B16_ROW;
                v8bf bk[4];
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    bk[st] = as_v8bf(*(const v4i *)(rowb + 16 * ((4 * st + kg) ^ r16)));
                v4f d[HB];
#pragma unroll
                for (int hb = 0; hb < HB; ++hb)
                    d[hb] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int hb = 0; hb < HB; ++hb)
                        d[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[hb][st], bk[st], d[hb], 0, 0, 0);
                float r = 0.f;
#pragma unroll
                for (int hb = 0; hb < HB; ++hb)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        r = fmaf(fmaxf(d[hb][i], 0.f), wv[hb][i], r);
                r += xor_lanes16(r);  // the other lane group of this token (GPT = 2)
                res[j] = r;
            }
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
                if (s0 + 64 <= interior_end) {
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
        if (k0 + IDX_STAGE < key_end)
            issue(k0 + IDX_STAGE, sKey1, sKs1);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0, sKey0, sKs0);
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
        if (k0 + IDX_STAGE >= key_hi)
            break;
        if (k0 + 2 * IDX_STAGE < key_end)
            issue(k0 + 2 * IDX_STAGE, sKey0, sKs0);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0 + IDX_STAGE, sKey1, sKs1);
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
    }
}

// MXFP4 keys at prefill: the fp8 kernel's structure with the fp8 x fp4
// scaled MFMA consuming the keys as stored.  For an fp4 operand the MFMA takes
// 16 contiguous bytes per lane: lane group g holds elements 32g .. 32g+31
// (element j in the low nibble of byte j/2 when j is even), which is exactly
// MX block g of a key, and it applies the E8M0 scale that lane group g
// supplies to that block - so each lane passes its key's scale for block g.
// The fp8 query operand keeps its own layout (dims 16g .. 16g+15 in
// registers 0-3, 64+16g .. in 4-7).  Key rows are 64 bytes in LDS, chunk c
// of row r at slot c ^ ((r >> 2) & 3), so the 16 rows of an operand read
// fall in 16 different bank groups.  Each key's block scales are divided by
// the largest of the four (E8M0 exponents minus the largest, clamped at
// 2^-127) and its key scale multiplied by that largest one, once per stage by
// the two waves that load them: with the query scale 2^-25 every product is
// then below 1 in magnitude and the epilogue is the fp8 kernel's clamping
// convert and dot product (4 VALU per MFMA).  Dividing by a power of two
// changes no rounding, so the scores are those of the unnormalised products.
constexpr int F4_ROW = 64;  // bytes of e2m1 codes per key (128 dims)

__global__ __launch_bounds__(256, 4) void index_scores_mxfp4_mfma(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs, int es,
    int nchunks, int key_chunk, int ntiles, const uint8_t *__restrict__ q, const float *__restrict__ q_scale,
    const uint8_t *__restrict__ kI, const uint8_t *__restrict__ k_bscale, const float *__restrict__ k_scale,
    const float *__restrict__ w, float *__restrict__ scores)
{
    constexpr int H = 64, TPW = 2, RPT = 16 / TPW, HB = H / RPT, TOK_TILE = 4 * TPW;
    __shared__ __attribute__((aligned(16))) uint8_t sKey0[IDX_STAGE * F4_ROW];
    __shared__ __attribute__((aligned(16))) uint8_t sKey1[IDX_STAGE * F4_ROW];
    __shared__ uint32_t sBs0[IDX_STAGE];  // the 4 E8M0 block scales of each key
    __shared__ uint32_t sBs1[IDX_STAGE];
    __shared__ float sKs0[IDX_STAGE];
    __shared__ float sKs1[IDX_STAGE];
    int slot, chunk, b, tile0;
    if (!xcd_tile_chunk(blockIdx.x, nchunks, ntiles, slot, chunk))
        return;
    if (!tile_slot(q_start, num_seqs, slot, TOK_TILE, b, tile0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = entries_of(M + N, es);
    const int key_lo = chunk * key_chunk;
    if (key_lo >= ctx)
        return;
    const int key_hi = min(ctx, key_lo + key_chunk);
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tw0 = tile0 + wave * TPW;
    const bool wave_on = tw0 < N;
    const int r16 = lane & 15, kg = lane >> 4;
    const int qrow0 = q_start[b];
    const int64_t kbase = ctx_start[b];
    const int block_lim = last_cand(M, min(tile0 + TOK_TILE - 1, N - 1), es);
    const int key_end = min(key_hi, block_lim + 1);

    // Key DMA: instruction i of wave `wave` fills stage bytes 4096i + 1024wave
    // + 16lane = key row 64i + 16wave + lane/4, slot lane%4, which holds chunk
    // (lane%4) ^ ((lane/16) & 3); waves 2 and 3 also load the block scales and
    // key scales of keys 64(wave-2) .. +63 (one dword per lane each)
    const uint32_t kvoff = 1024u * wave + 64u * (lane >> 2) + 16u * ((lane & 3) ^ ((lane >> 4) & 3));
    auto issue = [&](int k0, uint8_t *kdst, uint32_t *bdst, float *sdst) {
        const __amdgpu_buffer_rsrc_t krs =
            make_buffer_rsrc((void *)(kI + (kbase + k0) * F4_ROW), (uint32_t)(ctx - k0) * F4_ROW);
#pragma unroll
        for (int i = 0; i < IDX_STAGE * F4_ROW / 16 / 256; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lds_void_t *)(kdst + 4096 * i + 1024 * wave), 16,
                                                     kvoff + 4096u * i, 0, 0, 0);
        if (wave >= 2) {
            const __amdgpu_buffer_rsrc_t brs =
                make_buffer_rsrc((void *)(k_bscale + (kbase + k0) * 4), (uint32_t)(ctx - k0) << 2);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(brs, (lds_void_t *)(bdst + 64 * (wave - 2)), 4,
                                                     4u * (64 * (wave - 2) + lane), 0, 0, 0);
            if (k_scale) {
                const __amdgpu_buffer_rsrc_t srs =
                    make_buffer_rsrc((void *)(k_scale + kbase + k0), (uint32_t)(ctx - k0) << 2);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void_t *)(sdst + 64 * (wave - 2)), 4,
                                                         4u * (64 * (wave - 2) + lane), 0, 0, 0);
            }
        }
    };
    // Normalise the block scales of this wave's 64 keys in a stage whose
    // loads have landed (waves 2 and 3): exponents minus the key's largest
    // (at least 0), and the key scale times 2^(largest - 127).  The LDS writes
    // complete before the wave moves on.
    auto normalise = [&](uint32_t *bsb, float *ksb) {
        const int key = 64 * (wave - 2) + lane;
        const uint32_t e = bsb[key];
        const int e0 = (int)(e & 0xFFu), e1 = (int)((e >> 8) & 0xFFu), e2 = (int)((e >> 16) & 0xFFu),
                  e3 = (int)(e >> 24);
        const int em = max(max(e0, e1), max(e2, e3));
        const uint32_t n0 = (uint32_t)max(e0 + 127 - em, 0), n1 = (uint32_t)max(e1 + 127 - em, 0),
                       n2 = (uint32_t)max(e2 + 127 - em, 0), n3 = (uint32_t)max(e3 + 127 - em, 0);
        const float ks = k_scale ? ksb[key] : 1.0f;
        bsb[key] = n0 | (n1 << 8) | (n2 << 16) | (n3 << 24);
        ksb[key] = ks * __builtin_ldexpf(1.0f, em - 127);
        __builtin_amdgcn_s_waitcnt(IDX_LGKM0);
    };
    if (key_lo < key_end)
        issue(key_lo, sKey0, sBs0, sKs0);

    // A operand of head tile hb: row r16 = (token r16/RPT, head RPT*hb +
    // r16%RPT); registers 0-3 = query bytes 16kg .., 4-7 = bytes 64+16kg ..
    const int a_tok = tw0 + r16 / RPT;
    const bool a_ok = a_tok < N;
    const int64_t a_row = (int64_t)qrow0 + (a_ok ? a_tok : 0);
    v8i a[HB];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
        const uint8_t *qr = q + ((a_row * H + RPT * hb + (r16 % RPT)) << 7);
        const v4i lo = a_ok ? *(const v4i *)(qr + 16 * kg) : v4i{0, 0, 0, 0};
        const v4i hi = a_ok ? *(const v4i *)(qr + 64 + 16 * kg) : v4i{0, 0, 0, 0};
        a[hb] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
    // output rows 4kg..4kg+3 of every tile: token tw0 + 4kg/RPT, heads
    // RPT*hb + (4kg)%RPT + i.  Head weights times the token's query scale and
    // 2^25 (undoing the MFMA's query scale), rounded once to bf16, as the
    // head-sum MFMA's A operands (as in the fp8 prefill kernel)
    const int e_tok = tw0 + (4 * kg) / RPT;
    const bool e_ok = e_tok < N;
    const int64_t e_row = (int64_t)qrow0 + (e_ok ? e_tok : 0);
    const int hsub = (4 * kg) % RPT;
    const float sq = (q_scale ? q_scale[e_row] : 1.0f) * 0x1p25f;
    const bool hs_lane = r16 == 4 * (kg >> 1);
    v8bf wA[HB / 2];
#pragma unroll
    for (int p = 0; p < HB / 2; ++p) {
        const v4f t0 = *(const v4f *)(w + e_row * H + RPT * (2 * p) + hsub);
        const v4f t1 = *(const v4f *)(w + e_row * H + RPT * (2 * p + 1) + hsub);
        const float f = hs_lane ? sq : 0.0f;
        wA[p] = __builtin_convertvector((v8f){t0[0] * f, t0[1] * f, t0[2] * f, t0[3] * f, t1[0] * f, t1[1] * f,
                                              t1[2] * f, t1[3] * f},
                                        v8bf);
    }
    const int sa = IDX_SCALE_2M25;
    const int wave_lim = last_cand(M, min(tw0 + TPW - 1, N - 1), es);
    // token tw0 + t's sums come out in lane group t (t < 2): one store per 16-key block
    const int s_tok = tw0 + kg;
    const int lim = last_cand(M, s_tok, es);
    const int nrows_blk = max(0, min(TOK_TILE, N - tile0));
    const int64_t blk_off = score_start[b] + (int64_t)tile0 * ctx;
    const __amdgpu_buffer_rsrc_t rsrc = make_buffer_rsrc(scores + blk_off, (uint32_t)((int64_t)nrows_blk * ctx * 4));
    const bool row_ok = kg < TPW && s_tok < N && wave_on;
    const uint32_t lane_row_off = (uint32_t)((int64_t)(s_tok - tile0) * ctx * 4);
    constexpr int STORES_PER_GROUP = 4;
    constexpr int STAGE_STORES = (IDX_STAGE / 64) * STORES_PER_GROUP;
    const int interior_end = min(ctx, last_cand(M, tile0, es) + 1);
    // this lane's B chunk (key row r16 of a 16-key block, bytes 16kg ..)
    const int boff = r16 * F4_ROW + 16 * (kg ^ ((r16 >> 2) & 3));

    // one stage: compute the keys in (stg, bs, ks); waves 2 and 3 normalise
    // the next stage's scales (nbs, nks) half way through, once its loads
    // (issued before this stage's stores) have landed
    auto stage = [&](int k0, const uint8_t *stg, const uint32_t *bs, const float *ks, uint32_t *nbs, float *nks,
                     bool next) {
#pragma unroll
        for (int gsub = 0; gsub < IDX_STAGE / 64; ++gsub) {
            const int s0 = k0 + 64 * gsub;
            if (s0 >= key_hi)
                break;
            const bool skip = !wave_on || s0 > wave_lim;
#pragma unroll
            for (int j = 0; j < STORES_PER_GROUP; ++j) {
                // token tw0 + kg at key s0 + 16*j + r16 (kg < 2), before the key scale
                float v = -INFINITY;
                if (!skip) {
                    const int row = 64 * gsub + 16 * j;  // first key of the 16-key block
                    const v4i bk = *(const v4i *)(stg + row * F4_ROW + boff);
                    const int sb = (int)((bs[row + r16] >> (8 * kg)) & 0xFFu);  // normalised E8M0 of block kg
                    v4f hc;
                    head_sum_group_f4c<true>(hc, a[0], a[1], a[2], a[3], bk, sa, sb, wA[0], wA[1]);
                    head_sum_group_f4c<false>(hc, a[4], a[5], a[6], a[7], bk, sa, sb, wA[2], wA[3]);
                    v = hc[0];
                }
                const int s = s0 + 16 * j + r16;
                const float kscale = ks[64 * gsub + 16 * j + r16];
                uint32_t off;
                if (s0 + 64 <= interior_end) {
                    v *= kscale;
                    off = row_ok ? lane_row_off + 4u * (uint32_t)s : 0x80000000u;
                } else {
                    v = s > lim ? -INFINITY : v * kscale;
                    off = (row_ok && s < ctx) ? lane_row_off + 4u * (uint32_t)s : 0x80000000u;
                }
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rsrc, off, 0, 0);
            }
            if (gsub == 0 && next && wave >= 2) {
                // the next stage's loads precede this group's stores
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_waitcnt(vmcnt_only(STORES_PER_GROUP));
                normalise(nbs, nks);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    __builtin_amdgcn_s_waitcnt(0);
    if (key_lo < key_end && wave >= 2)
        normalise(sBs0, sKs0);
    __syncthreads();
    for (int k0 = key_lo; k0 < key_hi; k0 += 2 * IDX_STAGE) {
        const bool n1 = k0 + IDX_STAGE < key_end;
        if (n1)
            issue(k0 + IDX_STAGE, sKey1, sBs1, sKs1);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0, sKey0, sBs0, sKs0, sBs1, sKs1, n1);
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
        if (k0 + IDX_STAGE >= key_hi)
            break;
        const bool n0 = k0 + 2 * IDX_STAGE < key_end;
        if (n0)
            issue(k0 + 2 * IDX_STAGE, sKey0, sBs0, sKs0);
        __builtin_amdgcn_sched_barrier(0);
        stage(k0 + IDX_STAGE, sKey1, sBs1, sKs1, sBs0, sKs0, n0);
        __builtin_amdgcn_s_waitcnt(vmcnt_only(STAGE_STORES));
        lds_barrier();
    }
}

// Plain vector kernel for any dtype and shape: one (token, key) score per thread.
__global__ __launch_bounds__(256) void index_scores_vector(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs, int es,
    const void *__restrict__ q, int q_dt, const float *__restrict__ q_scale,
    const void *__restrict__ kI, int k_dt, const float *__restrict__ k_scale,
    const float *__restrict__ w, int H, int d, float *__restrict__ scores)
{
    int b, t0;
    if (!tile_slot(q_start, num_seqs, blockIdx.y, GEN_TOK_TILE, b, t0))
        return;
    const int N = q_start[b + 1] - q_start[b];
    const int M = hist_len[b];
    const int ctx = entries_of(M + N, es);
    const int i = t0 + threadIdx.x / GEN_KEY_TILE;
    const int s = blockIdx.x * GEN_KEY_TILE + threadIdx.x % GEN_KEY_TILE;
    if (i >= N || s >= ctx)
        return;
    float *dst = scores + score_start[b] + (int64_t)i * ctx + s;
    if (s > last_cand(M, i, es)) {
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

namespace janus {

// Row-tile kernel: a block takes up to NQ tokens of one session and one
// chunk of 1024, 2048 or 4096 keys (chosen per launch).  It serves
// decode-shaped batches (every session appends at most NQ tokens, as in the
// decode phase: the scores are a GEMV over each session's keys, bound by
// reading the keys once), with fp8 or MXFP4 keys.  The four waves take the
// chunk's 64-key groups in turn; a wave reads a group's keys (and their
// scales) straight from global memory one group ahead - each key is used by
// this block alone, so nothing is staged in LDS - and for every token runs
// one head group per 16-key block: four 16x16x128 MFMAs (16 heads x 16 keys
// each) and the epilogue.  fp8 keys: the tokens' head sums accumulate into
// one head-sum MFMA result whose lane group t holds token t's scores, and
// one store per 16-key block writes them.  MXFP4 keys: each token's head sum
// is completed across lanes, and lane group g stores 16-key block g of the
// group: one 256-byte store per token and group; groups wholly past every
// token's causal limit skip the MFMAs (their stores write -inf).
constexpr int ROWS_NQ = 4;
constexpr int ROWS_CHUNK_MAX = 4096;   // keys per block: 4096, 2048 or 1024
constexpr int ROWS_CHUNK_MIN = 1024;

template <int NQ, bool FP4>
__global__ __launch_bounds__(256, 2) void index_scores_rows(
    const int32_t *__restrict__ q_start, const int32_t *__restrict__ ctx_start,
    const int32_t *__restrict__ hist_len, const int64_t *__restrict__ score_start, int num_seqs, int es, int nchunks,
    int chunk, int one_tile, const uint8_t *__restrict__ q, const float *__restrict__ q_scale, const uint8_t *__restrict__ kI,
    const uint8_t *__restrict__ k_bscale, const float *__restrict__ k_scale, const float *__restrict__ w,
    float *__restrict__ scores)
{
    // block = (tile, chunk), chunk fastest; with one tile per session the
    // tile is the session
    const int tile = blockIdx.x / nchunks;
    const int c0 = (blockIdx.x - tile * nchunks) * chunk;
    int b = tile, t0 = 0;
    if (!one_tile && !tile_slot(q_start, num_seqs, tile, NQ, b, t0))
        return;
    const int qs = q_start[b], N = q_start[b + 1] - qs;
    const int M = hist_len[b], ctx = entries_of(M + N, es);
    const int nv = min(NQ, N - t0);  // tokens of this tile
    if (nv <= 0 || c0 >= ctx)
        return;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, kg = lane >> 4;
    // A operand of token t, head tile hb: row r16 = head 16hb + r16, bytes
    // 32kg .. 32kg+31 (for MXFP4 keys reordered by evens_odds); this lane's
    // output rows 4kg .. 4kg+3 are heads
    // 16hb + 4kg + i, whose weights (times the query scale, and for fp8 keys
    // times 2^25) it holds
    v8i a[NQ][4];
    v2bf wv[NQ][4][2];  // MXFP4 keys: the dot products' weight pairs
    // fp8 keys: the head-sum MFMA's A operands, tile pairs (0, 1) and (2, 3)
    // of token t in row 4t (lanes with r16 = 4t; zeros elsewhere), so that
    // lane group t receives token t's sums (as in the prefill kernel)
    v8bf wA[NQ][2];
    // MXFP4: the scaled MFMA takes K 16kg .. 16kg+15 from this lane's low 16
    // bytes, K 64+16kg .. from its high 16, and the E8M0 scale of K block b
    // (32 elements) from lane group b.  Lane group kg therefore holds half kg%2
    // of MX blocks kg/2 and 2+kg/2, so each hardware block is one MX block,
    // the one whose scale this lane supplies.
    const int f4_half = 32 * (kg >> 1) + 16 * (kg & 1);  // first element of the low half
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
        const bool ok = t < nv;
        const int64_t row = qs + t0 + (ok ? t : 0);
        const float sq = (q_scale ? q_scale[row] : 1.0f) * (FP4 ? 1.0f : 0x1p25f);
#pragma unroll
        for (int hb = 0; hb < 4; ++hb) {
            const uint8_t *qr = q + ((row * 64 + 16 * hb + r16) << 7);
            if constexpr (FP4) {
                const v4i lo = ok ? *(const v4i *)(qr + f4_half) : v4i{0, 0, 0, 0};
                const v4i hi = ok ? *(const v4i *)(qr + 64 + f4_half) : v4i{0, 0, 0, 0};
                a[t][hb] = evens_odds(v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
            } else {
                a[t][hb] = ok ? *(const v8i *)(qr + 32 * kg) : v8i{0, 0, 0, 0, 0, 0, 0, 0};
            }
            if constexpr (FP4) {
                const v4f tw = *(const v4f *)(w + row * 64 + 16 * hb + 4 * kg);
                wv[t][hb][0] = __builtin_convertvector((v2f){tw[0] * sq, tw[1] * sq}, v2bf);
                wv[t][hb][1] = __builtin_convertvector((v2f){tw[2] * sq, tw[3] * sq}, v2bf);
            }
        }
        if constexpr (!FP4) {
            const float f = r16 == 4 * t ? sq : 0.0f;
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const v4f t0w = *(const v4f *)(w + row * 64 + 16 * (2 * p) + 4 * kg);
                const v4f t1w = *(const v4f *)(w + row * 64 + 16 * (2 * p + 1) + 4 * kg);
                wA[t][p] = __builtin_convertvector((v8f){t0w[0] * f, t0w[1] * f, t0w[2] * f, t0w[3] * f, t1w[0] * f,
                                                         t1w[1] * f, t1w[2] * f, t1w[3] * f},
                                                   v8bf);
            }
        }
    }
    constexpr int KB = FP4 ? 64 : 128;  // key bytes
    // the session's keys (block scales, key scales) from c0 on: rows past the
    // context read as zeros; its score rows (row t at t * ctx): stores past
    // them drop
    const int64_t kbase = (int64_t)ctx_start[b] + c0;
    const __amdgpu_buffer_rsrc_t krs = make_buffer_rsrc((void *)(kI + kbase * KB), (uint32_t)(ctx - c0) * KB);
    const __amdgpu_buffer_rsrc_t bsr =
        make_buffer_rsrc((void *)(FP4 ? k_bscale + kbase * 4 : nullptr), FP4 ? (uint32_t)(ctx - c0) * 4u : 0u);
    const __amdgpu_buffer_rsrc_t ksr =
        make_buffer_rsrc((void *)(k_scale ? k_scale + kbase : nullptr), k_scale ? (uint32_t)(ctx - c0) << 2 : 0u);
    const __amdgpu_buffer_rsrc_t srs =
        make_buffer_rsrc(scores + score_start[b] + (int64_t)t0 * ctx, (uint32_t)(nv * ctx) << 2);
    const int ngroups = (min(chunk, ctx - c0) + 63) / 64;
    int lim[NQ];  // each token's last candidate (block-uniform)
#pragma unroll
    for (int t = 0; t < NQ; ++t)
        lim[t] = __builtin_amdgcn_readfirstlane(last_cand(M, t0 + t, es));
    const int last_lim = last_cand(M, t0 + nv - 1, es);  // largest causal limit in the tile
    const int lane_lim = last_cand(M, t0 + kg, es);       // fp8 keys: the causal limit of the token this lane stores

    struct Group {
        v4i k[8];   // 16-key block j: key row 16j + r16; fp8: bytes 32kg.. in k[2j], k[2j+1]; fp4: both halves in k[j]
        int bs[4];  // fp4: the E8M0 scales of key row 16j + r16, block kg in the low byte
        float ks[4];  // fp4: [0] = scale of key 16kg + r16 (the one this lane stores); fp8: key 16j + r16
    };
    auto load = [&](int g, Group &G) {
        const uint32_t row0 = (uint32_t)(64 * g + r16);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t row = row0 + 16u * j;
            if constexpr (FP4) {
                const v2i lo = __builtin_bit_cast(v2i, __builtin_amdgcn_raw_buffer_load_b64(krs, row * 64u + f4_half / 2, 0, 0));
                const v2i hi =
                    __builtin_bit_cast(v2i, __builtin_amdgcn_raw_buffer_load_b64(krs, row * 64u + 32u + f4_half / 2, 0, 0));
                G.k[j] = v4i{lo[0], lo[1], hi[0], hi[1]};
                G.bs[j] = (int)(__builtin_amdgcn_raw_buffer_load_b32(bsr, row * 4u, 0, 0) >> (8 * kg));
            } else {
                const uint32_t off = row0 * 128u + 32u * kg + 2048u * j;
                G.k[2 * j] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(krs, off, 0, 0));
                G.k[2 * j + 1] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(krs, off + 16u, 0, 0));
            }
        }
        if constexpr (FP4) {
            G.ks[0] = k_scale ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                          ksr, (uint32_t)(64 * g + 16 * kg + r16) * 4u, 0, 0))
                              : 1.0f;
        } else {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
                G.ks[jj] = k_scale ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                               ksr, (uint32_t)(64 * g + 16 * jj + r16) * 4u, 0, 0))
                                   : 1.0f;
        }
    };
    auto compute = [&](int g, const Group &G) {
        if constexpr (!FP4) {
            // per 16-key block: the tokens' head groups accumulate into one
            // head-sum result, lane group t holding token t's scores; one
            // store writes them all
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const v8i bk = v8i{G.k[2 * j][0], G.k[2 * j][1], G.k[2 * j][2], G.k[2 * j][3],
                                   G.k[2 * j + 1][0], G.k[2 * j + 1][1], G.k[2 * j + 1][2], G.k[2 * j + 1][3]};
                v4f hc;
                head_sum_group<true>(hc, a[0][0], a[0][1], a[0][2], a[0][3], bk, IDX_MFMA_SCALES, wA[0][0], wA[0][1]);
#pragma unroll
                for (int t = 1; t < NQ; ++t) {
                    if (t >= nv)  // block-uniform; a missing token's lanes store nothing
                        continue;
                    head_sum_group<false>(hc, a[t][0], a[t][1], a[t][2], a[t][3], bk, IDX_MFMA_SCALES, wA[t][0],
                                          wA[t][1]);
                }
                const int s = c0 + 64 * g + 16 * j + r16;  // the key this lane stores, for token kg
                const float v = s > lane_lim ? -INFINITY : hc[0] * G.ks[j];
                const uint32_t off = (kg < nv && s < ctx) ? (uint32_t)(kg * ctx + s) * 4u : 0x80000000u;
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), srs, off, 0, 0);
            }
        } else {
            // one vector per token, so that picking this lane's key below is a
            // register select (an array of floats picked by kg goes to scratch)
            v4f res[NQ];
            const bool masked = c0 + 64 * g > last_lim;  // block-uniform
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const v8i bk = expand_e2m1(G.k[j]);
#pragma unroll
                for (int t = 0; t < NQ; ++t) {
                    // block-uniform; a masked group's stores write -inf, a
                    // missing token's none
                    if (t >= nv || masked)
                        continue;
                    float r;
                    head_group_f4<true>(r, a[t][0], a[t][1], a[t][2], a[t][3], bk, F4_QUERY_SCALE, G.bs[j],
                                        &wv[t][0]);
                    r += xor_lanes16(r);
                    r += __shfl_xor(r, 32, 64);
                    res[t][j] = r;
                }
            }
            const int s = c0 + 64 * g + 16 * kg + r16;  // the key this lane stores
#pragma unroll
            for (int t = 0; t < NQ; ++t) {
                if (t >= nv)
                    continue;
                float v = res[t][kg];
                v = s > lim[t] ? -INFINITY : v * G.ks[0];
                const uint32_t off = s < ctx ? (uint32_t)(t * ctx + s) * 4u : 0x80000000u;
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), srs, off, 0, 0);
            }
        }
    };
    // The prefetch is unconditional (groups past the chunk read zeros through
    // the descriptor), so the compiler sees the same number of loads after
    // every group's and can wait for just that group.
    Group A, B;
    load(wave, A);
    for (int g = wave; g < ngroups; g += 8) {
        load(g + 4, B);
        compute(g, A);
        if (g + 4 >= ngroups)
            break;
        load(g + 8, A);
        compute(g + 4, B);
    }
}

}  // namespace janus

namespace janus {

// Tiles of the row-tile kernel: one per session when no session appends
// more than NQ tokens, else an upper bound (ceil(total_q / NQ) + sessions).
static int64_t rows_tiles(const janus_batch *bt, int nq)
{
    return bt->max_q <= nq ? bt->num_seqs : ceil_div(bt->total_q, nq) + (int64_t)bt->num_seqs;
}
static int rows_nq(const janus_batch *bt) { return bt->max_q <= 1 ? 1 : bt->max_q <= 2 ? 2 : ROWS_NQ; }
static bool rows_grid_ok(const janus_batch *bt)
{
    return rows_tiles(bt, rows_nq(bt)) * ceil_div(bt->max_ctx, ROWS_CHUNK_MIN) <= INT32_MAX;
}

// Keys per block.  A ragged batch's blocks fill the GPU's resident block
// slots in rounds, the last one part-empty, and few blocks leave CUs idle:
// of 4096, 2048 and 1024 keys, take the chunk whose estimated block count
// fills its rounds best (ties, within 5%, go to the longer chunk, which
// loads its tokens' queries once for more keys).  A session of C keys makes
// about C/chunk + 1/2 blocks per tile.
template <typename Kern>
static int rows_chunk(const janus_batch *bt, int64_t tiles, Kern kern)
{
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, 256, 0) != hipSuccess || cus < 1 || per < 1)
        return ROWS_CHUNK_MAX;
    const double slots = (double)per * cus;
    const double tiles_per_seq = (double)tiles / bt->num_seqs;
    int best = ROWS_CHUNK_MAX;
    double best_fill = -1.0;
    for (int c = ROWS_CHUNK_MAX; c >= ROWS_CHUNK_MIN; c /= 2) {
        const double blocks = tiles_per_seq * ((double)bt->total_ctx / c + 0.5 * bt->num_seqs);
        const double fill = blocks / (std::ceil(blocks / slots) * slots);
        if (fill > best_fill + 0.05) {
            best_fill = fill;
            best = c;
        }
    }
    return best;
}

// 1-D grid of the row-tile kernel: (tile, key chunk), chunk fastest
template <bool FP4>
static void launch_rows(const janus_batch *bt, const void *q, const float *q_scale, const void *kI,
                        const uint8_t *k_bscale, const float *k_scale, const float *w, float *scores, hipStream_t st)
{
    const int nq = rows_nq(bt);
    const int one_tile = bt->max_q <= nq;
    const int64_t tiles = rows_tiles(bt, nq);
    auto go = [&](auto kern) {
        const int chunk = rows_chunk(bt, tiles, kern);
        const int nchunks = ceil_div(bt->max_ctx, chunk);
        hipLaunchKernelGGL(kern, dim3((unsigned)(tiles * nchunks)), dim3(256), 0, st, bt->q_start, bt->ctx_start,
                           bt->hist_len, bt->score_start, bt->num_seqs, bt->entry_shift, nchunks, chunk, one_tile,
                           (const uint8_t *)q, q_scale, (const uint8_t *)kI, k_bscale, k_scale, w, scores);
    };
    if (nq == 1)
        go(index_scores_rows<1, FP4>);
    else if (nq == 2)
        go(index_scores_rows<2, FP4>);
    else
        go(index_scores_rows<ROWS_NQ, FP4>);
}

}  // namespace janus

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
    // the MFMA kernel addresses a session's keys and a block's score rows
    // with 32-bit buffer offsets: contexts up to 2^24 tokens
    if (q_dt == JANUS_FP8_E4M3 && d == 128 && H == 64 && bt->max_ctx <= (1 << 24) && bt->max_q <= ROWS_NQ &&
        rows_grid_ok(bt)) {
        // decode-shaped: one block per (session, 4096-key chunk)
        launch_rows<false>(bt, q, q_scale, kI, nullptr, k_scale, w, scores, st);
        return launch_status();
    }
    if (q_dt == JANUS_FP8_E4M3 && d == 128 && H == 64 && bt->max_ctx <= (1 << 24)) {
        // key chunks: a multiple of the XCD count, each a whole number of
        // stages and at most IDX_KEY_CHUNK keys long
        const int per_xcd_keys = ceil_div(bt->max_ctx, IDX_XCD);
        const int chunks_per_xcd = std::max(1, ceil_div(per_xcd_keys, IDX_KEY_CHUNK));
        const int key_chunk = ceil_div(ceil_div(per_xcd_keys, chunks_per_xcd), IDX_STAGE) * IDX_STAGE;
        const int nchunks = ceil_div(bt->max_ctx, key_chunk);
        constexpr int TPW = IDX_TPW;
        const int ntiles = ceil_div(bt->total_q, 4 * TPW) + nseq;
        const int per_xcd = ceil_div(nchunks, IDX_XCD) * ntiles;
        hipLaunchKernelGGL((index_scores_fp8_mfma<64, TPW>), dim3(IDX_XCD * per_xcd), dim3(256), 0, st, bt->q_start,
                           bt->ctx_start, bt->hist_len, bt->score_start, nseq, bt->entry_shift, nchunks, key_chunk, ntiles,
                           (const uint8_t *)q, q_scale, (const uint8_t *)kI, k_scale, w, scores);
        return launch_status();
    }
    if (q_dt == JANUS_BF16 && d == 128 && H == 64 && bt->max_ctx <= (1 << 23)) {
        // bf16 on bf16 MFMA: the fp8 kernel's key chunking (32-bit buffer
        // offsets over 256-byte key rows: contexts up to 2^23)
        const int per_xcd_keys = ceil_div(bt->max_ctx, IDX_XCD);
        const int chunks_per_xcd = std::max(1, ceil_div(per_xcd_keys, IDX_KEY_CHUNK));
        const int key_chunk = ceil_div(ceil_div(per_xcd_keys, chunks_per_xcd), IDX_STAGE) * IDX_STAGE;
        const int nchunks = ceil_div(bt->max_ctx, key_chunk);
        const int ntiles = ceil_div(bt->total_q, 8) + nseq;
        const int per_xcd = ceil_div(nchunks, IDX_XCD) * ntiles;
        hipLaunchKernelGGL(index_scores_bf16_mfma, dim3(IDX_XCD * per_xcd), dim3(256), 0, st, bt->q_start,
                           bt->ctx_start, bt->hist_len, bt->score_start, nseq, bt->entry_shift, nchunks, key_chunk,
                           ntiles, (const uint16_t *)q, q_scale, (const uint8_t *)kI, k_scale, w, scores);
        return launch_status();
    }
    dim3 grid(ceil_div(bt->max_ctx, GEN_KEY_TILE), ceil_div(bt->total_q, GEN_TOK_TILE) + nseq);
    hipLaunchKernelGGL(index_scores_vector, grid, dim3(GEN_TOK_TILE * GEN_KEY_TILE), 0, st, bt->q_start,
                       bt->ctx_start, bt->hist_len, bt->score_start, nseq, bt->entry_shift, q, (int)q_dt, q_scale, kI, (int)k_dt,
                       k_scale, w, H, d, scores);
    return launch_status();
}

extern "C" int janus_index_scores_mxfp4(const janus_batch *bt, const void *q, const float *q_scale, const void *kI,
                                        const uint8_t *k_block_scale, const float *k_scale, const float *w, int H,
                                        int d, float *scores, void *stream)
{
    if (!batch_ok(bt) || !bt->ctx_start || !bt->score_start || !q || !kI || !k_block_scale || !w || !scores ||
        H < 1 || d < 1 || d % 32 != 0)
        return JANUS_ERR_INVALID_ARG;
    // the row-tile kernel: 64 heads x 128 dims, 32-bit buffer offsets
    if (H != 64 || d != 128 || bt->max_ctx > (1 << 24) || !rows_grid_ok(bt))
        return JANUS_ERR_UNSUPPORTED;
    if (bt->total_q == 0 || bt->max_ctx == 0)
        return JANUS_OK;
    if (bt->max_q <= ROWS_NQ) {
        // decode-shaped: the row-tile kernel
        launch_rows<true>(bt, q, q_scale, kI, k_block_scale, k_scale, w, scores, as_stream(stream));
        return launch_status();
    }
    // prefill-shaped: keys staged through LDS, the fp8 kernel's chunking
    const int per_xcd_keys = ceil_div(bt->max_ctx, IDX_XCD);
    const int chunks_per_xcd = std::max(1, ceil_div(per_xcd_keys, IDX_KEY_CHUNK));
    const int key_chunk = ceil_div(ceil_div(per_xcd_keys, chunks_per_xcd), IDX_STAGE) * IDX_STAGE;
    const int nchunks = ceil_div(bt->max_ctx, key_chunk);
    const int ntiles = ceil_div(bt->total_q, 8) + bt->num_seqs;
    const int per_xcd = ceil_div(nchunks, IDX_XCD) * ntiles;
    hipLaunchKernelGGL(index_scores_mxfp4_mfma, dim3(IDX_XCD * per_xcd), dim3(256), 0, as_stream(stream),
                       bt->q_start, bt->ctx_start, bt->hist_len, bt->score_start, bt->num_seqs, bt->entry_shift,
                       nchunks, key_chunk, ntiles, (const uint8_t *)q, q_scale, (const uint8_t *)kI, k_block_scale,
                       k_scale, w, scores);
    return launch_status();
}
