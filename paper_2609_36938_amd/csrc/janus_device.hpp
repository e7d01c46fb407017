// Device-side helpers shared by the gfx950 kernels of libjanus.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "janus.h"

#define JANUS_DEV __device__ __forceinline__

namespace janus {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v8f __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef short v2s __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Entry granularity (2^es tokens per entry; es = 0: tokens).  Entries
// complete among a session's first n tokens, and the last candidate of the
// appended token at position M + i: the last entry complete there.
JANUS_DEV int entries_of(int n, int es) { return n >> es; }
JANUS_DEV int last_cand(int M, int i, int es) { return ((M + i + 1) >> es) - 1; }

// Session of global query row `row`: largest b with q_start[b] <= row.
JANUS_DEV int session_of_row(const int32_t *q_start, int num_seqs, int row)
{
    int lo = 0, hi = num_seqs - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (q_start[mid] <= row)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// OCP e4m3fn byte -> fp32 (exact).
JANUS_DEV float fp8e4m3_to_f32(uint32_t b)
{
    uint32_t sign = (b & 0x80u) << 24;
    uint32_t e = (b >> 3) & 15u, m = b & 7u;
    float v;
    if (e == 0) {
        v = (float)m * 0.001953125f; // m * 2^-9
        return __uint_as_float(__float_as_uint(v) | sign);
    }
    if (e == 15 && m == 7)
        return __uint_as_float(0x7fc00000u | sign);
    return __uint_as_float(sign | ((e + 120u) << 23) | (m << 20));
}

JANUS_DEV float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

JANUS_DEV float load_elem(const void *p, int dt, int64_t i)
{
    if (dt == JANUS_F32)
        return ((const float *)p)[i];
    if (dt == JANUS_BF16)
        return bf16_to_f32(((const uint16_t *)p)[i]);
    return fp8e4m3_to_f32(((const uint8_t *)p)[i]);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
JANUS_DEV uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Order-preserving map of an fp32 score to uint32 (larger score -> larger
// key); -0.0 is folded onto +0.0 so the two compare equal.
JANUS_DEV uint32_t score_key(float f)
{
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

} // namespace janus
