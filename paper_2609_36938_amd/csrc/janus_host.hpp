// Host-side helpers for the C ABI entry points: argument checks and launch
// status handling.  No entry point allocates or synchronises.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "janus.h"

namespace janus {

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Status of the most recent launch on this thread.
inline int launch_status()
{
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? JANUS_OK : JANUS_ERR_DEVICE;
}

inline bool batch_ok(const janus_batch *b)
{
    return b && b->num_seqs >= 1 && b->total_q >= 0 && b->max_q >= 0 && b->max_ctx >= 0 &&
           b->total_ctx >= 0 && b->q_start && b->hist_len && b->max_q <= b->total_q &&
           (int64_t)b->max_ctx <= b->total_ctx && b->entry_shift >= 0 && b->entry_shift <= 16;
}

inline bool dtype_ok(int dt) { return dt == JANUS_F32 || dt == JANUS_BF16 || dt == JANUS_FP8_E4M3; }

inline bool pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

// A page table of pt_ld entries per session covers every id of the longest
// session (ids are read through it up to max_ctx - 1).  page_size > 0.
inline bool table_covers(const janus_batch *b, int pt_ld, int page_size)
{
    return pt_ld >= 1 && (int64_t)pt_ld * page_size >= (int64_t)b->max_ctx;
}

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

} // namespace janus
