"""Python face of the plain CPU oracle (``janus_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the HIP library or its binding.  The
functions take numpy arrays from the input generator, hand them to the C
oracle and return numpy results; they add no arithmetic of their own beyond
slicing rows out of a score matrix.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "janus_oracle.c")
_LIB = os.path.join(_HERE, "libjanus_oracle.so")

DT = {"f32": 0, "bf16": 1, "fp8": 2}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        # JANUS_ORACLE_LIB: a separately built copy of the same source (the
        # tests' sanitizer run loads an AddressSanitizer/UBSan build this way)
        path = os.environ.get("JANUS_ORACLE_LIB")
        if not path:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            path = _LIB
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64, dbl = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.jo_fp8_e4m3fn_value.argtypes = [ctypes.c_uint8]
        L.jo_fp8_e4m3fn_value.restype = dbl
        L.jo_bf16_value.argtypes = [ctypes.c_uint16]
        L.jo_bf16_value.restype = dbl
        L.jo_index_scores.argtypes = [i32, P, P, i32, P, i32, P, P, i32, P, P, i32, i32, i32, P, P, i64]
        L.jo_index_scores_mxfp4.argtypes = [i32, P, P, i32, P, i32, P, P, P, P, P, i32, i32, i32, P, P, i64]
        L.jo_e2m1_value.argtypes = [ctypes.c_uint8]
        L.jo_e2m1_value.restype = dbl
        L.jo_e8m0_value.argtypes = [ctypes.c_uint8]
        L.jo_e8m0_value.restype = dbl
        L.jo_topk.argtypes = [i32, P, P, i32, i32, P, P, i64, i32, P]
        L.jo_topk_sharded.argtypes = [i32, P, P, i32, i32, P, P, i64, i32, i32, i32, P]
        L.jo_page_demand.argtypes = [i32, P, P, i32, P, i32, P, i32, i32, P, i32, P, P, P]
        L.jo_runs.argtypes = [P, i32, i32, P, P]
        L.jo_predict_diff.argtypes = [P, P, i32, i32, P, P, P]
        L.jo_sparse_attn.argtypes = [i32, P, P, i32, i32, P, P, i32, i32, i32, P, P, i64, i64,
                                     P, i32, i32, P, i32, dbl, P, P]
        L.jo_sparse_attn_fp8kv.argtypes = [i32, P, P, i32, i32, P, P, i32, P, i64, P, i32, i32, P, i32, dbl, P, P]
        for f in ("jo_index_scores", "jo_sparse_attn_fp8kv", "jo_topk", "jo_topk_sharded", "jo_page_demand", "jo_runs",
                  "jo_predict_diff", "jo_sparse_attn"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def fp8_value(b: int) -> float:
    return lib().jo_fp8_e4m3fn_value(int(b))


def e2m1_value(code: int) -> float:
    return lib().jo_e2m1_value(int(code))


def e8m0_value(e: int) -> float:
    return lib().jo_e8m0_value(int(e))


def index_scores_mxfp4(q_start, hist_len, q, q_dt, q_scale, kI, k_bscale, k_scale, w, rows, out_ld=None, entry=1):
    """Scores (float64) with MXFP4 indexer keys: kI [ctx rows, d/2] bytes,
    k_bscale [ctx rows, d/32] E8M0 bytes."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    H, d = q.shape[1], q.shape[2]
    if out_ld is None:
        out_ld = int(((hist_len + np.diff(q_start)) // entry).max())
    out = np.empty((rows.shape[0], out_ld), dtype=np.float64)
    rc = lib().jo_index_scores_mxfp4(len(hist_len), _p(q_start), _p(hist_len), entry, _p(np.ascontiguousarray(q)),
                                     DT[q_dt],
                                     _p(_c(q_scale, np.float32)), _p(_c(kI, np.uint8)), _p(_c(k_bscale, np.uint8)),
                                     _p(_c(k_scale, np.float32)), _p(_c(w, np.float32)), H, d, rows.shape[0],
                                     _p(rows), _p(out), out_ld)
    _check(rc, "index_scores_mxfp4")
    return out


def bf16_value(b: int) -> float:
    return lib().jo_bf16_value(int(b))


def index_scores(q_start, hist_len, q, q_dt, q_scale, kI, k_dt, k_scale, w, rows, out_ld=None, entry=1):
    """Scores (float64) of the given global query rows, [len(rows), out_ld].
    entry = tokens per entry (1: token granularity)."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    H, d = q.shape[1], q.shape[2]
    if out_ld is None:
        out_ld = int(((hist_len + np.diff(q_start)) // entry).max())
    out = np.empty((rows.shape[0], out_ld), dtype=np.float64)
    rc = lib().jo_index_scores(len(hist_len), _p(q_start), _p(hist_len), entry, _p(np.ascontiguousarray(q)), DT[q_dt],
                               _p(_c(q_scale, np.float32)), _p(np.ascontiguousarray(kI)), DT[k_dt],
                               _p(_c(k_scale, np.float32)), _p(_c(w, np.float32)), H, d,
                               rows.shape[0], _p(rows), _p(out), out_ld)
    _check(rc, "index_scores")
    return out


def topk(q_start, hist_len, rows, scores_rows, k, entry=1):
    """Top-k ids of the given rows; scores_rows [len(rows), ld] float32."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    sc = _c(scores_rows, np.float32)
    out = np.empty((rows.shape[0], k), dtype=np.int32)
    rc = lib().jo_topk(len(hist_len), _p(q_start), _p(hist_len), entry, rows.shape[0], _p(rows), _p(sc),
                       sc.shape[1], k, _p(out))
    _check(rc, "topk")
    return out


def topk_sharded(q_start, hist_len, rows, scores_rows, k, shards, align, entry=1):
    """Per-shard top-(k/shards) history ids of the given rows (Eq. 3);
    scores_rows [len(rows), ld] float32.  Returns [len(rows), k]."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    sc = _c(scores_rows, np.float32)
    out = np.empty((rows.shape[0], k), dtype=np.int32)
    rc = lib().jo_topk_sharded(len(hist_len), _p(q_start), _p(hist_len), entry, rows.shape[0], _p(rows), _p(sc),
                               sc.shape[1], k, shards, align, _p(out))
    _check(rc, "topk_sharded")
    return out


def page_demand(q_start, hist_len, topk_idx, page_table, page_size, num_phys_pages, limit=None, entry=1):
    """(bitmap uint32 [ceil(P/32)], ascending page list, count)."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    ti = _c(topk_idx, np.int32)
    pt = _c(page_table, np.int32)
    lim = _c(limit, np.int32)
    nw = (num_phys_pages + 31) // 32
    bm = np.zeros(max(nw, 1), dtype=np.uint32)
    lst = np.zeros(max(num_phys_pages, 1), dtype=np.int32)
    cnt = np.zeros(1, dtype=np.int32)
    rc = lib().jo_page_demand(len(hist_len), _p(q_start), _p(hist_len), entry, _p(ti), ti.shape[1], _p(pt),
                              pt.shape[1], page_size, _p(lim), num_phys_pages, _p(bm), _p(lst), _p(cnt))
    _check(rc, "page_demand")
    c = int(cnt[0])
    return bm[:nw], lst[:c].copy(), c


def runs(bitmap, num_phys_pages, max_run):
    """Packed reads: int32 [n_runs, 2] of (start, length)."""
    bm = _c(bitmap, np.uint32)
    out = np.zeros((max(num_phys_pages, 1), 2), dtype=np.int32)
    n = np.zeros(1, dtype=np.int32)
    rc = lib().jo_runs(_p(bm), num_phys_pages, max_run, _p(out), _p(n))
    _check(rc, "runs")
    return out[: int(n[0])].copy()


def predict_diff(actual, predicted, num_phys_pages, max_run):
    """(miss bitmap, miss runs [n, 2], counts {|A|,|P|,|A&P|,|miss|,#runs})."""
    a = _c(actual, np.uint32)
    p = _c(predicted, np.uint32)
    nw = (num_phys_pages + 31) // 32
    miss = np.zeros(max(nw, 1), dtype=np.uint32)
    mr = np.zeros((max(num_phys_pages, 1), 2), dtype=np.int32)
    counts = np.zeros(5, dtype=np.int32)
    rc = lib().jo_predict_diff(_p(a), _p(p), num_phys_pages, max_run, _p(miss), _p(mr), _p(counts))
    _check(rc, "predict_diff")
    return miss[:nw], mr[: int(counts[4])].copy(), counts


def sparse_attn(q_start, hist_len, rows, q_rows, k_pool, v_pool, k_row_stride, v_row_stride,
                page_table, page_size, sel_rows, scale, dv, entry=1):
    """Attention (float64) for the given rows.

    q_rows [len(rows), Hq, dqk] bf16 bits of those rows; sel_rows [len(rows), k].
    Returns (out [len(rows), Hq, dv], lse [len(rows), Hq]).
    """
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    q_rows = _c(q_rows, np.uint16)
    n, Hq, dqk = q_rows.shape
    out = np.empty((n, Hq, dv), dtype=np.float64)
    lse = np.empty((n, Hq), dtype=np.float64)
    kp = _c(k_pool, np.uint16)
    vp = kp if v_pool is None else _c(v_pool, np.uint16)
    pt = _c(page_table, np.int32)
    sel = _c(sel_rows, np.int32)
    rc = lib().jo_sparse_attn(len(hist_len), _p(q_start), _p(hist_len), entry, n, _p(rows), _p(q_rows), Hq, dqk, dv,
                              _p(kp), _p(vp), k_row_stride, v_row_stride, _p(pt), pt.shape[1], page_size,
                              _p(sel), sel.shape[1], float(scale), _p(out), _p(lse))
    _check(rc, "sparse_attn")
    return out, lse


def sparse_attn_fp8kv(q_start, hist_len, rows, q_rows, kv_pool, page_table, page_size, sel_rows, scale, entry=1):
    """MLA attention (float64) over fp8 KV rows: kv_pool uint8 [..., row_bytes],
    576 e4m3 bytes then the fp32 scale.  Returns (out [n, Hq, 512], lse [n, Hq])."""
    q_start = _c(q_start, np.int32)
    hist_len = _c(hist_len, np.int32)
    rows = _c(rows, np.int32)
    q_rows = _c(q_rows, np.uint16)
    n, Hq, _ = q_rows.shape
    kv = _c(kv_pool, np.uint8)
    row_bytes = kv.shape[-1]
    out = np.empty((n, Hq, 512), dtype=np.float64)
    lse = np.empty((n, Hq), dtype=np.float64)
    pt = _c(page_table, np.int32)
    sel = _c(sel_rows, np.int32)
    rc = lib().jo_sparse_attn_fp8kv(len(hist_len), _p(q_start), _p(hist_len), entry, n, _p(rows), _p(q_rows), Hq,
                                    _p(kv), row_bytes, _p(pt), pt.shape[1], page_size, _p(sel), sel.shape[1],
                                    float(scale), _p(out), _p(lse))
    _check(rc, "sparse_attn_fp8kv")
    return out, lse
