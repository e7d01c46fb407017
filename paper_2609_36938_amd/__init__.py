"""Python binding of libjanus (gfx950): the sparse-selection hot path of append
prefill for top-k sparse-attention LLMs.

Every function here only marshals arguments to the C ABI declared in
``include/janus.h``; all arithmetic runs in the library's HIP kernels.  Torch
provides device memory and the current stream.  There is no fallback: if the
library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libjanus.so")

JANUS_F32, JANUS_BF16, JANUS_FP8_E4M3 = 0, 1, 2
_DT_NAMES = {"f32": JANUS_F32, "bf16": JANUS_BF16, "fp8": JANUS_FP8_E4M3}


class JanusError(RuntimeError):
    pass


class _Batch(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("total_q", ctypes.c_int32),
        ("max_q", ctypes.c_int32),
        ("max_ctx", ctypes.c_int32),
        ("total_ctx", ctypes.c_int64),
        ("q_start", ctypes.c_void_p),
        ("ctx_start", ctypes.c_void_p),
        ("hist_len", ctypes.c_void_p),
        ("score_start", ctypes.c_void_p),
        ("entry_shift", ctypes.c_int32),
    ]


_lib = None


def lib():
    """The loaded libjanus; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise JanusError(f"{LIB_PATH} is missing: build it with python -m paper_2609_36938_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        BP = ctypes.POINTER(_Batch)
        SZ = ctypes.POINTER(ctypes.c_size_t)
        L.janus_index_scores.argtypes = [BP, P, i32, P, P, i32, P, P, i32, i32, P, P]
        L.janus_topk.argtypes = [BP, P, i32, P, P, SZ, P]
        L.janus_topk_sharded.argtypes = [BP, P, i32, i32, i32, P, P, SZ, P]
        L.janus_page_demand.argtypes = [BP, P, i32, P, i32, i32, P, i32, i32, P, P, P, P, P, SZ, P]
        L.janus_predict_diff.argtypes = [P, P, i32, i32, P, P, P, P]
        L.janus_sparse_attn.argtypes = [BP, P, i32, i32, i32, P, P, i64, i64, P, i32, i32, P, i32, f32, P, i32,
                                        P, P]
        L.janus_index_scores_mxfp4.argtypes = [BP, P, P, P, P, P, P, i32, i32, P, P]
        L.janus_sparse_attn_split.argtypes = [BP, P, i32, i32, i32, P, P, i64, i64, P, i32, i32, P, i32, f32, P,
                                              i32, P, i32, P, SZ, P]
        L.janus_sparse_attn_fp8kv.argtypes = [BP, P, i32, P, i64, P, i32, i32, P, i32, f32, P, i32, P, i32, P, SZ, P]
        L.janus_sparse_attn_split_noalloc.argtypes = [BP, P, i32, i32, i32, P, P, i64, i64, P, i32, i32, P, i32, f32,
                                                      P, i32, P, i32, P]
        for f in ("janus_index_scores", "janus_topk", "janus_topk_sharded", "janus_page_demand",
                  "janus_predict_diff", "janus_sparse_attn", "janus_sparse_attn_split", "janus_index_scores_mxfp4",
                  "janus_sparse_attn_fp8kv", "janus_sparse_attn_split_noalloc"):
            getattr(L, f).restype = ctypes.c_int
        L.janus_status_string.argtypes = [ctypes.c_int]
        L.janus_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        msg = lib().janus_status_string(rc).decode()
        raise JanusError(f"{what}: {msg} (status {rc})")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise JanusError("device tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t: torch.Tensor, dt: Optional[str]) -> int:
    if dt is not None:
        return _DT_NAMES[dt]
    if t.dtype in (torch.float8_e4m3fn, torch.uint8):
        return JANUS_FP8_E4M3
    if t.dtype in (torch.bfloat16, torch.int16):
        return JANUS_BF16
    if t.dtype == torch.float32:
        return JANUS_F32
    raise JanusError(f"unsupported dtype {t.dtype}")


def _table(batch: "Batch", page_table, page_size: int) -> int:
    """pt_ld of a [B, pt_ld] page table, which must cover the longest session."""
    pt_ld = int(page_table.shape[1])
    if pt_ld * int(page_size) < batch.max_ctx:
        raise JanusError(f"page table covers {pt_ld} x {page_size} ids, the longest session has {batch.max_ctx}")
    return pt_ld


class Batch:
    """A ragged batch of sessions: history lengths M_b and appended lengths N_b
    (tokens).  entry_shift = e > 0 selects entry granularity: candidates are
    entries of 2^e tokens, and session b holds (M_b + N_b) >> e of them."""

    def __init__(self, hist_len: Sequence[int], new_len: Sequence[int], device="cuda", entry_shift: int = 0):
        hl = np.asarray(hist_len, dtype=np.int64).reshape(-1)
        nl = np.asarray(new_len, dtype=np.int64).reshape(-1)
        if hl.shape != nl.shape or hl.size < 1:
            raise JanusError("hist_len and new_len must be equal-length, non-empty")
        self.entry_shift = int(entry_shift)
        ctx = (hl + nl) >> self.entry_shift
        self.hist_len_host = hl.astype(np.int32)
        self.new_len_host = nl.astype(np.int32)
        self.q_start_host = np.concatenate([[0], np.cumsum(nl)]).astype(np.int32)
        self.ctx_start_host = np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32)
        self.score_start_host = np.concatenate([[0], np.cumsum(nl * ctx)]).astype(np.int64)
        self.q_start = torch.from_numpy(self.q_start_host).to(device)
        self.ctx_start = torch.from_numpy(self.ctx_start_host).to(device)
        self.hist_len = torch.from_numpy(self.hist_len_host).to(device)
        self.score_start = torch.from_numpy(self.score_start_host).to(device)
        self.total_q = int(nl.sum())
        self.total_ctx = int(ctx.sum())
        self.max_ctx = int(ctx.max())
        self.total_scores = int(self.score_start_host[-1])
        self.c = _Batch(len(hl), self.total_q, int(nl.max()), self.max_ctx, self.total_ctx,
                        self.q_start.data_ptr(), self.ctx_start.data_ptr(), self.hist_len.data_ptr(),
                        self.score_start.data_ptr(), self.entry_shift)

    @property
    def ref(self):
        return ctypes.byref(self.c)


def index_scores(batch: Batch, q, kI, w, q_scale=None, k_scale=None, scores=None, dtype=None, stream=None):
    """janus_index_scores: returns the flat fp32 score buffer (batch.total_scores)."""
    H, d = int(q.shape[-2]), int(q.shape[-1])
    if scores is None:
        scores = torch.empty(batch.total_scores, dtype=torch.float32, device=q.device)
    qd, kd = _dtype_code(q, dtype), _dtype_code(kI, dtype)
    rc = lib().janus_index_scores(batch.ref, _ptr(q), qd, _ptr(q_scale), _ptr(kI), kd, _ptr(k_scale), _ptr(w), H, d,
                                  _ptr(scores), _stream(stream))
    _check(rc, "janus_index_scores")
    return scores


def index_scores_mxfp4(batch: Batch, q, kI, k_block_scale, w, q_scale=None, k_scale=None, scores=None, stream=None):
    """janus_index_scores_mxfp4: q fp8 bytes [total_q, H, d]; kI MXFP4 bytes
    [total_ctx, d/2] with E8M0 block scales [total_ctx, d/32]; returns the flat
    fp32 score buffer laid out as for index_scores."""
    H, d = int(q.shape[1]), int(q.shape[2])
    if scores is None:
        scores = torch.empty(batch.total_scores, dtype=torch.float32, device=q.device)
    rc = lib().janus_index_scores_mxfp4(batch.ref, _ptr(q), _ptr(q_scale), _ptr(kI), _ptr(k_block_scale),
                                        _ptr(k_scale), _ptr(w), H, d, _ptr(scores), _stream(stream))
    _check(rc, "janus_index_scores_mxfp4")
    return scores


def topk(batch: Batch, scores, k: int, out=None, stream=None):
    """janus_topk: [total_q, k] int32 ids, ascending, -1 padded."""
    if out is None:
        out = torch.empty((batch.total_q, k), dtype=torch.int32, device=scores.device)
    ws = ctypes.c_size_t(0)
    rc = lib().janus_topk(batch.ref, _ptr(scores), int(k), _ptr(out), None, ctypes.byref(ws), _stream(stream))
    _check(rc, "janus_topk")
    return out


def topk_sharded(batch: Batch, scores, k: int, num_shards: int, align: int, out=None, stream=None):
    """janus_topk_sharded: [total_q, k] int32; slots n*(k/num_shards) .. hold
    shard n's history ids, ascending, -1 padded."""
    if out is None:
        out = torch.empty((batch.total_q, k), dtype=torch.int32, device=scores.device)
    ws = ctypes.c_size_t(0)
    rc = lib().janus_topk_sharded(batch.ref, _ptr(scores), int(k), int(num_shards), int(align), _ptr(out), None,
                                  ctypes.byref(ws), _stream(stream))
    _check(rc, "janus_topk_sharded")
    return out


def page_demand(batch: Batch, topk_idx, page_table, page_size: int, num_phys_pages: int, max_run: int,
                limit=None, out=None, stream=None):
    """janus_page_demand: (bitmap, page_list, runs, counts) device tensors.

    page_list and runs are sized to the pool; counts = [num_pages, num_runs]."""
    dev = topk_idx.device
    nw = max(1, (num_phys_pages + 31) // 32)
    if out is None:
        out = (torch.empty(nw, dtype=torch.int32, device=dev),
               torch.empty(max(1, num_phys_pages), dtype=torch.int32, device=dev),
               torch.empty(max(1, 2 * num_phys_pages), dtype=torch.int32, device=dev),
               torch.empty(2, dtype=torch.int32, device=dev))
    bm, lst, runs, counts = out
    ws = ctypes.c_size_t(0)
    rc = lib().janus_page_demand(batch.ref, _ptr(topk_idx), int(topk_idx.shape[1]), _ptr(page_table),
                                 _table(batch, page_table, page_size), int(page_size), _ptr(limit), int(num_phys_pages),
                                 int(max_run), _ptr(bm), _ptr(lst), _ptr(runs), _ptr(counts), None,
                                 ctypes.byref(ws), _stream(stream))
    _check(rc, "janus_page_demand")
    return out


def predict_diff(actual, predicted, num_phys_pages: int, max_run: int, out=None, stream=None):
    """janus_predict_diff: (miss bitmap, miss runs, counts[5])."""
    dev = actual.device
    nw = max(1, (num_phys_pages + 31) // 32)
    if out is None:
        out = (torch.empty(nw, dtype=torch.int32, device=dev),
               torch.empty(max(1, 2 * num_phys_pages), dtype=torch.int32, device=dev),
               torch.empty(5, dtype=torch.int32, device=dev))
    miss, runs, counts = out
    rc = lib().janus_predict_diff(_ptr(actual), _ptr(predicted), int(num_phys_pages), int(max_run), _ptr(miss),
                                  _ptr(runs), _ptr(counts), _stream(stream))
    _check(rc, "janus_predict_diff")
    return out


def sparse_attn(batch: Batch, q, k_pool, v_pool, page_table, page_size: int, topk_idx, scale: float,
                k_row_stride: Optional[int] = None, v_row_stride: Optional[int] = None, dv: Optional[int] = None,
                out_dtype: str = "bf16", want_lse: bool = False, out=None, lse=None, stream=None):
    """janus_sparse_attn: returns (out [total_q, Hq, dv], lse or None).

    q is [total_q, Hq, dqk] bf16; pools are bf16 rows (k_row_stride / v_row_stride
    elements each; default: the pool's last dimension).  Pass v_pool = k_pool for
    the latent-KV layout, where V is the first dv elements of each row."""
    Hq, dqk = int(q.shape[-2]), int(q.shape[-1])
    krs = int(k_row_stride if k_row_stride is not None else k_pool.shape[-1])
    vrs = int(v_row_stride if v_row_stride is not None else v_pool.shape[-1])
    dv = int(dv if dv is not None else (v_pool.shape[-1] if v_pool is not k_pool else dqk))
    odt = {"bf16": (JANUS_BF16, torch.bfloat16), "f32": (JANUS_F32, torch.float32)}[out_dtype]
    if out is None:
        out = torch.empty((batch.total_q, Hq, dv), dtype=odt[1], device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((batch.total_q, Hq), dtype=torch.float32, device=q.device)
    rc = lib().janus_sparse_attn(batch.ref, _ptr(q), Hq, dqk, dv, _ptr(k_pool), _ptr(v_pool), krs, vrs,
                                 _ptr(page_table), _table(batch, page_table, page_size), int(page_size), _ptr(topk_idx),
                                 int(topk_idx.shape[1]), float(scale), _ptr(out), odt[0], _ptr(lse),
                                 _stream(stream))
    _check(rc, "janus_sparse_attn")
    return out, lse


def sparse_attn_split(batch: Batch, q, k_pool, v_pool, page_table, page_size: int, topk_idx, scale: float,
                      num_splits: int = 0, k_row_stride: Optional[int] = None, v_row_stride: Optional[int] = None,
                      dv: Optional[int] = None, out_dtype: str = "bf16", want_lse: bool = False, out=None,
                      lse=None, workspace=None, stream=None):
    """janus_sparse_attn_split: as sparse_attn, each row's selection split
    over num_splits blocks (0: the library picks); returns (out, lse or None).
    workspace: a device uint8 tensor of at least the byte count the library
    reports for these arguments (its NULL-workspace size query, made here
    first), or None to allocate one here."""
    Hq, dqk = int(q.shape[-2]), int(q.shape[-1])
    krs = int(k_row_stride if k_row_stride is not None else k_pool.shape[-1])
    vrs = int(v_row_stride if v_row_stride is not None else v_pool.shape[-1])
    dv = int(dv if dv is not None else (v_pool.shape[-1] if v_pool is not k_pool else dqk))
    odt = {"bf16": (JANUS_BF16, torch.bfloat16), "f32": (JANUS_F32, torch.float32)}[out_dtype]
    if out is None:
        out = torch.empty((batch.total_q, Hq, dv), dtype=odt[1], device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((batch.total_q, Hq), dtype=torch.float32, device=q.device)
    args = (batch.ref, _ptr(q), Hq, dqk, dv, _ptr(k_pool), _ptr(v_pool), krs, vrs, _ptr(page_table),
            _table(batch, page_table, page_size), int(page_size), _ptr(topk_idx), int(topk_idx.shape[1]),
            float(scale), _ptr(out), odt[0], _ptr(lse), int(num_splits))
    need = ctypes.c_size_t(0)
    _check(lib().janus_sparse_attn_split(*args, None, ctypes.byref(need), _stream(stream)), "janus_sparse_attn_split")
    if workspace is None:
        workspace = torch.empty(max(int(need.value), 1), dtype=torch.uint8, device=q.device)
    have = ctypes.c_size_t(workspace.numel() * workspace.element_size())
    rc = lib().janus_sparse_attn_split(*args, _ptr(workspace), ctypes.byref(have), _stream(stream))
    _check(rc, "janus_sparse_attn_split")
    return out, lse


def sparse_attn_split_noalloc(batch: Batch, q, k_pool, v_pool, page_table, page_size: int, topk_idx, scale: float,
                              num_splits: int = 0, k_row_stride: Optional[int] = None,
                              v_row_stride: Optional[int] = None, dv: Optional[int] = None, out_dtype: str = "bf16",
                              want_lse: bool = False, out=None, lse=None, stream=None):
    """janus_sparse_attn_split_noalloc: as sparse_attn_split, with the slices'
    partial results in the library's own per-GPU scratch array instead of a
    workspace (pass out, and lse if wanted, to allocate nothing here either);
    returns (out, lse or None)."""
    Hq, dqk = int(q.shape[-2]), int(q.shape[-1])
    krs = int(k_row_stride if k_row_stride is not None else k_pool.shape[-1])
    vrs = int(v_row_stride if v_row_stride is not None else v_pool.shape[-1])
    dv = int(dv if dv is not None else (v_pool.shape[-1] if v_pool is not k_pool else dqk))
    odt = {"bf16": (JANUS_BF16, torch.bfloat16), "f32": (JANUS_F32, torch.float32)}[out_dtype]
    if out is None:
        out = torch.empty((batch.total_q, Hq, dv), dtype=odt[1], device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((batch.total_q, Hq), dtype=torch.float32, device=q.device)
    rc = lib().janus_sparse_attn_split_noalloc(batch.ref, _ptr(q), Hq, dqk, dv, _ptr(k_pool), _ptr(v_pool), krs, vrs,
                                               _ptr(page_table), _table(batch, page_table, page_size),
                                               int(page_size), _ptr(topk_idx), int(topk_idx.shape[1]), float(scale),
                                               _ptr(out), odt[0], _ptr(lse), int(num_splits), _stream(stream))
    _check(rc, "janus_sparse_attn_split_noalloc")
    return out, lse


def sparse_attn_fp8kv(batch: Batch, q, kv_pool, page_table, page_size: int, topk_idx, scale: float,
                      num_splits: int = 1, out_dtype: str = "bf16", want_lse: bool = False, out=None, lse=None,
                      workspace=None, stream=None):
    """janus_sparse_attn_fp8kv: MLA attention (576/512) over fp8 KV rows
    (uint8 [..., row_bytes]: 576 e4m3 bytes, the fp32 scale at byte 576);
    num_splits as for sparse_attn_split (1: unsplit).  Returns (out, lse or None)."""
    Hq = int(q.shape[-2])
    row_bytes = int(kv_pool.shape[-1])
    odt = {"bf16": (JANUS_BF16, torch.bfloat16), "f32": (JANUS_F32, torch.float32)}[out_dtype]
    if out is None:
        out = torch.empty((batch.total_q, Hq, 512), dtype=odt[1], device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((batch.total_q, Hq), dtype=torch.float32, device=q.device)
    args = (batch.ref, _ptr(q), Hq, _ptr(kv_pool), row_bytes, _ptr(page_table),
            _table(batch, page_table, page_size), int(page_size), _ptr(topk_idx), int(topk_idx.shape[1]),
            float(scale), _ptr(out), odt[0], _ptr(lse), int(num_splits))
    need = ctypes.c_size_t(0)
    _check(lib().janus_sparse_attn_fp8kv(*args, None, ctypes.byref(need), _stream(stream)), "janus_sparse_attn_fp8kv")
    if workspace is None:
        workspace = torch.empty(max(int(need.value), 1), dtype=torch.uint8, device=q.device)
    have = ctypes.c_size_t(workspace.numel() * workspace.element_size())
    rc = lib().janus_sparse_attn_fp8kv(*args, _ptr(workspace), ctypes.byref(have), _stream(stream))
    _check(rc, "janus_sparse_attn_fp8kv")
    return out, lse
