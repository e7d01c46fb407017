"""Indexer scores (Eq. 1) with bf16 queries and keys on the bf16 MFMA kernel
(64 heads x 128 dims), against the oracle.

Cases: a ragged batch with an empty history and a history shorter than one
64-key group (every row), the same batch with per-token query and key scales
far from 1, a batch at entry granularity (E = 16), and the 32K-history +
2K-append layer shape in bf16 on sampled rows (each session's first and last
row included).  Compared: the causal -inf pattern exactly and, per row,
max |gpu - oracle| / max |oracle| <= 1e-3 (the bf16 tolerance); the GPU's
top-k on its own scores by the band check (every candidate more than 1e-3
of the row maximum above the oracle's k-th score selected, none that far
below it), with min(k, candidates) ascending ids.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import make_workload

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")

TOL = 1e-3


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _check(wl, rows, q_scale=None, k_scale=None):
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=wl.entry_shift)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=None if q_scale is None else T(q_scale),
                            k_scale=None if k_scale is None else T(k_scale), dtype="bf16")
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    E = 1 << wl.entry_shift
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "bf16", q_scale, wl.kI, "bf16", k_scale, wl.w, rows,
                              out_ld=wl.max_ctx, entry=E)
    flat = sc.cpu().numpy()
    gs = sel.cpu().numpy()
    b_of = wl.row_session(rows)
    worst = 0.0
    for j, (g, b) in enumerate(zip(rows, b_of)):
        ctx = int(wl.ctx_len[b])
        i = int(g) - int(wl.q_start[b])
        got = flat[wl.score_start[b] + i * ctx: wl.score_start[b] + (i + 1) * ctx].astype(np.float64)
        r = ref[j, :ctx]
        n = (int(wl.hist_len[b]) + i + 1) >> wl.entry_shift  # candidates 0 .. n-1
        assert np.all(np.isneginf(got[n:])) and np.all(np.isneginf(r[n:])), f"row {g}: causal pattern"
        if n == 0:
            assert np.all(gs[g] == -1)
            continue
        assert np.all(np.isfinite(got[:n])), f"row {g}: a candidate is not finite"
        top = np.abs(r[:n]).max()
        err = np.abs(got[:n] - r[:n]).max()
        worst = max(worst, err / top)
        assert err <= TOL * top, f"row {g}: rel err {err / top:.3e}"
        want = min(wl.k, n)
        ids = gs[g]
        assert np.all(ids[want:] == -1) and np.all(ids[:want] >= 0) and np.all(ids[:want] < n)
        assert np.all(np.diff(ids[:want]) > 0)
        if n <= wl.k:
            continue
        theta = np.partition(r[:n], n - wl.k)[n - wl.k]
        chosen = np.zeros(n, bool)
        chosen[ids[:want]] = True
        assert np.all(chosen[r[:n] > theta + TOL * top]), f"row {g}: a clear winner was dropped"
        assert not np.any(chosen[r[:n] < theta - TOL * top]), f"row {g}: a clear loser was selected"
    print(f"bf16 indexer: {len(rows)} rows, worst row-relative error {worst:.2e}", flush=True)


def test_bf16_mfma_ragged_every_row():
    wl = make_workload(hist_len=[4200, 1500, 0, 77, 9000], new_len=[37, 20, 10, 5, 3], H=64, d=128,
                       idx_dtype="bf16", k=512, seed=41, w_scale=0.125)
    _check(wl, np.arange(wl.total_q, dtype=np.int32))


def test_bf16_mfma_with_token_scales():
    wl = make_workload(hist_len=[3000, 260], new_len=[24, 9], H=64, d=128, idx_dtype="bf16", k=256, seed=42,
                       w_scale=0.125)
    rng = np.random.default_rng(3)
    q_scale = np.exp(rng.uniform(-4, 4, wl.total_q)).astype(np.float32)
    k_scale = np.exp(rng.uniform(-4, 4, wl.total_ctx)).astype(np.float32)
    _check(wl, np.arange(wl.total_q, dtype=np.int32), q_scale=q_scale, k_scale=k_scale)


def test_bf16_mfma_entries():
    wl = make_workload(hist_len=[40000, 100], new_len=[40, 30], H=64, d=128, idx_dtype="bf16", k=256, seed=43,
                       w_scale=0.125, entry_shift=4)
    _check(wl, np.arange(wl.total_q, dtype=np.int32))


def test_bf16_mfma_32k_layer_sampled():
    wl = make_workload(hist_len=[32768], new_len=[2048], H=64, d=128, idx_dtype="bf16", k=2048, seed=1,
                       w_scale=0.125)
    rows = np.unique(np.concatenate([[0, wl.total_q - 1], np.linspace(0, wl.total_q - 1, 22).astype(np.int32)]))
    _check(wl, rows.astype(np.int32))
