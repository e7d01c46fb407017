"""The fp8 indexer's row-tile kernel for sessions that append two to four
tokens (Eq. 1; the decode phase of Sec. 2.2 batches sessions that append a
few tokens each).  A batch whose sessions append at most two tokens runs the
two-token tile, at most four the four-token tile; these tests build ragged
batches of exactly those shapes at token granularity, with histories that
span several key chunks with ragged tails, an empty history and a history
shorter than one 64-key group.

Compared with the oracle on every row: the causal -inf pattern exactly, and
max |gpu - oracle| / max |oracle| <= 1e-2 over the row's candidates; the
GPU's top-k on those scores by the band check (every candidate more than
1e-2 of the row maximum above the oracle's k-th score is selected, none that
far below it), with exactly min(k, candidates) ids, ascending.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import make_workload

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


CASES = {
    # max appended tokens 2 -> the two-token tile
    "two": ([5000, 1200, 0, 77, 9000, 4097], [2, 1, 2, 2, 1, 2]),
    # max 3 -> the four-token tile with a partly empty tile
    "three": ([6100, 33, 2500, 0], [3, 1, 2, 3]),
    # max 4 -> the four-token tile, full and partial tiles mixed
    "four": ([8191, 4096, 1, 3000, 700], [4, 1, 3, 4, 2]),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("k", [256, 2048])
def test_rows_tile_scores_and_topk(case, k):
    hist, new = CASES[case]
    wl = make_workload(hist_len=hist, new_len=new, H=64, d=128, idx_dtype="fp8", k=k, seed=17, w_scale=0.125,
                       table="permuted")
    assert wl.max_q == max(new) and wl.max_q <= 4
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(wl.k_scale))
    sel = janus.topk(bt, sc, k)
    torch.cuda.synchronize()
    print(f"rows tile case {case} k={k}: {wl.total_q} rows", flush=True)
    rows = np.arange(wl.total_q, dtype=np.int32)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, "fp8", wl.k_scale, wl.w,
                              rows, out_ld=wl.max_ctx)
    flat = sc.cpu().numpy()
    gs = sel.cpu().numpy()
    for b in range(wl.num_seqs):
        ctx = int(wl.ctx_len[b])
        for i in range(int(wl.new_len[b])):
            g = int(wl.q_start[b]) + i
            got = flat[wl.score_start[b] + i * ctx: wl.score_start[b] + (i + 1) * ctx].astype(np.float64)
            r = ref[g, :ctx]
            n = int(wl.hist_len[b]) + i + 1  # candidates 0 .. M+i
            assert np.all(np.isneginf(got[n:])) and np.all(np.isneginf(r[n:])), f"row {g}: causal pattern"
            assert np.all(np.isfinite(got[:n])), f"row {g}: a candidate is not finite"
            err = np.abs(got[:n] - r[:n]).max()
            top = np.abs(r[:n]).max()
            assert err <= 1e-2 * top, f"row {g} ({case}): rel err {err / top:.3e}"
            ids = gs[g]
            want = min(k, n)
            assert np.all(ids[want:] == -1) and np.all(ids[:want] >= 0) and np.all(ids[:want] < n)
            assert np.all(np.diff(ids[:want]) > 0)
            if n <= k:
                continue  # every candidate selected
            theta = np.partition(r[:n], n - k)[n - k]
            tau = 1e-2 * top
            chosen = np.zeros(n, bool)
            chosen[ids[:want]] = True
            assert np.all(chosen[r[:n] > theta + tau]), f"row {g}: a clear winner was dropped"
            assert not np.any(chosen[r[:n] < theta - tau]), f"row {g}: a clear loser was selected"
