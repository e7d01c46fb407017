"""The five evaluation workloads at full size, in the launch configuration the
benchmark uses, checked on sampled rows against the CPU oracle.

Workloads (seed = workload number): tiny fp32 layer (M=4096, N=256); a
DeepSeek-V3.2-shaped layer at M=32K/N=2K and at M=128K/N=8K behind a random
page table; a ragged batch of 16 sessions; and the 8-layer prediction path
(M=128K, N=4K, predicted queries 0.9 q + sqrt(0.19) noise).

What is compared with the oracle:
  * indexer scores on sampled rows (row-relative error <= 1e-2 for fp8,
    <= 1e-5 for fp32), -inf pattern exact;
  * top-k on GPU scores: band check against the oracle's scores of the row;
  * page demand / runs / predict-diff: bit-exact, both sides fed the same
    generator-made selections (never the GPU's own ids);
  * attention on sampled rows fed generator-made selections: max abs error
    <= 2e-2 and <= 2e-2 of the row's largest output.
The GPU's own top-k is further checked by properties that hold at any size:
ids ascending, distinct, causal, exactly min(k, candidates) of them, and the
page set equal to the union of their pages.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, attention_q_rows, config, synth_topk

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _sample_rows(wl, n):
    rows = set()
    for b in range(wl.num_seqs):
        lo, hi = int(wl.q_start[b]), int(wl.q_start[b + 1])
        rows.update({lo, hi - 1})
    rows.update(np.linspace(0, wl.total_q - 1, n).astype(int).tolist())
    return np.array(sorted(rows), dtype=np.int32)


def _row_scores(flat, wl, rows):
    out = np.full((len(rows), wl.max_ctx), -np.inf, dtype=np.float32)
    b_of = wl.row_session(rows)
    for j, (g, b) in enumerate(zip(rows, b_of)):
        ctx = int(wl.ctx_len[b])
        i = int(g) - int(wl.q_start[b])
        st = int(wl.score_start[b]) + i * ctx
        out[j, :ctx] = flat[st: st + ctx].cpu().numpy()
    return out


def _check_selection_properties(wl, sel, bm, cnt, limit=None):
    bm = bm.cpu().numpy().view(np.uint32)
    pages = set()
    for b in range(wl.num_seqs):
        M = int(wl.hist_len[b])
        lim = M if limit is None else int(limit[b])
        for g in range(int(wl.q_start[b]), int(wl.q_start[b + 1])):
            n = M + (g - int(wl.q_start[b])) + 1
            want = min(wl.k, n)
            row = sel[g]
            assert np.all(row[want:] == -1) and np.all(row[:want] >= 0) and row[want - 1] < n
            assert np.all(np.diff(row[:want]) > 0)
            h = row[:want][row[:want] < lim]
            pages.update(wl.page_table[b, np.unique(h // wl.page_size)].tolist())
    got = set(np.flatnonzero(np.unpackbits(bm.view(np.uint8), bitorder="little")).tolist())
    assert got == pages and int(cnt[0]) == len(pages)


def _scores_topk(wl, bt, rows, tol, q=None, q_scale=None):
    q = wl.q if q is None else q
    q_scale = wl.q_scale if q_scale is None else q_scale
    sc = janus.index_scores(bt, T(q), T(wl.kI), T(wl.w), q_scale=None if q_scale is None else T(q_scale),
                            k_scale=None if wl.k_scale is None else T(wl.k_scale), dtype=wl.idx_dtype)
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    got = _row_scores(sc, wl, rows)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, q, wl.idx_dtype, q_scale, wl.kI, wl.idx_dtype,
                              wl.k_scale, wl.w, rows, out_ld=wl.max_ctx)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got))
    diff = np.zeros(ref.shape)
    diff[fin] = np.abs(got[fin].astype(np.float64) - ref[fin])  # masked cells are -inf on both sides
    err = diff.max(axis=1)
    rel = err / np.where(fin, np.abs(ref), 0.0).max(axis=1)
    assert rel.max() <= tol, rel.max()
    gsel = sel.cpu().numpy()
    for j, g in enumerate(rows):
        b = int(wl.row_session([g])[0])
        n = int(wl.hist_len[b]) + (int(g) - int(wl.q_start[b])) + 1
        r = ref[j, :n]
        tau = tol * np.abs(r).max()
        kk = min(wl.k, n)
        theta = np.partition(r, n - kk)[n - kk]
        chosen = np.zeros(n, bool)
        chosen[gsel[g][gsel[g] >= 0]] = True
        assert chosen.sum() == kk
        assert np.all(chosen[r > theta + tau]) and not np.any(chosen[r < theta - tau])
    return sc, sel, gsel


def _attn_parity(wl, bt, rows, seed=11):
    ai = attention_inputs(wl, with_q=False)
    sel = np.sort(synth_topk(wl, seed=seed, hot_frac=0.8), axis=1)
    sel = np.where(sel < 0, np.iinfo(np.int32).max, sel)
    sel = np.sort(sel, axis=1)
    sel = np.where(sel == np.iinfo(np.int32).max, -1, sel).astype(np.int32)
    # only the sampled rows carry their real queries; the others are zero
    # (valid inputs whose outputs are not compared)
    q_all = np.zeros((wl.total_q, ai.Hq, ai.dqk), dtype=np.uint16)
    q_all[rows] = attention_q_rows(wl, rows)
    kv = T(ai.k_pool)
    vp = kv if ai.v_pool is None else T(ai.v_pool)
    out, lse = janus.sparse_attn(bt, T(q_all), kv, vp, T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                 dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    ref, lref = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                   ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, sel[rows],
                                   ai.scale, ai.dv)
    got = out[torch.from_numpy(rows.astype(np.int64)).cuda()].cpu().numpy()
    err = np.abs(got - ref).max()
    assert err <= 2e-2 and err <= 2e-2 * np.abs(ref).max(), err
    assert np.allclose(lse[torch.from_numpy(rows.astype(np.int64)).cuda()].cpu().numpy(), lref, atol=2e-3)


def _demand_parity(wl, bt, seed=5, limit=None):
    sel = synth_topk(wl, seed=seed, pad_rows=2)
    lim_t = None if limit is None else T(np.asarray(limit, np.int32))
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), wl.page_size, wl.num_phys_pages,
                                           wl.max_run, limit=lim_t)
    torch.cuda.synchronize()
    rbm, rlst, rc = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, wl.page_size,
                                       wl.num_phys_pages, limit=limit)
    rr = oracle.runs(rbm, wl.num_phys_pages, wl.max_run)
    c = cnt.cpu().numpy()
    assert c[0] == rc and c[1] == rr.shape[0]
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm)
    assert np.array_equal(lst.cpu().numpy()[:rc], rlst)
    assert np.array_equal(runs.cpu().numpy()[: 2 * c[1]].reshape(-1, 2), rr)
    return rbm


@pytest.mark.parametrize("ci", [0, 1])
def test_workload_small_and_medium(ci):
    wl = config(ci)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    rows = _sample_rows(wl, 6)
    tol = 1e-5 if wl.idx_dtype == "f32" else 1e-2
    _, sel_t, gsel = _scores_topk(wl, bt, rows, tol)
    bm, lst, runs, cnt = janus.page_demand(bt, sel_t, T(wl.page_table), wl.page_size, wl.num_phys_pages,
                                           wl.max_run)
    torch.cuda.synchronize()
    _check_selection_properties(wl, gsel, bm, cnt.cpu().numpy())
    _demand_parity(wl, bt)
    _attn_parity(wl, bt, rows[:4])


def test_workload_128k_permuted():
    wl = config(2)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    rows = _sample_rows(wl, 4)
    _, sel_t, gsel = _scores_topk(wl, bt, rows, 1e-2)
    bm, lst, runs, cnt = janus.page_demand(bt, sel_t, T(wl.page_table), wl.page_size, wl.num_phys_pages,
                                           wl.max_run)
    torch.cuda.synchronize()
    _check_selection_properties(wl, gsel, bm, cnt.cpu().numpy())
    _demand_parity(wl, bt)
    _attn_parity(wl, bt, rows[:3])


def test_workload_ragged_batch():
    wl = config(3)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    rows = _sample_rows(wl, 4)[::3]
    _, sel_t, gsel = _scores_topk(wl, bt, rows, 1e-2)
    bm, lst, runs, cnt = janus.page_demand(bt, sel_t, T(wl.page_table), wl.page_size, wl.num_phys_pages,
                                           wl.max_run)
    torch.cuda.synchronize()
    _check_selection_properties(wl, gsel, bm, cnt.cpu().numpy())
    _demand_parity(wl, bt)
    _demand_parity(wl, bt, seed=6, limit=wl.ctx_len)
    _attn_parity(wl, bt, rows[:4])


@pytest.mark.parametrize("layer", [0, 5])
def test_workload_prediction_layers(layer):
    wl = config(4, layer=layer)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    rows = _sample_rows(wl, 3)
    _, sel_a, gsel = _scores_topk(wl, bt, rows, 1e-2)
    _, sel_p, _ = _scores_topk(wl, bt, rows, 1e-2, q=wl.q_pred, q_scale=wl.q_pred_scale)
    pt = T(wl.page_table)
    bma, _, _, cnta = janus.page_demand(bt, sel_a, pt, wl.page_size, wl.num_phys_pages, wl.max_run)
    bmp, _, _, _ = janus.page_demand(bt, sel_p, pt, wl.page_size, wl.num_phys_pages, wl.max_run)
    miss, mruns, mcnt = janus.predict_diff(bma, bmp, wl.num_phys_pages, wl.max_run)
    torch.cuda.synchronize()
    _check_selection_properties(wl, gsel, bma, cnta.cpu().numpy())
    a = bma.cpu().numpy().view(np.uint32)
    p = bmp.cpu().numpy().view(np.uint32)
    pc = lambda x: int(np.unpackbits(x.view(np.uint8)).sum())
    c = mcnt.cpu().numpy()
    assert c.tolist()[:4] == [pc(a), pc(p), pc(a & p), pc(a & ~p)]
    assert np.array_equal(miss.cpu().numpy().view(np.uint32), a & ~p)
    # predict-diff parity on generator-made page sets of this workload
    ra = _demand_parity(wl, bt, seed=7)
    rp = _demand_parity(wl, bt, seed=8)
    gm, gr, gc = janus.predict_diff(T(ra.view(np.int32)), T(rp.view(np.int32)), wl.num_phys_pages, wl.max_run)
    torch.cuda.synchronize()
    om, orr, oc = oracle.predict_diff(ra, rp, wl.num_phys_pages, wl.max_run)
    assert np.array_equal(gc.cpu().numpy(), oc) and np.array_equal(gm.cpu().numpy().view(np.uint32), om)
    assert np.array_equal(gr.cpu().numpy()[: 2 * oc[4]].reshape(-1, 2), orr)
