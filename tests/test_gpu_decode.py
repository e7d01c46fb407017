"""The decode phase (Sec. 2.2): each step is an append prefill with one
appended token per session, many sessions batched.  The KV to load before
attention is the selection's page set minus the pages already resident in
HBM, which is janus_predict_diff with the resident bitmap in the predicted
slot.  Attention with few rows runs split (janus_sparse_attn_split).

Workload: 16 sessions with histories log-uniform in 8K-48K, one new token
each, DeepSeek-V3.2-shaped indexer and MLA attention, k = 2048, a random page
table.  Compared with the oracle: scores on every row (row-relative 1e-2),
top-k by the band check, page demand and the load set bit-exact on
generator-made selections and resident bitmaps, attention on every row for
several slice counts (2e-2, absolute and relative to the row's largest
output)."""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, attention_q_rows, config, resident_pages, synth_topk

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(scope="module")
def wl():
    return config(5)


@pytest.fixture(scope="module")
def ai(wl):
    return attention_inputs(wl)


def test_decode_scores_and_topk(wl):
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(wl.k_scale))
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    rows = np.arange(wl.total_q, dtype=np.int32)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, "fp8", wl.k_scale, wl.w,
                              rows, out_ld=wl.max_ctx)
    flat = sc.cpu().numpy()
    gs = sel.cpu().numpy()
    for b in range(wl.num_seqs):
        n = int(wl.ctx_len[b])  # the single row sees the whole context
        got = flat[wl.score_start[b]: wl.score_start[b] + n].astype(np.float64)
        r = ref[b, :n]
        assert np.all(np.isfinite(got))
        assert np.abs(got - r).max() <= 1e-2 * np.abs(r).max()
        theta = np.partition(r, n - wl.k)[n - wl.k]
        tau = 1e-2 * np.abs(r).max()
        chosen = np.zeros(n, bool)
        chosen[gs[b][gs[b] >= 0]] = True
        assert chosen.sum() == wl.k and np.all(np.diff(gs[b]) > 0)
        assert np.all(chosen[r > theta + tau]) and not np.any(chosen[r < theta - tau])


@pytest.mark.parametrize("p", [0.0, 0.9, 1.0])
def test_decode_load_set_is_demand_minus_resident(wl, p):
    """Pages to load = demand & ~resident, with the counts and packed runs."""
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sel = synth_topk(wl, seed=3, hot_frac=0.7)
    res = resident_pages(wl, p=p, seed=1)
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), wl.page_size, wl.num_phys_pages, wl.max_run)
    load, lruns, lc = janus.predict_diff(bm, T(res.view(np.int32)), wl.num_phys_pages, wl.max_run)
    torch.cuda.synchronize()
    rbm, _, rc = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, wl.page_size, wl.num_phys_pages)
    om, orr, oc = oracle.predict_diff(rbm, res, wl.num_phys_pages, wl.max_run)
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm)
    assert np.array_equal(load.cpu().numpy().view(np.uint32), om)
    assert np.array_equal(lc.cpu().numpy(), oc)
    assert np.array_equal(lruns.cpu().numpy()[: 2 * oc[4]].reshape(-1, 2), orr)
    if p == 1.0:
        assert oc[3] == 0  # everything resident: nothing to load
    if p == 0.0:
        assert oc[3] == oc[0] == rc  # nothing resident: load the whole demand


def _attn_ref(wl, ai, sel):
    rows = np.arange(wl.total_q, dtype=np.int32)
    return oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                              ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, sel, ai.scale, ai.dv)


@pytest.fixture(scope="module")
def attn_case(wl, ai):
    sel = synth_topk(wl, seed=11, hot_frac=0.8)
    return sel, _attn_ref(wl, ai, sel)


@pytest.mark.parametrize("splits", [1, 2, 5, 16, 0])
def test_decode_split_attention(wl, ai, attn_case, splits):
    sel, (ref, lref) = attn_case
    bt = janus.Batch(wl.hist_len, wl.new_len)
    kv = T(ai.k_pool)
    out, lse = janus.sparse_attn_split(bt, T(ai.q), kv, kv, T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                       num_splits=splits, dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for r in range(wl.total_q):
        err = np.abs(got[r] - ref[r]).max()
        assert err <= 2e-2 and err <= 2e-2 * np.abs(ref[r]).max(), (splits, r, err)
    assert np.allclose(lse.cpu().numpy(), lref, atol=2e-3)


def test_split_matches_unsplit(wl, ai, attn_case):
    """Splitting changes only the order of the sums (and which max each bf16
    probability is rounded against)."""
    sel, _ = attn_case
    bt = janus.Batch(wl.hist_len, wl.new_len)
    kv, pt, s = T(ai.k_pool), T(wl.page_table), T(sel)
    a, la = janus.sparse_attn(bt, T(ai.q), kv, kv, pt, wl.page_size, s, ai.scale, dv=ai.dv, out_dtype="f32",
                              want_lse=True)
    b_, lb = janus.sparse_attn_split(bt, T(ai.q), kv, kv, pt, wl.page_size, s, ai.scale, num_splits=8, dv=ai.dv,
                                     out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    a, b_ = a.cpu().numpy(), b_.cpu().numpy()
    assert np.abs(a - b_).max() <= 1e-2 * np.abs(a).max()
    assert np.allclose(la.cpu().numpy(), lb.cpu().numpy(), atol=1e-3)


def test_split_with_empty_slices(wl, ai):
    """Rows whose valid ids sit in the first slice only: the other slices see
    padding only (their weight in the merge is zero); one row has no valid id
    at all (out = 0, lse = -inf)."""
    rng = np.random.default_rng(4)
    sel = np.full((wl.total_q, wl.k), -1, np.int32)
    for b in range(wl.num_seqs):
        n = int(wl.ctx_len[b])
        sel[b, :40] = rng.choice(n, 40, replace=False)
    sel[3, :] = -1
    sel[5, 100] = int(wl.ctx_len[5]) + 9  # out of range: padding
    ref, lref = _attn_ref(wl, ai, sel)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    kv = T(ai.k_pool)
    out, lse = janus.sparse_attn_split(bt, T(ai.q), kv, kv, T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                       num_splits=16, dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    got, gl = out.cpu().numpy(), lse.cpu().numpy()
    assert np.all(got[3] == 0) and np.all(np.isneginf(gl[3]))
    keep = np.arange(wl.total_q) != 3
    assert np.abs(got[keep] - ref[keep]).max() <= 2e-2 * np.abs(ref[keep]).max()
    assert np.allclose(gl[keep], lref[keep], atol=2e-3)


def test_split_attention_at_prefill_size():
    """The split entry point on a prefill-sized batch (sampled rows of the 32K
    workload) agrees with the oracle too."""
    wl = config(1)
    ai = attention_inputs(wl, with_q=False)
    rows = np.array([0, 777, wl.total_q - 1], dtype=np.int32)
    sel = np.sort(synth_topk(wl, seed=2, hot_frac=0.8), axis=1)
    q_all = np.zeros((wl.total_q, ai.Hq, ai.dqk), dtype=np.uint16)
    q_all[rows] = attention_q_rows(wl, rows)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    kv = T(ai.k_pool)
    out, _ = janus.sparse_attn_split(bt, T(q_all), kv, kv, T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                     num_splits=3, dv=ai.dv, out_dtype="f32")
    torch.cuda.synchronize()
    ref, _ = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, sel[rows], ai.scale,
                                ai.dv)
    got = out[torch.from_numpy(rows.astype(np.int64)).cuda()].cpu().numpy()
    err = np.abs(got - ref).max()
    assert err <= 2e-2 and err <= 2e-2 * np.abs(ref).max(), err
