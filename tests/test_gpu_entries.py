"""Entry granularity on the GPU against the oracle.  DeepSeek-V4 selects
entries (Sec. 2.2 footnote), each one cached row standing for E = 128
consecutive tokens that a token can select once all of them have arrived.

Batches: a ragged prefill-shaped batch (one session with 2048 history entries,
one whose 100-token history holds no whole entry, so its first appended
tokens have no candidate at all) and a decode-shaped batch of 12 sessions
appending 1 to 4 tokens.  Compared: scores row by row (row-relative 1e-2, the
-inf pattern exact) for fp8 and MXFP4 keys on both indexer kernels, top-k by
the band check, page demand and runs bit-exact, MLA attention whole and split
(2e-2)."""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, attention_q_rows, decode_lengths, make_workload, synth_topk
from workloads.gen import MLA_ATTN

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")

SHIFT = 7
E = 1 << SHIFT


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _prefill(key_format=None):
    return make_workload(hist_len=[262144, 70000, 100], new_len=[700, 300, 160], H=64, d=128, idx_dtype="fp8",
                         k=512, seed=21, w_scale=1 / 8, table="permuted", attn=MLA_ATTN, entry_shift=SHIFT,
                         key_format=key_format)


def _decode():
    M = decode_lengths(12, 40000, 300000, seed=4)
    N = np.array([1, 2, 3, 4] * 3, np.int32)
    return make_workload(hist_len=M, new_len=N, H=64, d=128, idx_dtype="fp8", k=512, seed=22, w_scale=1 / 8,
                         table="permuted", attn=MLA_ATTN, entry_shift=SHIFT)


def _rows(wl):
    """Every row of the small sessions, every 5th of the large one, and each
    session's first and last."""
    out = []
    for b in range(wl.num_seqs):
        lo, hi = int(wl.q_start[b]), int(wl.q_start[b + 1])
        step = 5 if hi - lo > 400 else 1
        out += list(range(lo, hi, step)) + [hi - 1]
    return np.unique(np.array(out, np.int32))


def _scores(wl, bt):
    if wl.k_bscale is not None:
        return janus.index_scores_mxfp4(bt, T(wl.q), T(wl.kI), T(wl.k_bscale), T(wl.w), q_scale=T(wl.q_scale))
    return janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(wl.k_scale))


def _ref_scores(wl, rows):
    if wl.k_bscale is not None:
        return oracle.index_scores_mxfp4(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, wl.k_bscale, None,
                                         wl.w, rows, out_ld=wl.max_ctx, entry=E)
    return oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, "fp8", wl.k_scale, wl.w,
                               rows, out_ld=wl.max_ctx, entry=E)


def _check_scores_and_topk(wl, flat, gsel, rows):
    ref = _ref_scores(wl, rows)
    b_of = wl.row_session(rows)
    empty = 0
    for j, (g, b) in enumerate(zip(rows, b_of)):
        C = int(wl.ctx_len[b])
        i = int(g) - int(wl.q_start[b])
        n = (int(wl.hist_len[b]) + i + 1) // E  # whole entries at this token
        st = int(wl.score_start[b]) + i * C
        got = flat[st: st + C].astype(np.float64)
        r = ref[j, :C]
        fin = np.isfinite(r)
        assert np.array_equal(fin, np.arange(C) < n) and np.array_equal(fin, np.isfinite(got)), (g,)
        s = gsel[g]
        if n == 0:
            empty += 1
            assert np.all(s == -1)
            continue
        assert np.abs(got[fin] - r[fin]).max() <= 1e-2 * np.abs(r[fin]).max(), (g,)
        chosen = np.zeros(C, bool)
        chosen[s[s >= 0]] = True
        if n <= wl.k:
            assert np.array_equal(chosen, fin) and np.sum(s == -1) == wl.k - n
            continue
        rv = r[:n]
        theta = np.partition(rv, n - wl.k)[n - wl.k]
        tau = 1e-2 * np.abs(rv).max()
        assert chosen.sum() == wl.k and not np.any(chosen[n:])
        assert np.all(chosen[:n][rv > theta + tau]) and not np.any(chosen[:n][rv < theta - tau])
    return empty


@pytest.mark.parametrize("key_format", [None, "mxfp4"])
def test_entry_prefill_scores_and_topk(key_format):
    wl = _prefill(key_format)
    assert list(wl.ctx_len) == [(262144 + 700) // E, (70000 + 300) // E, 260 // E]
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=SHIFT)
    assert bt.total_scores == wl.total_scores
    sc = _scores(wl, bt)
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    empty = _check_scores_and_topk(wl, sc.cpu().numpy(), sel.cpu().numpy(), _rows(wl))
    assert empty == 27  # session 3: tokens 0..26 precede its first whole entry


def test_entry_decode_scores_and_topk():
    wl = _decode()
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=SHIFT)
    sc = _scores(wl, bt)
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    _check_scores_and_topk(wl, sc.cpu().numpy(), sel.cpu().numpy(), np.arange(wl.total_q, dtype=np.int32))


def test_entry_page_demand_and_runs():
    wl = _prefill()
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=SHIFT)
    sel = synth_topk(wl, seed=5, hot_frac=0.5, pad_rows=3)
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), wl.page_size, wl.num_phys_pages,
                                           wl.max_run)
    torch.cuda.synchronize()
    rbm, rl, rc = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, wl.page_size, wl.num_phys_pages,
                                     entry=E)
    rr = oracle.runs(rbm, wl.num_phys_pages, wl.max_run)
    c = cnt.cpu().numpy()
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm)
    assert c[0] == rc and np.array_equal(lst.cpu().numpy()[:rc], rl)
    assert np.array_equal(runs.cpu().numpy()[: 2 * c[1]].reshape(-1, 2), rr)
    # the appended tokens' own entries never enter the demand
    hist_pages = {int(wl.page_table[b, p]) for b in range(wl.num_seqs)
                  for p in range(-(-int(wl.hist_ids[b]) // wl.page_size))}
    assert set(rl.tolist()) <= hist_pages


@pytest.mark.parametrize("shape", ["prefill", "decode"])
def test_entry_attention(shape):
    wl = _prefill() if shape == "prefill" else _decode()
    ai = attention_inputs(wl)
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=SHIFT)
    sel = synth_topk(wl, seed=9, hot_frac=0.6, pad_rows=2)
    rng = np.random.default_rng(1)
    sel[:, :4] = rng.integers(0, int(wl.ctx_len.max()), size=(wl.total_q, 4))  # some not yet whole
    kv, pt, s = T(ai.k_pool), T(wl.page_table), T(sel)
    if shape == "prefill":
        out, lse = janus.sparse_attn(bt, T(ai.q), kv, kv, pt, wl.page_size, s, ai.scale, dv=ai.dv, out_dtype="f32",
                                     want_lse=True)
        rows = _rows(wl)
    else:
        out, lse = janus.sparse_attn_split(bt, T(ai.q), kv, kv, pt, wl.page_size, s, ai.scale, num_splits=0,
                                           dv=ai.dv, out_dtype="f32", want_lse=True)
        rows = np.arange(wl.total_q, dtype=np.int32)
    torch.cuda.synchronize()
    ref, lref = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                   ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, sel[rows],
                                   ai.scale, ai.dv, entry=E)
    got, gl = out.cpu().numpy()[rows], lse.cpu().numpy()[rows]
    for j, g in enumerate(rows):
        if np.isneginf(lref[j]).all():  # no whole entry yet
            assert np.all(got[j] == 0) and np.all(np.isneginf(gl[j])), (g,)
            continue
        err = np.abs(got[j] - ref[j]).max()
        assert err <= 2e-2 and err <= 2e-2 * np.abs(ref[j]).max(), (g, err)
    fin = np.isfinite(lref)
    assert np.allclose(gl[fin], lref[fin], atol=2e-3)


def test_entry_vector_kernels_and_sharded_topk():
    """The generic kernels at entry granularity (E = 8): fp32 indexer scores
    (4 heads x 64), top-k and the sharded top-k on the GPU's own scores (exact
    against the oracle's selection over the same fp32 rows), and MQA attention
    with separate K and V pools at 24 heads (more than the MQA MFMA kernel
    takes); two sessions, one shorter than an entry."""
    from workloads.gen import MQA0_ATTN
    E = 8
    wl = make_workload(hist_len=[1500, 5], new_len=[70, 30], H=4, d=64, idx_dtype="f32", k=32, seed=51,
                       attn=dict(MQA0_ATTN, Hq=24), entry_shift=3, table="permuted", page_size=16)
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=3)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w))
    sel = janus.topk(bt, sc, wl.k)
    shd = janus.topk_sharded(bt, sc, wl.k, 4, wl.page_size)
    ai = attention_inputs(wl)
    out, lse = janus.sparse_attn(bt, T(ai.q), T(ai.k_pool), T(ai.v_pool), T(wl.page_table), wl.page_size, sel,
                                 ai.scale, dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    rows = np.arange(wl.total_q, dtype=np.int32)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "f32", None, wl.kI, "f32", None, wl.w, rows,
                              out_ld=wl.max_ctx, entry=E)
    flat = sc.cpu().numpy()
    got = np.full((wl.total_q, wl.max_ctx), -np.inf)
    for b in range(wl.num_seqs):
        C = int(wl.ctx_len[b])
        for i in range(int(wl.new_len[b])):
            st = int(wl.score_start[b]) + i * C
            got[wl.q_start[b] + i, :C] = flat[st: st + C]
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got))
    assert np.allclose(got[fin], ref[fin], rtol=1e-5, atol=1e-4)
    # selections on the GPU's own fp32 scores are exact
    g32 = got.astype(np.float32)
    assert np.array_equal(np.sort(sel.cpu().numpy(), axis=1),
                          np.sort(oracle.topk(wl.q_start, wl.hist_len, rows, g32, wl.k, entry=E), axis=1))
    want = oracle.topk_sharded(wl.q_start, wl.hist_len, rows, g32, wl.k, 4, wl.page_size, entry=E)
    gs = shd.cpu().numpy()
    kg = wl.k // 4
    for n in range(4):
        assert np.array_equal(np.sort(gs[:, n * kg:(n + 1) * kg], axis=1), np.sort(want[:, n * kg:(n + 1) * kg], axis=1))
    gsel = sel.cpu().numpy()
    oref, lref = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                    ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, gsel, ai.scale,
                                    ai.dv, entry=E)
    o = out.cpu().numpy()
    assert np.allclose(o, oref, atol=2e-3, rtol=1e-2)
    l = lse.cpu().numpy()
    assert np.array_equal(np.isneginf(l), np.isneginf(lref))
    assert np.allclose(l[np.isfinite(lref)], lref[np.isfinite(lref)], atol=1e-3)
    assert np.isneginf(lref).any()  # session 2's first tokens have no whole entry


def test_entry_mqa_mfma_attention():
    """The small config's MQA attention (8 heads, dqk = dv = 128, separate K
    and V pools) on the MFMA kernel at entry granularity (E = 8), with ids
    of entries not yet whole and a session shorter than one entry."""
    from workloads.gen import MQA0_ATTN
    E = 8
    wl = make_workload(hist_len=[1500, 5], new_len=[70, 30], H=4, d=64, idx_dtype="f32", k=96, seed=52,
                       attn=MQA0_ATTN, entry_shift=3, table="permuted", page_size=16)
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=3)
    ai = attention_inputs(wl)
    sel = synth_topk(wl, seed=9, hot_frac=0.6, pad_rows=2)
    rng = np.random.default_rng(2)
    sel[:, :4] = rng.integers(0, int(wl.ctx_len.max()), size=(wl.total_q, 4))  # some not yet whole
    out, lse = janus.sparse_attn(bt, T(ai.q), T(ai.k_pool), T(ai.v_pool), T(wl.page_table), wl.page_size, T(sel),
                                 ai.scale, dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    rows = np.arange(wl.total_q, dtype=np.int32)
    ref, lref = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                   ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, sel, ai.scale,
                                   ai.dv, entry=E)
    got, gl = out.cpu().numpy(), lse.cpu().numpy()
    assert np.isneginf(lref).any()
    for j in rows:
        if np.isneginf(lref[j]).all():  # no whole entry yet
            assert np.all(got[j] == 0) and np.all(np.isneginf(gl[j])), (j,)
            continue
        err = np.abs(got[j] - ref[j]).max()
        assert err <= 2e-2 and err <= 2e-2 * np.abs(ref[j]).max(), (j, err)
    fin = np.isfinite(lref)
    assert np.array_equal(fin, np.isfinite(gl))
    assert np.allclose(gl[fin], lref[fin], atol=2e-3)
