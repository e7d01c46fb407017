"""GPU parity of every entry point against the CPU oracle, through the C ABI.

Sizes are small enough for the oracle to finish in seconds but span several
kernel tiles and key chunks, with ragged tails, several sessions, an empty
history (the paper's initial prefill, P = 0) and misaligned score rows.

Tolerances (stated, not tuned):
  * indexer scores, per row over the causal candidates:
      max |gpu - oracle| / max |oracle|  <= 1e-2 (fp8), 1e-3 (bf16), 1e-5 (fp32);
    the -inf pattern must match exactly;
  * top-k fed the oracle's scores: the exact oracle set (bit-exact ids);
  * page demand, runs, predict-diff fed the same ids: bit-exact;
  * attention: max abs err <= 2e-2 and max abs err / max |oracle| <= 2e-2,
    fp32 accumulation.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, make_workload, synth_topk

pytestmark = pytest.mark.gpu

janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _batch(wl):
    return janus.Batch(wl.hist_len, wl.new_len)


def _rows_of(flat, wl):
    """Split the flat GPU score buffer into [total_q, max_ctx] (-inf padded)."""
    out = np.full((wl.total_q, wl.max_ctx), -np.inf, dtype=np.float32)
    ss = wl.score_start
    for b in range(wl.num_seqs):
        ctx = int(wl.ctx_len[b])
        blk = flat[ss[b]:ss[b + 1]].reshape(int(wl.new_len[b]), ctx)
        out[wl.q_start[b]:wl.q_start[b + 1], :ctx] = blk
    return out


def _score_check(wl, got_rows, tol):
    rows = np.arange(wl.total_q)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, wl.idx_dtype, wl.q_scale, wl.kI, wl.idx_dtype,
                              wl.k_scale, wl.w, rows, out_ld=wl.max_ctx)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got_rows)), "causal -inf pattern differs"
    assert np.all(np.isneginf(got_rows[~fin]))
    diff = np.zeros(ref.shape)
    diff[fin] = np.abs(got_rows[fin].astype(np.float64) - ref[fin])  # masked cells are -inf on both sides
    err = diff.max(axis=1)
    scale = np.where(fin, np.abs(ref), 0.0).max(axis=1)
    rel = err / np.maximum(scale, 1e-300)
    assert rel.max() <= tol, f"row rel err {rel.max():.3e} > {tol}"
    return ref, rel.max()


@pytest.mark.parametrize("dt,H,d,tol", [("fp8", 64, 128, 1e-2), ("bf16", 16, 32, 1e-3), ("f32", 4, 64, 1e-5),
                                        ("fp8", 8, 24, 1e-2)])
def test_index_scores_parity_ragged(dt, H, d, tol):
    if dt == "fp8" and H == 64:
        hist, new = [4200, 1500, 0, 77], [37, 20, 10, 5]
    else:
        hist, new = [700, 0, 65], [13, 6, 3]
    wl = make_workload(hist_len=hist, new_len=new, H=H, d=d, idx_dtype=dt, k=16, seed=31, w_scale=0.125)
    bt = _batch(wl)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=None if wl.q_scale is None else T(wl.q_scale),
                            k_scale=None if wl.k_scale is None else T(wl.k_scale), dtype=dt)
    torch.cuda.synchronize()
    _score_check(wl, _rows_of(sc.cpu().numpy(), wl), tol)


@pytest.mark.parametrize("hist,new", [([4200, 1500, 0], [37, 20, 10]), ([9000, 300, 64], [1, 3, 2])])
def test_fp8_index_scores_without_scales(hist, new):
    """fp8 keys and queries with both scale arrays NULL (every scale 1): the
    prefill kernel (sessions appending more than 4 tokens) and the row-tile
    kernel (at most 4), against the oracle over the same bytes."""
    wl = make_workload(hist_len=hist, new_len=new, H=64, d=128, idx_dtype="fp8", k=16, seed=37, w_scale=0.125)
    bt = _batch(wl)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=None, k_scale=None, dtype="fp8")
    torch.cuda.synchronize()
    got = _rows_of(sc.cpu().numpy(), wl)
    rows = np.arange(wl.total_q)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", None, wl.kI, "fp8", None, wl.w, rows,
                              out_ld=wl.max_ctx)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got))
    diff = np.where(fin, np.abs(got.astype(np.float64) - np.where(fin, ref, 0.0)), 0.0)
    scale = np.where(fin, np.abs(ref), 0.0).max(axis=1)
    assert (diff.max(axis=1) <= 1e-2 * np.maximum(scale, 1e-300)).all()


def _topk_case(hist, new, k, fill, seed=0):
    """A batch plus a synthetic flat score buffer built by `fill(rng, b, i, n)`."""
    rng = np.random.default_rng(seed)
    hist = np.asarray(hist, np.int32)
    new = np.asarray(new, np.int32)
    ctx = hist + new
    flat = []
    rows = []
    for b in range(len(hist)):
        for i in range(int(new[b])):
            n = int(hist[b]) + i + 1
            r = np.full(int(ctx[b]), -np.inf, np.float32)
            r[:n] = fill(rng, b, i, n).astype(np.float32)
            flat.append(r)
            rows.append(r)
    return hist, new, np.concatenate(flat)


FILLS = {
    "normal": lambda rng, b, i, n: rng.standard_normal(n),
    "hot": lambda rng, b, i, n: np.where((np.arange(n) // 700) % 9 == 3, 3.0, 1.0) * np.abs(rng.normal(18, 4, n)),
    "ascending": lambda rng, b, i, n: np.arange(n, dtype=np.float64),
    "descending": lambda rng, b, i, n: -np.arange(n, dtype=np.float64),
    "all_equal": lambda rng, b, i, n: np.full(n, 2.5),
    "all_zero": lambda rng, b, i, n: np.where(rng.random(n) < 0.5, 0.0, -0.0),
    "few_levels": lambda rng, b, i, n: rng.integers(0, 5, n).astype(np.float64),
    "uniform": lambda rng, b, i, n: rng.random(n),
    "inf_mix": lambda rng, b, i, n: np.where(rng.random(n) < 0.01, np.inf,
                                             np.where(rng.random(n) < 0.3, -np.inf, rng.standard_normal(n))),
    "sample_trap": lambda rng, b, i, n: _sample_trap(rng, n),
}


def _sample_trap(rng, n):
    """High values exactly where a strided sample of 32-element lines looks
    (8 per sampled line), too few to fill k: a threshold taken from such a
    sample sits above the k-th score, which the kernel must detect."""
    stride = max(1, (n >> 5) // 128)
    idx = np.arange(n)
    hot = ((idx >> 5) % stride == 0) & ((idx & 31) < 8)
    return rng.random(n) + np.where(hot, 10.0, 0.0)


@pytest.mark.parametrize("fill", list(FILLS))
@pytest.mark.parametrize("hist,new,k", [([20000, 9000], [3, 2], 2048), ([5000], [4], 6144), ([3000, 131], [2, 3], 1),
                                        ([130000], [1], 2048)])
def test_topk_exact_on_oracle_scores(fill, hist, new, k):
    hist, new, flat = _topk_case(hist, new, k, FILLS[fill])
    wl_q_start = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    bt = janus.Batch(hist, new)
    sel = janus.topk(bt, T(flat), k)
    torch.cuda.synchronize()
    got = sel.cpu().numpy()
    ctx = hist + new
    ss = bt.score_start_host
    for b in range(len(hist)):
        for i in range(int(new[b])):
            g = wl_q_start[b] + i
            row = flat[ss[b] + i * ctx[b]: ss[b] + (i + 1) * ctx[b]]
            ref = oracle.topk([0, 1], [hist[b] + i], [0], row[None, :], k)[0]
            n = int(hist[b]) + i + 1
            want = min(k, n)
            gv = got[g]
            assert np.all(gv[want:] == -1) and np.all(gv[:want] >= 0)
            assert np.all(np.diff(gv[:want]) > 0), "ids must be ascending"
            assert np.array_equal(np.sort(gv[:want]), np.sort(ref[:want])), f"{fill} row {g}"


def test_topk_band_on_gpu_scores():
    wl = make_workload(hist_len=[9000, 3000], new_len=[20, 12], H=64, d=128, idx_dtype="fp8", k=512, seed=5,
                       w_scale=0.125)
    bt = _batch(wl)
    sc = janus.index_scores(bt, T(wl.q), T(wl.kI), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(wl.k_scale))
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    got = sel.cpu().numpy()
    rows = np.arange(wl.total_q)
    ref = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, "fp8", wl.k_scale, wl.w, rows,
                              out_ld=wl.max_ctx)
    for g in rows:
        b = int(wl.row_session([g])[0])
        n = int(wl.hist_len[b]) + (g - int(wl.q_start[b])) + 1
        r = ref[g, :n]
        tau = 1e-2 * np.abs(r).max()
        theta = np.sort(r)[::-1][wl.k - 1]
        chosen = np.zeros(n, bool)
        chosen[got[g][got[g] >= 0]] = True
        assert chosen.sum() == wl.k
        assert np.all(chosen[r > theta + tau]), "a clear winner was dropped"
        assert not np.any(chosen[r < theta - tau]), "a clear loser was selected"


def _pd_ref(wl, sel, limit=None, max_run=None):
    max_run = max_run or wl.max_run
    bm, lst, c = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, wl.page_size, wl.num_phys_pages,
                                    limit=limit)
    return bm, lst, c, oracle.runs(bm, wl.num_phys_pages, max_run)


@pytest.mark.parametrize("table,page_size,max_run", [("permuted", 64, 32), ("identity", 16, 5), ("identity", 64, 32)])
def test_page_demand_bit_exact(table, page_size, max_run):
    wl = make_workload(hist_len=[30000, 5000, 0, 777], new_len=[300, 40, 16, 9], H=2, d=8, idx_dtype="f32",
                       k=512, page_size=page_size, seed=8, table=table, max_run=max_run)
    sel = synth_topk(wl, seed=2, pad_rows=3)
    bt = _batch(wl)
    for limit in (None, wl.ctx_len):
        bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), page_size, wl.num_phys_pages, max_run,
                                               limit=None if limit is None else T(limit.astype(np.int32)))
        torch.cuda.synchronize()
        rbm, rlst, rc, rruns = _pd_ref(wl, sel, limit, max_run)
        c = cnt.cpu().numpy()
        assert c[0] == rc and c[1] == rruns.shape[0]
        assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm)
        assert np.array_equal(lst.cpu().numpy()[:rc], rlst)
        assert np.array_equal(runs.cpu().numpy()[: 2 * c[1]].reshape(-1, 2), rruns)


def test_page_demand_largest_pool():
    """The largest pool the call takes (2^19 pages: a 64 KB bitmap, staged
    whole in LDS by the run walk), with the selection's pages spread over it
    by a sparse page table; bit-exact against the oracle."""
    P = 1 << 19
    wl = make_workload(hist_len=[30000, 777], new_len=[40, 9], H=2, d=8, idx_dtype="f32", k=512, seed=4)
    rng = np.random.default_rng(12)
    table = rng.choice(P - 16, size=wl.page_table.size, replace=False).astype(np.int32)
    table = table.reshape(wl.page_table.shape)
    # the short session (786 tokens in 13 pages, 512 of them selected per
    # row) sits on the pool's last pages: a run that ends at the pool's end
    table[1, :13] = np.arange(P - 13, P, dtype=np.int32)
    sel = synth_topk(wl, seed=5)
    bt = _batch(wl)
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(table), wl.page_size, P, 32)
    torch.cuda.synchronize()
    rbm, rlst, rc = oracle.page_demand(wl.q_start, wl.hist_len, sel, table, wl.page_size, P)
    rruns = oracle.runs(rbm, P, 32)
    c = cnt.cpu().numpy()
    assert c[0] == rc and c[1] == rruns.shape[0]
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm)
    assert np.array_equal(lst.cpu().numpy()[:rc], rlst)
    assert np.array_equal(runs.cpu().numpy()[: 2 * c[1]].reshape(-1, 2), rruns)


def test_page_demand_edges():
    wl = make_workload(hist_len=[4096], new_len=[8], H=2, d=8, idx_dtype="f32", k=64, seed=1)
    bt = _batch(wl)
    # nothing selected
    sel = np.full((8, 64), -1, np.int32)
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), 64, wl.num_phys_pages, 32)
    torch.cuda.synchronize()
    assert cnt.cpu().tolist() == [0, 0] and not bm.cpu().numpy().any()
    # every history token selected: pages 0..63 set, runs of 32
    sel = np.stack([np.arange(64) * 64 + i for i in range(8)]).astype(np.int32)
    bm, lst, runs, cnt = janus.page_demand(bt, T(sel), T(wl.page_table), 64, wl.num_phys_pages, 32)
    torch.cuda.synchronize()
    assert cnt.cpu().tolist() == [64, 2]
    assert runs.cpu().numpy()[:4].tolist() == [0, 32, 32, 32]


def test_predict_diff_bit_exact():
    rng = np.random.default_rng(9)
    for P, max_run in [(2176, 32), (7557, 32), (100, 1), (33, 4), (1, 32), (1 << 19, 32)]:
        nw = (P + 31) // 32
        for dens in (0.05, 0.5, 0.97):
            A = (rng.random(nw * 32) < dens).reshape(nw, 32)
            Q = (rng.random(nw * 32) < dens).reshape(nw, 32)
            pack = lambda m: (m.astype(np.uint64) << np.arange(32, dtype=np.uint64)).sum(1).astype(np.uint32)
            a, q = pack(A), pack(Q)
            miss, mruns, cnt = janus.predict_diff(T(a.view(np.int32)), T(q.view(np.int32)), P, max_run)
            torch.cuda.synchronize()
            rmiss, rruns, rcnt = oracle.predict_diff(a, q, P, max_run)
            c = cnt.cpu().numpy()
            assert np.array_equal(c, rcnt)
            assert np.array_equal(miss.cpu().numpy().view(np.uint32), rmiss)
            assert np.array_equal(mruns.cpu().numpy()[: 2 * c[4]].reshape(-1, 2), rruns)


def _attn_check(wl, ai, sel, out_dtype="f32"):
    bt = _batch(wl)
    vp = ai.k_pool if ai.v_pool is None else ai.v_pool
    kp_t = T(ai.k_pool)
    vp_t = kp_t if ai.v_pool is None else T(vp)
    out, lse = janus.sparse_attn(bt, T(ai.q), kp_t, vp_t, T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                 dv=ai.dv, out_dtype=out_dtype, want_lse=True)
    torch.cuda.synchronize()
    rows = np.arange(wl.total_q)
    ref, lref = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                                   ai.v_row_stride, wl.page_table, wl.page_size, sel, ai.scale, ai.dv)
    got = out.float().cpu().numpy()
    err = np.abs(got - ref).max()
    assert err <= 2e-2, f"max abs err {err}"
    assert err <= 2e-2 * np.abs(ref).max(), f"normalised err {err / np.abs(ref).max()}"
    lg = lse.cpu().numpy()
    fin = np.isfinite(lref)
    assert np.array_equal(fin, np.isfinite(lg))
    assert np.allclose(lg[fin], lref[fin], atol=2e-3, rtol=1e-4)
    return got, ref


MLA_SMALL = dict(Hq=128, dqk=576, dv=512, mla=True, q_std=1.0, kv_std=1.0 / 24.0, scale=1.0 / 24.0)


@pytest.mark.parametrize("kv_std,scale", [(1.0 / 24.0, 1.0 / 24.0), (1.0, 1.0 / 24.0), (1.0 / 24.0, 8.0)])
def test_sparse_mla_parity(kv_std, scale):
    attn = dict(MLA_SMALL, kv_std=kv_std, scale=scale)
    wl = make_workload(hist_len=[1500, 300], new_len=[6, 5], H=2, d=8, idx_dtype="f32", k=200, seed=4,
                       table="permuted", attn=attn)
    sel = synth_topk(wl, seed=3, pad_rows=2)
    _attn_check(wl, attention_inputs(wl), sel)


def test_sparse_mla_full_selection_is_dense_and_bf16_out():
    wl = make_workload(hist_len=[90], new_len=[7], H=2, d=8, idx_dtype="f32", k=128, seed=6, table="permuted",
                       attn=MLA_SMALL)
    sel = np.full((7, 128), -1, np.int32)
    for i in range(7):
        sel[i, :91 + i] = np.arange(91 + i)
    ai = attention_inputs(wl)
    got, ref = _attn_check(wl, ai, sel)
    gb, _ = _attn_check(wl, ai, sel, out_dtype="bf16")
    assert np.abs(gb - got).max() <= np.abs(ref).max() * 2 ** -7


@pytest.mark.parametrize("Hq,k", [(8, 300), (1, 64), (16, 1024), (5, 33)])
def test_sparse_mqa_mfma(Hq, k):
    """MQA with separate K and V pools at dqk = dv = 128 (the small config's
    attention: 8 heads sharing one KV head) on the MFMA kernel: one head,
    16 heads, a ragged tile (k = 33) and the largest k it takes, with padded
    rows and ids past the causal limit."""
    attn = dict(Hq=Hq, dqk=128, dv=128, mla=False, q_std=1.0, kv_std=1.0, scale=1.0 / math.sqrt(128.0))
    wl = make_workload(hist_len=[1800, 100, 0], new_len=[9, 4, 3], H=2, d=8, idx_dtype="f32", k=k, seed=2 + Hq,
                       table="permuted", attn=attn)
    sel = synth_topk(wl, seed=5, pad_rows=2)
    got, ref = _attn_check(wl, attention_inputs(wl), sel)
    gb, _ = _attn_check(wl, attention_inputs(wl), sel, out_dtype="bf16")
    assert np.abs(gb - got).max() <= np.abs(ref).max() * 2 ** -7


@pytest.mark.parametrize("Hq,dqk,dv,k", [(8, 64, 96, 200), (24, 128, 128, 200), (8, 128, 128, 1100)])
def test_sparse_attn_vector_kernel(Hq, dqk, dv, k):
    """Shapes outside the MFMA kernels (other head dims, more than 16 MQA
    heads, k above 1024 at dqk = 128) run on the plain vector kernel."""
    attn = dict(Hq=Hq, dqk=dqk, dv=dv, mla=False, q_std=1.0, kv_std=1.0, scale=1.0 / math.sqrt(dqk))
    wl = make_workload(hist_len=[1500, 100], new_len=[5, 4], H=2, d=8, idx_dtype="f32", k=k, seed=3, attn=attn)
    sel = synth_topk(wl, seed=5, pad_rows=2)
    _attn_check(wl, attention_inputs(wl), sel)


def test_empty_selection_row_gives_zero_and_neg_inf():
    wl = make_workload(hist_len=[64], new_len=[3], H=2, d=8, idx_dtype="f32", k=32, seed=6, attn=MLA_SMALL)
    sel = np.full((3, 32), -1, np.int32)
    sel[1, :5] = np.arange(5)
    got, ref = _attn_check(wl, attention_inputs(wl), sel)
    assert not got[0].any() and not got[2].any()
