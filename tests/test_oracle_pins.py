"""Pins for the CPU oracle: it is checked against things other than itself.

Library routines (torch casts, numpy matmul, torch.topk, numpy lexsort/unique,
torch scaled_dot_product_attention), closed forms and special cases, the
paper's read-packing example, and invariants.  Each test is chosen so that a
plausible slip in the oracle (a dropped term, a ReLU in the wrong place, a
transposed weight, a wrong session base, a wrong tie rule, an off-by-one in
the causal limit or in run splitting) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workloads import make_workload, synth_topk, attention_inputs, to_bf16_bits


# ----------------------------------------------------------------------------- decoders
def test_fp8_decoder_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.fp8_value(c) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(ref[~nan], got[~nan])
    assert oracle.fp8_value(0x7E) == 448.0 and oracle.fp8_value(0x01) == 2.0 ** -9


def test_bf16_decoder_matches_torch():
    rng = np.random.default_rng(0)
    bits = np.concatenate([rng.integers(0, 1 << 16, 4000), [0x0000, 0x8000, 0x3F80, 0x7F7F, 0x0001]]).astype(np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]  # finite only
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.bf16_value(b) for b in bits])
    assert np.array_equal(ref, got)


# ----------------------------------------------------------------------------- scores
def _f64(wl, a, dt):
    if dt == "f32":
        return a.astype(np.float64)
    if dt == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    return torch.from_numpy(a).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _scores(wl, rows=None, q=None):
    rows = np.arange(wl.total_q) if rows is None else rows
    return oracle.index_scores(wl.q_start, wl.hist_len, wl.q if q is None else q, wl.idx_dtype, wl.q_scale,
                               wl.kI, wl.idx_dtype, wl.k_scale, wl.w, rows)


def test_scores_single_head_unit_weight_is_relu_gemm():
    wl = make_workload(hist_len=[57], new_len=[9], H=1, d=12, idx_dtype="f32", k=8, seed=11)
    wl.w[:] = 1.0
    S = _scores(wl)
    ref = np.maximum(wl.q[:, 0, :].astype(np.float64) @ wl.kI.astype(np.float64).T, 0.0)
    for i in range(wl.total_q):
        lim = 57 + i
        assert np.allclose(S[i, :lim + 1], ref[i, :lim + 1], rtol=1e-13, atol=1e-12)
        assert np.all(np.isneginf(S[i, lim + 1:]))


@pytest.mark.parametrize("dt", ["f32", "bf16", "fp8"])
def test_scores_negation_identity_is_weighted_gemm(dt):
    # ReLU(x) - ReLU(-x) = x per head, so S(q) - S(-q) = sq*sk*sum_h w[t,h] x_h:
    # a plain weighted GEMM computed with numpy.
    wl = make_workload(hist_len=[70, 33], new_len=[5, 7], H=3, d=16, idx_dtype=dt, k=8, seed=5)
    if dt == "f32":
        qneg = -wl.q
    elif dt == "bf16":
        qneg = wl.q ^ np.uint16(0x8000)
    else:
        qneg = wl.q ^ np.uint8(0x80)
    S_pos = _scores(wl)
    S_neg = _scores(wl, q=qneg)
    qf = _f64(wl, wl.q, dt)
    kf = _f64(wl, wl.kI, dt)
    sq = wl.q_scale.astype(np.float64) if wl.q_scale is not None else np.ones(wl.total_q)
    sk = wl.k_scale.astype(np.float64) if wl.k_scale is not None else np.ones(wl.total_ctx)
    for b in range(wl.num_seqs):
        k0 = wl.ctx_start[b]
        for i in range(wl.new_len[b]):
            g = wl.q_start[b] + i
            lim = wl.hist_len[b] + i
            x = qf[g] @ kf[k0:k0 + lim + 1].T                     # [H, lim+1]
            ref = sq[g] * sk[k0:k0 + lim + 1] * (wl.w[g].astype(np.float64) @ x)
            got = S_pos[g, :lim + 1] - S_neg[g, :lim + 1]
            assert np.allclose(got, ref, rtol=1e-10, atol=1e-9 * np.abs(ref).max())
            assert np.all(S_pos[g, :lim + 1] >= 0.0)


def test_scores_zero_weight_and_key_scaling():
    wl = make_workload(hist_len=[40], new_len=[6], H=4, d=8, idx_dtype="fp8", k=8, seed=3)
    base = _scores(wl)
    w0 = wl.w.copy()
    wl.w[:] = 0.0
    z = _scores(wl)
    for i in range(6):
        assert np.all(z[i, :41 + i] == 0.0) and np.all(np.isneginf(z[i, 41 + i:]))
    wl.w[:] = w0
    c = np.float32(2.5)
    wl.k_scale[7] *= c
    sc = _scores(wl)
    assert np.allclose(sc[:, 7], base[:, 7] * float(c), rtol=1e-6)
    mask = np.ones(base.shape[1], bool)
    mask[7] = False
    assert np.array_equal(sc[:, mask], base[:, mask])


def test_scores_ragged_batch_equals_sessions_alone():
    wl = make_workload(hist_len=[30, 45, 12], new_len=[4, 2, 5], H=2, d=8, idx_dtype="bf16", k=4, seed=9)
    S = _scores(wl)
    for b in range(3):
        ks = slice(wl.ctx_start[b], wl.ctx_start[b + 1])
        qs = slice(wl.q_start[b], wl.q_start[b + 1])
        one = oracle.index_scores([0, wl.new_len[b]], [wl.hist_len[b]], wl.q[qs], "bf16", None, wl.kI[ks], "bf16",
                                  None, wl.w[qs], np.arange(wl.new_len[b]))
        ctx = int(wl.ctx_len[b])
        assert np.array_equal(S[qs, :ctx], one[:, :ctx])


def test_scores_brute_force_tiny():
    wl = make_workload(hist_len=[6], new_len=[3], H=2, d=3, idx_dtype="fp8", k=4, seed=21)
    S = _scores(wl)
    qf, kf = _f64(wl, wl.q, "fp8"), _f64(wl, wl.kI, "fp8")
    for i in range(3):
        for s in range(9):
            if s > 6 + i:
                assert math.isinf(S[i, s]) and S[i, s] < 0
                continue
            tot = 0.0
            for h in range(2):
                x = sum(qf[i, h, j] * kf[s, j] for j in range(3))
                tot += float(wl.w[i, h]) * max(x, 0.0)
            ref = float(wl.q_scale[i]) * float(wl.k_scale[s]) * tot
            assert S[i, s] == pytest.approx(ref, rel=1e-12, abs=1e-15)


# ----------------------------------------------------------------------------- top-k
def _topk_rows(scores, M, k):
    n = scores.shape[0]
    return oracle.topk([0, n], [M], np.arange(n), scores, k)


def test_topk_matches_torch_topk_distinct_values():
    rng = np.random.default_rng(1)
    M, N, k = 300, 20, 37
    sc = rng.permutation(M + N).astype(np.float32)[None, :].repeat(N, 0) + rng.standard_normal((N, M + N)).astype(np.float32) * 0
    sc = np.stack([rng.permutation(M + N).astype(np.float32) for _ in range(N)])
    got = _topk_rows(sc, M, k)
    for i in range(N):
        n = M + i + 1
        ref = torch.topk(torch.from_numpy(sc[i, :n]), k).indices.numpy()
        assert np.array_equal(got[i], ref)


def test_topk_ties_prefer_lower_index_and_padding():
    M, N = 10, 4
    sc = np.zeros((N, M + N), np.float32)
    sc[:, 3] = -0.0
    got = _topk_rows(sc, M, 6)
    for i in range(N):
        assert list(got[i]) == [0, 1, 2, 3, 4, 5]
    got = _topk_rows(sc, M, 13)
    for i in range(N):
        n = M + i + 1
        exp = list(range(min(n, 13))) + [-1] * (13 - min(n, 13))
        assert list(got[i]) == exp


def test_topk_lexsort_brute_force_with_ties():
    rng = np.random.default_rng(2)
    M, N, k = 200, 16, 50
    sc = rng.integers(0, 12, size=(N, M + N)).astype(np.float32)
    got = _topk_rows(sc, M, k)
    for i in range(N):
        n = M + i + 1
        order = np.lexsort((np.arange(n), -sc[i, :n].astype(np.float64)))
        assert np.array_equal(got[i], order[:k])
        sel = np.zeros(n, bool)
        sel[got[i]] = True
        assert sc[i, :n][sel].min() >= sc[i, :n][~sel].max()


# ----------------------------------------------------------------------------- sharded prediction (Eq. 3)
def _shards(M, G, align):
    L = align * (-(-(-(-M // align)) // G))
    return [(n * L, min(M, (n + 1) * L)) for n in range(G)]


@pytest.mark.parametrize("M,G,align,k", [(1000, 1, 1, 64), (1000, 4, 64, 64), (777, 8, 16, 40), (130, 4, 64, 64),
                                         (5000, 16, 64, 256)])
def test_topk_sharded_is_per_shard_lexsort(M, G, align, k):
    """Each shard's selection is the (score desc, id asc) head of its own
    history range, by numpy.lexsort; appended tokens are never candidates."""
    rng = np.random.default_rng(M + G)
    N = 5
    sc = rng.integers(0, 9, size=(N, M + N)).astype(np.float32) + rng.standard_normal((N, M + N)).astype(np.float32) * 0.5 * (G % 2)
    got = oracle.topk_sharded([0, N], [M], np.arange(N), sc, k, G, align)
    kg = k // G
    for i in range(N):
        for n, (lo, hi) in enumerate(_shards(M, G, align)):
            part = got[i, n * kg:(n + 1) * kg]
            cnt = max(0, hi - lo)
            if cnt:
                order = lo + np.lexsort((np.arange(cnt), -sc[i, lo:hi].astype(np.float64)))
                exp = order[:kg]
            else:
                exp = np.zeros(0, int)
            assert np.array_equal(part[:len(exp)], exp)
            assert np.all(part[len(exp):] == -1)


def test_topk_sharded_closed_forms():
    rng = np.random.default_rng(9)
    M, N, ps = 640, 3, 64
    sc = rng.standard_normal((N, M + N)).astype(np.float32)
    # one shard per page and k/G >= page size: every history token is selected
    got = oracle.topk_sharded([0, N], [M], np.arange(N), sc, 10 * 64, 10, ps)
    for i in range(N):
        assert sorted(got[i][got[i] >= 0].tolist()) == list(range(M))
    # shards are disjoint, page aligned and inside the history
    got = oracle.topk_sharded([0, N], [M], np.arange(N), sc, 32, 4, ps)
    for i in range(N):
        ids = got[i][got[i] >= 0]
        assert len(set(ids.tolist())) == len(ids) and ids.max() < M
        for n, (lo, hi) in enumerate(_shards(M, 4, ps)):
            assert lo % ps == 0
            part = got[i, n * 8:(n + 1) * 8]
            assert np.all((part >= lo) & (part < hi))
    # k not divisible by the shard count is rejected
    with pytest.raises(ValueError):
        oracle.topk_sharded([0, N], [M], np.arange(N), sc, 30, 4, ps)


def test_topk_sharded_one_shard_is_history_topk():
    """G = 1 is Eq. 2's selection over the history keys: the top-k of the
    history part of the row, by torch.topk on distinct values."""
    rng = np.random.default_rng(10)
    M, N, k = 500, 6, 50
    sc = np.stack([rng.permutation(M + N).astype(np.float32) for _ in range(N)])
    got = oracle.topk_sharded([0, N], [M], np.arange(N), sc, k, 1, 64)
    for i in range(N):
        ref = torch.topk(torch.from_numpy(sc[i, :M]), k).indices.numpy()
        assert np.array_equal(got[i], ref)


# ----------------------------------------------------------------------------- page demand, runs, diff
def test_page_demand_identity_and_permuted_tables():
    wl = make_workload(hist_len=[1000, 700], new_len=[40, 30], H=2, d=8, idx_dtype="f32", k=64, page_size=16, seed=4)
    sel = synth_topk(wl, seed=1, pad_rows=3)
    bm, lst, c = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, 16, wl.num_phys_pages)
    exp = set()
    for b in range(2):
        rows = sel[wl.q_start[b]:wl.q_start[b + 1]].ravel()
        rows = rows[(rows >= 0) & (rows < wl.hist_len[b])]
        exp |= set((wl.page_table[b, np.unique(rows // 16)]).tolist())
    assert lst.tolist() == sorted(exp) and c == len(exp)
    assert int(sum(bin(int(x)).count("1") for x in bm)) == c
    # a permuted table maps the identity result through the permutation
    perm = np.random.default_rng(7).permutation(wl.num_phys_pages).astype(np.int32)
    pt2 = perm[wl.page_table]
    _, lst2, c2 = oracle.page_demand(wl.q_start, wl.hist_len, sel, pt2, 16, wl.num_phys_pages)
    assert sorted(perm[lst].tolist()) == lst2.tolist() and c2 == c
    # limit 0 gives nothing; limit = context adds the new tokens' pages
    _, l0, c0 = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, 16, wl.num_phys_pages, limit=[0, 0])
    assert c0 == 0 and l0.size == 0
    _, lall, call = oracle.page_demand(wl.q_start, wl.hist_len, sel, wl.page_table, 16, wl.num_phys_pages,
                                       limit=wl.ctx_len)
    exp_all = set()
    for b in range(2):
        rows = sel[wl.q_start[b]:wl.q_start[b + 1]].ravel()
        rows = rows[(rows >= 0) & (rows < wl.ctx_len[b])]
        exp_all |= set((wl.page_table[b, np.unique(rows // 16)]).tolist())
    assert lall.tolist() == sorted(exp_all)


def _bitmap(pages, P):
    bm = np.zeros((P + 31) // 32, np.uint32)
    for p in pages:
        bm[p // 32] |= np.uint32(1 << (p % 32))
    return bm


def test_runs_paper_worked_example(golden_dir):
    cases = json.load(open(os.path.join(golden_dir, "read_packing.json")))["cases"]
    for c in cases:
        r = oracle.runs(_bitmap(c["selected"], c["num_pages"]), c["num_pages"], c["max_run"])
        assert r.tolist() == c["runs"], c["what"]


def test_runs_invariants_random_and_full():
    rng = np.random.default_rng(3)
    for P, max_run, density in [(1000, 32, 0.9), (777, 5, 0.5), (64, 32, 1.0), (100, 1, 0.7), (2176, 32, 0.05)]:
        pages = np.flatnonzero(rng.random(P) < density)
        bm = _bitmap(pages, P)
        r = oracle.runs(bm, P, max_run)
        covered = np.zeros(P, bool)
        prev_end = -1
        prev_len = 0
        for s, ln in r:
            assert 1 <= ln <= max_run and s > prev_end - 1 and s >= prev_end
            assert not covered[s:s + ln].any()
            covered[s:s + ln] = True
            if s == prev_end:
                assert prev_len == max_run          # touching runs only after a full piece
            elif s > 0:
                assert s - 1 not in set(pages.tolist()) or prev_end == s  # maximal start
            prev_end, prev_len = s + ln, ln
        assert np.array_equal(np.flatnonzero(covered), pages)
    r = oracle.runs(_bitmap(range(100), 100), 100, 32)
    assert r.tolist() == [[0, 32], [32, 32], [64, 32], [96, 4]]


def test_predict_diff_golden_and_set_algebra(golden_dir):
    for c in json.load(open(os.path.join(golden_dir, "recall_precision.json")))["cases"]:
        P = c["num_pages"]
        miss, mr, counts = oracle.predict_diff(_bitmap(c["actual"], P), _bitmap(c["predicted"], P), P, c["max_run"])
        assert counts.tolist() == c["counts"]
        assert np.array_equal(miss, _bitmap(c["miss"], P))
        assert mr.tolist() == c["miss_runs"]
        if c["recall"] is not None:
            assert counts[2] / counts[0] == pytest.approx(c["recall"])
        if c["precision"] is not None:
            assert counts[2] / counts[1] == pytest.approx(c["precision"])
    rng = np.random.default_rng(5)
    P = 2176
    for _ in range(5):
        A = rng.integers(0, 1 << 32, (P + 31) // 32, dtype=np.uint64).astype(np.uint32)
        Q = rng.integers(0, 1 << 32, (P + 31) // 32, dtype=np.uint64).astype(np.uint32)
        miss, _, counts = oracle.predict_diff(A, Q, P, 32)
        assert np.array_equal(miss, A & ~Q)
        pc = lambda x: int(sum(bin(int(v)).count("1") for v in x))
        assert counts.tolist()[:4] == [pc(A), pc(Q), pc(A & Q), pc(A & ~Q)]
        assert counts[3] == counts[0] - counts[2]
        zero = np.zeros_like(A)
        m0, _, c0 = oracle.predict_diff(A, zero, P, 32)
        assert np.array_equal(m0, A) and c0[3] == c0[0]
        m1, r1, c1 = oracle.predict_diff(A, A | Q, P, 32)
        assert not m1.any() and c1[3] == 0 and c1[4] == 0 and c1[2] == c1[0]


# ----------------------------------------------------------------------------- attention
def _attn_wl(hist, new, Hq=4, dqk=24, dv=16, mla=False, page_size=8, table="identity", seed=0):
    attn = dict(Hq=Hq, dqk=dqk, dv=dv, mla=mla, q_std=1.0, kv_std=1.0, scale=1.0 / math.sqrt(dqk))
    wl = make_workload(hist_len=hist, new_len=new, H=1, d=4, idx_dtype="f32", k=4, page_size=page_size,
                       seed=seed, table=table, attn=attn)
    return wl, attention_inputs(wl)


def _bf(x):
    return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(torch.float64)


def _logical_kv(wl, ai, b):
    ctx = int(wl.ctx_len[b])
    s = np.arange(ctx)
    slot = wl.page_table[b, s // wl.page_size] * wl.page_size + s % wl.page_size
    K = _bf(ai.k_pool.reshape(-1, ai.k_row_stride)[slot, :ai.dqk])
    vp = ai.k_pool if ai.v_pool is None else ai.v_pool
    V = _bf(vp.reshape(-1, vp.shape[2])[slot, :ai.dv])
    return K, V


@pytest.mark.parametrize("mla,table", [(False, "identity"), (True, "permuted")])
def test_attention_full_selection_is_dense_causal_sdpa(mla, table):
    wl, ai = _attn_wl([50, 29], [6, 9], mla=mla, dqk=24 if not mla else 20, dv=16, table=table)
    kk = int(wl.ctx_len.max()) + 3
    rows = np.arange(wl.total_q)
    sel = np.full((wl.total_q, kk), -1, np.int32)
    rng = np.random.default_rng(0)
    for b in range(wl.num_seqs):
        for i in range(wl.new_len[b]):
            n = wl.hist_len[b] + i + 1
            sel[wl.q_start[b] + i, :n] = rng.permutation(n)
    out, lse = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                                  ai.v_row_stride, wl.page_table, wl.page_size, sel, ai.scale, ai.dv)
    for b in range(wl.num_seqs):
        K, V = _logical_kv(wl, ai, b)
        M, N = int(wl.hist_len[b]), int(wl.new_len[b])
        Q = _bf(ai.q[wl.q_start[b]:wl.q_start[b + 1]]).permute(1, 0, 2)      # [Hq, N, dqk]
        mask = torch.arange(M + N)[None, :] <= (M + torch.arange(N))[:, None]  # bottom-right aligned
        ref = torch.nn.functional.scaled_dot_product_attention(
            Q, K[None].expand(ai.Hq, -1, -1), V[None].expand(ai.Hq, -1, -1), attn_mask=mask, scale=ai.scale)
        got = torch.from_numpy(out[wl.q_start[b]:wl.q_start[b + 1]]).permute(1, 0, 2)
        assert torch.allclose(got, ref, rtol=1e-10, atol=1e-12)
        logits = (Q @ K.T) * ai.scale
        logits = logits.masked_fill(~mask, -math.inf)
        assert np.allclose(lse[wl.q_start[b]:wl.q_start[b + 1]].T, torch.logsumexp(logits, -1).numpy(), rtol=1e-12)


def test_attention_closed_forms():
    wl, ai = _attn_wl([40], [5])
    rows = np.arange(5)
    K, V = _logical_kv(wl, ai, 0)
    # one selected id: output is that value row
    sel = np.full((5, 7), -1, np.int32)
    sel[:, 3] = np.array([2, 17, 30, 41, 44])
    out, lse = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                                  ai.v_row_stride, wl.page_table, wl.page_size, sel, ai.scale, ai.dv)
    for i in range(5):
        assert np.allclose(out[i], V[sel[i, 3]].numpy()[None, :].repeat(ai.Hq, 0), rtol=0, atol=0)
    # zero query: the plain mean of the selected values
    sel2 = np.stack([np.arange(10) * 3 + i for i in range(5)]).astype(np.int32)
    q0 = np.zeros_like(ai.q)
    out0, lse0 = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, q0, ai.k_pool, ai.v_pool, ai.k_row_stride,
                                    ai.v_row_stride, wl.page_table, wl.page_size, sel2, ai.scale, ai.dv)
    for i in range(5):
        assert np.allclose(out0[i], V[sel2[i]].mean(0).numpy()[None, :], rtol=1e-12, atol=1e-14)
        assert np.allclose(lse0[i], math.log(10.0))
    # ids past the causal limit and -1 are padding; permuting a row changes nothing
    sel3 = sel2.copy()
    sel3[:, 9] = 44 + 1  # beyond every row's limit (M + i <= 44)
    sel3 = np.concatenate([sel3, np.full((5, 2), -1, np.int32)], 1)
    a, _ = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                              ai.v_row_stride, wl.page_table, wl.page_size, sel3, ai.scale, ai.dv)
    perm = np.random.default_rng(1).permutation(sel3.shape[1])
    b_, _ = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                               ai.v_row_stride, wl.page_table, wl.page_size, sel3[:, perm], ai.scale, ai.dv)
    c_, _ = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, ai.k_pool, ai.v_pool, ai.k_row_stride,
                               ai.v_row_stride, wl.page_table, wl.page_size, sel2[:, :9], ai.scale, ai.dv)
    assert np.allclose(a, b_, rtol=1e-12, atol=1e-15) and np.allclose(a, c_, rtol=1e-12, atol=1e-15)


# ----------------------------------------------------------------------------- decode step
def test_decode_step_is_append_prefill_with_one_token():
    """A decode step is an append prefill with one appended token (Sec. 2.2,
    decode phase): row i of a session with history M and N appended tokens is
    the single row of a session with history M + i whose keys are the same
    first M + i + 1 keys - for scores and for attention over the same ids."""
    rng = np.random.default_rng(12)
    M, N, H, d, ps = 300, 5, 2, 16, 16
    q = rng.standard_normal((N, H, d)).astype(np.float32)
    kI = rng.standard_normal((M + N, d)).astype(np.float32)
    w = rng.random((N, H)).astype(np.float32)
    pre = oracle.index_scores([0, N], [M], q, "f32", None, kI, "f32", None, w, np.arange(N), out_ld=M + N)
    dec_hist = [M + i for i in range(N)]
    dec_keys = np.concatenate([kI[:M + i + 1] for i in range(N)])
    dec = oracle.index_scores(np.arange(N + 1), dec_hist, q, "f32", None, dec_keys, "f32", None, w, np.arange(N),
                              out_ld=M + N)
    assert np.array_equal(pre, dec)
    # attention through one pool: every decode session maps its pages like the prefill session
    Hq, dqk = 4, 32
    pages = (M + N + ps - 1) // ps
    pool = to_bf16_bits(rng.standard_normal((pages * ps, dqk)).astype(np.float32))
    pt = np.arange(pages, dtype=np.int32)[None, :]
    qa = to_bf16_bits(rng.standard_normal((N, Hq, dqk)).astype(np.float32))
    sel = np.stack([rng.choice(M + i + 1, 40, replace=False) for i in range(N)]).astype(np.int32)
    o1, l1 = oracle.sparse_attn([0, N], [M], np.arange(N), qa, pool, None, dqk, dqk, pt, ps, sel, 0.2, dqk)
    o2, l2 = oracle.sparse_attn(np.arange(N + 1), dec_hist, np.arange(N), qa, pool, None, dqk, dqk,
                                np.repeat(pt, N, axis=0), ps, sel, 0.2, dqk)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


# ----------------------------------------------------------------------------- MXFP4 indexer keys
# OCP MX v1.0, FP4 (E2M1) element encodings: code -> value (sign in bit 3)
OCP_E2M1 = {0b0000: 0.0, 0b0001: 0.5, 0b0010: 1.0, 0b0011: 1.5, 0b0100: 2.0, 0b0101: 3.0, 0b0110: 4.0, 0b0111: 6.0}


def test_e2m1_and_e8m0_tables():
    for c, v in OCP_E2M1.items():
        assert oracle.e2m1_value(c) == v and oracle.e2m1_value(c | 8) == -v
    assert math.copysign(1.0, oracle.e2m1_value(8)) == -1.0  # negative zero
    assert oracle.e8m0_value(127) == 1.0 and oracle.e8m0_value(130) == 8.0 and oracle.e8m0_value(120) == 2.0 ** -7
    assert oracle.e8m0_value(0) == 2.0 ** -127 and oracle.e8m0_value(254) == 2.0 ** 127
    assert math.isnan(oracle.e8m0_value(255))


def _decode_mxfp4_table(packed, E):
    """MXFP4 keys to float32 through the OCP table (exact: e2m1 x 2^k)."""
    n, half = packed.shape
    codes = np.empty((n, 2 * half), np.uint8)
    codes[:, 0::2], codes[:, 1::2] = packed & 15, packed >> 4
    mag = np.array([OCP_E2M1[c & 7] for c in range(16)])[codes]
    val = np.where(codes & 8, -mag, mag) * np.repeat(np.exp2(E.astype(np.float64) - 127), 32, axis=1)
    return val.astype(np.float32)


@pytest.mark.parametrize("H,d", [(2, 64), (4, 128)])
def test_mxfp4_scores_are_the_f32_scores_of_the_decoded_keys(H, d):
    """The MXFP4 path equals the (separately pinned) f32 path fed the decoded
    key values, bit for bit; queries are fp8 with per-token scales in both."""
    from workloads import quantize_mxfp4
    rng = np.random.default_rng(H + d)
    hist, new = [300, 90], [4, 3]
    ctx = sum(hist) + sum(new)
    kf = (rng.standard_normal((ctx, d)) * rng.choice([0.01, 1.0, 50.0], size=(ctx, 1))).astype(np.float32)
    packed, E = quantize_mxfp4(kf)
    from workloads import quantize_fp8_per_row
    q, qs = quantize_fp8_per_row(rng.standard_normal((sum(new), H, d)).astype(np.float32))
    w = rng.random((sum(new), H)).astype(np.float32)
    ks = rng.uniform(0.5, 2.0, ctx).astype(np.float32)
    qst = np.array([0, new[0], sum(new)])
    rows = np.arange(sum(new))
    got = oracle.index_scores_mxfp4(qst, hist, q, "fp8", qs, packed, E, ks, w, rows)
    ref = oracle.index_scores(qst, hist, q, "fp8", qs, _decode_mxfp4_table(packed, E), "f32", ks, w, rows)
    assert np.array_equal(got, ref)


def test_mxfp4_constant_keys_closed_form():
    """Every key element = code 0b0010 (1.0) at block scale 2^3: k = 8 * ones,
    so S[t,s] = sq[t] * sum_h w[t,h] * max(0, 8 * sum_j q[t,h,j])."""
    rng = np.random.default_rng(31)
    H, d, M, N = 3, 64, 50, 2
    packed = np.full((M + N, d // 2), 0x22, np.uint8)
    E = np.full((M + N, d // 32), 130, np.uint8)
    q = rng.standard_normal((N, H, d)).astype(np.float32)
    from workloads import quantize_fp8_per_row
    q8, qs = quantize_fp8_per_row(q)
    w = rng.random((N, H)).astype(np.float32)
    got = oracle.index_scores_mxfp4([0, N], [M], q8, "fp8", qs, packed, E, None, w, np.arange(N))
    qd = np.array([oracle.fp8_value(b) for b in q8.reshape(-1)]).reshape(N, H, d)
    for t in range(N):
        want = qs[t] * (w[t] * np.maximum(0.0, 8.0 * qd[t].sum(axis=1))).sum()
        assert np.allclose(got[t, :M + t + 1], want, rtol=1e-12, atol=0)
        assert np.all(np.isneginf(got[t, M + t + 1:]))


def test_mxfp4_generator_rounding():
    """The key generator's MXFP4 encoding (input bytes, not method
    arithmetic): the block exponent is the smallest that fits amax within 6,
    elements round to the nearest e2m1 value with ties to the even code, and
    decoding through the OCP table returns every representable input as is."""
    from workloads import quantize_mxfp4
    x = np.zeros((2, 32), np.float32)
    x[0, :9] = [0.75, 0.25, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, -0.75]
    x[1, :4] = [12.0, -3.0, 1.0, 8.0]  # amax 12 -> exponent 1
    packed, E = quantize_mxfp4(x)
    assert E[0, 0] == 127 and E[1, 0] == 128
    codes = [(packed[0, j // 2] >> (4 * (j % 2))) & 15 for j in range(9)]
    assert codes == [0b0010, 0b0000, 0b0010, 0b0100, 0b0100, 0b0110, 0b0110, 0b0111, 0b1010]
    dec = _decode_mxfp4_table(packed, E)
    assert np.array_equal(dec[1, :4], x[1, :4])


# ----------------------------------------------------------------------------- entry granularity
# An entry j stands for tokens E*j .. E*j+E-1 (DeepSeek-V4 selects entries;
# the notation table applies to them unchanged).  The pins below enumerate an
# entry's tokens one by one, instead of the oracle's region-end comparison.

def _entry_ok(j, E, pos):
    """Every token of entry j is at or before position pos."""
    return all(t <= pos for t in range(E * j, E * j + E))


SMALL_MQA = dict(Hq=4, dqk=32, dv=32, mla=False, q_std=1.0, kv_std=1.0, scale=0.2)


@pytest.mark.parametrize("E", [4, 16])
def test_entry_scores_are_token_scores_with_entry_masks(E):
    """Entry scores equal token-granularity scores over the same key rows
    (under a history so long that every row is a candidate), with exactly the
    entries whose tokens have all arrived kept and the rest -inf."""
    M, N = 203, 37
    wl = make_workload(hist_len=[M], new_len=[N], H=2, d=32, idx_dtype="f32", k=8, seed=E,
                       entry_shift=int(math.log2(E)), hot=False)
    C = int(wl.ctx_len[0])
    assert C == (M + N) // E and wl.kI.shape[0] == C
    rows = np.arange(N, dtype=np.int32)
    got = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "f32", None, wl.kI, "f32", None, wl.w, rows,
                              entry=E)
    keys = np.concatenate([wl.kI, np.zeros((N, wl.d), np.float32)])  # rows C.. are never read below
    every = oracle.index_scores([0, N], [C], wl.q, "f32", None, keys, "f32", None, wl.w, rows)[:, :C]
    assert got.shape == (N, C)
    for i in range(N):
        ok = np.array([_entry_ok(j, E, M + i) for j in range(C)])
        assert np.array_equal(got[i, ok], every[i, ok])
        assert np.all(np.isneginf(got[i, ~ok]))
    # one new entry completes every E appended tokens
    counts = np.isfinite(got).sum(axis=1)
    assert counts[0] == (M + 1) // E and counts[-1] == C


@pytest.mark.parametrize("E", [4, 16])
def test_entry_topk_and_sharded_over_entry_candidates(E):
    M, N, k = 150, 20, 12
    rng = np.random.default_rng(E)
    C = (M + N) // E
    sc = rng.integers(0, 5, size=(N, C)).astype(np.float32)  # many ties
    rows = np.arange(N, dtype=np.int32)
    got = oracle.topk([0, N], [M], rows, sc, k, entry=E)
    for i in range(N):
        cand = [j for j in range(C) if _entry_ok(j, E, M + i)]
        order = [cand[t] for t in np.lexsort((np.array(cand), -sc[i, cand]))] if cand else []
        want = (order + [-1] * k)[:k]
        assert list(got[i]) == want
    # sharded: only the entries wholly in the history are candidates
    G, align = 2, 4
    gs = oracle.topk_sharded([0, N], [M], rows, sc, k, G, align, entry=E)
    hist = [j for j in range(C) if _entry_ok(j, E, M - 1)]
    units = -(-len(hist) // align)
    L = align * (-(-units // G))
    for i in range(N):
        for n in range(G):
            part = [j for j in hist if n * L <= j < (n + 1) * L]
            order = [part[t] for t in np.lexsort((np.array(part), -sc[i, part]))] if part else []
            assert list(gs[i, n * (k // G):(n + 1) * (k // G)]) == (order + [-1] * (k // G))[:k // G]


def test_entry_page_demand_keeps_history_entries_only():
    E, M, N, ps = 8, 100, 30, 4
    C = (M + N) // E
    rng = np.random.default_rng(3)
    sel = rng.integers(-1, C + 2, size=(N, 6)).astype(np.int32)
    pt = rng.permutation(8).astype(np.int32).reshape(1, 8)
    bm, lst, cnt = oracle.page_demand([0, N], [M], sel, pt, ps, 8, entry=E)
    want = sorted({int(pt[0, s // ps]) for s in sel.reshape(-1) if 0 <= s < C and _entry_ok(s, E, M - 1)})
    assert list(lst) == want and cnt == len(want)


@pytest.mark.parametrize("E", [2, 8])
def test_entry_attention_equals_token_attention_with_entry_masks(E):
    """Attention over entries equals token-granularity attention over the
    same rows (every id a candidate) after the not-yet-complete entries are
    turned into padding."""
    M, N = 90, 21
    wl = make_workload(hist_len=[M], new_len=[N], H=2, d=32, idx_dtype="f32", k=10, page_size=4, seed=E,
                       entry_shift=int(math.log2(E)), attn=SMALL_MQA)
    ai = attention_inputs(wl)
    sel = synth_topk(wl, seed=1)
    C = int(wl.ctx_len[0])
    rng = np.random.default_rng(E)
    sel[:, :3] = rng.integers(0, C, size=(N, 3))  # some ids past each token's entries
    rows = np.arange(N, dtype=np.int32)
    args = (ai.k_pool.reshape(-1, ai.dqk), ai.v_pool.reshape(-1, ai.dv), ai.dqk, ai.dv, wl.page_table,
            wl.page_size)
    o1, l1 = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, ai.q, *args, sel, ai.scale, ai.dv, entry=E)
    masked = np.array([[s if 0 <= s < C and _entry_ok(int(s), E, M + i) else -1 for s in sel[i]]
                       for i in range(N)], dtype=np.int32)
    o2, l2 = oracle.sparse_attn([0, N], [C], rows, ai.q, *args, masked, ai.scale, ai.dv)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    assert np.any(masked != sel)


# ----------------------------------------------------------------------------- FP8 KV cache
def test_fp8kv_attention_equals_bf16_attention_on_decoded_rows():
    """With power-of-two row scales every stored value e4m3 * 2^e is a bf16
    value, so attention over the fp8 rows equals the (separately pinned)
    bf16 attention over the decoded rows bit for bit: the fp8 decode, the
    scale's place in the row and V being the row's first 512 elements."""
    from workloads import to_fp8_bytes
    rng = np.random.default_rng(8)
    M, N, ps, Hq = 60, 5, 8, 4
    P = (M + N + ps - 1) // ps
    x = rng.standard_normal((P * ps, 576)).astype(np.float32)
    e = rng.integers(-12, 4, size=P * ps)
    pool8 = np.zeros((P * ps, 592), np.uint8)
    pool8[:, :576] = to_fp8_bytes(x * 16)
    pool8[:, 576:580] = np.exp2(e).astype(np.float32).view(np.uint8).reshape(-1, 4)
    dec = np.array([oracle.fp8_value(b) for b in range(256)])[pool8[:, :576]] * np.exp2(e)[:, None]
    bf = to_bf16_bits(dec.astype(np.float32))
    assert np.array_equal(np.array([oracle.bf16_value(b) for b in bf.reshape(-1)[:2000]]), dec.reshape(-1)[:2000])
    pt = rng.permutation(P).astype(np.int32).reshape(1, P)
    q = to_bf16_bits(rng.standard_normal((N, Hq, 576)).astype(np.float32))
    sel = rng.integers(-1, M + N, size=(N, 16)).astype(np.int32)
    rows = np.arange(N, dtype=np.int32)
    o8, l8 = oracle.sparse_attn_fp8kv([0, N], [M], rows, q, pool8.reshape(P, ps, 592), pt, ps, sel, 0.05)
    ob, lb = oracle.sparse_attn([0, N], [M], rows, q, bf, None, 576, 576, pt, ps, sel, 0.05, 512)
    assert np.array_equal(o8, ob) and np.array_equal(l8, lb)
