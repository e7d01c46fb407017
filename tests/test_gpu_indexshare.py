"""IndexShare (the GLM-5 series' layer grouping, Sec. 2.2): four consecutive
sparse-attention layers share one selection.  Only the first runs the indexer
and top-k, and each layer attends over its own KV cache and queries with the
shared ids.  The four layers' pools share the page table, so one page-demand
call serves the group.

Workload: one session, history 20000 + 300 new tokens, fp8 indexer (64 x 128),
k = 2048, MLA attention, a random page table; each layer's queries and KV are
drawn from its own generator streams.  Compared with the oracle per layer on
every 3rd row (2e-2, absolute and relative to the row's largest output), and
the shared page set bit-exact."""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, attention_q_rows, make_workload
from workloads.gen import MLA_ATTN

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")

LAYERS = 4


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _layer(l):
    return make_workload(hist_len=[20000], new_len=[300], H=64, d=128, idx_dtype="fp8", k=2048, seed=31, layer=l,
                         w_scale=1 / 8, table="permuted", attn=MLA_ATTN)


def test_indexshare_group_matches_each_layer():
    wls = [_layer(l) for l in range(LAYERS)]
    assert all(np.array_equal(w.page_table, wls[0].page_table) for w in wls)
    lead = wls[0]
    bt = janus.Batch(lead.hist_len, lead.new_len)
    sc = janus.index_scores(bt, T(lead.q), T(lead.kI), T(lead.w), q_scale=T(lead.q_scale), k_scale=T(lead.k_scale))
    sel = janus.topk(bt, sc, lead.k)
    pt = T(lead.page_table)
    bm, lst, runs, cnt = janus.page_demand(bt, sel, pt, lead.page_size, lead.num_phys_pages, lead.max_run)
    outs = []
    for wl in wls:
        ai = attention_inputs(wl)
        kv = T(ai.k_pool)
        o, l_ = janus.sparse_attn(bt, T(ai.q), kv, kv, pt, wl.page_size, sel, ai.scale, dv=ai.dv, out_dtype="f32",
                                  want_lse=True)
        outs.append((o.cpu().numpy(), ai))
    torch.cuda.synchronize()
    gsel = sel.cpu().numpy()
    rbm, rl, rc = oracle.page_demand(lead.q_start, lead.hist_len, gsel, lead.page_table, lead.page_size,
                                     lead.num_phys_pages)
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), rbm) and int(cnt.cpu()[0]) == rc
    rows = np.arange(0, lead.total_q, 3, dtype=np.int32)
    prev = None
    for l, (wl, (got, ai)) in enumerate(zip(wls, outs)):
        ref, _ = oracle.sparse_attn(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), ai.k_pool, ai.v_pool,
                                    ai.k_row_stride, ai.v_row_stride, wl.page_table, wl.page_size, gsel[rows],
                                    ai.scale, ai.dv)
        for j, g in enumerate(rows):
            err = np.abs(got[g] - ref[j]).max()
            assert err <= 2e-2 and err <= 2e-2 * np.abs(ref[j]).max(), (l, g, err)
        if prev is not None:  # the layers' own KV and queries give different outputs
            assert not np.allclose(got[rows], prev)
        prev = got[rows]
