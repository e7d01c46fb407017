"""janus_sparse_attn_split_noalloc, the split attention for callers that
cannot allocate: through the C ABI, two calls in a row on one GPU (the second
with a smaller batch, while the library's scratch array still holds the first
call's partial results), each compared with janus_sparse_attn_split on the
same inputs and slice count (same kernels: identical output and lse) and, for
the smaller call, with the oracle (max abs error <= 2e-2 and <= 2e-2 of the
largest output)."""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, make_workload, synth_topk

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")

MLA = dict(Hq=128, dqk=576, dv=512, mla=True, q_std=1.0, kv_std=1.0 / 24.0, scale=1.0 / 24.0)


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(hist, new, k, seed):
    wl = make_workload(hist_len=hist, new_len=new, H=2, d=8, idx_dtype="f32", k=k, seed=seed, table="permuted",
                       attn=MLA)
    return wl, attention_inputs(wl), synth_topk(wl, seed=seed, pad_rows=1)


def _run_both(wl, ai, sel, num_splits):
    bt = janus.Batch(wl.hist_len, wl.new_len)
    q, kv, pt, s = T(ai.q), T(ai.k_pool), T(wl.page_table), T(sel)
    out = torch.empty((wl.total_q, ai.Hq, ai.dv), dtype=torch.float32, device="cuda")
    lse = torch.empty((wl.total_q, ai.Hq), dtype=torch.float32, device="cuda")
    janus.sparse_attn_split_noalloc(bt, q, kv, kv, pt, wl.page_size, s, ai.scale, num_splits=num_splits, dv=ai.dv,
                                    out_dtype="f32", out=out, lse=lse)
    ref_out, ref_lse = janus.sparse_attn_split(bt, q, kv, kv, pt, wl.page_size, s, ai.scale, num_splits=num_splits,
                                               dv=ai.dv, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy(), ref_out.cpu().numpy(), ref_lse.cpu().numpy()


def test_noalloc_split_matches_the_workspace_split_twice():
    # first call: 20 rows, 6 slices each (120 slice blocks of partials)
    wl, ai, sel = _case([1500, 300, 4000], [6, 5, 9], 384, seed=21)
    print("noalloc call 1: 20 rows, k=384, 6 slices", flush=True)
    o, l, ro, rl = _run_both(wl, ai, sel, 6)
    assert np.array_equal(o, ro) and np.array_equal(l, rl, equal_nan=True)
    # second call: smaller (3 rows, 3 slices); the scratch still holds call 1's partials
    wl2, ai2, sel2 = _case([700], [3], 96, seed=22)
    print("noalloc call 2: 3 rows, k=96, 3 slices", flush=True)
    o2, l2, ro2, rl2 = _run_both(wl2, ai2, sel2, 3)
    assert np.array_equal(o2, ro2) and np.array_equal(l2, rl2, equal_nan=True)
    rows = np.arange(wl2.total_q)
    ref, lref = oracle.sparse_attn(wl2.q_start, wl2.hist_len, rows, ai2.q, ai2.k_pool, None, ai2.k_row_stride,
                                   ai2.v_row_stride, wl2.page_table, wl2.page_size, sel2, ai2.scale, ai2.dv)
    err = np.abs(o2 - ref).max()
    assert err <= 2e-2 and err <= 2e-2 * np.abs(ref).max(), err
    fin = np.isfinite(lref)
    assert np.array_equal(fin, np.isfinite(l2)) and np.allclose(l2[fin], lref[fin], atol=2e-3, rtol=1e-4)


def test_noalloc_split_automatic_slice_count():
    wl, ai, sel = _case([2500, 900], [4, 3], 512, seed=23)
    print("noalloc automatic slices: 7 rows, k=512", flush=True)
    o, l, ro, rl = _run_both(wl, ai, sel, 0)
    assert np.array_equal(o, ro) and np.array_equal(l, rl, equal_nan=True)


def test_noalloc_split_rejects_more_than_its_scratch():
    """A launch needing more than JANUS_NOALLOC_SCRATCH_BYTES of partials is
    refused before anything is enqueued (2048 rows x 16 slices x 128 heads)."""
    wl, ai, sel = _case([600], [8], 512, seed=24)
    bt = janus.Batch([600], [2048])  # only the host sizes matter: the call returns before launching
    q = torch.empty((2048, 128, 576), dtype=torch.bfloat16, device="cuda")
    kv = T(ai.k_pool)
    pt = torch.zeros((1, 64), dtype=torch.int32, device="cuda")
    s = torch.full((2048, 512), -1, dtype=torch.int32, device="cuda")
    with pytest.raises(janus.JanusError, match="workspace too small"):
        janus.sparse_attn_split_noalloc(bt, q, kv, kv, pt, 64, s, 0.1, num_splits=16, dv=512)
