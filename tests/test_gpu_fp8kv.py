"""MLA attention over an FP8 KV cache (KV states kept in FP8, Sec. 5.1) on
the GPU against the oracle.  Pool rows: 576 e4m3 bytes, the row's fp32 scale
at byte 576, 592 bytes in all.  The pools come from the same draws as the
bf16 pools (each row quantised with amax/448).  Compared per row: 2e-2
absolute and relative to the row's largest output, lse to 2e-3, on a
prefill-shaped batch (sampled rows, whole and split), the decode batch (split
over the CUs), entry granularity, and rows with padding or no valid id."""
import numpy as np
import pytest
import torch

import oracle
from workloads import attention_inputs, attention_kv_fp8, attention_q_rows, config, make_workload, synth_topk
from workloads.gen import MLA_ATTN

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _check(wl, pool8, sel, rows, got, gl, entry=1):
    ref, lref = oracle.sparse_attn_fp8kv(wl.q_start, wl.hist_len, rows, attention_q_rows(wl, rows), pool8,
                                         wl.page_table, wl.page_size, sel[rows], wl.attn_cfg["scale"], entry=entry)
    for j, g in enumerate(rows):
        if np.isneginf(lref[j]).all():
            assert np.all(got[g] == 0) and np.all(np.isneginf(gl[g])), (g,)
            continue
        err = np.abs(got[g] - ref[j]).max()
        assert err <= 2e-2 and err <= 2e-2 * np.abs(ref[j]).max(), (g, err)
    fin = np.isfinite(lref)
    assert np.allclose(gl[rows][fin], lref[fin], atol=2e-3)


@pytest.fixture(scope="module")
def prefill():
    wl = make_workload(hist_len=[30000, 5000], new_len=[400, 90], H=64, d=128, idx_dtype="fp8", k=2048, seed=41,
                       w_scale=1 / 8, table="permuted", attn=MLA_ATTN)
    sel = synth_topk(wl, seed=2, hot_frac=0.6, pad_rows=3)
    return wl, attention_kv_fp8(wl), sel


@pytest.mark.parametrize("splits", [1, 4])
def test_fp8kv_prefill(prefill, splits):
    wl, pool8, sel = prefill
    ai = attention_inputs(wl, with_q=True)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    out, lse = janus.sparse_attn_fp8kv(bt, T(ai.q), T(pool8), T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                       num_splits=splits, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, wl.total_q, 7), wl.q_start[1:] - 1])).astype(np.int32)
    _check(wl, pool8, sel, rows, out.cpu().numpy(), lse.cpu().numpy())


def test_fp8kv_decode_split():
    wl = config(5)
    pool8 = attention_kv_fp8(wl)
    ai = attention_inputs(wl)
    sel = synth_topk(wl, seed=12, hot_frac=0.8)
    sel[0, :] = -1  # a row with no valid id
    bt = janus.Batch(wl.hist_len, wl.new_len)
    out, lse = janus.sparse_attn_fp8kv(bt, T(ai.q), T(pool8), T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                       num_splits=0, out_dtype="f32", want_lse=True)
    torch.cuda.synchronize()
    _check(wl, pool8, sel, np.arange(wl.total_q, dtype=np.int32), out.cpu().numpy(), lse.cpu().numpy())


def test_fp8kv_entries_and_bf16_out():
    wl = make_workload(hist_len=[70000, 100], new_len=[300, 160], H=64, d=128, idx_dtype="fp8", k=512, seed=43,
                       w_scale=1 / 8, table="permuted", attn=MLA_ATTN, entry_shift=7)
    pool8 = attention_kv_fp8(wl)
    ai = attention_inputs(wl)
    sel = synth_topk(wl, seed=4, hot_frac=0.5)
    sel[:, :3] = np.random.default_rng(0).integers(0, int(wl.ctx_len.max()), size=(wl.total_q, 3))
    bt = janus.Batch(wl.hist_len, wl.new_len, entry_shift=7)
    out, lse = janus.sparse_attn_fp8kv(bt, T(ai.q), T(pool8), T(wl.page_table), wl.page_size, T(sel), ai.scale,
                                       want_lse=True)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()  # bf16 output: one more rounding, 2^-9 relative
    rows = np.unique(np.concatenate([np.arange(0, wl.total_q, 3), [wl.total_q - 1]])).astype(np.int32)
    _check(wl, pool8, sel, rows, got, lse.cpu().numpy(), entry=128)


def test_fp8kv_rejects_bad_rows():
    wl = config(5)
    bt = janus.Batch(wl.hist_len, wl.new_len)
    q = torch.zeros((wl.total_q, 128, 576), dtype=torch.bfloat16, device="cuda")
    pt = T(wl.page_table)
    sel = torch.zeros((wl.total_q, 64), dtype=torch.int32, device="cuda")
    short = torch.zeros((64, 584), dtype=torch.uint8, device="cuda")
    with pytest.raises(janus.JanusError):
        janus.sparse_attn_fp8kv(bt, q, short, pt, wl.page_size, sel, 0.1)
    odd = torch.zeros((64, 600), dtype=torch.uint8, device="cuda")  # not a multiple of 16
    with pytest.raises(janus.JanusError):
        janus.sparse_attn_fp8kv(bt, q, odd, pt, wl.page_size, sel, 0.1)
