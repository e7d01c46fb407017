"""MXFP4 indexer keys (DeepSeek-V4 keeps its indexer keys in FP4) on the GPU
against the CPU oracle.  Queries are fp8 e4m3fn with per-token scales; keys
are OCP MXFP4 (e2m1 elements, one E8M0 scale per 32) made by the generator.
Scores compare per row, max|g - r| / max|r| <= 1e-2 (the per-term bf16
rounding bounds the error by 2^-8), with the -inf pattern exact."""
import numpy as np
import pytest
import torch

import oracle
from workloads import make_workload, quantize_mxfp4

pytestmark = pytest.mark.gpu
janus = pytest.importorskip("paper_2609_36938_amd")


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _check_rows(wl, flat, rows, kI=None, bs=None):
    kI = wl.kI if kI is None else kI
    bs = wl.k_bscale if bs is None else bs
    ref = oracle.index_scores_mxfp4(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, kI, bs, wl.k_scale, wl.w,
                                    rows, out_ld=wl.max_ctx)
    b_of = wl.row_session(rows)
    for j, (g, b) in enumerate(zip(rows, b_of)):
        ctx = int(wl.ctx_len[b])
        i = int(g) - int(wl.q_start[b])
        st = int(wl.score_start[b]) + i * ctx
        got = flat[st: st + ctx].astype(np.float64)
        r = ref[j, :ctx]
        fin = np.isfinite(r)
        assert np.array_equal(fin, np.isfinite(got)), (g,)
        assert np.array_equal(fin, np.arange(ctx) <= int(wl.hist_len[b]) + i)
        err = np.abs(got[fin] - r[fin]).max()
        assert err <= 1e-2 * np.abs(r[fin]).max(), (g, err)


@pytest.mark.parametrize("hist,new", [([2000, 700, 64], [3, 130, 1]), ([5000], [1]), ([300, 9000], [2, 2]),
                                      ([4100, 17], [9, 4])])
def test_mxfp4_scores_exact_rows(hist, new):
    wl = make_workload(hist_len=hist, new_len=new, H=64, d=128, idx_dtype="fp8", k=64, seed=len(hist) + new[0],
                       w_scale=0.125, key_format="mxfp4")
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores_mxfp4(bt, T(wl.q), T(wl.kI), T(wl.k_bscale), T(wl.w), q_scale=T(wl.q_scale))
    torch.cuda.synchronize()
    _check_rows(wl, sc.cpu().numpy(), np.arange(wl.total_q, dtype=np.int32))


def test_mxfp4_wide_block_scales_and_key_scale():
    """Keys whose magnitudes span 2^-60 .. 2^40 (block scales far from 1) and a
    per-token key scale on top: no clamping or overflow in the epilogue."""
    wl = make_workload(hist_len=[3000], new_len=[5], H=64, d=128, idx_dtype="fp8", k=64, seed=77, w_scale=0.125,
                       key_format="mxfp4")
    rng = np.random.default_rng(5)
    kf = rng.standard_normal((wl.total_ctx, 128)).astype(np.float32)
    kf *= np.exp2(rng.choice([-60.0, -10.0, 0.0, 20.0, 40.0], size=(wl.total_ctx, 1))).astype(np.float32)
    kI, bs = quantize_mxfp4(kf)
    ks = rng.uniform(0.5, 2.0, wl.total_ctx).astype(np.float32)
    wl.k_scale = ks
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores_mxfp4(bt, T(wl.q), T(kI), T(bs), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(ks))
    torch.cuda.synchronize()
    _check_rows(wl, sc.cpu().numpy(), np.arange(wl.total_q, dtype=np.int32), kI, bs)


def test_mxfp4_block_scales_differ_within_a_key():
    """Each 32-element block of a key with its own magnitude (2^-60 .. 2^40,
    so a key's block scales differ by up to 2^100) and a key scale: the
    prefill kernel divides each key's block scales by the largest and
    multiplies it back into the key scale, which must leave every score as
    the oracle's."""
    wl = make_workload(hist_len=[2500, 700], new_len=[12, 7], H=64, d=128, idx_dtype="fp8", k=64, seed=78,
                       w_scale=0.125, key_format="mxfp4")
    rng = np.random.default_rng(6)
    kf = rng.standard_normal((wl.total_ctx, 128)).astype(np.float32)
    kf *= np.repeat(np.exp2(rng.choice([-60.0, -25.0, -5.0, 0.0, 15.0, 40.0], size=(wl.total_ctx, 4))), 32,
                    axis=1).astype(np.float32)
    kI, bs = quantize_mxfp4(kf)
    e = bs.astype(np.int32)
    assert (e.max(1) - e.min(1)).max() >= 90  # keys with far-apart block scales are present
    ks = rng.uniform(0.5, 2.0, wl.total_ctx).astype(np.float32)
    wl.k_scale = ks
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores_mxfp4(bt, T(wl.q), T(kI), T(bs), T(wl.w), q_scale=T(wl.q_scale), k_scale=T(ks))
    torch.cuda.synchronize()
    _check_rows(wl, sc.cpu().numpy(), np.arange(wl.total_q, dtype=np.int32), kI, bs)


def test_mxfp4_decode_batch():
    from workloads import decode_lengths
    M = decode_lengths(12, 4096, 40000, seed=9)
    wl = make_workload(hist_len=M, new_len=np.ones(12, np.int32), H=64, d=128, idx_dtype="fp8", k=2048, seed=9,
                       w_scale=0.125, key_format="mxfp4")
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores_mxfp4(bt, T(wl.q), T(wl.kI), T(wl.k_bscale), T(wl.w), q_scale=T(wl.q_scale))
    sel = janus.topk(bt, sc, wl.k)
    torch.cuda.synchronize()
    _check_rows(wl, sc.cpu().numpy(), np.arange(wl.total_q, dtype=np.int32))
    gs = sel.cpu().numpy()
    assert np.all(np.diff(gs, axis=1) > 0)  # every row has >= k candidates: k ascending distinct ids


def test_mxfp4_prefill_size_sampled_rows():
    wl = make_workload(hist_len=[32768], new_len=[2048], H=64, d=128, idx_dtype="fp8", k=2048, seed=1,
                       w_scale=0.125, key_format="mxfp4")
    bt = janus.Batch(wl.hist_len, wl.new_len)
    sc = janus.index_scores_mxfp4(bt, T(wl.q), T(wl.kI), T(wl.k_bscale), T(wl.w), q_scale=T(wl.q_scale))
    torch.cuda.synchronize()
    _check_rows(wl, sc.cpu().numpy(), np.array([0, 1, 2, 3, 777, 1500, 2044, 2045, 2046, 2047], dtype=np.int32))
