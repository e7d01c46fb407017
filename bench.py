"""Benchmark: one layer's append-prefill hot path on one MI355X.

Workload: history M = 131072 tokens + N = 8192 appended tokens, lightning
indexer 64 heads x 128 dims in fp8 e4m3fn with per-token scales, k = 2048,
64-token pages behind a seeded random page table, sparse MLA attention with
128 query heads over 576-dim bf16 latent+rope rows (V = first 512 dims).

A step is the whole path for the layer on one stream:
    janus_index_scores -> janus_topk -> janus_page_demand (bitmap, list, runs)
    -> janus_predict_diff (against the predicted set of this layer, produced
       before the timed region by the same three calls on the predicted
       query, as a lookahead run at an earlier layer would have)
    -> janus_sparse_attn.
value = appended tokens per second per layer (N * steps / time).

Printed as one JSON line (see the keys below), with the roofline of the
dominant kernel (index scores, fp8 MFMA) from HIP events on the launch stream
(medians over the timed steps), and the CPU oracle timed on bounded row
samples on the host cores, multi- and single-threaded.  Further fields (left
out by --core-only): the attention with selections spread over the pool, the
sharded-prediction sweep (Eq. 3) on workloads whose selection does not
saturate, the predicted path of Eq. 2 over 8 layers of the prediction
workload, the decode step, an IndexShare group and the attention over FP8 KV.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP8 = 5.0e15      # dense fp8 MFMA, FLOP/s
PEAK_BF16 = 2.5e15     # dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12      # bytes/s


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode", action="store_true", help="skip the decode-phase measurement")
    p.add_argument("--core-only", action="store_true",
                   help="time the one-layer step only: no sharded sweep, decode, IndexShare or fp8-KV fields "
                        "(for profiler passes)")
    p.add_argument("--cpu-rows", type=int, default=128, help="query rows in the oracle's multi-threaded sample")
    p.add_argument("--cpu-rows-1t", type=int, default=16, help="query rows in the oracle's single-threaded sample")
    p.add_argument("--spread-only", action="store_true",
                   help="time only the attention with selections spread over the whole pool (one JSON field), "
                        "for the HBM counter passes of that kernel")
    p.add_argument("--c4-layers", type=int, default=8,
                   help="layers of the prediction workload (history 131072 + 4096) in the predicted-path field")
    p.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "index_scores_traffic.json"))
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (known bytes) for HBM counter calibration")
    p.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="write --traffic from the counter_collection CSVs of a FETCH_SIZE and a WRITE_SIZE "
                        "rocprofv3 pass over 'bench.py --copy-calibration', then exit (no GPU needed)")
    return p.parse_args()


def main():
    args = parse()
    if args.record_traffic:
        record_traffic(*args.record_traffic, args.traffic)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path, so --gpus must be 1.",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2609_36938_amd as janus
    from workloads import attention_inputs, config

    t_gen = time.time()
    wl = config(2, with_pred=True)
    ai = attention_inputs(wl)
    t_gen = time.time() - t_gen
    dev = torch.device("cuda:0")
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bt = janus.Batch(wl.hist_len, wl.new_len, device=dev)
    q, kI, w, sq, sk = T(wl.q), T(wl.kI), T(wl.w), T(wl.q_scale), T(wl.k_scale)
    qp, sqp = T(wl.q_pred), T(wl.q_pred_scale)
    pt = T(wl.page_table)
    qa = T(ai.q)
    kv = T(ai.k_pool)
    P, ps, k, mr = wl.num_phys_pages, wl.page_size, wl.k, wl.max_run
    N, M = wl.total_q, int(wl.hist_len[0])
    if args.spread_only:
        print(json.dumps({"sparse_attn_spread": spread_attention(janus, torch, wl, bt, qa, kv, pt, ai,
                                                                 max(args.steps, 5))}))
        return

    scores = torch.empty(bt.total_scores, dtype=torch.float32, device=dev)
    sel = torch.empty((N, k), dtype=torch.int32, device=dev)
    nw = (P + 31) // 32
    pd_out = (torch.empty(nw, dtype=torch.int32, device=dev), torch.empty(P, dtype=torch.int32, device=dev),
              torch.empty(2 * P, dtype=torch.int32, device=dev), torch.empty(2, dtype=torch.int32, device=dev))
    diff_out = (torch.empty(nw, dtype=torch.int32, device=dev), torch.empty(2 * P, dtype=torch.int32, device=dev),
                torch.empty(5, dtype=torch.int32, device=dev))
    out = torch.empty((N, ai.Hq, ai.dv), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((N, ai.Hq), dtype=torch.float32, device=dev)

    # predicted set of this layer (lookahead run, outside the timed region)
    janus.index_scores(bt, qp, kI, w, q_scale=sqp, k_scale=sk, scores=scores)
    sel_p = janus.topk(bt, scores, k)
    pred_bm = janus.page_demand(bt, sel_p, pt, ps, P, mr)[0].clone()
    torch.cuda.synchronize()

    names = ["index_scores", "topk", "page_demand", "predict_diff", "sparse_attn"]

    def step(ev=None):
        if ev:
            ev[0].record()
        janus.index_scores(bt, q, kI, w, q_scale=sq, k_scale=sk, scores=scores)
        if ev:
            ev[1].record()
        janus.topk(bt, scores, k, out=sel)
        if ev:
            ev[2].record()
        janus.page_demand(bt, sel, pt, ps, P, mr, out=pd_out)
        if ev:
            ev[3].record()
        janus.predict_diff(pd_out[0], pred_bm, P, mr, out=diff_out)
        if ev:
            ev[4].record()
        janus.sparse_attn(bt, qa, kv, kv, pt, ps, sel, ai.scale, dv=ai.dv, out=out, lse=lse)
        if ev:
            ev[5].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)  # reads 1 GiB, writes 1 GiB
        torch.cuda.synchronize()
        del src, dst
    print(f"# inputs generated in {t_gen:.1f}s; warmup done", file=sys.stderr, flush=True)

    # timed region: K steps, bracketed by synchronisation
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # per-kernel durations: HIP events on the launch stream, separate pass
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    for e in evs:
        step(e)
    torch.cuda.synchronize()
    # median over the timed steps (the mean is kept beside it)
    per = {n: float(np.median([e[j].elapsed_time(e[j + 1]) for e in evs])) for j, n in enumerate(names)}
    per_mean = {n: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in evs])) for j, n in enumerate(names)}

    # algorithmic work
    pairs = N * (M + 1) + N * (N - 1) // 2                  # causal (token, candidate) pairs
    idx_flop = 2.0 * wl.H * wl.d * pairs
    topk_bytes = 4.0 * pairs + 4.0 * N * k
    attn_rows = N * k                                         # every row of this workload selects k ids
    gather_bytes = attn_rows * ai.dqk * 2.0
    attn_flop = 2.0 * N * ai.Hq * k * (ai.dqk + ai.dv)
    t_idx = per["index_scores"] * 1e-3
    ach = idx_flop / t_idx
    traffic = measured_traffic(args.traffic)

    ms_step = wall / args.steps * 1e3
    counts = diff_out[2].cpu().tolist()
    extras = not args.core_only
    spread = spread_attention(janus, torch, wl, bt, qa, kv, pt, ai, max(args.steps, 5)) if extras else None
    mxfp4 = mxfp4_prefill(janus, torch, bt, scores, max(args.steps, 5), per["index_scores"], idx_flop) \
        if extras else None
    sweep = prediction_sweep(janus, torch, max(args.steps, 5)) if extras else None
    predicted = predicted_path(janus, torch, args.c4_layers) if extras and args.c4_layers > 0 else None
    decode = decode_step(janus, torch, max(args.steps, 5)) if extras and not args.no_decode else None
    kv8 = fp8kv_attention(janus, torch, bt, qa, kv, pt, ps, sel, ai, max(args.steps, 5), per["sparse_attn"]) \
        if extras else None
    share = indexshare_group(janus, torch, step_calls=(bt, q, kI, w, sq, sk, pt, ps, P, mr, k, scores, sel, qa, kv,
                                                       pd_out, diff_out, pred_bm, out, lse, ai),
                             steps=max(args.steps, 3)) if extras else None
    peaks = measured_peaks(torch) if extras else None
    rec = {
        "metric": "new tokens/s per layer (indexer+top-k+sparse attn) at 128K history; % MFMA/HBM peak",
        "value": N * args.steps / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8+bf16",
        "data": "synthetic",
        "config": {"workload": "DeepSeek-V3.2-shaped layer, history 131072 + 8192 new tokens, k=2048, "
                               "64-token pages behind a random page table",
                   "history": M, "new_tokens": N, "indexer": "64 heads x 128 fp8 e4m3fn, per-token scales",
                   "k": k, "page_size": ps, "attention": "MLA-MQA 128 heads, 576/512 bf16"},
        "roofline": {"bound": "mfma", "kernel": "index_scores", "achieved": ach / 1e12, "peak": PEAK_FP8 / 1e12,
                     "unit": "TFLOP/s", "frac": ach / PEAK_FP8, "traffic": traffic},
        "kernels_ms": per,
        "kernels_ms_mean": per_mean,
        "kernel_rates": {
            "index_scores_TFLOPs": idx_flop / t_idx / 1e12,
            "topk_GBps": topk_bytes / (per["topk"] * 1e-3) / 1e9,
            "topk_frac_hbm": topk_bytes / (per["topk"] * 1e-3) / PEAK_HBM,
            "sparse_attn_gather_GBps_logical": gather_bytes / (per["sparse_attn"] * 1e-3) / 1e9,
            "sparse_attn_gather_frac_hbm": gather_bytes / (per["sparse_attn"] * 1e-3) / PEAK_HBM,
            "sparse_attn_TFLOPs": attn_flop / (per["sparse_attn"] * 1e-3) / 1e12,
            "sparse_attn_frac_bf16_mfma": attn_flop / (per["sparse_attn"] * 1e-3) / PEAK_BF16,
        },
        "demand": {"pages": int(pd_out[3][0]), "runs": int(pd_out[3][1]), "pred_counts": counts},
        "sparse_attn_spread": spread,
        "mxfp4_prefill": mxfp4,
        "prediction_sweep": sweep,
        "predicted_path": predicted,
        "decode": decode,
        "indexshare": share,
        "fp8_kv": kv8,
        "measured_peaks": peaks,
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, ai, args.cpu_rows, args.cpu_rows_1t, sel.cpu().numpy(),
                                           pred_bm.cpu().numpy().view(np.uint32))
    print(json.dumps(rec))


def measured_traffic(path):
    """HBM bytes per launch of the index-scores kernel from the committed
    FETCH_SIZE / WRITE_SIZE passes, or None when the kernel's sources have
    changed since those counters were taken."""
    import hashlib
    try:
        tr = json.load(open(path))
        h = hashlib.sha256()
        for f in tr["sources"]:
            h.update(open(os.path.join(ROOT, f), "rb").read())
        return tr["bytes_per_launch"] if h.hexdigest() == tr["sources_sha256"] else None
    except (OSError, KeyError, ValueError):
        return None


TRAFFIC_SOURCES = ["paper_2609_36938_amd/csrc/index_scores.hip", "paper_2609_36938_amd/csrc/janus_device.hpp"]


def record_traffic(fetch_csv, write_csv, out_path):
    """HBM bytes per launch of the index-scores kernel from one FETCH_SIZE and
    one WRITE_SIZE pass, each counter scaled by what it reads for the 1 GiB
    copy (1 GiB read, 1 GiB written) that --copy-calibration adds; stored with
    the sha256 of the kernel's sources so that a later change voids it."""
    import csv
    import hashlib

    def per_kernel(path, counter):
        acc = {}
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return acc

    fetch, write = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    gib_kib = float(1 << 20)
    copy_f = max(v for k, vs in fetch.items() if "copyBuffer" in k for v in vs)
    copy_w = max(v for k, vs in write.items() if "copyBuffer" in k for v in vs)
    fs, ws = round(gib_kib / copy_f, 2), round(gib_kib / copy_w, 2)
    name = next(k for k in fetch if "index_scores_fp8_mfma" in k)
    f_kib = float(np.mean(fetch[name]))
    w_kib = float(np.mean(write[name]))
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    rec = {"kernel": name.split("(")[0].replace("void ", ""),
           "workload": "history 131072 + 8192 new tokens, 64 heads x 128 fp8",
           "fetch_kib_raw": f_kib, "write_kib_raw": w_kib, "fetch_scale": fs, "write_scale": ws,
           "fetch_bytes": f_kib * 1024 * fs, "write_bytes": w_kib * 1024 * ws,
           "bytes_per_launch": f_kib * 1024 * fs + w_kib * 1024 * ws,
           "copy_calibration_kib": {"fetch": copy_f, "write": copy_w},
           "sources": TRAFFIC_SOURCES, "sources_sha256": h.hexdigest()}
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def _pct(a, b):
    return a / b if b else 1.0


def spread_attention(janus, torch, wl, bt, qa, kv, pt, ai, steps):
    """The 128K attention with selections spread over the whole causal range
    (every row's 2048 ids uniform over its candidates, no hot spans), so that
    the gathered rows cover the whole 160 MB pool instead of ~111 hot pages.
    Same queries and pool as the step."""
    from workloads import synth_topk
    sel = torch.from_numpy(synth_topk(wl, seed=5, hot_frac=0.0)).to(qa.device)
    out = torch.empty((bt.total_q, ai.Hq, ai.dv), dtype=torch.bfloat16, device=qa.device)
    f = lambda: janus.sparse_attn(bt, qa, kv, kv, pt, wl.page_size, sel, ai.scale, dv=ai.dv, out=out)
    f()
    torch.cuda.synchronize()
    ts = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        f()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = float(np.median(ts))
    gather = bt.total_q * sel.shape[1] * ai.dqk * 2.0
    return {"workload": "sparse attention of the 128K workload, each row's 2048 ids uniform over its causal "
                        "range (the whole 160 MB pool is gathered)",
            "ms": ms, "gather_GBps_logical": gather / (ms * 1e-3) / 1e9,
            "gather_frac_hbm": gather / (ms * 1e-3) / PEAK_HBM}


def mxfp4_prefill(janus, torch, bt, scores, steps, fp8_ms, flop):
    """The indexer of the 128K workload with its keys in MXFP4 (DeepSeek-V4
    keeps indexer keys in FP4, Sec. 5.1): the same draws quantised to e2m1
    codes with one E8M0 scale per 32 elements, fp8 queries; times the
    prefill kernel against the fp8-key indexer of the step."""
    from workloads import make_workload
    wl = make_workload(hist_len=[131072], new_len=[8192], H=64, d=128, idx_dtype="fp8", k=2048, seed=2,
                       w_scale=1.0 / 8, key_format="mxfp4")
    dev = scores.device
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    q, kI, bs, w, sq = T(wl.q), T(wl.kI), T(wl.k_bscale), T(wl.w), T(wl.q_scale)
    f = lambda: janus.index_scores_mxfp4(bt, q, kI, bs, w, q_scale=sq, scores=scores)
    f()
    torch.cuda.synchronize()
    ts = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        f()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = float(np.median(ts))
    return {"workload": "index scores of the 128K workload with MXFP4 keys (64 B of e2m1 + 4 E8M0 scales per key)",
            "ms": ms, "TFLOPs": flop / ms / 1e9, "frac_fp8_peak": flop / (ms * 1e-3) / PEAK_FP8,
            "fp8_keys_ms": fp8_ms, "ratio_to_fp8_keys": ms / fp8_ms}


SWEEP_LAYOUTS = (("hot spans 1% of the history (fewer tokens than k), one in each eighth", 0.01, "even"),
                 ("hot spans 5% of the history, all in its most recent quarter", 0.05, "recent"))


def prediction_sweep(janus, torch, steps):
    """Synchronization-free sharded prediction (Eq. 3) against the exact
    selection, for G = 1, 2, 4, 8 history shards, on workloads where the
    selection does not saturate: one session, history 131072, 64 appended
    tokens, the 64 x 128 fp8 indexer, k = 2048, predicted queries
    0.9 q + sqrt(0.19) N(0, 1).  Recall = |A & P| / |A| and precision =
    |A & P| / |P| (Sec. 4.2) of the history sets, at token granularity and at
    64-token pages (identity page table); the sharded top-k time is for all G
    shards on this GPU (one GPU's share is 1/G of it)."""
    from workloads import make_workload
    dev = torch.device("cuda:0")
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    out = []
    for name, frac, layout in SWEEP_LAYOUTS:
        wl = make_workload(hist_len=[131072], new_len=[64], H=64, d=128, idx_dtype="fp8", k=2048, seed=7,
                           w_scale=1.0 / 8, table="identity", q_pred_corr=0.9, hot_frac=frac, hot_layout=layout)
        bt = janus.Batch(wl.hist_len, wl.new_len, device=dev)
        kI, w, sk = T(wl.kI), T(wl.w), T(wl.k_scale)
        M, ctx = int(wl.hist_len[0]), int(wl.ctx_len[0])
        levels = {"token": (1, T(np.arange(ctx, dtype=np.int32)[None, :]), ctx),
                  "page64": (64, T(wl.page_table), wl.num_phys_pages)}
        sc = janus.index_scores(bt, T(wl.q), kI, w, q_scale=T(wl.q_scale), k_scale=sk)
        sel = janus.topk(bt, sc, wl.k)
        actual = {lv: janus.page_demand(bt, sel, tab, psz, npg, 32)[0].clone()
                  for lv, (psz, tab, npg) in levels.items()}
        janus.index_scores(bt, T(wl.q_pred), kI, w, q_scale=T(wl.q_pred_scale), k_scale=sk, scores=sc)
        rows = {}
        for G in (1, 2, 4, 8):
            janus.topk_sharded(bt, sc, wl.k, G, 64)
            ts = []
            for _ in range(steps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                psel = janus.topk_sharded(bt, sc, wl.k, G, 64)
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            r = {"topk_sharded_ms": float(np.median(ts))}
            for lv, (psz, tab, npg) in levels.items():
                bm = janus.page_demand(bt, psel, tab, psz, npg, 32)[0]
                c = janus.predict_diff(actual[lv], bm, npg, 32)[2].cpu().tolist()
                r[lv] = {"actual": c[0], "predicted": c[1], "recall": _pct(c[2], c[0]),
                         "precision": _pct(c[2], c[1]), "miss": c[3], "miss_runs": c[4]}
            rows[str(G)] = r
        out.append({"workload": name, "history": M, "new_tokens": int(wl.total_q), "k": wl.k, "shards": rows})
        del sc, sel, kI
    return out


def predicted_path(janus, torch, layers):
    """The prediction workload over several layers: history 131072 + 4096
    appended tokens, the 64 x 128 fp8 indexer with the same hot-span positions
    in every layer, k = 2048, identity page table, max run 32.  Per layer the
    actual path (scores -> top-k -> page demand and runs -> sparse MLA
    attention over the actual set) and the predicted path of Eq. 2 (scores ->
    top-k -> page demand on q_pred = 0.9 q + sqrt(0.19) N(0, 1)) and the
    corrective set (predict_diff).  Indexer inputs come from the shared
    generator; attention queries and the KV pool of each layer are drawn on
    the GPU from a seeded generator (nothing here is compared with the
    oracle).  Times are medians of HIP-event timings over two passes."""
    from workloads import config
    dev = torch.device("cuda:0")
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(4)
    L = []
    for layer in range(layers):
        wl = config(4, layer=layer)
        L.append(dict(q=T(wl.q), sq=T(wl.q_scale), qp=T(wl.q_pred), sqp=T(wl.q_pred_scale), kI=T(wl.kI),
                      sk=T(wl.k_scale), w=T(wl.w),
                      qa=torch.randn((wl.total_q, 128, 576), generator=g, device=dev).to(torch.bfloat16),
                      kv=(torch.randn((wl.num_phys_pages * wl.page_size, 576), generator=g, device=dev)
                          / 24.0).to(torch.bfloat16)))
    bt = janus.Batch(wl.hist_len, wl.new_len, device=dev)
    pt, P, ps, k, mr = T(wl.page_table), wl.num_phys_pages, wl.page_size, wl.k, wl.max_run
    scores = torch.empty(bt.total_scores, dtype=torch.float32, device=dev)
    sel = torch.empty((bt.total_q, k), dtype=torch.int32, device=dev)
    psel = torch.empty_like(sel)
    out = torch.empty((bt.total_q, 128, 512), dtype=torch.bfloat16, device=dev)
    mk = lambda: (torch.empty((P + 31) // 32, dtype=torch.int32, device=dev),
                  torch.empty(P, dtype=torch.int32, device=dev),
                  torch.empty(2 * P, dtype=torch.int32, device=dev), torch.empty(2, dtype=torch.int32, device=dev))
    pd_a, pd_p = mk(), mk()
    diff = (torch.empty((P + 31) // 32, dtype=torch.int32, device=dev),
            torch.empty(2 * P, dtype=torch.int32, device=dev), torch.empty(5, dtype=torch.int32, device=dev))
    ev = lambda: torch.cuda.Event(enable_timing=True)
    per_layer = []
    for rep in range(2):
        for li, x in enumerate(L):
            e = [ev() for _ in range(10)]
            e[0].record()
            janus.index_scores(bt, x["q"], x["kI"], x["w"], q_scale=x["sq"], k_scale=x["sk"], scores=scores)
            e[1].record()
            janus.topk(bt, scores, k, out=sel)
            e[2].record()
            janus.page_demand(bt, sel, pt, ps, P, mr, out=pd_a)
            e[3].record()
            janus.sparse_attn(bt, x["qa"], x["kv"], x["kv"], pt, ps, sel, 1.0 / 24.0, dv=512, out=out)
            e[4].record()
            janus.index_scores(bt, x["qp"], x["kI"], x["w"], q_scale=x["sqp"], k_scale=x["sk"], scores=scores)
            e[5].record()
            janus.topk(bt, scores, k, out=psel)
            e[6].record()
            janus.page_demand(bt, psel, pt, ps, P, mr, out=pd_p)
            e[7].record()
            janus.predict_diff(pd_a[0], pd_p[0], P, mr, out=diff)
            e[8].record()
            torch.cuda.synchronize()
            d = [e[j].elapsed_time(e[j + 1]) for j in range(8)]
            c = diff[2].cpu().tolist()
            if rep == 0:
                per_layer.append({"t": [], "counts": c, "runs": int(pd_a[3][1])})
            per_layer[li]["t"].append(d)
    names = ["index_scores", "topk", "page_demand", "sparse_attn", "pred_index_scores", "pred_topk",
             "pred_page_demand", "predict_diff"]
    layers_out = []
    for li, rec in enumerate(per_layer):
        t = np.median(np.array(rec["t"]), axis=0)
        actual, pred = float(t[0] + t[1] + t[2] + t[3]), float(t[4] + t[5] + t[6])
        c = rec["counts"]
        layers_out.append({"layer": li, "actual_path_ms": actual, "predicted_path_ms": pred,
                           "predict_diff_ms": float(t[7]), "prediction_overhead": (pred + float(t[7])) / actual,
                           "actual_pages": c[0], "predicted_pages": c[1], "recall": _pct(c[2], c[0]),
                           "precision": _pct(c[2], c[1]), "miss_pages": c[3], "miss_runs": c[4],
                           "actual_runs": rec["runs"], "kernels_ms": dict(zip(names, map(float, t)))})
    mean = lambda key: float(np.mean([r[key] for r in layers_out]))
    # the first layer again behind a seeded random page table: the same sets
    # of pages up to the permutation, but adjacent logical pages are no longer
    # adjacent physically, so runs shrink to single pages
    perm = torch.randperm(P, generator=g, device=dev).to(torch.int32).reshape(1, P)
    x = L[0]
    janus.index_scores(bt, x["q"], x["kI"], x["w"], q_scale=x["sq"], k_scale=x["sk"], scores=scores)
    janus.topk(bt, scores, k, out=sel)
    janus.page_demand(bt, sel, perm, ps, P, mr, out=pd_a)
    janus.index_scores(bt, x["qp"], x["kI"], x["w"], q_scale=x["sqp"], k_scale=x["sk"], scores=scores)
    janus.topk(bt, scores, k, out=psel)
    janus.page_demand(bt, psel, perm, ps, P, mr, out=pd_p)
    janus.predict_diff(pd_a[0], pd_p[0], P, mr, out=diff)
    torch.cuda.synchronize()
    c = diff[2].cpu().tolist()
    permuted = {"layer": 0, "actual_pages": c[0], "actual_runs": int(pd_a[3][1]), "predicted_pages": c[1],
                "recall": _pct(c[2], c[0]), "precision": _pct(c[2], c[1]), "miss_pages": c[3], "miss_runs": c[4]}
    return {"workload": f"{layers} layers, history 131072 + 4096 new tokens, k=2048, identity page table, "
                        "q_pred = 0.9 q + sqrt(0.19) N(0,1)",
            "per_layer_actual_ms": mean("actual_path_ms"), "per_layer_predicted_ms": mean("predicted_path_ms"),
            "per_layer_predict_diff_ms": mean("predict_diff_ms"),
            "prediction_overhead": mean("prediction_overhead"), "layers": layers_out,
            "permuted_table": permuted}


def measured_peaks(torch, reps=5):
    """What this GPU reaches on plain library work, beside the published
    peaks the rooflines use: a 2 GiB device copy (HBM read + write) and a sum
    over the same 2 GiB (read only), and
    8192^3 GEMMs through hipBLASLt in fp8 e4m3 (torch._scaled_mm, bf16 out)
    and bf16 (torch.matmul).  Medians of HIP-event timings."""
    dev = torch.device("cuda:0")

    def timed(f):
        f()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            f()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts)) * 1e-3

    out = {}
    try:
        src = torch.empty(1 << 29, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        t = timed(lambda: dst.copy_(src))
        out["hbm_copy_TBps"] = 2.0 * src.numel() * 4 / t / 1e12
        t = timed(lambda: torch.sum(src))
        out["hbm_read_TBps"] = src.numel() * 4 / t / 1e12
        del src, dst
    except RuntimeError as e:
        out["hbm_copy_TBps"] = None
        out["hbm_copy_error"] = str(e)[:200]
    n = 8192
    try:
        g = torch.Generator(device=dev)
        g.manual_seed(0)
        a = torch.randn((n, n), generator=g, device=dev).to(torch.float8_e4m3fn)
        b = torch.randn((n, n), generator=g, device=dev).to(torch.float8_e4m3fn).t()
        one = torch.ones((), device=dev)
        t = timed(lambda: torch._scaled_mm(a, b, scale_a=one, scale_b=one, out_dtype=torch.bfloat16))
        out["fp8_gemm_TFLOPs"] = 2.0 * n ** 3 / t / 1e12
        del a, b
    except (RuntimeError, AttributeError, TypeError) as e:
        out["fp8_gemm_TFLOPs"] = None
        out["fp8_gemm_error"] = str(e)[:200]
    try:
        a = torch.randn((n, n), device=dev, dtype=torch.bfloat16)
        b = torch.randn((n, n), device=dev, dtype=torch.bfloat16)
        t = timed(lambda: torch.matmul(a, b))
        out["bf16_gemm_TFLOPs"] = 2.0 * n ** 3 / t / 1e12
        del a, b
    except RuntimeError as e:
        out["bf16_gemm_TFLOPs"] = None
        out["bf16_gemm_error"] = str(e)[:200]
    return out


def fp8kv_attention(janus, torch, bt, qa, kv, pt, ps, sel, ai, steps, bf16_ms):
    """Attention of the 128K workload over the KV cache kept in FP8 (Sec. 5.1):
    the bf16 pool quantised on the GPU, one fp32 scale per row (amax/448),
    rows of 576 e4m3 bytes + the scale, 592 bytes.  Same queries and ids."""
    rows = kv.shape[0] * kv.shape[1]
    x = kv.reshape(rows, -1).float()
    scale = (x.abs().amax(dim=1).clamp_min(1e-12) / 448.0).float()
    pool8 = torch.zeros((rows, 592), dtype=torch.uint8, device=kv.device)
    pool8[:, :576] = (x / scale[:, None]).to(torch.float8_e4m3fn).view(torch.uint8)
    pool8[:, 576:580] = scale.view(torch.uint8).reshape(rows, 4)
    del x
    out = torch.empty((bt.total_q, ai.Hq, ai.dv), dtype=torch.bfloat16, device=kv.device)
    ws = torch.empty(1, dtype=torch.uint8, device=kv.device)
    f = lambda: janus.sparse_attn_fp8kv(bt, qa, pool8, pt, ps, sel, ai.scale, out=out, workspace=ws)
    f()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        f()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    gather = bt.total_q * sel.shape[1] * 592.0
    return {"workload": "sparse attention of the 128K workload over fp8 KV rows (576 e4m3 + fp32 scale)",
            "ms": ms, "bf16_ms": bf16_ms, "speedup_vs_bf16": bf16_ms / ms,
            "gather_GBps_logical": gather / (ms * 1e-3) / 1e9,
            "gather_frac_hbm": gather / (ms * 1e-3) / PEAK_HBM}


def indexshare_group(janus, torch, step_calls, steps):
    """IndexShare (GLM-5 series, Sec. 2.2): four consecutive sparse-attention
    layers share one selection, and only the first runs the indexer and top-k.
    One group at the 128K workload: scores -> top-k -> page demand ->
    corrective set (once: the four layers' KV pools share the page table, so
    their page sets coincide) -> attention of four layers, each over its own
    queries and KV pool (layers 1-3 drawn on the GPU from a seeded generator)
    with the shared ids.  Reported per layer: the group's time over four."""
    (bt, q, kI, w, sq, sk, pt, ps, P, mr, k, scores, sel, qa, kv, pd_out, diff_out, pred_bm, out, lse, ai) = step_calls
    dev = qa.device
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    layers = [(qa, kv)]
    for _ in range(3):
        layers.append((torch.randn(qa.shape, generator=g, device=dev).to(torch.bfloat16),
                       (torch.randn(kv.shape, generator=g, device=dev) / 24.0).to(torch.bfloat16)))

    def group():
        janus.index_scores(bt, q, kI, w, q_scale=sq, k_scale=sk, scores=scores)
        janus.topk(bt, scores, k, out=sel)
        janus.page_demand(bt, sel, pt, ps, P, mr, out=pd_out)
        janus.predict_diff(pd_out[0], pred_bm, P, mr, out=diff_out)
        for ql, kvl in layers:
            janus.sparse_attn(bt, ql, kvl, kvl, pt, ps, sel, ai.scale, dv=ai.dv, out=out, lse=lse)

    group()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        group()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / steps * 1e3
    del layers
    N = bt.total_q
    return {"workload": "4 sparse layers sharing one selection (IndexShare) at the 128K workload",
            "layers": 4, "ms_per_group": ms, "ms_per_layer": ms / 4,
            "value": N / (ms / 4) * 1e3, "unit": "new tokens/s per layer"}


def decode_step(janus, torch, steps):
    """The decode phase (Sec. 2.2) at one layer: 64 sessions with histories
    log-uniform in 32K-160K tokens, one new token each.  A step is scores ->
    top-k -> page demand -> load set (demand minus the resident pages, 90% of
    the pool) -> attention split over the CUs.  Indexer inputs come from the
    shared generator; the KV pool (80K pages, 6 GB) and the attention queries
    are drawn on the GPU from a seeded generator, since nothing here is
    compared with the oracle."""
    from workloads import decode_lengths, make_workload, resident_pages

    B, k = 64, 2048
    M = decode_lengths(B, 32768, 163840, seed=6)
    wl = make_workload(hist_len=M, new_len=np.ones(B, np.int32), H=64, d=128, idx_dtype="fp8", k=k, seed=6,
                       w_scale=1.0 / 8, table="permuted", name="decode-64")
    dev = torch.device("cuda:0")
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bt = janus.Batch(wl.hist_len, wl.new_len, device=dev)
    q, kI, w, sq, sk, pt = T(wl.q), T(wl.kI), T(wl.w), T(wl.q_scale), T(wl.k_scale), T(wl.page_table)
    res = T(resident_pages(wl, p=0.9).view(np.int32))
    g = torch.Generator(device=dev)
    g.manual_seed(6)
    P, ps = wl.num_phys_pages, wl.page_size
    pool = (torch.randn((P * ps, 576), generator=g, device=dev) / 24.0).to(torch.bfloat16)
    qa = torch.randn((B, 128, 576), generator=g, device=dev).to(torch.bfloat16)
    scores = torch.empty(wl.total_scores, dtype=torch.float32, device=dev)
    sel = torch.empty((B, k), dtype=torch.int32, device=dev)
    out = torch.empty((B, 128, 512), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(B * 16 * 128 * 514 * 4, dtype=torch.uint8, device=dev)
    pd = janus.page_demand(bt, sel, pt, ps, P, wl.max_run)
    calls = [
        ("index_scores", lambda: janus.index_scores(bt, q, kI, w, q_scale=sq, k_scale=sk, scores=scores)),
        ("topk", lambda: janus.topk(bt, scores, k, out=sel)),
        ("page_demand", lambda: janus.page_demand(bt, sel, pt, ps, P, wl.max_run, out=pd)),
        ("load_set", lambda: janus.predict_diff(pd[0], res, P, wl.max_run)),
        ("sparse_attn_split", lambda: janus.sparse_attn_split(bt, qa, pool, pool, pt, ps, sel, 1.0 / 24.0,
                                                              num_splits=0, dv=512, out=out, workspace=ws)),
    ]
    for _, f in calls:  # warm-up
        f()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        for _, f in calls:
            f()
    torch.cuda.synchronize()
    step_ms = (time.perf_counter() - t0) / steps * 1e3
    kms = {}
    for name, f in calls:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            f()
        e1.record()
        torch.cuda.synchronize()
        kms[name] = e0.elapsed_time(e1) / steps
    counts = janus.predict_diff(pd[0], res, P, wl.max_run)[2].cpu().tolist()
    idx_bytes = wl.kI.nbytes + wl.k_scale.nbytes + wl.total_scores * 4
    gather = B * k * 1152
    return {
        "workload": f"{B} decoding sessions, histories log-uniform in 32K-160K (mean {int(M.mean())}), one new "
                    f"token each, k={k}, 90% of the pool resident",
        "unit": "decode tokens/s per layer", "value": B / step_ms * 1e3, "ms_per_step": step_ms, "kernels_ms": kms,
        "index_scores_GBps": idx_bytes / kms["index_scores"] / 1e6,
        "index_scores_frac_hbm": idx_bytes / kms["index_scores"] / 1e6 / (PEAK_HBM / 1e9),
        "sparse_attn_gather_GBps_logical": gather / kms["sparse_attn_split"] / 1e6,
        "demand_pages": counts[0], "load_pages": counts[3],
    }


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, ai, nrows, nrows_1t, gpu_sel, pred_bm):
    """The oracle, untuned, on stride samples of query rows of the same
    workload: scores over all candidates, top-k and attention for each sampled
    row, timed stage by stage; page demand, runs and the corrective set over
    the full selection (the GPU's ids, as in the parity tests).  Run with this
    process's OpenMP thread count (OMP_NUM_THREADS, else the CPUs this
    process may use) and again single-threaded on a smaller sample.
    tokens/s = 1 / (row-stage seconds per row + set-stage seconds / N)."""
    import ctypes

    import oracle
    from workloads import attention_q_rows

    oracle.lib()
    gomp = ctypes.CDLL("libgomp.so.1")
    threads = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))
    P = wl.num_phys_pages

    def run(n, nthreads, with_sets):
        gomp.omp_set_num_threads(nthreads)
        rows = np.linspace(0, wl.total_q - 1, n).astype(np.int32)
        qr = attention_q_rows(wl, rows)
        t0 = time.perf_counter()
        sc = oracle.index_scores(wl.q_start, wl.hist_len, wl.q, "fp8", wl.q_scale, wl.kI, "fp8", wl.k_scale, wl.w,
                                 rows)
        t1 = time.perf_counter()
        sel = oracle.topk(wl.q_start, wl.hist_len, rows, sc.astype(np.float32), wl.k)
        t2 = time.perf_counter()
        oracle.sparse_attn(wl.q_start, wl.hist_len, rows, qr, ai.k_pool, None, ai.k_row_stride, ai.v_row_stride,
                           wl.page_table, wl.page_size, sel, ai.scale, ai.dv)
        t3 = time.perf_counter()
        stages = {"index_scores": (t1 - t0) / n, "topk": (t2 - t1) / n, "sparse_attn": (t3 - t2) / n}
        sets = 0.0
        if with_sets:
            s0 = time.perf_counter()
            bm, _, _ = oracle.page_demand(wl.q_start, wl.hist_len, gpu_sel, wl.page_table, wl.page_size, P)
            oracle.runs(bm, P, wl.max_run)
            oracle.predict_diff(bm, pred_bm, P, wl.max_run)
            sets = time.perf_counter() - s0
        return stages, sets, t3 - t0

    stages, sets, dt = run(nrows, threads, True)
    per_token = sum(stages.values()) + sets / wl.total_q
    stages1, sets1, dt1 = run(nrows_1t, 1, True)
    per_token1 = sum(stages1.values()) + sets1 / wl.total_q
    gomp.omp_set_num_threads(threads)
    return {"value": 1.0 / per_token, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{nrows} evenly spaced query rows of the same workload (scores over all ~139K candidates, "
                      f"top-k, attention over k=2048; {dt:.1f} s) plus page demand, runs and the corrective set "
                      f"over all 8192 rows' ids ({sets:.2f} s)",
            "cpu_model": _cpu_model(), "nproc": os.cpu_count(), "cpus_allowed": len(os.sched_getaffinity(0)),
            "seconds_per_token": stages, "set_stages_s": sets,
            "single_thread": {"value": 1.0 / per_token1, "unit": "tokens/s", "cores": 1,
                              "sample": f"{nrows_1t} evenly spaced rows ({dt1:.1f} s) plus the set stages over all "
                                        f"rows ({sets1:.2f} s)", "seconds_per_token": stages1,
                              "set_stages_s": sets1}}


if __name__ == "__main__":
    main()
