"""Seeded synthetic workloads for append prefill with top-k sparse attention.

The shapes follow the workloads the method is evaluated on: one layer of a
DeepSeek-V3.2-like model (lightning-indexer 64 heads x 128 dims in fp8 e4m3fn
with per-token scales, MLA latent KV of 512 + 64 rope dims kept as one 576-dim
bf16 row per token, 128 query heads), long agentic histories (the trace table
of the evaluation reports histories of 77K-131K tokens at the median and
appends of 0.9K-12K tokens), and 64-token KV pages behind a page table.

Draw order and streams.  Every tensor comes from its own PCG64 stream keyed by
``SeedSequence([seed, stream, layer, ...])`` so tensors can be regenerated on
their own, and the large attention query is drawn in 64-row chunks so a sample
of rows can be regenerated without the rest:

    1 hot spans, 2 history indexer keys, 3 new-token indexer keys,
    4 indexer queries, 5 indexer head weights, 6 prediction noise,
    7 attention queries, 8 KV rows, 9 page table, 10 session lengths,
    11 synthetic selections, 12 resident-page bitmaps.

"Hot spans" stand in for concentrated relevance: 5% of each session's history
sits in 8 contiguous spans whose indexer keys are multiplied by 3 before
quantisation (one span placed uniformly inside each eighth of the history).

Quantisation to fp8 e4m3fn uses one fp32 scale per token (amax / 448, floored
at 1e-12 / 448) and round-to-nearest-even through torch's float8_e4m3fn cast;
bf16 uses torch's round-to-nearest-even cast.  These produce the input bytes;
the method never re-quantises.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

S_HOT, S_KHIST, S_KNEW, S_Q, S_W, S_QNOISE, S_QATT, S_KV, S_PT, S_SESS, S_SEL, S_RES = range(1, 13)

FP8_MAX = 448.0
ATTN_Q_CHUNK = 64

CONFIG_NAMES = {
    0: "tiny-fp32-M4096-N256",
    1: "dsv32-layer-M32768-N2048",
    2: "dsv32-layer-M131072-N8192-permuted",
    3: "ragged-16-sessions-M8K-64K",
    4: "prediction-8-layers-M131072-N4096",
    5: "decode-16-sessions-M8K-48K-N1",
}


def _rng(seed: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, *extra])))


def to_fp8_bytes(x: np.ndarray) -> np.ndarray:
    """float32 -> OCP fp8 e4m3fn bytes (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def quantize_fp8_per_row(x: np.ndarray):
    """One fp32 scale per leading index: bytes = fp8(x / scale), scale = amax / 448."""
    flat = x.reshape(x.shape[0], -1).astype(np.float32)
    amax = np.abs(flat).max(axis=1)
    scale = (np.maximum(amax, np.float32(1e-12)) / np.float32(FP8_MAX)).astype(np.float32)
    q = to_fp8_bytes(flat / scale[:, None]).reshape(x.shape)
    return q, scale


# OCP MX FP4 (e2m1) element magnitudes by code 0..7 (the sign is bit 3)
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def quantize_mxfp4(x: np.ndarray):
    """float32 [n, d] -> (bytes [n, d/2], E8M0 scales [n, d/32]) in OCP MXFP4.

    Per 32-element block the shared exponent is ceil(log2(amax / 6)), the
    smallest that fits the block's largest magnitude within the e2m1 maximum
    of 6, stored as E8M0 (biased by 127, clamped to [0, 254]); elements are
    divided by 2^exponent, rounded to the nearest e2m1 value (ties to the
    even code) and clamped to +-6.  Element j sits in the
    low nibble of byte j/2 when j is even, the high nibble when odd."""
    n, d = x.shape
    blk = x.astype(np.float64).reshape(n, d // 32, 32)
    amax = np.abs(blk).max(axis=2)
    e = np.where(amax > 0, np.ceil(np.log2(np.where(amax > 0, amax, 6.0) / 6.0)), 0)
    E = np.clip(e + 127, 0, 254).astype(np.uint8)
    v = blk / np.exp2(E.astype(np.float64) - 127)[:, :, None]
    mag = np.minimum(np.abs(v), 6.0)
    dist = np.abs(mag[..., None] - E2M1_MAGNITUDES)
    nearest = dist == dist.min(axis=-1, keepdims=True)  # one code, or two on a tie
    even_first = nearest & ((np.arange(8) & 1) == 0)
    code = np.where(even_first.any(axis=-1), np.argmax(even_first, axis=-1), np.argmax(nearest, axis=-1))
    code = code.astype(np.uint8) | np.where(v < 0, 8, 0).astype(np.uint8)
    code = code.reshape(n, d)
    packed = (code[:, 0::2] | (code[:, 1::2] << 4)).astype(np.uint8)
    return packed, E


def _encode(x: np.ndarray, dtype: str):
    if dtype == "fp8":
        return quantize_fp8_per_row(x)
    if dtype == "bf16":
        return to_bf16_bits(x), None
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32), None
    raise ValueError(dtype)


@dataclass
class AttnInputs:
    q: np.ndarray            # uint16 bf16 bits [total_q, Hq, dqk]
    k_pool: np.ndarray       # uint16 [num_phys_pages, page_size, k_row]
    v_pool: Optional[np.ndarray]  # None when V is the first dv elements of the K rows
    Hq: int
    dqk: int
    dv: int
    scale: float

    @property
    def k_row_stride(self) -> int:
        return int(self.k_pool.shape[2])

    @property
    def v_row_stride(self) -> int:
        return int((self.v_pool if self.v_pool is not None else self.k_pool).shape[2])


@dataclass
class Workload:
    name: str
    seed: int
    layer: int
    hist_len: np.ndarray     # int32 [B]  M_b
    new_len: np.ndarray      # int32 [B]  N_b
    H: int
    d: int
    idx_dtype: str           # "f32" | "bf16" | "fp8"
    q: np.ndarray            # [total_q, H, d]
    q_scale: Optional[np.ndarray]
    kI: np.ndarray           # [total_ctx, d]
    k_scale: Optional[np.ndarray]
    w: np.ndarray            # float32 [total_q, H]
    k: int
    page_size: int
    max_run: int
    page_table: np.ndarray   # int32 [B, pt_ld] logical page -> physical page
    num_phys_pages: int
    hot_spans: list          # per session: list of (start, length)
    attn_cfg: dict = field(default_factory=dict)
    q_pred: Optional[np.ndarray] = None
    q_pred_scale: Optional[np.ndarray] = None
    k_bscale: Optional[np.ndarray] = None   # MXFP4 keys: E8M0 [total_ctx, d/32]; kI is then [total_ctx, d/2]
    entry_shift: int = 0     # ids are entries of 2^entry_shift tokens (0: tokens)

    # ---- derived batch description -------------------------------------
    @property
    def num_seqs(self) -> int:
        return int(self.hist_len.shape[0])

    @property
    def ctx_len(self) -> np.ndarray:
        """Ids (key rows, score row length) per session: tokens, or whole entries."""
        return ((self.hist_len + self.new_len) >> self.entry_shift).astype(np.int32)

    @property
    def hist_ids(self) -> np.ndarray:
        """History ids per session: tokens, or entries wholly in the history."""
        return (self.hist_len >> self.entry_shift).astype(np.int32)

    @property
    def q_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.new_len)]).astype(np.int32)

    @property
    def ctx_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.ctx_len)]).astype(np.int32)

    @property
    def score_start(self) -> np.ndarray:
        per = self.new_len.astype(np.int64) * self.ctx_len.astype(np.int64)
        return np.concatenate([[0], np.cumsum(per)]).astype(np.int64)

    @property
    def total_q(self) -> int:
        return int(self.new_len.sum())

    @property
    def total_ctx(self) -> int:
        return int(self.ctx_len.sum())

    @property
    def max_q(self) -> int:
        return int(self.new_len.max())

    @property
    def max_ctx(self) -> int:
        return int(self.ctx_len.max())

    @property
    def total_scores(self) -> int:
        return int(self.score_start[-1])

    def row_session(self, rows) -> np.ndarray:
        return np.searchsorted(self.q_start, np.asarray(rows), side="right") - 1


def _hot_spans(rng: np.random.Generator, M: int, n_spans: int = 8, frac: float = 0.05, layout: str = "even"):
    """frac of the M history tokens in n_spans equal spans, one placed
    uniformly inside each of n_spans equal segments of the region: the whole
    history ("even") or its most recent quarter ("recent")."""
    span = int(math.floor(frac * M / n_spans))
    spans = []
    if span <= 0:
        return spans
    if layout == "even":
        base, region = 0, M
    elif layout == "recent":
        base, region = M - M // 4, M // 4
    else:
        raise ValueError(layout)
    seg = region // n_spans
    for j in range(n_spans):
        lo = base + j * seg
        start = lo + int(rng.integers(0, max(seg - span, 0) + 1))
        spans.append((start, min(span, M - start)))
    return spans


def make_workload(*, hist_len, new_len, H, d, idx_dtype, k, page_size=64, max_run=32,
                  seed=0, layer=0, w_scale=1.0, hot=True, table="identity",
                  attn=None, q_pred_corr=None, name="custom", key_format=None, entry_shift=0,
                  hot_frac=0.05, hot_layout="even") -> Workload:
    """Build one layer's indexer inputs for a (possibly ragged) batch of sessions.

    With ``entry_shift`` = e > 0 the keys, hot spans, pages and KV rows are
    per entry of 2^e tokens: session b has (M_b + N_b) >> e of them, the first
    M_b >> e from the history.  Queries stay per token.

    ``table`` is "identity" (logical page p of session b -> physical page
    base_b + p) or "permuted" (one seeded permutation of the pool, sliced
    consecutively per session).  ``q_pred_corr`` = rho adds a predicted query
    rho * q + sqrt(1 - rho^2) * N(0, 1), quantised on its own.  ``hot_frac``
    and ``hot_layout`` set the share of history tokens in hot spans and where
    the spans sit ("even": one in each eighth of the history; "recent": all
    in its last quarter).
    """
    hist_len = np.asarray(hist_len, dtype=np.int32).reshape(-1)
    new_len = np.asarray(new_len, dtype=np.int32).reshape(-1)
    B = hist_len.shape[0]
    ctx = (hist_len + new_len) >> entry_shift   # ids per session
    hist_ids = hist_len >> entry_shift
    pages_per = (ctx + page_size - 1) // page_size
    num_phys = int(pages_per.sum())
    pt_ld = int(max(1, pages_per.max()))

    # 1. hot spans (layer independent: the same positions in every layer)
    spans = []
    for b in range(B):
        spans.append(_hot_spans(_rng(seed, S_HOT, b), int(hist_ids[b]), frac=hot_frac, layout=hot_layout)
                     if hot else [])

    # 2./3. indexer keys, history then new tokens, per session
    keys = []
    for b in range(B):
        kh = _rng(seed, S_KHIST, layer, b).standard_normal((int(hist_ids[b]), d), dtype=np.float32)
        for (s0, ln) in spans[b]:
            kh[s0:s0 + ln] *= np.float32(3.0)
        kn = _rng(seed, S_KNEW, layer, b).standard_normal((int(ctx[b] - hist_ids[b]), d), dtype=np.float32)
        keys.append(kh)
        keys.append(kn)
    kI_f = np.concatenate(keys, axis=0) if keys else np.zeros((0, d), np.float32)

    # 4. queries, 5. head weights
    total_q = int(new_len.sum())
    q_f = _rng(seed, S_Q, layer).standard_normal((total_q, H, d), dtype=np.float32)
    w = (_rng(seed, S_W, layer).random((total_q, H), dtype=np.float32) * np.float32(w_scale)).astype(np.float32)

    q, q_scale = _encode(q_f, idx_dtype)
    k_bscale = None
    if key_format == "mxfp4":  # FP4 indexer keys with per-32 E8M0 scales (no per-token scale)
        kI, k_bscale = quantize_mxfp4(kI_f)
        k_scale = None
    else:
        kI, k_scale = _encode(kI_f, idx_dtype)

    q_pred = q_pred_scale = None
    if q_pred_corr is not None:
        rho = np.float32(q_pred_corr)
        eps = _rng(seed, S_QNOISE, layer).standard_normal((total_q, H, d), dtype=np.float32)
        qp = rho * q_f + np.float32(math.sqrt(1.0 - float(rho) ** 2)) * eps
        q_pred, q_pred_scale = _encode(qp.astype(np.float32), idx_dtype)
        del eps, qp
    del q_f, kI_f

    # 9. page table
    pt = np.zeros((B, pt_ld), dtype=np.int32)
    if table == "identity":
        phys = np.arange(num_phys, dtype=np.int32)
    elif table == "permuted":
        phys = _rng(seed, S_PT).permutation(num_phys).astype(np.int32)
    else:
        raise ValueError(table)
    base = 0
    for b in range(B):
        n = int(pages_per[b])
        pt[b, :n] = phys[base:base + n]
        base += n

    return Workload(name=name, seed=seed, layer=layer, hist_len=hist_len, new_len=new_len,
                    H=H, d=d, idx_dtype=idx_dtype, q=q, q_scale=q_scale, kI=kI, k_scale=k_scale,
                    w=w, k=k, page_size=page_size, max_run=max_run, page_table=pt,
                    num_phys_pages=num_phys, hot_spans=spans, attn_cfg=dict(attn or {}),
                    q_pred=q_pred, q_pred_scale=q_pred_scale, k_bscale=k_bscale, entry_shift=int(entry_shift))


MLA_ATTN = dict(Hq=128, dqk=576, dv=512, mla=True, q_std=1.0, kv_std=1.0 / math.sqrt(576.0),
                scale=1.0 / math.sqrt(576.0))
MQA0_ATTN = dict(Hq=8, dqk=128, dv=128, mla=False, q_std=1.0, kv_std=1.0, scale=1.0 / math.sqrt(128.0))


def config(i: int, layer: int = 0, with_pred: Optional[bool] = None) -> Workload:
    """The five evaluation workloads (seed = config index)."""
    if i == 0:
        return make_workload(hist_len=[4096], new_len=[256], H=4, d=64, idx_dtype="f32", k=256,
                             seed=0, layer=layer, attn=MQA0_ATTN, name=CONFIG_NAMES[0])
    if i == 1:
        return make_workload(hist_len=[32768], new_len=[2048], H=64, d=128, idx_dtype="fp8", k=2048,
                             seed=1, layer=layer, w_scale=1.0 / 8, attn=MLA_ATTN, name=CONFIG_NAMES[1])
    if i == 2:
        return make_workload(hist_len=[131072], new_len=[8192], H=64, d=128, idx_dtype="fp8", k=2048,
                             seed=2, layer=layer, w_scale=1.0 / 8, table="permuted", attn=MLA_ATTN,
                             q_pred_corr=0.9 if with_pred else None, name=CONFIG_NAMES[2])
    if i == 3:
        rng = _rng(3, S_SESS)
        M = np.floor(np.exp(rng.uniform(math.log(8192), math.log(65536), size=16))).astype(np.int32)
        N = rng.integers(512, 4096, size=16, endpoint=True).astype(np.int32)
        return make_workload(hist_len=M, new_len=N, H=64, d=128, idx_dtype="fp8", k=2048, seed=3,
                             layer=layer, w_scale=1.0 / 8, table="permuted", attn=MLA_ATTN,
                             name=CONFIG_NAMES[3])
    if i == 4:
        return make_workload(hist_len=[131072], new_len=[4096], H=64, d=128, idx_dtype="fp8", k=2048,
                             seed=4, layer=layer, w_scale=1.0 / 8, table="identity", attn=MLA_ATTN,
                             q_pred_corr=0.9 if with_pred is None else (0.9 if with_pred else None),
                             name=CONFIG_NAMES[4])
    if i == 5:
        # decode: one appended token per session (the step of the decode
        # phase), many sessions batched
        rng = _rng(5, S_SESS)
        M = np.floor(np.exp(rng.uniform(math.log(8192), math.log(49152), size=16))).astype(np.int32)
        return make_workload(hist_len=M, new_len=np.ones(16, np.int32), H=64, d=128, idx_dtype="fp8", k=2048,
                             seed=5, layer=layer, w_scale=1.0 / 8, table="permuted", attn=MLA_ATTN,
                             name=CONFIG_NAMES[5])
    raise ValueError(i)


def decode_lengths(B: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """History lengths of a batch of decoding sessions, log-uniform in [lo, hi]."""
    rng = _rng(seed, S_SESS)
    return np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=B))).astype(np.int32)


def resident_pages(wl: Workload, p: float = 0.9, seed: int = 0) -> np.ndarray:
    """A bitmap of pages already in HBM (bit j%32 of word j/32, LSB first):
    each physical page independently with probability p."""
    rng = _rng(wl.seed, S_RES, wl.layer, seed)
    bits = rng.random(wl.num_phys_pages) < p
    words = np.zeros((wl.num_phys_pages + 31) // 32 * 32, dtype=np.uint8)
    words[:wl.num_phys_pages] = bits
    return np.packbits(words.reshape(-1, 8), axis=1, bitorder="little").reshape(-1).view(np.uint32).copy()


def attention_q_rows(wl: Workload, rows) -> np.ndarray:
    """bf16 bits of the attention query for the given global rows, [len(rows), Hq, dqk]."""
    a = wl.attn_cfg
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((rows.shape[0], a["Hq"], a["dqk"]), dtype=np.uint16)
    chunks = {}
    for j, r in enumerate(rows):
        c = int(r) // ATTN_Q_CHUNK
        if c not in chunks:
            chunks[c] = _attn_q_chunk(wl, c)
        out[j] = chunks[c][int(r) - c * ATTN_Q_CHUNK]
    return out


def _attn_q_chunk(wl: Workload, c: int) -> np.ndarray:
    a = wl.attn_cfg
    lo = c * ATTN_Q_CHUNK
    n = min(ATTN_Q_CHUNK, wl.total_q - lo)
    x = _rng(wl.seed, S_QATT, wl.layer, c).standard_normal((n, a["Hq"], a["dqk"]), dtype=np.float32)
    if a["q_std"] != 1.0:
        x *= np.float32(a["q_std"])
    return to_bf16_bits(x)


def attention_inputs(wl: Workload, with_q: bool = True) -> AttnInputs:
    """Attention query and the paged KV pool (physically placed through the page table)."""
    a = wl.attn_cfg
    Hq, dqk, dv = a["Hq"], a["dqk"], a["dv"]
    q = None
    if with_q:
        nch = (wl.total_q + ATTN_Q_CHUNK - 1) // ATTN_Q_CHUNK
        q = np.empty((wl.total_q, Hq, dqk), dtype=np.uint16)
        for c in range(nch):
            lo = c * ATTN_Q_CHUNK
            blk = _attn_q_chunk(wl, c)
            q[lo:lo + blk.shape[0]] = blk
    P, ps = wl.num_phys_pages, wl.page_size
    mla = a["mla"]
    krow = dqk
    k_pool = np.zeros((P, ps, krow), dtype=np.uint16)
    v_pool = None if mla else np.zeros((P, ps, dv), dtype=np.uint16)
    kv_std = np.float32(a["kv_std"])
    for b in range(wl.num_seqs):
        npg = (int(wl.ctx_len[b]) + ps - 1) // ps
        for lp in range(npg):
            pp = int(wl.page_table[b, lp])
            x = _rng(wl.seed, S_KV, wl.layer, b, lp, 0).standard_normal((ps, krow), dtype=np.float32)
            if kv_std != 1.0:
                x *= kv_std
            k_pool[pp] = to_bf16_bits(x)
            if not mla:
                y = _rng(wl.seed, S_KV, wl.layer, b, lp, 1).standard_normal((ps, dv), dtype=np.float32)
                if kv_std != 1.0:
                    y *= kv_std
                v_pool[pp] = to_bf16_bits(y)
    return AttnInputs(q=q, k_pool=k_pool, v_pool=v_pool, Hq=Hq, dqk=dqk, dv=dv, scale=float(a["scale"]))


KV8_ROW_BYTES = 592  # 576 e4m3 bytes, the fp32 scale at byte 576, padding


def attention_kv_fp8(wl: Workload) -> np.ndarray:
    """The MLA KV pool of attention_inputs (the same draws) kept in fp8: uint8
    [num_phys_pages, page_size, 592], each row 576 e4m3 bytes (amax/448 scale,
    round-to-nearest-even cast) followed by its fp32 scale and zero padding."""
    a = wl.attn_cfg
    assert a["mla"] and a["dqk"] == 576
    P, ps = wl.num_phys_pages, wl.page_size
    pool = np.zeros((P, ps, KV8_ROW_BYTES), dtype=np.uint8)
    kv_std = np.float32(a["kv_std"])
    for b in range(wl.num_seqs):
        npg = (int(wl.ctx_len[b]) + ps - 1) // ps
        for lp in range(npg):
            pp = int(wl.page_table[b, lp])
            x = _rng(wl.seed, S_KV, wl.layer, b, lp, 0).standard_normal((ps, 576), dtype=np.float32)
            if kv_std != 1.0:
                x *= kv_std
            q8, sc = quantize_fp8_per_row(x)
            pool[pp, :, :576] = q8
            pool[pp, :, 576:580] = sc.astype(np.float32).view(np.uint8).reshape(ps, 4)
    return pool


def synth_topk(wl: Workload, seed: int = 0, hot_frac: float = 0.6, pad_rows: int = 0) -> np.ndarray:
    """Selections shaped like real ones, without scoring anything.

    Row i of session b gets min(k, n) distinct ids in [0, n), n = M_b + i + 1
    (entries: (M_b + i + 1) >> entry_shift):
    a hot_frac share drawn from the session's hot spans, the rest uniformly,
    in random order, padded with -1.  The last ``pad_rows`` rows of each
    session also get a few -1 holes and out-of-range ids in place of real ones.
    """
    rng = _rng(wl.seed, S_SEL, wl.layer, seed)
    k = wl.k
    out = np.full((wl.total_q, k), -1, dtype=np.int32)
    qs = wl.q_start
    for b in range(wl.num_seqs):
        M = int(wl.hist_len[b])
        hot = np.concatenate([np.arange(s, s + n) for (s, n) in wl.hot_spans[b]]) if wl.hot_spans[b] else np.zeros(0, np.int64)
        for i in range(int(wl.new_len[b])):
            n = (M + i + 1) >> wl.entry_shift  # ids that exist at this token
            if n == 0:
                continue
            want = min(k, n)
            nh = min(int(hot_frac * want), hot.shape[0])
            sel = rng.choice(hot, nh, replace=False) if nh else np.zeros(0, np.int64)
            extra = rng.integers(0, n, size=2 * want + 16)
            cand = np.concatenate([sel, extra])
            _, first = np.unique(cand, return_index=True)
            uniq = cand[np.sort(first)]
            if uniq.shape[0] < want:
                rest = np.setdiff1d(np.arange(n), uniq)
                uniq = np.concatenate([uniq, rest])
            row = uniq[:want].astype(np.int32)
            rng.shuffle(row)
            out[qs[b] + i, :want] = row
            if pad_rows and i >= int(wl.new_len[b]) - pad_rows:
                holes = rng.choice(want, size=min(4, want), replace=False)
                out[qs[b] + i, holes[:2]] = -1
                out[qs[b] + i, holes[2:3]] = int(wl.ctx_len[b]) + 3
                out[qs[b] + i, holes[3:]] = -7
    return out
