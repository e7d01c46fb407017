"""The C ABI library loads, exports every declared entry point, and rejects bad
arguments on the host (these calls return before touching a device)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "janus.h")
LIB = os.path.join(ROOT, "paper_2609_36938_amd", "libjanus.so")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced on the host


def _ensure_lib():
    if not os.path.exists(LIB):
        from paper_2609_36938_amd import build
        build.build()
    return LIB


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(janus_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_five_calls():
    syms = declared_symbols()
    for s in ("janus_index_scores", "janus_topk", "janus_topk_sharded", "janus_page_demand",
              "janus_predict_diff", "janus_sparse_attn", "janus_sparse_attn_split", "janus_index_scores_mxfp4",
              "janus_sparse_attn_fp8kv", "janus_status_string"):
        assert s in syms


def test_library_exports_every_declared_symbol():
    out = subprocess.check_output(["nm", "-D", "--defined-only", _ensure_lib()], text=True)
    exported = set(l.split()[-1] for l in out.splitlines() if " T " in l)
    missing = [s for s in declared_symbols() if s not in exported]
    assert not missing, missing
    L = ctypes.CDLL(LIB)
    for s in declared_symbols():
        assert hasattr(L, s)


def test_header_compiles_as_c():
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


@pytest.fixture(scope="module")
def L():
    import paper_2609_36938_amd as janus
    _ensure_lib()
    return janus.lib()


def _batch(total_q=4, max_ctx=100, B=1):
    import paper_2609_36938_amd as janus
    return janus._Batch(B, total_q, total_q, max_ctx, max_ctx, FAKE.value, FAKE.value, FAKE.value, FAKE.value)


def test_status_strings(L):
    assert L.janus_status_string(0) == b"ok"
    assert L.janus_status_string(1) == b"invalid argument"
    assert L.janus_status_string(2) == b"unsupported shape or dtype"
    assert L.janus_status_string(99) == b"unknown status"


def test_invalid_arguments_are_rejected_on_host(L):
    b = _batch()
    ws = ctypes.c_size_t(123)
    # NULL batch / pointers
    assert L.janus_topk(None, FAKE, 8, FAKE, None, ctypes.byref(ws), None) == 1
    assert L.janus_topk(ctypes.byref(b), None, 8, FAKE, None, ctypes.byref(ws), None) == 1
    assert L.janus_topk(ctypes.byref(b), FAKE, 0, FAKE, None, ctypes.byref(ws), None) == 1
    assert ws.value == 0  # top-k needs no workspace
    # k above the supported maximum
    assert L.janus_topk(ctypes.byref(b), FAKE, 7000, FAKE, None, ctypes.byref(ws), None) == 2
    # sharded top-k: shard count must divide k; align >= 1
    assert L.janus_topk_sharded(ctypes.byref(b), FAKE, 30, 4, 64, FAKE, None, ctypes.byref(ws), None) == 1
    assert L.janus_topk_sharded(ctypes.byref(b), FAKE, 32, 0, 64, FAKE, None, ctypes.byref(ws), None) == 1
    assert L.janus_topk_sharded(ctypes.byref(b), FAKE, 32, 4, 0, FAKE, None, ctypes.byref(ws), None) == 1
    assert L.janus_topk_sharded(ctypes.byref(b), FAKE, 8 * 7000, 8, 64, FAKE, None, ctypes.byref(ws), None) == 2
    # mismatched indexer dtypes, bad dtype code, bad sizes
    assert L.janus_index_scores(ctypes.byref(b), FAKE, 2, None, FAKE, 1, None, FAKE, 64, 128, FAKE, None) == 2
    assert L.janus_index_scores(ctypes.byref(b), FAKE, 7, None, FAKE, 7, None, FAKE, 64, 128, FAKE, None) == 1
    assert L.janus_index_scores(ctypes.byref(b), FAKE, 2, None, FAKE, 2, None, FAKE, 0, 128, FAKE, None) == 1
    # page size must be a power of two; max_run >= 1
    args = [ctypes.byref(b), FAKE, 8, FAKE, 4, 48, None, 100, 32, FAKE, FAKE, FAKE, FAKE, None,
            ctypes.byref(ws), None]
    assert L.janus_page_demand(*args) == 1
    args[5], args[8] = 64, 0
    assert L.janus_page_demand(*args) == 1
    args[8], args[7] = 32, (1 << 19) + 1
    assert L.janus_page_demand(*args) == 2
    assert L.janus_predict_diff(FAKE, None, 10, 32, FAKE, FAKE, FAKE, None) == 1
    assert L.janus_predict_diff(FAKE, FAKE, 10, 0, FAKE, FAKE, FAKE, None) == 1
    # attention: output dtype, row strides shorter than the head dims
    assert L.janus_sparse_attn(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, 4, 64, FAKE,
                               8, ctypes.c_float(0.1), FAKE, 2, None, None) == 2
    assert L.janus_sparse_attn(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 500, 576, FAKE, 4, 64, FAKE,
                               8, ctypes.c_float(0.1), FAKE, 1, None, None) == 1


def test_mxfp4_scores_rejections(L):
    b = _batch()
    assert L.janus_index_scores_mxfp4(ctypes.byref(b), FAKE, None, FAKE, None, None, FAKE, 64, 128, FAKE, None) == 1
    assert L.janus_index_scores_mxfp4(ctypes.byref(b), FAKE, None, FAKE, FAKE, None, FAKE, 64, 100, FAKE, None) == 1
    assert L.janus_index_scores_mxfp4(ctypes.byref(b), FAKE, None, FAKE, FAKE, None, FAKE, 32, 128, FAKE, None) == 2
    assert L.janus_index_scores_mxfp4(ctypes.byref(b), FAKE, None, FAKE, FAKE, None, FAKE, 64, 64, FAKE, None) == 2


def test_split_attention_workspace_and_rejections(L):
    """janus_sparse_attn_split: the workspace query (nothing launched with an
    explicit slice count), a short workspace, and argument errors."""
    b = _batch()  # total_q rows of the host-only batch
    f = ctypes.c_float(0.1)

    def call(nsplit, ws, ws_bytes, Hq=128, dqk=576, dv=512, k=2048, v=FAKE, odt=1):
        return L.janus_sparse_attn_split(ctypes.byref(b), FAKE, Hq, dqk, dv, FAKE, v, 576, 576, FAKE, 4, 64, FAKE, k,
                                         f, FAKE, odt, None, nsplit, ws, ctypes.byref(ws_bytes), None)

    need = ctypes.c_size_t(0)
    assert call(4, None, need) == 0
    assert need.value == b.total_q * 4 * 128 * 514 * 4
    assert call(1, None, need) == 0 and need.value == 0          # one slice: no workspace
    assert call(16, None, need, k=64) == 0                        # at most one slice per 32 ids
    assert need.value == b.total_q * 2 * 128 * 514 * 4
    short = ctypes.c_size_t(b.total_q * 4 * 128 * 514 * 4 - 1)
    assert call(4, FAKE, short) == 3                              # JANUS_ERR_WORKSPACE
    assert call(17, None, need) == 1 and call(-1, None, need) == 1
    assert L.janus_sparse_attn_split(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, 4, 64, FAKE,
                                     8, f, FAKE, 1, None, 2, None, None, None) == 1  # no size pointer
    assert call(2, None, need, dqk=128, dv=128) == 2              # only the MFMA shape splits
    assert call(2, None, need, v=ctypes.c_void_p(0x2000)) == 2    # separate V pool
    assert call(2, None, need, odt=2) == 2                        # fp8 output
    big = ctypes.c_size_t(1 << 40)
    assert call(4, ctypes.c_void_p(0x1008), big) == 2             # slice merge needs a 16-byte aligned workspace
    assert L.janus_sparse_attn_split(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, 4, 64, FAKE,
                                     2048, f, ctypes.c_void_p(0x1004), 1, None, 4, FAKE, ctypes.byref(big),
                                     None) == 2                  # ... and a 16-byte aligned output


def test_product_path_does_not_touch_the_oracle():
    pkg = os.path.join(ROOT, "paper_2609_36938_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "janus_oracle" not in text, f


def test_batch_layout_matches_the_header(tmp_path):
    """The binding's janus_batch has the header's size and field offsets."""
    import paper_2609_36938_amd as janus
    src = tmp_path / "layout.c"
    names = [f[0] for f in janus._Batch._fields_]
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "janus.h"\nint main(void){\n'
                   + 'printf("%zu\\n", sizeof(janus_batch));\n'
                   + "".join(f'printf("%zu\\n", offsetof(janus_batch, {n}));\n' for n in names) + "return 0;}\n")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), "-o", str(exe), str(src)])
    got = [int(x) for x in subprocess.check_output([str(exe)], text=True).split()]
    assert got[0] == ctypes.sizeof(janus._Batch)
    assert got[1:] == [getattr(janus._Batch, n).offset for n in names]


def test_entry_shift_out_of_range_is_rejected(L):
    ws = ctypes.c_size_t(0)
    for shift in (-1, 17):
        b = _batch()
        b.entry_shift = shift
        assert L.janus_topk(ctypes.byref(b), FAKE, 8, FAKE, None, ctypes.byref(ws), None) == 1
        assert L.janus_index_scores(ctypes.byref(b), FAKE, 2, None, FAKE, 2, None, FAKE, 64, 128, FAKE, None) == 1
    b = _batch()
    b.entry_shift = 16
    assert L.janus_topk(ctypes.byref(b), FAKE, 7000, FAKE, None, ctypes.byref(ws), None) == 2  # accepted shift


def test_fp8kv_attention_rejections(L):
    b = _batch()
    ws = ctypes.c_size_t(0)
    call = lambda **kw: L.janus_sparse_attn_fp8kv(
        ctypes.byref(b), kw.get("q", FAKE), kw.get("Hq", 128), kw.get("kv", FAKE), kw.get("rb", 592), FAKE, 4, 64,
        FAKE, kw.get("k", 64), ctypes.c_float(0.1), FAKE, kw.get("odt", 1), None, kw.get("ns", 1), None,
        ctypes.byref(ws), None)
    assert call() == 0 and ws.value == 0  # size query: unsplit needs no workspace
    assert call(rb=576) == 1              # row shorter than 576 bytes + scale
    assert call(kv=None) == 1
    assert call(ns=17) == 1
    assert call(rb=600) == 2              # rows must be 16-byte multiples
    assert call(Hq=48) == 2
    assert call(k=5000) == 2
    assert call(odt=2) == 2               # out dtype fp8
    assert call(q=ctypes.c_void_p(0x1008)) == 2  # misaligned q


def test_page_table_narrower_than_the_context_is_rejected(L):
    """Every call that reads a page table checks on the host that pt_ld pages
    cover the longest session (max_ctx = 100 ids here: 2 pages of 64 do, 1
    does not); a narrower table would be read past its end on the device."""
    b = _batch()
    ws = ctypes.c_size_t(0)
    f = ctypes.c_float(0.1)
    for pt_ld, want in ((1, 1), (2, 0)):
        # page demand and unsplit attention launch once the table is wide
        # enough, so only their rejection is exercised here
        if want:
            assert L.janus_page_demand(ctypes.byref(b), FAKE, 8, FAKE, pt_ld, 64, None, 100, 32, FAKE, FAKE, FAKE,
                                       FAKE, None, ctypes.byref(ws), None) == 1
            assert L.janus_sparse_attn(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, pt_ld, 64,
                                       FAKE, 8, f, FAKE, 1, None, None) == 1
        # the split and fp8-KV calls stop at their size query when the table is wide enough
        rc = L.janus_sparse_attn_split(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, pt_ld, 64,
                                       FAKE, 2048, f, FAKE, 1, None, 4, None, ctypes.byref(ws), None)
        assert rc == want
        rc = L.janus_sparse_attn_fp8kv(ctypes.byref(b), FAKE, 128, FAKE, 592, FAKE, pt_ld, 64, FAKE, 64, f, FAKE, 1,
                                       None, 1, None, ctypes.byref(ws), None)
        assert rc == want
    # entries: max_ctx counts entries, so 1 page of 128 entries covers 100 of them
    assert L.janus_sparse_attn_fp8kv(ctypes.byref(b), FAKE, 128, FAKE, 592, FAKE, 1, 128, FAKE, 64, f, FAKE, 1,
                                     None, 1, None, ctypes.byref(ws), None) == 0


def test_null_workspace_is_always_a_size_query(L):
    """A NULL workspace only reports the size, also when 0 bytes are needed
    (one slice): the call returns ok without launching (on this host, which has
    no GPU, a launch would have returned JANUS_ERR_DEVICE)."""
    b = _batch()
    f = ctypes.c_float(0.1)
    ws = ctypes.c_size_t(777)
    assert L.janus_sparse_attn_fp8kv(ctypes.byref(b), FAKE, 128, FAKE, 592, FAKE, 4, 64, FAKE, 64, f, FAKE, 1,
                                     None, 1, None, ctypes.byref(ws), None) == 0
    assert ws.value == 0
    ws = ctypes.c_size_t(777)
    assert L.janus_sparse_attn_split(ctypes.byref(b), FAKE, 128, 576, 512, FAKE, FAKE, 576, 576, FAKE, 4, 64, FAKE,
                                     2048, f, FAKE, 1, None, 1, None, ctypes.byref(ws), None) == 0
    assert ws.value == 0


def test_noalloc_split_attention_host_checks(L):
    """janus_sparse_attn_split_noalloc refuses, before touching a device, a
    launch whose slice partials exceed its scratch array, and argument errors."""
    f = ctypes.c_float(0.1)

    def call(b, nsplit, Hq=128, dqk=576, pt_ld=4096, k=2048):
        return L.janus_sparse_attn_split_noalloc(ctypes.byref(b), FAKE, Hq, dqk, 512, FAKE, FAKE, 576, 576, FAKE,
                                                 pt_ld, 64, FAKE, k, f, FAKE, 1, None, nsplit, None)

    big = _batch(total_q=2048)
    assert 2048 * 16 * 128 * 514 * 4 > (128 << 20)
    assert call(big, 16) == 3                      # JANUS_ERR_WORKSPACE: more than the scratch holds
    assert call(big, 17) == 1 and call(big, -1) == 1
    assert call(big, 2, dqk=128) == 2              # only the MLA shape splits
    assert call(_batch(max_ctx=100), 2, pt_ld=1) == 1  # page table narrower than the context
