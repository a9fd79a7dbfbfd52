"""The C ABI on the host: the built library loads, exports every function include/flashloop.h declares,
and rejects bad arguments with the documented status before anything is enqueued (no GPU needed: every
call here fails host-side validation, and pointers are never dereferenced on the host)."""
import ctypes
import os
import re

import pytest

from paper_2609_29812_amd import flashloop as fl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashloop.h")

FL_OK, FL_E_NULL, FL_E_SHAPE, FL_E_RANGE, FL_E_UNSUPPORTED, FL_E_WORKSPACE = 0, 1, 2, 3, 4, 5
DUMMY = ctypes.c_void_p(0x1000)     # a non-NULL device pointer stand-in, never dereferenced on the host
DUMMY2 = ctypes.c_void_p(0x2000)    # a second, distinct stand-in


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\**\s*(fl_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fl.LIB_PATH):
        from paper_2609_29812_amd import build
        build.build(verbose=False)
    return fl.load()


def test_library_loads_and_exports_every_declared_function(lib):
    names = declared_functions()
    assert len(names) >= 11
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(fl.EXPORTS) == names        # the binding covers exactly the header


def test_version_and_status_strings(lib):
    assert lib.fl_abi_version() == 1
    for code in range(8):
        assert lib.fl_status_str(code)
    assert b"OK" in lib.fl_status_str(FL_OK).upper()


def test_workspace_queries(lib):
    # records: list + compacted updated list per (b, h), every column and every row per batch, a sentinel;
    # then one count per (b, h)
    B, N, H, d, k, c, w = 2, 100, 3, 64, 10, 8, 4
    want = (2 * B * H * c + B * N + B * k + 1) * 8 + B * H * 4
    assert lib.fl_loop_sparse_attn_ws(B, N, H, d, k, c, w, 0) == want
    assert lib.fl_loop_sparse_attn_ws(B, N, H, d, N, 0, 0, fl.ATTN_DENSE) == 0
    # list pruning: fp64 partial sums per 256-row chunk of the updated rows and per non-sink entry
    assert lib.fl_prune_columns_ws(1, 16, 1638, 1536, 4) == 16 * 7 * 1532 * 8
    assert lib.fl_prune_columns_ws(2, 3, 0, 10, 20) == 0          # all sinks: nothing to rank


def _attn(lib, **kw):
    a = dict(q_cur=DUMMY, q_prev=DUMMY, k_cache=DUMMY, v_cache=DUMMY, k_new=DUMMY, v_new=DUMMY, slot=DUMMY,
             rows=DUMMY, k=4, cols=DUMMY, c_list=8, window=4, B=1, N=64, H=2, d=64, scale=0.125, flags=0,
             lse=DUMMY, o=DUMMY, ws=DUMMY, ws_bytes=1 << 20)
    a.update(kw)
    return lib.fl_loop_sparse_attn(a["q_cur"], a["q_prev"], a["k_cache"], a["v_cache"], a["k_new"], a["v_new"],
                                   a["slot"], a["rows"], a["k"], a["cols"], a["c_list"], a["window"], a["B"], a["N"],
                                   a["H"], a["d"], a["scale"], a["flags"], a["lse"], a["o"], a["ws"], a["ws_bytes"],
                                   None)


def test_attention_rejects_bad_arguments(lib):
    assert _attn(lib, flags=8) == FL_E_UNSUPPORTED
    assert _attn(lib, q_cur=None) == FL_E_NULL
    assert _attn(lib, d=96) == FL_E_SHAPE
    assert _attn(lib, N=1 << 20, H=16, d=128) == FL_E_SHAPE      # N * H * d above 2^30
    assert _attn(lib, scale=0.0) == FL_E_RANGE
    assert _attn(lib, k=65) == FL_E_RANGE
    assert _attn(lib, q_prev=None) == FL_E_NULL
    assert _attn(lib, window=-1) == FL_E_RANGE
    assert _attn(lib, ws=None) == FL_E_WORKSPACE
    assert _attn(lib, ws_bytes=16) == FL_E_WORKSPACE
    assert _attn(lib, flags=fl.ATTN_DENSE, rows=DUMMY, k=64) == FL_E_SHAPE   # dense takes rows == NULL
    assert _attn(lib, k_new=None, v_new=None) == FL_E_NULL   # no new rows: only with reused terms
    assert _attn(lib, v_new=None) == FL_E_NULL               # new rows come in pairs
    assert b"fl_loop_sparse_attn" in lib.fl_last_error()


def test_select_and_codec_reject_bad_arguments(lib):
    sel = lambda **kw: lib.fl_select_tokens(
        kw.get("kc", DUMMY), DUMMY, kw.get("vc", DUMMY), DUMMY, 1, 64, kw.get("D", 128), None, 64, kw.get("k", 8),
        1, 1e-6, DUMMY, DUMMY, DUMMY, None)
    assert sel(kc=None) == FL_E_NULL
    assert sel(vc=None) == FL_E_NULL          # one pair half-given
    assert sel(D=12) == FL_E_SHAPE
    assert sel(k=65) == FL_E_RANGE
    assert b"fl_select_tokens" in lib.fl_last_error()

    q = lambda **kw: lib.fl_kv_residual_quant(DUMMY, DUMMY, DUMMY, 8, 1, 64, 2, kw.get("d", 64), kw.get("bits", 4),
                                              kw.get("G", 32), kw.get("axis", fl.AXIS_TOKEN), DUMMY, DUMMY, DUMMY,
                                              None, None)
    assert q(bits=3) == FL_E_UNSUPPORTED
    assert q(axis=2) == FL_E_UNSUPPORTED
    assert q(G=48) == FL_E_UNSUPPORTED
    assert q(d=96) == FL_E_SHAPE
    assert q(d=64, G=128, axis=fl.AXIS_CHANNEL) == FL_E_SHAPE    # CHANNEL groups must divide d
    qc = lambda **kw: lib.fl_kv_residual_quant_commit(DUMMY, kw.get("x_hat", DUMMY), DUMMY, 8, 1, 64, 2, 64,
                                                      kw.get("bits", 4), 32, fl.AXIS_TOKEN, DUMMY, DUMMY, DUMMY,
                                                      None)
    assert qc(x_hat=None) == FL_E_NULL
    assert qc(bits=3) == FL_E_UNSUPPORTED
    assert b"fl_kv_residual_quant_commit" in lib.fl_last_error()
    qkv = lambda **kw: lib.fl_kv_residual_quant_kv(
        DUMMY, kw.get("kr", DUMMY), DUMMY, kw.get("vr", DUMMY2), DUMMY, 8, 1, 64, 2, 64, kw.get("bits", 4), 32,
        DUMMY, DUMMY, DUMMY, kw.get("vc", DUMMY2), DUMMY, DUMMY, kw.get("krows"), kw.get("vrows"),
        kw.get("mode", fl.DQ_COMPACT), None)
    assert qkv(mode=2) == FL_E_UNSUPPORTED
    assert qkv(bits=3) == FL_E_UNSUPPORTED
    assert qkv(mode=fl.DQ_COMMIT, vr=None) == FL_E_NULL           # commit needs both caches
    assert qkv(mode=fl.DQ_COMMIT, krows=DUMMY2) == FL_E_NULL      # commit takes no compact rows
    assert qkv(mode=fl.DQ_COMMIT, vr=DUMMY) == FL_E_SHAPE         # one cache for keys and values
    assert qkv(krows=DUMMY) == FL_E_SHAPE                         # rows alias the reference with idx
    assert qkv(vc=DUMMY) == FL_E_SHAPE                            # shared code buffer
    assert b"fl_kv_residual_quant_kv" in lib.fl_last_error()
    dqkv = lambda **kw: lib.fl_kv_residual_dequant_kv(
        DUMMY, DUMMY, DUMMY, DUMMY2, DUMMY2, DUMMY2, DUMMY, 8, 1, 64, 2, 64, kw.get("bits", 4), 32,
        kw.get("mode", fl.DQ_COMMIT), DUMMY, kw.get("vh", DUMMY2), kw.get("kr"), kw.get("vr"), None)
    assert dqkv(mode=5) == FL_E_UNSUPPORTED
    assert dqkv(bits=3) == FL_E_UNSUPPORTED
    assert dqkv(kr=DUMMY2) == FL_E_NULL                           # commit takes no compact rows
    assert dqkv(mode=fl.DQ_COMPACT, kr=DUMMY2) == FL_E_NULL       # compact needs both row buffers
    assert dqkv(vh=DUMMY) == FL_E_SHAPE                           # one cache for keys and values
    assert b"fl_kv_residual_dequant_kv" in lib.fl_last_error()
    dq = lib.fl_kv_residual_dequant(DUMMY, DUMMY, DUMMY, DUMMY, 8, 1, 64, 2, 64, 4, 32, fl.AXIS_TOKEN, 7, DUMMY,
                                    None, None)
    assert dq == FL_E_UNSUPPORTED                                   # unknown mode


def test_decode_workspace_and_argument_checks(lib):
    # workspace: fp64 logits, chunk parts, fp32 keys and selection parts; 0 for unsupported shapes
    assert lib.fl_decode_step_ws(1, 4096, 16, 128, 0, 2048) > 4096 * 16 * 12
    assert lib.fl_decode_step_ws(1, 4096, 16, 96, 0, 2048) == 0
    assert lib.fl_decode_step_ws(0, 4096, 16, 128, 0, 2048) == 0
    WS = ctypes.c_size_t(1 << 40)

    def dec(**kw):
        return lib.fl_decode_step(
            kw.get("q", DUMMY), DUMMY, DUMMY, kw.get("cols"), kw.get("c", 0), kw.get("mass"), kw.get("sub"),
            1, kw.get("T", 64), 2, kw.get("d", 64), ctypes.c_float(kw.get("scale", 0.125)), DUMMY, None,
            kw.get("n_sink", 4), 8, kw.get("c_next", 16), kw.get("cn", DUMMY), DUMMY, DUMMY,
            kw.get("ws", DUMMY), kw.get("wsb", WS), None)
    assert dec(q=None) == FL_E_NULL
    assert dec(d=96) == FL_E_SHAPE
    assert dec(scale=0.0) == FL_E_RANGE
    assert dec(c=5) == FL_E_SHAPE                               # dense: c must be 0 or T
    assert dec(cols=DUMMY, c=65, mass=DUMMY, sub=DUMMY) == FL_E_RANGE
    assert dec(cols=DUMMY, c=10) == FL_E_NULL                    # sparse needs mass and sub
    assert dec(c_next=65) == FL_E_RANGE
    assert dec(cn=None) == FL_E_NULL                             # a selection needs its outputs
    assert dec(n_sink=-1) == FL_E_RANGE
    assert dec(T=70000) == FL_E_SHAPE                            # more columns than the selection takes
    assert dec(ws=None) == FL_E_WORKSPACE
    assert dec(wsb=ctypes.c_size_t(16)) == FL_E_WORKSPACE
    assert b"fl_decode_step" in lib.fl_last_error()


def test_decode_noalloc_argument_checks(lib):
    # the same host-side checks as fl_decode_step, before the scratch array is looked up, plus its size limit
    assert lib.fl_decode_step_ws(1, 8192, 16, 128, 0, 2048) <= 32 << 20      # a dense 8K step fits
    assert lib.fl_decode_step_ws(4, 65536, 16, 128, 0, 2048) > 32 << 20      # B * H * T = 4M does not

    def dec(**kw):
        return lib.fl_decode_step_noalloc(
            kw.get("q", DUMMY), DUMMY, DUMMY, kw.get("cols"), kw.get("c", 0), kw.get("mass"), kw.get("sub"),
            kw.get("B", 1), kw.get("T", 64), kw.get("H", 2), kw.get("d", 64), ctypes.c_float(0.125), DUMMY, None,
            4, 8, kw.get("c_next", 16), kw.get("cn", DUMMY), DUMMY, DUMMY, None)
    assert dec(q=None) == FL_E_NULL
    assert dec(d=96) == FL_E_SHAPE
    assert dec(c=5) == FL_E_SHAPE
    assert dec(cn=None) == FL_E_NULL
    assert dec(B=64, T=65536, H=16, d=128) == FL_E_RANGE                     # beyond the scratch array
    assert b"scratch" in lib.fl_last_error()


def test_attention_kernel_names(lib):
    """The host-side query names the kernel each pass launches (no device call)."""
    name = fl.attn_kernel_name
    # 32K workload: band 512, list 2048, 1638 rows, 16 heads -> the two-team segment kernels
    assert name(fl.PASS_ADD, 1638, 2048, 512, 1, 32768, 16, 128) == "seg_cur_kernel"
    assert name(fl.PASS_SUBTRACT, 1638, 2048, 512, 1, 32768, 16, 128) == "seg_sub_kernel"
    assert name(fl.PASS_BOTH, 1638, 2048, 512, 1, 32768, 16, 128) == "loop_attn_kernel"
    # no band: one team from about 1.5 full 128-row segments per CU (ceil(k / 128) * B * H >= 384), else two
    assert name(fl.PASS_ADD, 706, 1024, 0, 4, 16384, 16, 128) == "seg1_cur_kernel"      # 6 * 64 = 384
    assert name(fl.PASS_SUBTRACT, 706, 1024, 0, 4, 16384, 16, 128) == "seg1_sub_kernel"
    assert name(fl.PASS_ADD, 640, 1024, 0, 4, 16384, 16, 128) == "seg_cur_kernel"       # 5 * 64 = 320
    assert name(fl.PASS_ADD, 410, 512, 0, 1, 4096, 16, 128) == "seg_cur_kernel"
    # lists beyond the segment kernels' LDS copy: the 64-row kernels, then the record-driven one
    assert name(fl.PASS_ADD, 500, 2049, 64, 1, 8192, 16, 128) == "cur_attn_kernel"
    assert name(fl.PASS_SUBTRACT, 500, 3072, 0, 1, 8192, 16, 64) == "cur_sub_kernel"
    assert name(fl.PASS_ADD, 500, 3073, 64, 1, 8192, 16, 128) == "reuse_attn_kernel"
    assert name(fl.PASS_SUBTRACT, 500, 3073, 64, 1, 8192, 16, 128) is None
    # arguments outside the domain
    assert name(fl.PASS_ADD, 0, 512, 0, 1, 4096, 16, 128) is None
    assert name(fl.PASS_ADD, 100, 512, 0, 1, 4096, 16, 96) is None
    assert name(7, 100, 512, 0, 1, 4096, 16, 128) is None
    # the subtract query agrees with the name
    for args in [(1638, 2048, 512, 32768, 128), (100, 512, 0, 4096, 128), (100, 3073, 0, 4096, 128)]:
        k, c, w, N, d = args
        assert fl.subtract_terms_supported(k, c, w, N, d) == (name(fl.PASS_SUBTRACT, k, c, w, 1, N, 16, d) is not None)
