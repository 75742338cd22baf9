"""The C ABI library: it loads, exports what include/zeta.h declares, sizes
workspaces, and rejects bad arguments before any GPU work (no GPU needed).

Every call below breaks exactly one rule and must return before touching the
HIP runtime; pointers are dummies that the library never dereferences.
"""

import ctypes
import os
import re

import pytest

import paper_2501_14577_amd as zeta
from paper_2501_14577_amd import zeta as zb

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "zeta.h")
P = ctypes.c_void_p(0x10000)  # dummy, 256-byte aligned, never dereferenced
P2 = ctypes.c_void_p(0x20000)
P3 = ctypes.c_void_p(0x30000)
P4 = ctypes.c_void_p(0x40000)
NULL = None
BIG = 1 << 40
INV, UNS, WSP = zb.ZETA_ERR_INVALID_ARG, zb.ZETA_ERR_UNSUPPORTED, zb.ZETA_ERR_WORKSPACE


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\S.*?\b(zeta_\w+)\(", text, flags=re.M)))


def test_header_declares_the_four_calls_and_helpers():
    syms = declared_symbols()
    assert syms == sorted(zeta.EXPORTED), syms


def test_library_exports_every_declared_symbol():
    lib = zeta.load_library()
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_library_is_in_tree():
    assert os.path.dirname(zeta.library_path()) == os.path.dirname(os.path.abspath(zb.__file__))


def test_status_strings():
    names = ["ZETA_OK", "ZETA_ERR_INVALID_ARG", "ZETA_ERR_UNSUPPORTED", "ZETA_ERR_WORKSPACE", "ZETA_ERR_HIP"]
    for code, name in enumerate(names):
        assert zeta.zeta_status_string(code) == name
    assert zeta.zeta_status_string(99) == "ZETA_ERR_UNKNOWN"


def test_workspace_size():
    ws = zeta.zeta_workspace_size
    assert ws(0, 1, 10, 3, 10, 4, 1) == 0
    assert ws(1, 1, 10, 3, 11, 4, 1) == 0  # 33 code bits
    assert ws(1, 1, 10, 0, 10, 4, 1) == 0
    assert ws(1, 1, 10, 3, 10, 0, 1) == 0
    # Long-context shape: the forward's joint sort needs 2 x 16 x 65536 x 8 B;
    # the one-pass call's lists, bounds and list-order key rows stay below 64 MB.
    big = ws(1, 16, 65536, 3, 6, 128, 1)
    assert big >= 2 * 16 * 65536 * 8
    assert big < 64 << 20
    assert big % 256 == 0
    assert ws(1, 16, 65536, 3, 6, 128, 0) <= big
    # One tiny segment still gets a buffer for the range partials.
    assert ws(1, 1, 1, 3, 10, 1, 1) > 0


def test_bwd_workspace_size():
    ws = zeta.zeta_bwd_workspace_size
    assert ws(0, 1, 10, 3, 64, 4, 0) == 0
    assert ws(1, 1, 10, 3, 64, 0, 0) == 0
    assert ws(1, 1, 10, 3, 64, 1025, 0) == 0
    assert ws(1, 1, 10, 9, 64, 4, 0) == 0
    assert ws(1, 1, 10, 3, 48, 4, 0) == 0
    assert ws(1, 1, 1 << 22, 3, 64, 1024, 0) == 0  # N * topk = 2^32 slots
    # Long-context shape: the window slots (keys, sorted keys, sorted slots:
    # 3 x 16 x 65536 x 128 x 4 B) plus the slot sort's own buffers; the
    # history-mean candidate adds (3 + 128) x 4 B per row.
    big = ws(1, 16, 65536, 3, 128, 128, 0)
    assert big >= 3 * 16 * 65536 * 128 * 4
    assert big % 256 == 0
    assert ws(1, 16, 65536, 3, 128, 128, 1) >= big + 16 * 65536 * 131 * 4
    assert ws(1, 1, 1, 1, 32, 1, 0) > 0


def _hist(**kw):
    a = dict(k=P, v=P2, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, d_v=64, causal=1,
             mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0000), ws=ctypes.c_void_p(0x80000),
             ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_history_mean(*a.values())


HIST_CASES = [
    (dict(k=NULL), INV), (dict(v=NULL), INV), (dict(mean_k=NULL), INV), (dict(mean_v=NULL), INV),
    (dict(B=0), INV), (dict(N=0), INV), (dict(d_k=0), INV), (dict(d_v=0), INV), (dict(causal=2), INV),
    (dict(v=ctypes.c_void_p(0x20008)), INV), (dict(mean_v=ctypes.c_void_p(0xC0004)), INV),
    (dict(mean_v=ctypes.c_void_p(0xB0000)), INV),  # mean_v is mean_k
    (dict(mean_k=P), INV),  # mean_k is k
    (dict(dtype=4), UNS), (dict(d_k=9), UNS), (dict(d_v=100), UNS),
    (dict(ws=NULL), WSP), (dict(ws_bytes=64), WSP),
]


@pytest.mark.parametrize("kw,code", HIST_CASES, ids=[str(c[0]) for c in HIST_CASES])
def test_history_mean_rejects(kw, code):
    assert _hist(**kw) == code


def _knn(**kw):
    a = dict(q=P, k=P2, dtype=zb.ZETA_F32, B=1, H=2, N=100, d_k=3, kn=8, causal=0, out=P3, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_exact_knn(*a.values())


KNN_CASES = [
    (dict(q=NULL), INV), (dict(k=NULL), INV), (dict(out=NULL), INV), (dict(B=0), INV), (dict(N=0), INV),
    (dict(d_k=0), INV), (dict(kn=0), INV), (dict(causal=2), INV),
    (dict(dtype=3), UNS), (dict(d_k=9), UNS), (dict(kn=1025), UNS), (dict(N=4097), UNS),
]


@pytest.mark.parametrize("kw,code", KNN_CASES, ids=[str(c[0]) for c in KNN_CASES])
def test_exact_knn_rejects(kw, code):
    assert _knn(**kw) == code


def _ovl(**kw):
    a = dict(a=P, ka=8, b=P2, kb=8, rows=100, N=100, counts=P3, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_index_overlap(*a.values())


OVERLAP_CASES = [
    (dict(a=NULL), INV), (dict(b=NULL), INV), (dict(counts=NULL), INV), (dict(ka=0), INV), (dict(kb=-1), INV),
    (dict(rows=0), INV), (dict(N=0), INV), (dict(ka=1025), UNS), (dict(kb=2000), UNS), (dict(N=65537), UNS),
]


@pytest.mark.parametrize("kw,code", OVERLAP_CASES, ids=[str(c[0]) for c in OVERLAP_CASES])
def test_index_overlap_rejects(kw, code):
    assert _ovl(**kw) == code


def test_workspace_covers_history_mean():
    # The forward workspace also serves zeta_history_mean at the widest d_v:
    # float32 sums per (segment, chunk of 32 rows, column of k and v) and totals.
    for B, H, N in ((1, 16, 65536), (32, 4, 2048), (1, 1, 1), (3, 1, 65)):
        ws = zeta.zeta_workspace_size(B, H, N, 3, 10, 32, 1)
        assert ws >= B * H * (-(-N // 32) + 1) * (8 + 256) * 4
    assert _hist(d_v=256, ws_bytes=64) == WSP


def _enc(**kw):
    a = dict(q=P, k=P2, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, bits=10, range_lohi=NULL,
             range_out=NULL, q_codes=P3, k_codes=P4, ws=P, ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_morton_encode(*a.values())


def _sort(**kw):
    a = dict(k_codes=P, S=2, N=100, code_bits=30, sorted_codes=P2, perm=P3, ws=P4, ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_sort_keys(*a.values())


def _qord(**kw):
    a = dict(q_order=P, S=2, N=100, topk=8, causal=1, chunk=0, order_out=P2, ws=P3, ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_query_order(*a.values())


def _sel(**kw):
    a = dict(q_codes=P, sorted_codes=P2, perm=P3, S=2, N=100, topk=8, causal=1, chunk=0, q_order=NULL, idx=P4, ws=P,
             ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_select_topk(*a.values())


def _att(**kw):
    a = dict(q=P, k=P2, v=P3, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, d_v=64, topk=8, idx=P4,
             q_order=NULL, score=0, eps=0.5, mean_k=NULL, mean_v=NULL, out=ctypes.c_void_p(0x50000), stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_topk_attn_fwd(*a.values())


ENCODE_CASES = [
    (dict(q=NULL), INV), (dict(k=NULL), INV), (dict(q_codes=NULL), INV), (dict(k_codes=NULL), INV),
    (dict(B=0), INV), (dict(H=-1), INV), (dict(N=0), INV), (dict(N=1 << 31), INV), (dict(B=1 << 20, N=1 << 12), INV),
    (dict(d_k=0), INV), (dict(bits=0), INV), (dict(bits=11), INV), (dict(d_k=4, bits=9), INV),
    (dict(k_codes=P3), INV), (dict(dtype=7), UNS), (dict(d_k=9, bits=3), UNS), (dict(d_k=1, bits=25), UNS),
    (dict(ws=NULL), WSP), (dict(ws_bytes=8), WSP),
]


@pytest.mark.parametrize("kw,code", ENCODE_CASES, ids=[str(c[0]) for c in ENCODE_CASES])
def test_encode_rejects(kw, code):
    assert _enc(**kw) == code


def _enc_static(**kw):
    a = dict(q=P, k=P2, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, bits=10, range_lohi=NULL,
             range_out=NULL, q_codes=P3, k_codes=P4, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_morton_encode_static(*a.values())


@pytest.mark.parametrize("kw,code", [c for c in ENCODE_CASES if "ws" not in c[0] and "ws_bytes" not in c[0]],
                         ids=[str(c[0]) for c in ENCODE_CASES if "ws" not in c[0] and "ws_bytes" not in c[0]])
def test_encode_static_rejects(kw, code):
    """The allocation-free encode validates exactly as the workspace one."""
    assert _enc_static(**kw) == code


def test_encode_static_scratch_limit():
    """Range partials beyond the library's per-GPU array are refused before
    any GPU work: 24 bytes per segment and 512-row chunk at d_k = 3."""
    limit = zb.ZETA_ENCODE_STATIC_SCRATCH_BYTES
    assert limit == 1 << 20
    chunks = 500
    over = limit // (24 * chunks) + 1  # segments whose partials just exceed the array
    assert _enc_static(H=over, N=512 * chunks) == UNS
    assert 24 * (over - 1) * chunks <= limit


SORT_CASES = [
    (dict(k_codes=NULL), INV), (dict(sorted_codes=NULL), INV), (dict(perm=NULL), INV),
    (dict(S=0), INV), (dict(N=0), INV), (dict(N=1 << 31), INV), (dict(code_bits=0), INV), (dict(code_bits=33), INV),
    (dict(sorted_codes=P), INV), (dict(perm=P), INV), (dict(perm=P2), INV),
    (dict(ws=NULL), WSP), (dict(ws_bytes=100), WSP),
]


@pytest.mark.parametrize("kw,code", SORT_CASES, ids=[str(c[0]) for c in SORT_CASES])
def test_sort_rejects(kw, code):
    assert _sort(**kw) == code


SELECT_CASES = [
    (dict(q_codes=NULL), INV), (dict(sorted_codes=NULL), INV), (dict(perm=NULL), INV), (dict(idx=NULL), INV),
    (dict(S=0), INV), (dict(N=0), INV), (dict(topk=0), INV), (dict(causal=2), INV),
    (dict(chunk=-1), INV), (dict(causal=0, chunk=4), INV),  # the chunked rule is causal
    (dict(topk=1025), UNS), (dict(ws=NULL), WSP), (dict(ws_bytes=64), WSP),
    (dict(causal=0, ws=NULL), WSP),  # the window bounds need room even without prefix lists
    (dict(ws=ctypes.c_void_p(0x10008)), INV),  # not 16-byte aligned
]


@pytest.mark.parametrize("kw,code", SELECT_CASES, ids=[str(c[0]) for c in SELECT_CASES])
def test_select_rejects(kw, code):
    assert _sel(**kw) == code


ATTEND_CASES = [
    (dict(q=NULL), INV), (dict(k=NULL), INV), (dict(v=NULL), INV), (dict(idx=NULL), INV), (dict(out=NULL), INV),
    (dict(B=0), INV), (dict(N=0), INV), (dict(d_k=0), INV), (dict(d_v=0), INV), (dict(topk=0), INV),
    (dict(eps=0.0), INV), (dict(eps=-1.0), INV), (dict(eps=float("inf")), INV), (dict(eps=float("nan")), INV),
    (dict(v=ctypes.c_void_p(0x30008)), INV), (dict(out=ctypes.c_void_p(0x50004)), INV), (dict(out=P3), INV),
    (dict(dtype=5), UNS), (dict(d_k=9), UNS), (dict(d_v=96), UNS), (dict(d_v=512), UNS), (dict(topk=2000), UNS),
    (dict(score=5), UNS), (dict(score=-1), UNS),
    (dict(mean_k=ctypes.c_void_p(0xB0000)), INV),  # history means come in pairs
    (dict(mean_v=ctypes.c_void_p(0xC0000)), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0004)), INV),  # mean_v misaligned
]


@pytest.mark.parametrize("kw,code", ATTEND_CASES, ids=[str(c[0]) for c in ATTEND_CASES])
def test_attend_rejects(kw, code):
    assert _att(**kw) == code


QORDER_CASES = [
    (dict(order_out=NULL), INV), (dict(S=0), INV), (dict(N=0), INV), (dict(topk=0), INV), (dict(causal=3), INV),
    (dict(chunk=-1), INV), (dict(causal=0, chunk=8), INV),
    (dict(topk=1025), UNS), (dict(ws=NULL), WSP), (dict(ws_bytes=16), WSP),
    (dict(order_out=ctypes.c_void_p(0x10000 + 64)), INV),  # partial overlap with q_order
]


@pytest.mark.parametrize("kw,code", QORDER_CASES, ids=[str(c[0]) for c in QORDER_CASES])
def test_query_order_rejects(kw, code):
    assert _qord(**kw) == code


def _fused(**kw):
    a = dict(q=P, k=P2, v=P3, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, d_v=64, topk=8, causal=1, chunk=0,
             q_codes=P4, sorted_codes=ctypes.c_void_p(0x60000), perm=ctypes.c_void_p(0x70000), q_order=NULL, score=0,
             eps=0.5,
             mean_k=NULL, mean_v=NULL, out=ctypes.c_void_p(0x50000), idx_out=NULL, ws=ctypes.c_void_p(0x80000),
             ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_select_attend_fwd(*a.values())


FUSED_CASES = [
    (dict(q=NULL), INV), (dict(v=NULL), INV), (dict(out=NULL), INV), (dict(q_codes=NULL), INV),
    (dict(sorted_codes=NULL), INV), (dict(perm=NULL), INV), (dict(B=0), INV), (dict(N=0), INV),
    (dict(d_k=0), INV), (dict(topk=0), INV), (dict(causal=-1), INV), (dict(eps=0.0), INV),
    (dict(eps=float("nan")), INV), (dict(v=ctypes.c_void_p(0x30004)), INV), (dict(out=P), INV),
    (dict(dtype=9), UNS), (dict(d_k=9), UNS), (dict(d_v=48), UNS), (dict(topk=1025), UNS),
    (dict(ws=NULL), WSP), (dict(ws_bytes=32), WSP),
    (dict(ws=ctypes.c_void_p(0x80008)), INV),  # bf16 one pass keeps 8-byte bounds in the workspace
    (dict(mean_v=ctypes.c_void_p(0xC0000)), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0008)), INV),
    (dict(chunk=-2), INV), (dict(causal=0, chunk=16), INV), (dict(score=7), UNS),
    # A score variant with d_k = 3 runs on the matrix-core tiles too, so it
    # needs the one-pass layout: none at all (non-causal needs no lists),
    # 2304 bytes (the select-only layout of this shape: 2 segments x 120 list
    # entries, under the one-pass layout's 7936), or a misaligned buffer.
    (dict(score=1, causal=0, ws=NULL), WSP), (dict(score=1, ws_bytes=2304), WSP),
    (dict(score=2, ws=ctypes.c_void_p(0x80008)), INV),
]


@pytest.mark.parametrize("kw,code", FUSED_CASES, ids=[str(c[0]) for c in FUSED_CASES])
def test_select_attend_rejects(kw, code):
    assert _fused(**kw) == code


def _bwd(**kw):
    a = dict(q=P, k=P2, v=P3, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, d_v=64, topk=8, idx=P4, q_order=NULL,
             dout=ctypes.c_void_p(0x50000), eps=0.5, mean_k=NULL, mean_v=NULL, causal=1,
             dq=ctypes.c_void_p(0x60000), dk=ctypes.c_void_p(0x70000),
             dv=ctypes.c_void_p(0x80000), deps=ctypes.c_void_p(0x90000), ws=ctypes.c_void_p(0xA0000), ws_bytes=BIG,
             stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_topk_attn_bwd(*a.values())


BWD_CASES = [
    (dict(q=NULL), INV), (dict(idx=NULL), INV), (dict(dout=NULL), INV), (dict(dq=NULL), INV), (dict(dk=NULL), INV),
    (dict(dv=NULL), INV), (dict(deps=NULL), INV), (dict(B=0), INV), (dict(N=0), INV), (dict(d_k=0), INV),
    (dict(topk=0), INV), (dict(eps=0.0), INV), (dict(eps=float("inf")), INV),
    (dict(dout=ctypes.c_void_p(0x50004)), INV), (dict(v=ctypes.c_void_p(0x30008)), INV),
    (dict(dk=ctypes.c_void_p(0x60000)), INV),  # dk aliases dq
    (dict(dv=P3), INV),  # dv aliases v
    (dict(deps=P4), INV),  # deps aliases idx
    (dict(dtype=7), UNS), (dict(d_k=9), UNS), (dict(d_v=48), UNS), (dict(topk=1025), UNS),
    (dict(ws=NULL), WSP), (dict(ws_bytes=64), WSP), (dict(causal=2), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000)), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0000), dv=ctypes.c_void_p(0x80004)), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0000), dq=ctypes.c_void_p(0xB0000)), INV),
]


@pytest.mark.parametrize("kw,code", BWD_CASES, ids=[str(c[0]) for c in BWD_CASES])
def test_attend_bwd_rejects(kw, code):
    assert _bwd(**kw) == code


def _obwd(**kw):
    a = dict(q=P, k=P2, v=P3, dtype=zb.ZETA_BF16, B=1, H=2, N=100, d_k=3, d_v=64, topk=8, causal=1, chunk=0,
             q_codes=P4, sorted_codes=ctypes.c_void_p(0xD0000), perm=ctypes.c_void_p(0xE0000), q_order=NULL,
             dout=ctypes.c_void_p(0x50000), eps=0.5, mean_k=NULL, mean_v=NULL, dq=ctypes.c_void_p(0x60000),
             dk=ctypes.c_void_p(0x70000), dv=ctypes.c_void_p(0x80000), deps=ctypes.c_void_p(0x90000),
             ws=ctypes.c_void_p(0xA0000), ws_bytes=BIG, stream=NULL)
    a.update(kw)
    return zeta.load_library().zeta_select_attend_bwd(*a.values())


OBWD_CASES = [
    (dict(q=NULL), INV), (dict(k=NULL), INV), (dict(dout=NULL), INV), (dict(q_codes=NULL), INV),
    (dict(sorted_codes=NULL), INV), (dict(perm=NULL), INV), (dict(dq=NULL), INV), (dict(dk=NULL), INV),
    (dict(dv=NULL), INV), (dict(deps=NULL), INV), (dict(B=0), INV), (dict(N=0), INV), (dict(d_k=0), INV),
    (dict(topk=0), INV), (dict(causal=2), INV), (dict(chunk=-1), INV), (dict(causal=0, chunk=8), INV),
    (dict(eps=0.0), INV), (dict(eps=float("nan")), INV),
    (dict(dout=ctypes.c_void_p(0x50004)), INV), (dict(v=ctypes.c_void_p(0x30008)), INV),
    (dict(dv=ctypes.c_void_p(0x80008)), INV),  # dv is written with 16-byte stores
    (dict(dk=ctypes.c_void_p(0x60000)), INV),  # dk aliases dq
    (dict(dv=P3), INV),  # dv aliases v
    (dict(deps=ctypes.c_void_p(0xE0000)), INV),  # deps aliases perm
    (dict(dtype=7), UNS), (dict(dtype=zb.ZETA_F32), UNS), (dict(d_k=2), UNS), (dict(d_k=4), UNS),
    (dict(d_v=48), UNS), (dict(d_v=512), UNS), (dict(topk=1025), UNS),
    (dict(ws=NULL), WSP), (dict(ws_bytes=64), WSP), (dict(ws=ctypes.c_void_p(0xA0008)), INV),
    (dict(mean_k=ctypes.c_void_p(0xB0000)), INV),  # means come in pairs
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0008)), INV),  # mean_v 16-byte aligned
    (dict(mean_k=ctypes.c_void_p(0xB0000), mean_v=ctypes.c_void_p(0xC0000), dq=ctypes.c_void_p(0xB0000)), INV),
]


@pytest.mark.parametrize("kw,code", OBWD_CASES, ids=[str(c[0]) for c in OBWD_CASES])
def test_select_attend_bwd_rejects(kw, code):
    assert _obwd(**kw) == code


def test_select_attend_bwd_workspace_size():
    ws = zeta.zeta_select_attend_bwd_workspace_size
    assert ws(0, 1, 10, 64, 4, 1) == 0
    assert ws(1, 1, 10, 64, 0, 1) == 0
    assert ws(1, 1, 10, 48, 4, 1) == 0
    assert zeta.load_library().zeta_select_attend_bwd_workspace_size(1, 1, 10, 64, 4, 2, 0) == 0  # causal not 0/1
    # Long-context shape: the one-pass call's buffers plus, per row, the
    # 32-byte record, the dout copy (2 x 128 B) and the deps part.
    big = ws(1, 16, 65536, 128, 128, 1)
    rows = 16 * 65536
    assert big >= rows * (32 + 256 + 4)
    assert big < rows * (32 + 256 + 4) + (96 << 20)
    assert big % 256 == 0
    assert ws(1, 1, 1, 32, 1, 0) > 0
    # The history-mean candidate adds (3 + 128) x 4 B per row and the scan's sums.
    assert ws(1, 16, 65536, 128, 128, 1, True) >= big + rows * 131 * 4
