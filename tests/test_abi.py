"""C-ABI tests that need no GPU: the library loads, exports what include/fa.h declares, and rejects
every invalid argument on the host before any HIP call (so nothing is launched)."""

import ctypes
import os
import shutil
import subprocess
import re

import pytest

import paper_2609_21264_amd as fa
from paper_2609_21264_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fa.h")

# Fake, 256-byte-aligned addresses: never dereferenced because every call below returns before any
# HIP call.
P = 0x7F0000000000
QP, KP, VP, OP, LP = P, P + 0x1000, P + 0x2000, P + 0x3000, P + 0x4000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fa_\w+)\s*\(", text)))


def call(**kw):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, B=1, Hq=4, Hkv=2, Sq=100, Sk=100, d_qk=128, d_v=128,
             scale=0.125, causal=1, stream=None)
    a.update(kw)
    return fa.fa_fwd_ex(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"], a["Sq"],
                        a["Sk"], a["d_qk"], a["d_v"], a["scale"], a["causal"], a["stream"])


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_21264_amd import build
        build.build()
    return _lib.load()


def test_library_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(_lib.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n
    # dynamic symbol table of the shared object itself
    out = os.popen(f"nm -D --defined-only {_lib.LIB_PATH}").read()
    for n in names:
        assert re.search(rf"\bT {n}$", out, flags=re.M), n


def test_status_strings(lib):
    assert fa.fa_status_str(0) == "FA_OK"
    assert fa.fa_status_str(5) == "FA_ERR_HIP"
    assert fa.fa_status_str(99) == "unknown status"


def test_block_rows(lib):
    for dq, dv in ((64, 64), (128, 128), (192, 128)):
        bm = fa.fa_block_rows(dq, dv, True)
        assert bm > 0 and bm % 32 == 0
    assert fa.fa_block_rows(96, 96, False) == 0
    assert fa.fa_block_rows(128, 64, False) == 0


def _fwd_rows_expected(blocks, d, causal):
    """The dispatch fa.h states for (d, d) problems of `blocks` 256-row blocks."""
    half = (320 if causal else 64) if d == 64 else (192 if causal else 128)
    short = 1024 if d == 64 else 256
    return 64 if blocks <= half else 128 if blocks <= short else 256


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_fwd_rows_follows_the_grid(lib, d, causal):
    # B * Hq * ceil(Sq / 256) blocks, reached through each of the three factors, on both sides of
    # every switch
    for blocks in (1, 2, 63, 64, 65, 128, 129, 192, 193, 255, 256, 257, 320, 321, 1024, 1025, 5000):
        for B, Hq, Sq in ((blocks, 1, 256), (1, blocks, 200), (1, 1, 256 * blocks - 255)):
            assert fa.fa_fwd_rows(B, Hq, Sq, d, d, causal) == _fwd_rows_expected(blocks, d, causal), (B, Hq, Sq)
    assert fa.fa_fwd_rows(0, 8, 100, d, d, causal) in (64, 128, 256)


def test_fwd_rows_other_dims(lib):
    assert fa.fa_fwd_rows(1, 1, 64, 192, 128, True) == fa.fa_block_rows(192, 128, True) == 256
    assert fa.fa_fwd_rows(1, 1, 64, 96, 96, True) == 0
    assert fa.fa_fwd_rows(1, 1, 64, 128, 64, False) == 0
    assert fa.fa_fwd_rows(-1, 1, 64, 64, 64, False) == 0
    assert fa.fa_fwd_rows(1, 1, -64, 64, 64, False) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), fa.FA_ERR_BAD_SHAPE),
    (dict(Hq=-4), fa.FA_ERR_BAD_SHAPE),
    (dict(Sq=-1), fa.FA_ERR_BAD_SHAPE),
    (dict(Sk=-5), fa.FA_ERR_BAD_SHAPE),
    (dict(Hkv=0), fa.FA_ERR_BAD_SHAPE),
    (dict(Hq=4, Hkv=3), fa.FA_ERR_BAD_SHAPE),
    (dict(Hq=2, Hkv=4), fa.FA_ERR_BAD_SHAPE),
    (dict(d_qk=96, d_v=96), fa.FA_ERR_UNSUPPORTED),
    (dict(d_qk=128, d_v=64), fa.FA_ERR_UNSUPPORTED),
    (dict(d_qk=0, d_v=0), fa.FA_ERR_UNSUPPORTED),
    (dict(Q=None), fa.FA_ERR_NULL_POINTER),
    (dict(K=None), fa.FA_ERR_NULL_POINTER),
    (dict(V=None), fa.FA_ERR_NULL_POINTER),
    (dict(O=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("nan")), fa.FA_ERR_BAD_SCALE),
    (dict(scale=float("inf")), fa.FA_ERR_BAD_SCALE),
    (dict(scale=-float("inf")), fa.FA_ERR_BAD_SCALE),
    (dict(scale=3.0e38), fa.FA_ERR_BAD_SCALE),
    (dict(Q=QP + 8), fa.FA_ERR_UNSUPPORTED),
    (dict(K=KP + 2), fa.FA_ERR_UNSUPPORTED),
    (dict(V=VP + 4), fa.FA_ERR_UNSUPPORTED),
    (dict(O=OP + 8), fa.FA_ERR_UNSUPPORTED),
    (dict(LSE=LP + 2), fa.FA_ERR_UNSUPPORTED),
    (dict(Sq=20_000_000), fa.FA_ERR_BAD_SHAPE),       # Sq * d >= 2^31 inside one head
    (dict(Sk=20_000_000), fa.FA_ERR_BAD_SHAPE),
    (dict(B=2_000_000, Hq=4096, Hkv=4096, Sq=1000), fa.FA_ERR_BAD_SHAPE),  # too many workgroups
])
def test_invalid_arguments_are_rejected_on_host(lib, kw, status):
    assert call(**kw) == status


@pytest.mark.parametrize("kw", [dict(B=0), dict(Hq=0, Hkv=0), dict(Sq=0), dict(B=0, Q=None, O=None),
                                dict(Sq=0, Q=None, O=None, LSE=None)])
def test_empty_problems_are_noops_without_hip(lib, kw):
    # returns FA_OK without touching memory or the HIP runtime (no GPU here)
    assert call(**kw) == fa.FA_OK


def test_null_kv_is_allowed_when_there_are_no_keys(lib):
    # Sk == 0 with NULL K/V passes the pointer checks; a size error later proves no launch happened.
    assert call(K=None, V=None, Sk=0, Sq=20_000_000) == fa.FA_ERR_BAD_SHAPE


def test_check_order(lib):
    # several faults at once: the first in the documented order is reported
    assert call(B=-1, d_qk=96, Q=None, scale=float("nan")) == fa.FA_ERR_BAD_SHAPE
    assert call(d_qk=96, Q=None, scale=float("nan")) == fa.FA_ERR_UNSUPPORTED
    assert call(Q=None, scale=float("nan")) == fa.FA_ERR_NULL_POINTER
    assert call(scale=float("nan"), Q=QP + 2) == fa.FA_ERR_BAD_SCALE


def test_fa_fwd_entry_point_validates_on_host(lib):
    L = lib
    assert L.fa_fwd(QP, KP, VP, OP, 1, 4, 2, 64, 64, 100, 0.1, 0, None) == fa.FA_ERR_UNSUPPORTED
    assert L.fa_fwd(QP, KP, VP, None, 1, 4, 2, 64, 64, 64, 0.1, 0, None) == fa.FA_ERR_NULL_POINTER
    assert L.fa_fwd(QP, KP, VP, OP, 0, 4, 2, 64, 64, 64, 0.1, 0, None) == fa.FA_OK


def test_python_forward_rejects_cpu_tensors(lib):
    import torch
    q = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        fa.forward(q, q, q)
    with pytest.raises(ValueError):
        fa.forward(q.float(), q, q)


def test_python_forward_rejects_out_and_lse_on_another_device(lib, monkeypatch):
    """out / lse on another device than q, k, v raise ValueError before any launch. The inputs here
    are CPU tensors with the input check stubbed out (no GPU in this test); out / lse live on the
    meta device, a device different from the inputs'."""
    import torch

    q = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    monkeypatch.setattr(fa, "_check_qkv", lambda q_, k_, v_: (1, 2, 2, 8, 8, 64, 64))
    monkeypatch.setattr(fa, "fa_fwd_ex", lambda *a: pytest.fail("launched despite a bad out / lse"))
    bad_out = torch.empty(1, 2, 8, 64, dtype=torch.bfloat16, device="meta")
    with pytest.raises(ValueError, match="out must be on"):
        fa.forward(q, q, q, out=bad_out)
    bad_lse = torch.empty(1, 2, 8, dtype=torch.float32, device="meta")
    with pytest.raises(ValueError, match="lse must be on"):
        fa.forward(q, q, q, out=torch.empty_like(q), lse=bad_lse)
    with pytest.raises(ValueError, match="out must be a contiguous"):
        fa.forward(q, q, q, out=torch.empty(1, 2, 8, 64, dtype=torch.float32))


# ---- split mode (fa_fwd_split): host-side checks only ----------------------------------------------

WSP = P + 0x10000  # fake, 16-byte aligned workspace address


def call_split(**kw):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, B=1, Hq=4, Hkv=2, Sq=100, Sk=1000, d_qk=128, d_v=128,
             scale=0.125, causal=1, n_split=4, ws=WSP, ws_bytes=None, stream=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = fa.fa_fwd_split_workspace_bytes(max(a["B"], 0), max(a["Hq"], 0), max(a["Sq"], 0),
                                                        max(a["d_v"], 0), max(a["n_split"], 0))
    return fa.fa_fwd_split(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"],
                           a["d_qk"], a["d_v"], a["scale"], a["causal"], a["n_split"], a["ws"], a["ws_bytes"],
                           a["stream"])


def test_split_workspace_bytes(lib):
    assert fa.fa_fwd_split_workspace_bytes(2, 3, 5, 128, 4) == 4 * 2 * 3 * 5 * 129 * 4
    assert fa.fa_fwd_split_workspace_bytes(1, 1, 1, 64, 1) == 65 * 4
    for args in ((0, 3, 5, 128, 4), (2, 0, 5, 128, 4), (2, 3, 0, 128, 4), (2, 3, 5, 0, 4), (2, 3, 5, 128, 0),
                 (-1, 3, 5, 128, 4)):
        assert fa.fa_fwd_split_workspace_bytes(*args) == 0
    assert fa.fa_fwd_split_workspace_bytes(2**31 - 1, 2**31 - 1, 2**31 - 1, 128, 2**31 - 1) == 2**64 - 1


@pytest.mark.parametrize("kw,status", [
    (dict(n_split=0), fa.FA_ERR_BAD_SHAPE),
    (dict(n_split=-3), fa.FA_ERR_BAD_SHAPE),
    (dict(n_split=0, B=-1, Q=None), fa.FA_ERR_BAD_SHAPE),
    (dict(ws=None), fa.FA_ERR_WORKSPACE),
    (dict(ws_bytes=100), fa.FA_ERR_WORKSPACE),
    (dict(ws=WSP + 8), fa.FA_ERR_UNSUPPORTED),
    # the fa_fwd_ex checks come first
    (dict(d_qk=96, d_v=96, ws=None), fa.FA_ERR_UNSUPPORTED),
    (dict(Q=None, ws=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("nan"), ws=None), fa.FA_ERR_BAD_SCALE),
    (dict(Sq=20_000_000, ws=None), fa.FA_ERR_BAD_SHAPE),
    (dict(B=1, Hq=4096, Hkv=4096, Sq=4096 * 64, Sk=64, d_qk=64, d_v=64, n_split=2**20), fa.FA_ERR_BAD_SHAPE),
])
def test_split_invalid_arguments_are_rejected_on_host(lib, kw, status):
    assert call_split(**kw) == status


def test_split_empty_problems_need_no_workspace(lib):
    assert call_split(B=0, ws=None, ws_bytes=0) == fa.FA_OK
    assert call_split(Sq=0, Q=None, O=None, ws=None, ws_bytes=0) == fa.FA_OK


def test_split_status_string(lib):
    assert fa.fa_status_str(6) == "FA_ERR_WORKSPACE"


def test_split_parts_heuristic(lib):
    # decode: 32 query blocks on 256 CUs, 2048 key tiles -> 16 parts (two workgroups per CU)
    assert fa.fa_fwd_split_parts(256, 1, 32, 1, 131072, 128, 128, 0) == 16
    # many query blocks: no split
    assert fa.fa_fwd_split_parts(256, 1, 32, 8192, 8192, 128, 128, 1) == 1
    # 256 blocks: two parts
    assert fa.fa_fwd_split_parts(256, 8, 32, 1, 8192, 128, 128, 0) == 2
    # short keys cap the parts at 8 tiles each
    assert fa.fa_fwd_split_parts(256, 1, 1, 256, 256, 64, 64, 0) == 1
    assert fa.fa_fwd_split_parts(256, 1, 1, 256, 2048, 64, 64, 0) == 4
    # invalid
    assert fa.fa_fwd_split_parts(256, 1, 1, 1, 64, 96, 96, 0) == 0
    assert fa.fa_fwd_split_parts(0, 1, 1, 1, 64, 64, 64, 0) == 0
    assert fa.fa_fwd_split_parts(256, 1, 0, 1, 64, 64, 64, 0) == 0


# ---- layer-by-layer operators: host-side checks only --------------------------------------------

SP = P + 0x20000  # fake, 16-byte aligned spill buffers
PP = P + 0x40000


def call_unfused(**kw):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, B=1, Hq=4, Hkv=2, Sq=300, Sk=500, d_qk=128, d_v=128,
             scale=0.125, causal=1, ws=WSP, ws_bytes=None, stream=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = fa.fa_lbl_workspace_bytes(max(a["B"], 0), max(a["Hq"], 0), max(a["Sq"], 0), max(a["Sk"], 0))
    return fa.fa_fwd_unfused(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"],
                             a["d_qk"], a["d_v"], a["scale"], a["causal"], a["ws"], a["ws_bytes"], a["stream"])


def test_lbl_row_stride_and_workspace_bytes(lib):
    assert [fa.fa_lbl_ld(s) for s in (0, 1, 64, 65, 8192)] == [0, 64, 64, 128, 8192]
    assert fa.fa_lbl_ld(-1) == -1 and fa.fa_lbl_ld(2**22) == 2**22 and fa.fa_lbl_ld(2**22 + 1) == -1
    assert fa.fa_lbl_workspace_bytes(2, 3, 5, 100) == 2 * 3 * 5 * 128 * 2
    for args in ((0, 3, 5, 100), (2, 0, 5, 100), (2, 3, 0, 100), (2, 3, 5, 0), (-1, 3, 5, 100)):
        assert fa.fa_lbl_workspace_bytes(*args) == 0
    assert fa.fa_lbl_workspace_bytes(1, 1, 1, 2**22 + 1) == 2**64 - 1
    assert fa.fa_lbl_workspace_bytes(2**31 - 1, 2**31 - 1, 2**31 - 1, 2**22) == 2**64 - 1


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), fa.FA_ERR_BAD_SHAPE),
    (dict(Hkv=3), fa.FA_ERR_BAD_SHAPE),
    (dict(Sk=2**22 + 64), fa.FA_ERR_BAD_SHAPE),
    (dict(d_qk=96), fa.FA_ERR_UNSUPPORTED),
    (dict(d_v=192), fa.FA_ERR_UNSUPPORTED),
    (dict(Q=None), fa.FA_ERR_NULL_POINTER),
    (dict(V=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("inf")), fa.FA_ERR_BAD_SCALE),
    (dict(O=OP + 2), fa.FA_ERR_UNSUPPORTED),
    (dict(LSE=LP + 2), fa.FA_ERR_UNSUPPORTED),
    (dict(ws=None), fa.FA_ERR_WORKSPACE),
    (dict(ws_bytes=128 * 512 * 2 - 1), fa.FA_ERR_WORKSPACE),
    (dict(ws=WSP + 8), fa.FA_ERR_UNSUPPORTED),
    # checks in order: shape before dims before pointers before scale before alignment before workspace
    (dict(Hkv=3, d_qk=96, Q=None), fa.FA_ERR_BAD_SHAPE),
    (dict(d_qk=96, Q=None, scale=float("nan")), fa.FA_ERR_UNSUPPORTED),
    (dict(Q=None, scale=float("nan"), ws=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("nan"), O=OP + 2), fa.FA_ERR_BAD_SCALE),
    (dict(O=OP + 2, ws=None), fa.FA_ERR_UNSUPPORTED),
])
def test_unfused_invalid_arguments_are_rejected_on_host(lib, kw, status):
    assert call_unfused(**kw) == status


def test_unfused_least_workspace_is_accepted_on_host(lib):
    # one block of 128 rows (all of Sq when shorter) of spill buffer is the least accepted size; the call
    # would launch, so only the rejection side is exercised here
    assert call_unfused(ws_bytes=128 * 512 * 2 - 2) == fa.FA_ERR_WORKSPACE
    assert call_unfused(Sq=50, ws_bytes=50 * 512 * 2 - 2) == fa.FA_ERR_WORKSPACE


def test_unfused_empty_problems_need_no_workspace(lib):
    assert call_unfused(B=0, ws=None, ws_bytes=0) == fa.FA_OK
    assert call_unfused(Sq=0, Q=None, O=None, ws=None, ws_bytes=0) == fa.FA_OK


@pytest.mark.parametrize("name,args,status", [
    ("scores", dict(Q=None), fa.FA_ERR_NULL_POINTER),
    ("scores", dict(S=None), fa.FA_ERR_NULL_POINTER),
    ("scores", dict(d=160), fa.FA_ERR_UNSUPPORTED),
    ("scores", dict(S=SP + 4), fa.FA_ERR_UNSUPPORTED),
    ("scores", dict(scale=float("nan")), fa.FA_ERR_BAD_SCALE),
    ("scores", dict(Sk=2**22 + 1), fa.FA_ERR_BAD_SHAPE),
    ("softmax", dict(S=None), fa.FA_ERR_NULL_POINTER),
    ("softmax", dict(P=None), fa.FA_ERR_NULL_POINTER),
    ("softmax", dict(P=PP + 8), fa.FA_ERR_UNSUPPORTED),
    ("softmax", dict(Hq=-2), fa.FA_ERR_BAD_SHAPE),
    ("pv", dict(P=None), fa.FA_ERR_NULL_POINTER),
    ("pv", dict(V=None), fa.FA_ERR_NULL_POINTER),
    ("pv", dict(d=192), fa.FA_ERR_UNSUPPORTED),
    ("pv", dict(Hkv=0), fa.FA_ERR_BAD_SHAPE),
    # empty problems: nothing to do, no launch
    ("scores", dict(B=0, Q=None, S=None), fa.FA_OK),
    ("scores", dict(Sk=0, K=None, S=None), fa.FA_OK),
    ("softmax", dict(Sq=0, S=None, P=None), fa.FA_OK),
    ("pv", dict(Hq=0, Hkv=0, P=None, O=None), fa.FA_OK),
])
def test_lbl_operators_reject_on_host(lib, name, args, status):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, S=SP, P=PP, B=1, Hq=4, Hkv=2, Sq=200, Sk=300, d=128, scale=0.1,
             causal=1, stream=None)
    a.update(args)
    if name == "scores":
        st = fa.fa_lbl_scores(a["Q"], a["K"], a["S"], a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"], a["d"], a["scale"],
                              a["causal"], a["stream"])
    elif name == "softmax":
        st = fa.fa_lbl_softmax(a["S"], a["P"], a["LSE"], a["B"], a["Hq"], a["Sq"], a["Sk"], a["causal"], a["stream"])
    else:
        st = fa.fa_lbl_pv(a["P"], a["V"], a["O"], a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"], a["d"], a["causal"],
                          a["stream"])
    assert st == status


# ---- decode-shaped path: host-side checks only ----------------------------------------------------

def call_decode(**kw):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, B=1, Hq=32, Hkv=8, Sq=1, Sk=4096, d_qk=128, d_v=128,
             scale=0.125, causal=0, n_parts=4, ws=WSP, ws_bytes=None, stream=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = fa.fa_fwd_split_workspace_bytes(max(a["B"], 0), max(a["Hq"], 0), max(a["Sq"], 0),
                                                        max(a["d_v"], 0), max(a["n_parts"], 0))
    return fa.fa_fwd_decode(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"],
                            a["d_qk"], a["d_v"], a["scale"], a["causal"], a["n_parts"], a["ws"], a["ws_bytes"],
                            a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(n_parts=0), fa.FA_ERR_BAD_SHAPE),
    (dict(n_parts=0, Q=None), fa.FA_ERR_BAD_SHAPE),
    (dict(Hkv=5), fa.FA_ERR_BAD_SHAPE),
    (dict(d_qk=96, d_v=96), fa.FA_ERR_UNSUPPORTED),
    (dict(K=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("nan")), fa.FA_ERR_BAD_SCALE),
    (dict(V=VP + 4), fa.FA_ERR_UNSUPPORTED),
    (dict(Sk=20_000_000), fa.FA_ERR_BAD_SHAPE),
    (dict(ws=None), fa.FA_ERR_WORKSPACE),
    (dict(ws_bytes=64), fa.FA_ERR_WORKSPACE),
    (dict(ws=WSP + 4), fa.FA_ERR_UNSUPPORTED),
    (dict(B=1, Hq=4096, Hkv=4096, Sq=1, n_parts=2 ** 20), fa.FA_ERR_BAD_SHAPE),
])
def test_decode_invalid_arguments_are_rejected_on_host(lib, kw, status):
    assert call_decode(**kw) == status


def test_decode_empty_problems_need_no_workspace(lib):
    assert call_decode(B=0, ws=None, ws_bytes=0) == fa.FA_OK
    assert call_decode(Sq=0, Q=None, O=None, ws=None, ws_bytes=0) == fa.FA_OK


def test_decode_parts_heuristic(lib):
    # 8 key/value heads, one 32-column block each, 1024 tiles of 128 keys: 32 parts (one workgroup per CU)
    assert fa.fa_fwd_decode_parts(256, 1, 32, 8, 1, 131072) == 32
    # 16 rows per query head, 4 heads per group: two column blocks -> 16 parts
    assert fa.fa_fwd_decode_parts(256, 1, 32, 8, 16, 131072) == 16
    # few tiles cap the parts at 4 tiles each
    assert fa.fa_fwd_decode_parts(256, 1, 32, 8, 1, 1024) == 2
    assert fa.fa_fwd_decode_parts(256, 1, 32, 8, 1, 100) == 1
    for args in ((0, 1, 32, 8, 1, 100), (256, 0, 32, 8, 1, 100), (256, 1, 32, 5, 1, 100), (256, 1, 32, 8, 0, 100),
                 (256, 1, 32, 8, 1, -1)):
        assert fa.fa_fwd_decode_parts(*args) == 0


# ---- allocation-free decode entry point: host-side checks only ------------------------------------

def call_noalloc(**kw):
    a = dict(Q=QP, K=KP, V=VP, O=OP, LSE=LP, B=1, Hq=32, Hkv=8, Sq=1, Sk=4096, d_qk=128, d_v=128,
             scale=0.125, causal=0, n_parts=4, stream=None)
    a.update(kw)
    return fa.fa_fwd_decode_noalloc(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"], a["Sq"],
                                    a["Sk"], a["d_qk"], a["d_v"], a["scale"], a["causal"], a["n_parts"], a["stream"])


def test_noalloc_scratch_size_matches_header(lib):
    m = re.search(r"#define\s+FA_NOALLOC_SCRATCH_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == fa.FA_NOALLOC_SCRATCH_BYTES


# Largest partial-result count that fits: rows * n_parts * (d_v + 1) * 4 <= 32 MiB.
_ROWS_FIT = fa.FA_NOALLOC_SCRATCH_BYTES // (129 * 4)


@pytest.mark.parametrize("kw,status", [
    (dict(n_parts=0), fa.FA_ERR_BAD_SHAPE),
    (dict(n_parts=0, Q=None), fa.FA_ERR_BAD_SHAPE),
    (dict(Hkv=5), fa.FA_ERR_BAD_SHAPE),
    (dict(d_qk=96, d_v=96), fa.FA_ERR_UNSUPPORTED),
    (dict(K=None), fa.FA_ERR_NULL_POINTER),
    (dict(scale=float("nan")), fa.FA_ERR_BAD_SCALE),
    (dict(V=VP + 4), fa.FA_ERR_UNSUPPORTED),
    (dict(Sk=20_000_000), fa.FA_ERR_BAD_SHAPE),
    (dict(B=1, Hq=4096, Hkv=4096, Sq=1, n_parts=2 ** 20), fa.FA_ERR_BAD_SHAPE),
    # partial results one row past the scratch (B*Hq*Sq rows, one part): rejected before any HIP call
    (dict(B=1, Hq=1, Hkv=1, Sq=_ROWS_FIT + 1, n_parts=1), fa.FA_ERR_WORKSPACE),
    (dict(B=1, Hq=32, Hkv=8, Sq=64, n_parts=_ROWS_FIT // (32 * 64) + 1), fa.FA_ERR_WORKSPACE),
    # an invalid argument still wins over the size
    (dict(B=1, Hq=1, Hkv=1, Sq=_ROWS_FIT + 1, n_parts=1, scale=float("inf")), fa.FA_ERR_BAD_SCALE),
])
def test_noalloc_invalid_arguments_are_rejected_on_host(lib, kw, status):
    assert call_noalloc(**kw) == status


def test_noalloc_empty_problems_are_noops_without_hip(lib):
    assert call_noalloc(B=0) == fa.FA_OK
    assert call_noalloc(Sq=0, Q=None, O=None) == fa.FA_OK
    assert call_noalloc(Hq=0, Hkv=0) == fa.FA_OK


def _compile(cmd, source, suffix, tmp_path):
    path = tmp_path / f"t{suffix}"
    path.write_text(source)
    res = subprocess.run(cmd + [str(path)], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr


def test_header_compiles_as_c99(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = '#include "fa.h"\nint main(void) { hipStream_t s = NULL; return (int)fa_fwd(0, 0, 0, 0, 0, 0, 0, 0, 0, 64, 1.0f, 0, s); }\n'
    _compile(["gcc", "-x", "c", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I", os.path.dirname(HEADER)],
             src, ".c", tmp_path)


@pytest.mark.parametrize("hip_first", [True, False], ids=["hip-header-first", "fa-header-first"])
def test_header_stream_type_is_hips(tmp_path, hip_first):
    """fa.h declares hipStream_t exactly as HIP does, so either header may come first."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    inc = ['#include <hip/hip_runtime_api.h>', '#include "fa.h"']
    if not hip_first:
        inc.reverse()
    src = "\n".join(inc) + "\nint main() { hipStream_t s = nullptr; hipStreamCreate(&s); return (int)fa_fwd(0, 0, 0, 0, 0, 0, 0, 0, 0, 64, 1.f, 0, s); }\n"
    _compile([hipcc, "-fsyntax-only", "-Wno-unused-command-line-argument", "-I", os.path.dirname(HEADER)],
             src, ".cpp", tmp_path)
