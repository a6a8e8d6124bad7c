"""The C ABI without a GPU: the library loads, exports every entry point of
include/cold.h, validates model descriptions, sizes arenas and workspaces,
and rejects bad calls before touching the device."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2007_16122_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cold.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cold_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert header_functions() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = B.lib()
    for name in header_functions():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (cold_[a-z_]+)\b", out))
    assert set(header_functions()) <= exported


def desc(**kw):
    base = dict(n_user=12, n_seq=0, n_ad=24, n_cross=12, emb_dim=16, dtype="bf16",
                se_reduction=4, widths=[768, 1024, 512, 256, 128, 64, 2],
                table_rows=[1000] * 48)
    base.update(kw)
    return B.make_desc(**base)


def create_status(**kw):
    d, keep = desc(**kw)
    h = ctypes.c_void_p()
    st = B.lib().cold_create_model(ctypes.byref(d), ctypes.byref(h))
    if st == B.COLD_OK:
        B.cold_destroy_model(h)
    return st


@pytest.mark.parametrize("kw,status", [
    (dict(), B.COLD_OK),
    (dict(dtype="f16", linear_log=True), B.COLD_OK),
    (dict(dtype="f32", emb_dim=8, widths=[384, 64, 1]), B.COLD_OK),
    (dict(hashed=True), B.COLD_OK),
    (dict(topk_k=10), B.COLD_OK),
    (dict(n_user=-1), B.COLD_ERR_INVALID_ARG),
    (dict(se_reduction=0), B.COLD_ERR_INVALID_ARG),
    (dict(dtype=7), B.COLD_ERR_DTYPE),
    (dict(emb_dim=12), B.COLD_ERR_DTYPE),            # 24 bytes per row: not 16-byte chunks
    (dict(widths=[700, 1024, 2]), B.COLD_ERR_SHAPE),  # D_in != M * d
    (dict(widths=[768, 1024, 3]), B.COLD_ERR_SHAPE),  # head must be 1 or 2
    (dict(widths=[768, 1020, 2]), B.COLD_ERR_DTYPE),  # half hidden width % 8
    (dict(table_rows=[0] + [1000] * 47), B.COLD_ERR_SHAPE),
    (dict(table_rows=[2**31] + [1000] * 47), B.COLD_ERR_SHAPE),
    (dict(cross_pairs=[(f, f) for f in range(12)]), B.COLD_OK),
    (dict(cross_pairs=[(12, 0)] + [(0, 0)] * 11), B.COLD_ERR_SHAPE),   # user field >= n_user
    (dict(cross_pairs=[(0, 24)] + [(0, 0)] * 11), B.COLD_ERR_SHAPE),   # ad field >= n_ad
    (dict(cross_pairs=[(-1, 0)] + [(0, 0)] * 11), B.COLD_ERR_SHAPE),
    (dict(se_form=B.COLD_SE_LITERAL), B.COLD_OK),
    (dict(se_form=2), B.COLD_ERR_INVALID_ARG),
])
def test_create_model_validation(kw, status):
    assert create_status(**kw) == status


def test_create_model_null_args():
    L = B.lib()
    h = ctypes.c_void_p()
    assert L.cold_create_model(None, ctypes.byref(h)) == B.COLD_ERR_INVALID_ARG
    d, keep = desc()
    assert L.cold_create_model(ctypes.byref(d), None) == B.COLD_ERR_INVALID_ARG


def test_sizes():
    d, keep = desc()
    h = B.cold_create_model(d)
    try:
        arena = B.cold_weight_arena_bytes(h)
        # SE + MLP weights in bf16 + biases, at least
        mlp = sum(a * b for a, b in zip(d.widths[:6], [1024, 512, 256, 128, 64, 2])) * 2
        assert arena >= mlp + 4 * 2 * 12 * 48 and arena % 256 == 0
        w0 = B.cold_workspace_bytes(h, 0, 0)
        w1 = B.cold_workspace_bytes(h, 64000, 32)
        assert w1 > w0 and w1 % 256 == 0
        assert w1 >= 64000 * 768 * 2 + 2 * 64000 * 1024 * 2   # X + two activation buffers
        assert B.cold_workspace_bytes(h, -1, 0) == 0
        assert B.lib().cold_workspace_bytes(None, 10, 1) == 0
        assert B.lib().cold_weight_arena_bytes(None) == 0
    finally:
        B.cold_destroy_model(h)


def test_noalloc_array_holds_one_wide_request():
    """The no-allocation entry point's array holds the workspace of the wide
    top-k model's 5,000-row request (compacted first-layer input and weight
    columns included) and of eight 2,000-ad requests of the serving model."""
    d, keep = desc(n_user=50, n_ad=100, n_cross=50, widths=[3200, 1024, 512, 256, 128, 64, 2],
                   table_rows=[1000] * 200, topk_k=100)
    h = B.cold_create_model(d)
    try:
        assert B.cold_workspace_bytes(h, 5000, 1) <= B.COLD_NOALLOC_WORKSPACE_BYTES
        # the compacted input and weight columns are part of it
        d2, keep2 = desc(n_user=50, n_ad=100, n_cross=50, widths=[3200, 1024, 512, 256, 128, 64, 2],
                         table_rows=[1000] * 200, topk_k=200)
        h2 = B.cold_create_model(d2)
        try:
            grow = B.cold_workspace_bytes(h, 5000, 1) - B.cold_workspace_bytes(h2, 5000, 1)
            assert grow >= 2 * (5000 * 1600 + 1024 * 1600)
        finally:
            B.cold_destroy_model(h2)
    finally:
        B.cold_destroy_model(h)
    d, keep = desc()
    h = B.cold_create_model(d)
    try:
        assert B.cold_workspace_bytes(h, 16000, 8) <= B.COLD_NOALLOC_WORKSPACE_BYTES
        assert B.cold_workspace_bytes(h, 18000, 9) > B.COLD_NOALLOC_WORKSPACE_BYTES
    finally:
        B.cold_destroy_model(h)


def test_score_before_load_and_bad_calls():
    d, keep = desc()
    h = B.cold_create_model(d)
    try:
        b = B.cold_batch(n_requests=1, n_rows=10)
        st = B.cold_score(h, b, None, 0, None, None, None, None, None, 0, None)
        assert st == B.COLD_ERR_NOT_LOADED
        assert "before cold_load_weights" in B.cold_last_error(h)
        st = B.lib().cold_score(h, None, None, 0, None, None, None, None, None, 0, None)
        assert st == B.COLD_ERR_INVALID_ARG
        st = B.cold_score(h, b, None, 0, None, None, None, None, None, 0x10, None)
        assert st == B.COLD_ERR_INVALID_ARG
        assert B.lib().cold_score(None, ctypes.byref(b), None, 0, None, None, None, None, None, 0,
                                  None) == B.COLD_ERR_INVALID_ARG
        w = B.cold_weights()
        assert B.cold_load_weights(h, w, None, 0, None) == B.COLD_ERR_INVALID_ARG
        assert "null" in B.cold_last_error(h)
    finally:
        B.cold_destroy_model(h)


def test_status_strings():
    for st in range(0, -8, -1):
        s = B.cold_status_string(st)
        assert s and s != "unknown status"
    assert B.cold_status_string(-99) == "unknown status"
    assert B.lib().cold_last_error(None) == b"null model"
    B.lib().cold_destroy_model(None)   # no-op


def test_select_topn_rejects_bad_calls_before_the_device():
    fake = 0x1000   # never dereferenced: every call below fails its host checks
    sel = B.cold_select_topn
    assert sel(fake, fake, fake, 1, 10, 0, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, fake, 1, 10, B.COLD_TOPN_MAX + 1, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, fake, -1, 10, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, fake, 1, -1, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, fake, 1, 1 << 31, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, None, 1, 10, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, fake, fake, 1, 10, 5, None, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(None, fake, fake, 1, 10, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    assert sel(fake, None, fake, 1, 10, 5, fake, None, None) == B.COLD_ERR_INVALID_ARG
    # no requests: nothing to do, nothing enqueued
    assert sel(None, None, None, 0, 0, 5, None, None, None) == B.COLD_OK


def test_literal_se_arena_holds_the_full_layer():
    sizes = {}
    for form in (B.COLD_SE_SQUEEZE, B.COLD_SE_LITERAL):
        d, keep = desc(se_form=form)
        h = B.cold_create_model(d)
        try:
            sizes[form] = B.cold_weight_arena_bytes(h)
        finally:
            B.cold_destroy_model(h)
    # literal: W [48][768] + b [48] fp32 instead of W1 [12][48], b1, W2 [48][12], b2,
    # the transposed copies of W1 and W2 and the two 4 KB operand-order copies
    # that the squeeze form keeps
    grow = 4 * (48 * 768 + 48) - 4 * (2 * 12 * 48 + 12 + 2 * 48 * 12 + 48) - 2 * 4096
    assert sizes[B.COLD_SE_LITERAL] - sizes[B.COLD_SE_SQUEEZE] >= grow - 4 * 256


def test_probe_library_exports_its_declared_symbol():
    """libcold_probe.so (the row-gather measurement aid beside the scoring
    library) exports what include/cold_probe.h declares, and rejects bad
    arguments before anything is enqueued."""
    from paper_2007_16122_amd import build as hip_build
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "cold_probe.h")).read(),
                  flags=re.S)
    names = sorted(set(re.findall(r"\b(cold_[a-z_]+)\s*\(", text)))
    assert names == ["cold_probe_row_gather"]
    out = subprocess.run(["nm", "-D", "--defined-only", hip_build.PROBE_LIB], capture_output=True,
                         text=True, check=True).stdout
    assert set(names) <= set(re.findall(r"\bT (cold_[a-z_]+)\b", out))
    L = ctypes.CDLL(hip_build.PROBE_LIB)
    f = L.cold_probe_row_gather
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_void_p]
    p = ctypes.c_void_p(16)          # never dereferenced: each call is rejected on the host
    assert f(None, 10, p, p, 4, None) == -1
    assert f(p, 0, p, p, 4, None) == -1
    assert f(p, 10, p, p, -1, None) == -1
    assert f(p, 10, None, p, 4, None) == -1
    assert f(p, 10, p, p, 0, None) == 0   # nothing to gather: nothing enqueued
