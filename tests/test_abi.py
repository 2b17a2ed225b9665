"""The C-ABI library loads and exports every function include/oc.h declares;
argument errors are reported before any device work (runs without a GPU)."""
import ctypes as C
import os
import re

import pytest

import paper_1712_01537_amd as oc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "oc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(oc_[a-z0-9_]+)\s*\(", src)))


def test_header_matches_binding():
    names = _declared()
    assert "oc_build" in names and "oc_conv_bwd" in names
    assert sorted(oc.EXPORTS) == names


def test_library_exports_every_symbol():
    L = oc.load()
    for name in _declared():
        assert hasattr(L, name), name


def test_argument_errors_without_device():
    L = oc.load()
    out = C.c_void_p()
    offs = (C.c_int32 * 3)(0, 0, 0)
    assert L.oc_build(None, None, offs, 0, 3, 2, None, None, C.byref(out)) == 1   # batch 0
    assert L.oc_build(None, None, offs, 2, 9, 2, None, None, C.byref(out)) == 1   # depth 9
    assert L.oc_build(None, None, offs, 2, 3, 4, None, None, C.byref(out)) == 1   # full > depth
    assert L.oc_build(None, None, None, 2, 3, 2, None, None, C.byref(out)) == 1   # no offsets
    bad = (C.c_int32 * 3)(0, 5, 2)
    assert L.oc_build(None, None, bad, 2, 3, 2, None, None, C.byref(out)) == 1    # decreasing
    assert b"decrease" in L.oc_last_error()
    assert L.oc_build(None, None, (C.c_int32 * 2)(0, 4), 1, 3, 2, None, None, C.byref(out)) == 1
    job = C.c_void_p(1)
    assert L.oc_build_async(None, None, offs, 0, 3, 2, None, None, C.byref(job)) == 1
    assert not job.value  # no job on failure
    assert L.oc_build_async(None, None, bad, 2, 3, 2, None, None, C.byref(job)) == 1
    assert L.oc_build_async(None, None, offs, 2, 3, 2, None, None, None) == 1
    assert L.oc_build_finish(None, None, C.byref(out)) == 1
    L.oc_build_cancel(None)
    assert L.oc_conv_fwd(None, 1, 3, 1, 0, None, 3, None, 4, None, None, 0, 0, None) == 1
    assert L.oc_pool_fwd(None, 1, None, 3, None, None, None) == 1
    assert L.oc_deconv_fwd(None, 1, 3, 1, 0, None, 4, None, 3, None, None, 0, 0, None) == 1
    assert L.oc_deconv_bwd(None, 1, 3, 1, 0, None, 4, None, 3, None, None, None, None, 0, 0,
                           None) == 1
    assert L.oc_deconv_fwd_workspace(None, 1, 3, 1, 0, 4, 3) == 0
    assert L.oc_gpool_fwd(None, 1, 3, 1, 0, None, 4, None, None, None) == 1
    assert L.oc_gpool_bwd(None, 1, 3, 1, 1, None, None, 4, None, None) == 1
    off, npart, cnt = C.c_size_t(), C.c_int32(), C.c_int64()
    assert L.oc_conv_dw_partials(None, 1, 3, 1, 0, 4, 4, C.byref(off), C.byref(npart),
                                 C.byref(cnt)) == 1
    assert L.oc_sum_partials(-1, None, None, None, None, None) == 1
    assert L.oc_sum_partials(0, None, None, None, None, None) == 0
    one = (C.c_void_p * 1)(None)
    assert L.oc_sum_partials(1, one, (C.c_int32 * 1)(0), (C.c_int64 * 1)(4), one, None) == 1
    assert L.oc_sum_partials(1, None, (C.c_int32 * 1)(2), (C.c_int64 * 1)(4), one, None) == 1
    assert L.oc_round_bf16(-1, None, None, None) == 1
    assert L.oc_round_bf16(0, None, None, None) == 0
    assert L.oc_round_bf16(4, None, None, None) == 1
    assert L.oc_octree_signal(None) is None
    assert L.oc_status_str(2) == b"point outside the unit cube"
    L.oc_octree_free(None)


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(oc, "_lib", None)
    monkeypatch.setattr(oc, "lib_path", lambda: str(tmp_path / "liboc.so"))
    with pytest.raises(oc.OcError):
        oc.load()
