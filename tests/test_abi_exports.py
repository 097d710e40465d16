"""The C-ABI library loads without a GPU and exports every function that
include/buddy.h declares; the host-only helpers answer correctly."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    src = open(os.path.join(ROOT, "include", "buddy.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(buddy_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared()
    for n in ("buddy_pool_route", "buddy_select_topk", "buddy_decode_step",
              "buddy_model_create", "buddy_model_destroy"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2606_09514_amd import lib as blib
    L = blib.lib()
    missing = [n for n in declared() if not hasattr(L, n)]
    assert not missing, missing


def test_host_helpers():
    from paper_2606_09514_amd import lib as blib
    from paper_2606_09514_amd import costmodel
    for b in (0.3, 0.5, 0.625, 0.75, 0.875, 1.0):
        assert blib.budget_to_k(b, 32) == costmodel.budget_to_k(b, 32)
    assert blib.budget_to_k(0.0, 32) == -1 and blib.budget_to_k(1.5, 32) == -1
    L = blib.lib()
    for s in range(7):
        assert L.buddy_status_string(s)
    assert L.buddy_last_error(None) == b""


def test_entry_points_reject_null_handles_without_a_device():
    from paper_2606_09514_amd import lib as blib
    L = blib.lib()
    kv = blib.KV(None, None)
    assert L.buddy_decode_step(None, ctypes.byref(kv), None, None, None, 1, 0,
                               None, None, None, None) == blib.EINVAL
    assert L.buddy_pool_route(None, ctypes.byref(kv), None, None, 1, None, None) == blib.EINVAL
    assert L.buddy_select_topk(None, None, 1, 4, None, None) == blib.EINVAL
    out = ctypes.c_void_p(1)
    assert L.buddy_model_create(None, None, None, ctypes.byref(out)) == blib.EINVAL
    assert out.value is None


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    """No fallback: with the shared library absent, the binding raises
    instead of computing anything."""
    from paper_2606_09514_amd import lib as blib
    monkeypatch.setattr(blib, "_SO", str(tmp_path / "libbuddy.so"))
    monkeypatch.setattr(blib, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        blib.lib()
