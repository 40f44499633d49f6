"""The C-ABI library loads and exports every entry point its header declares
(no GPU calls here)."""
import ctypes
import os
import re

import pytest

import paper_2609_32166_amd as pf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in os.listdir(inc):
        if f.endswith(".h"):
            text = open(os.path.join(inc, f)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(pf_[a-z0-9_]+)\s*\(", text))
    return names


def test_header_declares_the_step_calls():
    d = _declared()
    for n in ("pf_store_build", "pf_draft_lookup", "pf_verify_step", "pf_kv_commit", "pf_prefill"):
        assert n in d


def test_library_exports_every_declared_symbol():
    if not os.path.exists(pf.LIB_PATH):
        pytest.fail("libpf.so not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(pf.LIB_PATH)
    missing = [n for n in sorted(_declared()) if not hasattr(lib, n)]
    assert not missing, missing
    assert set(pf.EXPORTED) <= _declared()


def test_record_layouts_match_header():
    assert pf.DRAFT_DTYPE.itemsize == 1384
    assert pf.RESULT_DTYPE.itemsize == 808
    assert ctypes.sizeof(pf.pf_kv_cache) == 56
    assert ctypes.sizeof(pf.pf_context) == 32
    assert ctypes.sizeof(pf.pf_model_config) == 48
    assert ctypes.sizeof(pf.pf_ctl_params) == 32
    assert ctypes.sizeof(pf.pf_ctl_state) == 168
    assert ctypes.sizeof(pf.pf_iteration) == 40


def test_error_paths_without_gpu():
    """Argument checks happen on the host before any launch."""
    lib = pf.lib()
    out = ctypes.c_void_p()
    assert lib.pf_store_build(None, None, 0, 3, None, ctypes.byref(out)) == pf.PF_EINVAL
    assert "offsets" in pf.last_error()
    assert lib.pf_model_create(None, None, None, ctypes.byref(out)) == pf.PF_EINVAL
    cfg = pf.pf_model_config(2, 256, 4, 2, 96, 688, 4096, pf.PF_DTYPE_F32, 1e4, 1e-6)
    w = pf.pf_model_weights(*([1] * 9))
    assert lib.pf_model_create(ctypes.byref(cfg), ctypes.byref(w), None,
                               ctypes.byref(out)) == pf.PF_EUNSUPPORTED
    assert lib.pf_verify_step(None, None, None, 9, 0, None, None, None) == pf.PF_EINVAL
    assert lib.pf_kv_commit(None, None, None, None) == pf.PF_EINVAL
    assert lib.pf_kv_carry(None, None, 0, None, None, None, None) == pf.PF_EINVAL
    assert lib.pf_store_reserve(None, 1, 1, None) == pf.PF_EINVAL
    assert lib.pf_store_append_verified(None, None, None, None, None) == pf.PF_EINVAL
    assert lib.pf_decode_iteration(*([None] * 6), 0, 0, *([None] * 5)) == pf.PF_EINVAL
    assert lib.pf_ctl_create(None, ctypes.byref(out)) == pf.PF_EINVAL
