"""The C-ABI library loads and exports every function include/netkv.h
declares (no compute calls: runs without a GPU)."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "netkv.h")) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(netkv_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("netkv_oracle_load", "netkv_cache_load", "netkv_select_batch", "netkv_rank_sweep",
              "netkv_create", "netkv_destroy", "netkv_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    import torch  # noqa: F401  (the binding maps torch's HIP runtime first)
    from paper_2606_03910_amd import netkv
    lib = netkv.load_library()
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(netkv._SIGS) == set(_declared())


def test_binding_has_the_same_names():
    from paper_2606_03910_amd import netkv
    for n in _declared():
        assert callable(getattr(netkv, n)), n


def test_create_without_gpu_fails_cleanly():
    import torch
    from paper_2606_03910_amd import netkv
    if torch.cuda.is_available():
        return
    h = ctypes.c_void_p()
    st = netkv.load_library().netkv_create(ctypes.byref(h), 0)
    assert st == -1 and not h.value
    assert netkv.load_library().netkv_last_error(None) == b"NULL handle"


def test_library_is_native_gfx950():
    from paper_2606_03910_amd import netkv
    with open(netkv.LIB_PATH, "rb") as f:
        blob = f.read()
    assert b"gfx950" in blob
