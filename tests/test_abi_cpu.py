"""CPU-side checks of the boundary: the built library loads without a GPU and
exports every function include/*.h declares; the binding declares the same
set; no product module imports the oracle."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]
LIB = os.path.join(ROOT, "paper_2202_11836_amd", "libskystage.so")


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b((?:stage|alloc)_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_header_declares_the_stage_calls():
    names = declared_functions()
    for n in ("stage_init", "stage_forward", "stage_backward", "stage_param", "stage_grad",
              "stage_destroy", "stage_last_error", "alloc_coarse", "alloc_fine", "alloc_workloads"):
        assert n in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_binding_covers_every_declared_symbol():
    from paper_2202_11836_amd import binding
    assert sorted(binding.EXPORTED) == declared_functions()


def test_product_path_does_not_import_oracle():
    pkg = os.path.join(ROOT, "paper_2202_11836_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", txt, flags=re.M), f
                assert "oracle/" not in txt, f


def test_missing_library_fails_loudly(tmp_path):
    from paper_2202_11836_amd import binding
    with pytest.raises(RuntimeError):
        binding.load_library.__wrapped__(str(tmp_path / "nope.so")) if hasattr(binding.load_library, "__wrapped__") \
            else _load_fresh(binding, str(tmp_path / "nope.so"))


def _load_fresh(binding, path):
    saved = binding._lib
    binding._lib = None
    try:
        binding.load_library(path)
    finally:
        binding._lib = saved


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")
def test_mfma_peak_rejects_bad_arguments():
    # argument checks come before any device call
    lib = ctypes.CDLL(LIB)
    t, g = ctypes.c_double(0.0), ctypes.c_double(0.0)
    f = lib.stage_mfma_peak
    f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                  ctypes.POINTER(ctypes.c_double)]
    f.restype = ctypes.c_int
    assert f(None, 0, ctypes.byref(t), ctypes.byref(g)) == 1
    assert f(None, 1 << 25, ctypes.byref(t), ctypes.byref(g)) == 1
    assert f(None, 100, None, ctypes.byref(g)) == 1


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")
def test_init_units_rejects_bad_arguments():
    # unit-range and dims checks come before any device call
    lib = ctypes.CDLL(LIB)
    f = lib.stage_init_units
    f.argtypes = [ctypes.c_int] * 5 + [ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_void_p)]
    f.restype = ctypes.c_int
    out = ctypes.c_void_p(1)
    for u0, n, h, H, ffn in [(-1, 2, 128, 2, 256), (0, 0, 128, 2, 256), (3, -1, 128, 2, 256),
                             ((1 << 30) - 1, 2, 128, 2, 256), (0, 2, 100, 2, 256),
                             (1, 3, 128, 3, 256), (0, 1, 128, 2, 500)]:
        assert f(u0, n, h, H, ffn, 0, 1, None, ctypes.byref(out)) == 1, (u0, n, h, H, ffn)
        assert out.value is None
    assert f(0, 2, 128, 2, 256, 0, 1, None, None) == 1
    init = lib.stage_init
    init.argtypes = [ctypes.c_int] * 4 + [ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_void_p)]
    init.restype = ctypes.c_int
    assert init(0, 128, 2, 256, 0, 1, None, ctypes.byref(out)) == 1
    assert init((1 << 29) + 1, 128, 2, 256, 0, 1, None, ctypes.byref(out)) == 1
