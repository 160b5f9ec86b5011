"""The C-ABI library loads and exports every function include/dpa4c.h
declares (no GPU needed: nothing is called)."""
import ctypes
import os
import re

import paper_2608_19041_amd as dp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "dpa4c.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?(?:int|void|char|const char)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("build_neighbors", "compute_energy_forces", "verlet_step",
                     "dpa4c_model_create", "dpa4c_model_destroy", "dpa4c_last_error"):
        assert required in names
    assert sorted(dp.exported_symbols()) == names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(dp.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    # the binding wires argument types for all of them
    dp.library()


def test_error_path_without_device():
    # a null blob is rejected before any device work
    lib = dp.library()
    h = ctypes.c_void_p()
    rc = lib.dpa4c_model_create(None, 0, 0, ctypes.byref(h))
    assert rc < 0
    assert lib.dpa4c_last_error()
