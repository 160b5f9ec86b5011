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


def test_too_many_species_rejected_before_device_work():
    # the per-call species bitmask covers 128 type rows: a header with more is
    # refused as unsupported, before any device call
    import struct

    import synth

    spec, weights = synth.model_weights("small")
    blob = bytearray(synth.pack_blob(spec, weights))
    assert blob[:8] == b"DPA4CW01"
    struct.pack_into("<i", blob, 36, 200)   # n_types, the seventh int32 after the version
    lib = dp.library()
    h = ctypes.c_void_p()
    buf = (ctypes.c_char * len(blob)).from_buffer(blob)
    rc = lib.dpa4c_model_create(buf, len(blob), 0, ctypes.byref(h))
    assert rc == -2
    assert b"127 species" in lib.dpa4c_last_error()
