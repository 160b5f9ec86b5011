"""Oracle neighbour list (test infrastructure only).

Thin ctypes wrapper around ``neighbors.c`` (the brute-force definition of
Eq. (neighbor-set) with an exact fixed-point predicate), plus a pure-Python
version of the same definition for tiny systems that pins the C code.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "neighbors.c")
_LIB = os.path.join(_HERE, "_neighbors.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile neighbors.c with gcc into oracle/_neighbors.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_neighbors_brute.restype = ctypes.c_int
        lib.oracle_neighbors_brute.argtypes = [
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double,
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]
        _lib = lib
    return _lib


def neighbor_list(pos, cell, pbc, r, centres=None):
    """Edges (i, j, n) of Eq. (neighbor-set) in canonical order.

    Returns (i int64 [E], j int64 [E], n int64 [E, 3]).
    """
    lib = _load()
    pos = np.ascontiguousarray(pos, dtype=np.float64)
    cell = np.ascontiguousarray(cell, dtype=np.float64).reshape(9)
    pbc = np.ascontiguousarray(pbc, dtype=np.int32)
    n = pos.shape[0]
    if centres is not None:
        centres = np.ascontiguousarray(centres, dtype=np.int64)
        nc = centres.shape[0]
        cptr = centres.ctypes.data
    else:
        nc, cptr = n, None
    cap = max(1024, int(nc * 200))
    while True:
        oi = np.empty(cap, np.int64)
        oj = np.empty(cap, np.int32)
        on = np.empty((cap, 3), np.int32)
        cnt = ctypes.c_int64(0)
        rc = lib.oracle_neighbors_brute(pos.ctypes.data, n, cell.ctypes.data, pbc.ctypes.data,
                                        float(r), cptr, nc, cap, oi.ctypes.data, oj.ctypes.data,
                                        on.ctypes.data, ctypes.byref(cnt))
        if rc == 2:
            raise ValueError("bad neighbour-list input")
        if rc == 0:
            e = cnt.value
            return oi[:e].copy(), oj[:e].astype(np.int64), on[:e].astype(np.int64)
        cap = cnt.value


def neighbor_list_python(pos, cell, pbc, r, n_image: int = 3):
    """Same definition with Python integers and a fixed wide image box.

    For tiny systems only: every image with |n_a| <= n_image on periodic
    axes is tested.  Used to pin the C implementation.
    """
    q = lambda x: int(np.rint(np.float64(x) * 1048576.0))
    n = len(pos)
    qp = [[q(pos[i][a]) for a in range(3)] for i in range(n)]
    qh = [[q(cell[b][a]) for a in range(3)] for b in range(3)]
    qr = q(r)
    rng = [range(-n_image, n_image + 1) if pbc[a] else range(0, 1) for a in range(3)]
    out = []
    for i in range(n):
        for j in range(n):
            for nx in rng[0]:
                for ny in rng[1]:
                    for nz in rng[2]:
                        if i == j and nx == 0 and ny == 0 and nz == 0:
                            continue
                        d = [qp[j][a] + nx * qh[0][a] + ny * qh[1][a] + nz * qh[2][a] - qp[i][a]
                             for a in range(3)]
                        if d[0] * d[0] + d[1] * d[1] + d[2] * d[2] < qr * qr:
                            out.append((i, j, nx, ny, nz))
    return out


def edge_vectors(pos, cell, i, j, n):
    """r_ij = (r_j + n.h) - r_i in float64 from the unquantised positions."""
    return pos[j] + n @ np.asarray(cell) - pos[i]
