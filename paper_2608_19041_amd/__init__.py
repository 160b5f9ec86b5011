"""Python binding of libdpa4c (the C ABI in include/dpa4c.h).

Argument marshalling only: every step of the energy-and-force path runs in
the HIP kernels of the library.  torch supplies device memory and the
current stream.  Importing works without a GPU; calling anything that needs
the library raises :class:`DPA4CError` if libdpa4c.so has not been built
(``python -m paper_2608_19041_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdpa4c.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_CAPACITY = -3
ERR_HIP = -4
ERR_NONFINITE = -5
ERR_SKIN = -6
ERR_OOM = -7

_lib = None


class DPA4CError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"dpa4c error {code}: {msg}")
        self.code = code


def library():
    """The loaded libdpa4c.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DPA4CError(ERR_UNSUPPORTED, f"{LIB_PATH} is missing; build it with "
                                              "python -m paper_2608_19041_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double
        sig = {
            "dpa4c_model_create": (i32, [vp, ctypes.c_size_t, i32, ctypes.POINTER(vp)]),
            "dpa4c_model_destroy": (None, [vp]),
            "dpa4c_model_info": (i32, [vp, vp]),
            "build_neighbors": (i32, [vp, i64, vp, vp, dbl, vp, vp, vp, i64,
                                      ctypes.POINTER(i64), vp]),
            "compute_energy_forces": (i32, [vp, vp, vp, i64, vp, vp, dbl, vp, vp, vp, i64,
                                            vp, vp, vp, vp]),
            "compute_energy_forces_virial": (i32, [vp, vp, vp, i64, vp, vp, dbl, vp, vp, vp,
                                                   i64, vp, vp, vp, vp, vp, vp]),
            "compute_energy_forces_noalloc": (i32, [vp, vp, vp, i64, vp, vp, dbl, vp, vp, vp, i64,
                                                    vp, vp, vp, vp]),
            "verlet_step": (i32, [vp, vp, vp, vp, vp, i64, vp, vp, dbl, dbl, dbl, i32, i32,
                                  vp, vp, vp, ctypes.POINTER(i64), vp]),
            "nvt_step": (i32, [vp, vp, vp, vp, vp, i64, vp, vp, dbl, dbl, dbl, i32, i32, dbl, dbl,
                               i32, vp, vp, vp, vp, vp, vp, ctypes.POINTER(i64), vp]),
            "dpa4c_debug_stages": (i32, [vp, i64, vp, vp, vp, vp]),
            "dpa4c_set_timing": (i32, [vp, i64]),
            "dpa4c_get_timings": (i32, [vp, vp, vp, i32]),
            "dpa4c_stage_name": (ctypes.c_char_p, [i32]),
            "dpa4c_debug_gemm": (i32, [vp, vp, vp, i32, i32, i32, vp]),
            "dpa4c_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def exported_symbols() -> list[str]:
    return ["dpa4c_model_create", "dpa4c_model_destroy", "dpa4c_model_info", "build_neighbors",
            "compute_energy_forces", "compute_energy_forces_virial",
            "compute_energy_forces_noalloc", "verlet_step", "nvt_step",
            "dpa4c_debug_stages", "dpa4c_set_timing",
            "dpa4c_get_timings", "dpa4c_stage_name", "dpa4c_debug_gemm", "dpa4c_last_error"]


def stage_names() -> list[str]:
    """Names of the timed stages, in stage-index order."""
    lib = library()
    names = []
    while True:
        name = lib.dpa4c_stage_name(len(names)).decode()
        if name == "?":
            return names
        names.append(name)


def _check(rc: int):
    if rc != OK:
        raise DPA4CError(rc, library().dpa4c_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _host_f64(a, n):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64).reshape(-1))
    if a.size != n:
        raise ValueError(f"expected {n} float64 values")
    return a


def _cell_arg(cell):
    """Host float64 [9] (rows = lattice vectors) and its pointer; None (an
    open system) passes a null pointer."""
    if cell is None:
        return None, None
    a = _host_f64(cell, 9)
    return a, a.ctypes.data


def _pbc_arg(pbc):
    if pbc is None:
        return None, None
    a = np.ascontiguousarray(np.asarray(pbc, dtype=np.int32).reshape(3))
    return a, a.ctypes.data


def _require(t, dtype, shape, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous CUDA tensor of {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def build_neighbors(pos, cell, pbc, r_list: float, cap: int | None = None, stream=None):
    """Skin list at radius r_list: (row_ptr int64 [N+1], nbr_j int32, nbr_shift int32, n_pairs).

    ``cap`` is the initial capacity guess; on DPA4C_ERR_CAPACITY the arrays
    are reallocated to the reported size and the call repeated.
    """
    import torch
    _require(pos, torch.float64, None, "pos")
    n = pos.shape[0]
    cellh, cellp = _cell_arg(cell)
    pbch, pbcp = _pbc_arg(pbc)
    dev = pos.device
    row_ptr = torch.empty(n + 1, dtype=torch.int64, device=dev)
    cap = int(cap if cap is not None else max(1024, 160 * n))
    lib = library()
    for _ in range(2):
        nbr_j = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
        nbr_s = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
        npairs = ctypes.c_int64(0)
        rc = lib.build_neighbors(_ptr(pos), n, cellp, pbcp, float(r_list),
                                 _ptr(row_ptr), _ptr(nbr_j), _ptr(nbr_s), cap, ctypes.byref(npairs),
                                 _stream(stream))
        if rc == ERR_CAPACITY:
            cap = int(npairs.value)
            continue
        _check(rc)
        e = int(npairs.value)
        return row_ptr, nbr_j[:e], nbr_s[:e], e
    raise DPA4CError(ERR_CAPACITY, "neighbour list did not fit after resizing")


def unpack_shift(s):
    """Packed image shift -> (n_x, n_y, n_z) int arrays."""
    s = np.asarray(s, dtype=np.int64)
    return np.stack([((s >> 16) & 0xFF) - 128, ((s >> 8) & 0xFF) - 128, (s & 0xFF) - 128], -1)


def debug_gemm(A, B, stream=None):
    import torch
    _require(A, torch.float32, None, "A")
    _require(B, torch.float32, None, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    C = torch.empty(M, N, dtype=torch.float32, device=A.device)
    _check(library().dpa4c_debug_gemm(_ptr(A), _ptr(B), _ptr(C), M, N, K, _stream(stream)))
    return C


class Model:
    """A model handle on one device (weights, radial table, pair cache)."""

    INFO_KEYS = ("C0", "L", "R", "S", "D_out", "F", "n_layers", "n_types", "table_rows", "C1",
                 "C2", "K1", "fold_words")

    def __init__(self, blob: bytes, device: int = 0):
        lib = library()
        h = ctypes.c_void_p()
        buf = ctypes.create_string_buffer(bytes(blob), len(blob))
        _check(lib.dpa4c_model_create(buf, len(blob), int(device), ctypes.byref(h)))
        self._h = h
        self.device = device
        info = (ctypes.c_int64 * 13)()
        _check(lib.dpa4c_model_info(self._h, info))
        self.info = dict(zip(self.INFO_KEYS, list(info)))

    def close(self):
        if getattr(self, "_h", None):
            library().dpa4c_model_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def compute_energy_forces(self, pos, species, cell, pbc, r_c, row_ptr, nbr_j, nbr_shift,
                              n_pairs, e_atom=None, forces=None, e_total=None, stream=None):
        import torch
        n = pos.shape[0]
        _require(pos, torch.float64, (n, 3), "pos")
        _require(species, torch.int32, (n,), "species")
        dev = pos.device
        e_atom = e_atom if e_atom is not None else torch.empty(n, dtype=torch.float64, device=dev)
        forces = forces if forces is not None else torch.empty(n, 3, dtype=torch.float64, device=dev)
        e_total = e_total if e_total is not None else torch.empty(1, dtype=torch.float64, device=dev)
        cellh, cellp = _cell_arg(cell)
        pbch, pbcp = _pbc_arg(pbc)
        _check(library().compute_energy_forces(
            self._h, _ptr(pos), _ptr(species), n, cellp, pbcp, float(r_c),
            _ptr(row_ptr), _ptr(nbr_j), _ptr(nbr_shift), int(n_pairs), _ptr(e_atom), _ptr(forces),
            _ptr(e_total), _stream(stream)))
        return e_atom, forces, e_total

    def compute_energy_forces_noalloc(self, pos, species, cell, pbc, r_c, row_ptr, nbr_j,
                                      nbr_shift, n_pairs, e_atom, forces, e_total, stream=None):
        """compute_energy_forces into caller buffers, with no device allocation
        in the library (its per-call buffers are a fixed device array)."""
        import torch
        n = pos.shape[0]
        _require(pos, torch.float64, (n, 3), "pos")
        _require(species, torch.int32, (n,), "species")
        _require(e_atom, torch.float64, (n,), "e_atom")
        _require(forces, torch.float64, (n, 3), "forces")
        _require(e_total, torch.float64, (1,), "e_total")
        cellh, cellp = _cell_arg(cell)
        pbch, pbcp = _pbc_arg(pbc)
        _check(library().compute_energy_forces_noalloc(
            self._h, _ptr(pos), _ptr(species), n, cellp, pbcp, float(r_c),
            _ptr(row_ptr), _ptr(nbr_j), _ptr(nbr_shift), int(n_pairs), _ptr(e_atom), _ptr(forces),
            _ptr(e_total), _stream(stream)))
        return e_atom, forces, e_total

    def compute_energy_forces_virial(self, pos, species, cell, pbc, r_c, row_ptr, nbr_j,
                                     nbr_shift, n_pairs, atom_virial=False, stream=None):
        """(e_atom, forces, e_total, virial [3, 3], atom_virial [N, 3, 3] or None)."""
        import torch
        n = pos.shape[0]
        _require(pos, torch.float64, (n, 3), "pos")
        _require(species, torch.int32, (n,), "species")
        dev = pos.device
        e_atom = torch.empty(n, dtype=torch.float64, device=dev)
        forces = torch.empty(n, 3, dtype=torch.float64, device=dev)
        e_total = torch.empty(1, dtype=torch.float64, device=dev)
        virial = torch.empty(3, 3, dtype=torch.float64, device=dev)
        w_atom = torch.empty(n, 3, 3, dtype=torch.float64, device=dev) if atom_virial else None
        cellh, cellp = _cell_arg(cell)
        pbch, pbcp = _pbc_arg(pbc)
        _check(library().compute_energy_forces_virial(
            self._h, _ptr(pos), _ptr(species), n, cellp, pbcp, float(r_c),
            _ptr(row_ptr), _ptr(nbr_j), _ptr(nbr_shift), int(n_pairs), _ptr(e_atom), _ptr(forces),
            _ptr(e_total), _ptr(virial), _ptr(w_atom), _stream(stream)))
        return e_atom, forces, e_total, virial, w_atom

    def nvt_step(self, pos, vel, species, mass_by_species, cell, pbc, r_c, skin, dt_fs, nsteps,
                 rebuild_every, forces, temperature, t_damp_fs, chain, virial=False, out=None,
                 stream=None):
        """NVT steps; ``chain`` is a float64 device tensor [2M] (in/out).
        ``out``: optional preallocated (e_pot, e_kin, e_thermo, virial [k, 3, 3]
        or None) with k >= nsteps.
        Returns (e_pot, e_kin, e_thermo, virial [nsteps, 3, 3] or None, n_rebuilds)."""
        import torch
        n = pos.shape[0]
        _require(pos, torch.float64, (n, 3), "pos")
        _require(vel, torch.float64, (n, 3), "vel")
        _require(forces, torch.float64, (n, 3), "forces")
        _require(species, torch.int32, (n,), "species")
        _require(chain, torch.float64, None, "chain")
        if chain.dim() != 1 or chain.shape[0] % 2:
            raise ValueError("chain must hold 2M values")
        dev = pos.device
        k = max(nsteps, 1)
        if out is not None:
            e_pot, e_kin, e_th, vir = out
            for x in (e_pot, e_kin, e_th):
                _require(x, torch.float64, None, "energy output")
                if x.numel() < nsteps:
                    raise ValueError("output buffers shorter than nsteps")
            if vir is not None and (vir.dtype != torch.float64 or vir.numel() < 9 * nsteps
                                    or not vir.is_contiguous()):
                raise ValueError("virial output must be contiguous float64 [k, 3, 3], k >= nsteps")
        else:
            e_pot = torch.empty(k, dtype=torch.float64, device=dev)
            e_kin = torch.empty(k, dtype=torch.float64, device=dev)
            e_th = torch.empty(k, dtype=torch.float64, device=dev)
            vir = torch.empty(k, 3, 3, dtype=torch.float64, device=dev) if virial else None
        masses = _host_f64(mass_by_species, self.info["n_types"] + 1)
        cellh, cellp = _cell_arg(cell)
        pbch, pbcp = _pbc_arg(pbc)
        nreb = ctypes.c_int64(0)
        _check(library().nvt_step(
            self._h, _ptr(pos), _ptr(vel), _ptr(species), masses.ctypes.data, n, cellp,
            pbcp, float(r_c), float(skin), float(dt_fs), int(nsteps), int(rebuild_every),
            float(temperature), float(t_damp_fs), int(chain.shape[0] // 2), _ptr(chain),
            _ptr(e_pot), _ptr(e_kin), _ptr(e_th), _ptr(vir), _ptr(forces), ctypes.byref(nreb),
            _stream(stream)))
        return (e_pot[:nsteps], e_kin[:nsteps], e_th[:nsteps],
                None if vir is None else vir[:nsteps], int(nreb.value))

    def verlet_step(self, pos, vel, species, mass_by_species, cell, pbc, r_c, skin, dt_fs,
                    nsteps, rebuild_every, forces, e_pot=None, e_kin=None, stream=None):
        import torch
        n = pos.shape[0]
        _require(pos, torch.float64, (n, 3), "pos")
        _require(vel, torch.float64, (n, 3), "vel")
        _require(forces, torch.float64, (n, 3), "forces")
        _require(species, torch.int32, (n,), "species")
        dev = pos.device
        e_pot = e_pot if e_pot is not None else torch.empty(max(nsteps, 1), dtype=torch.float64, device=dev)
        e_kin = e_kin if e_kin is not None else torch.empty(max(nsteps, 1), dtype=torch.float64, device=dev)
        masses = _host_f64(mass_by_species, self.info["n_types"] + 1)
        cellh, cellp = _cell_arg(cell)
        pbch, pbcp = _pbc_arg(pbc)
        nreb = ctypes.c_int64(0)
        _check(library().verlet_step(
            self._h, _ptr(pos), _ptr(vel), _ptr(species), masses.ctypes.data, n, cellp,
            pbcp, float(r_c), float(skin), float(dt_fs), int(nsteps), int(rebuild_every),
            _ptr(e_pot), _ptr(e_kin), _ptr(forces), ctypes.byref(nreb), _stream(stream)))
        return e_pot[:nsteps], e_kin[:nsteps], int(nreb.value)

    def debug_stages(self, n, stream=None):
        import torch
        dev = torch.device("cuda", self.device)
        node = torch.empty(n, self.info["S"] + 2, dtype=torch.float32, device=dev)
        desc = torch.empty(n, self.info["D_out"], dtype=torch.float32, device=dev)
        cnt = torch.empty(n, dtype=torch.int32, device=dev)
        _check(library().dpa4c_debug_stages(self._h, n, _ptr(node), _ptr(desc), _ptr(cnt),
                                            _stream(stream)))
        return node, desc, cnt

    def set_timing(self, on=True):
        """True: time every stage; False: none; a list of stage names: those."""
        if on is True:
            mask = -1
        elif not on:
            mask = 0
        else:
            names = stage_names()
            mask = 0
            for name in on:
                mask |= 1 << names.index(name)
        _check(library().dpa4c_set_timing(self._h, mask))

    def timings(self) -> dict:
        """{stage name: (milliseconds, launches)} since the last read."""
        lib = library()
        ms = (ctypes.c_double * 32)()
        cnt = (ctypes.c_int64 * 32)()
        k = lib.dpa4c_get_timings(self._h, ms, cnt, 32)
        if k < 0:
            _check(k)
        return {lib.dpa4c_stage_name(s).decode(): (ms[s], cnt[s]) for s in range(k)}
