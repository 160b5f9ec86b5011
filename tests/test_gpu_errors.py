"""Error paths of the C ABI, each forced from the host (every kernel still
runs to completion): a neighbour capacity that is too small, a non-finite
position, a skin violation with rebuilds disabled, and device memory that
cannot hold the workspace.  After each error the model stays usable."""
import ctypes

import numpy as np
import pytest
import torch

import synth
from oracle import neighbors as onb

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return torch.device("cuda", 0)


@pytest.fixture(scope="module")
def dp():
    import paper_2608_19041_amd as m
    m.library()
    return m


def raw_build(dp, pos, s, r, cap):
    """build_neighbors through the C ABI with the caller's capacity."""
    n = pos.shape[0]
    row_ptr = torch.empty(n + 1, dtype=torch.int64, device=pos.device)
    nbr_j = torch.empty(max(cap, 1), dtype=torch.int32, device=pos.device)
    nbr_s = torch.empty(max(cap, 1), dtype=torch.int32, device=pos.device)
    cell = np.ascontiguousarray(s.cell, dtype=np.float64).reshape(9)
    pbc = np.ascontiguousarray(s.pbc, dtype=np.int32)
    npairs = ctypes.c_int64(-1)
    rc = dp.library().build_neighbors(
        ctypes.c_void_p(pos.data_ptr()), n, cell.ctypes.data, pbc.ctypes.data, float(r),
        ctypes.c_void_p(row_ptr.data_ptr()), ctypes.c_void_p(nbr_j.data_ptr()),
        ctypes.c_void_p(nbr_s.data_ptr()), int(cap), ctypes.byref(npairs),
        dp._stream(None))
    torch.cuda.synchronize()
    return rc, int(npairs.value), row_ptr


def test_capacity_too_small_reports_the_need(dev, dp):
    s = synth.fcc_copper(4, 0.05, seed=3)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    ref_i, _, _ = onb.neighbor_list(s.pos, s.cell, s.pbc, 7.0)
    rc, need, row_ptr = raw_build(dp, pos, s, 7.0, 100)
    assert rc == dp.ERR_CAPACITY and need == len(ref_i)
    assert int(row_ptr[-1]) == need            # the count pass wrote the rows
    rc, got, _ = raw_build(dp, pos, s, 7.0, need)
    assert rc == 0 and got == need


def test_nonfinite_position_is_reported(dev, dp):
    s = synth.fcc_copper(3, 0.05, seed=4)
    p = s.pos.copy()
    p[7, 1] = np.nan
    pos = torch.tensor(p, dtype=torch.float64, device=dev)
    rc, _, _ = raw_build(dp, pos, s, 7.0, 20000)
    assert rc == dp.ERR_NONFINITE
    # the dynamics refuse it as well, before any step
    spec, w = synth.model_weights("small")
    model = dp.Model(synth.pack_blob(spec, w))
    vel = torch.zeros_like(pos)
    F = torch.zeros_like(pos)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    with pytest.raises(dp.DPA4CError) as ei:
        model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 1.0, 1.0, 5, 0, F)
    assert ei.value.code == dp.ERR_NONFINITE


def test_skin_violation_without_rebuilds(dev, dp):
    spec, w = synth.model_weights("small")
    model = dp.Model(synth.pack_blob(spec, w))
    s = synth.fcc_copper(3, 0.05, seed=0)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    vel = torch.tensor(synth.maxwell_boltzmann(s, 3000.0), dtype=torch.float64, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 6.02)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    # a 0.02 A skin is crossed within a few steps at 3000 K
    with pytest.raises(dp.DPA4CError) as ei:
        model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 0.02, 1.0, 50,
                          -1, F)
    assert ei.value.code == dp.ERR_SKIN
    # with rebuilds on, the same run goes through and rebuilds
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    vel = torch.tensor(synth.maxwell_boltzmann(s, 3000.0), dtype=torch.float64, device=dev)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    _, _, nreb = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 0.02,
                                   1.0, 50, 0, F)
    assert nreb >= 3


def test_workspace_beyond_device_memory_is_out_of_memory(dev, dp):
    """A pair count far beyond the device's memory: the workspace request
    fails before any kernel runs, and the model works afterwards."""
    spec, w = synth.model_weights("small")
    model = dp.Model(synth.pack_blob(spec, w))
    s = synth.fcc_copper(3, 0.05, seed=0)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    with pytest.raises(dp.DPA4CError) as ei:
        model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, 1 << 42)
    assert ei.value.code == dp.ERR_OOM
    ea, F, et = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    torch.cuda.synchronize()
    assert np.isfinite(F.cpu().numpy()).all() and abs(float(F.sum(0).abs().max())) < 1e-9


def test_malformed_caller_lists_are_refused(dev, dp):
    """A list with more entries than n_pairs, and a list where one entry lost
    its reverse, are refused with INVALID_ARG before any output is written;
    the intact list then evaluates normally."""
    spec, w = synth.model_weights("small")
    model = dp.Model(synth.pack_blob(spec, w))
    s = synth.fcc_copper(3, 0.05, seed=4)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, spec.r_c + 1.0)
    e_atom = torch.full((s.n,), 7.0, dtype=torch.float64, device=dev)
    F = torch.full((s.n, 3), 7.0, dtype=torch.float64, device=dev)
    et = torch.full((1,), 7.0, dtype=torch.float64, device=dev)
    # row_ptr[N] beyond n_pairs
    with pytest.raises(dp.DPA4CError) as ex:
        model.compute_energy_forces(pos, species, s.cell, s.pbc, spec.r_c, rp, nj, ns, e - 5,
                                    e_atom, F, et)
    assert ex.value.code == dp.ERR_INVALID_ARG and "n_pairs" in str(ex.value)
    # drop the first entry of row 5: its partner in the other row has no reverse
    rph = rp.cpu().numpy().copy()
    k = int(rph[5])
    keep = np.ones(e, bool)
    keep[k] = False
    rph[6:] -= 1
    rp2 = torch.tensor(rph, device=dev)
    nj2 = nj[torch.tensor(keep, device=dev)].contiguous()
    ns2 = ns[torch.tensor(keep, device=dev)].contiguous()
    with pytest.raises(dp.DPA4CError) as ex:
        model.compute_energy_forces(pos, species, s.cell, s.pbc, spec.r_c, rp2, nj2, ns2, e - 1,
                                    e_atom, F, et)
    assert ex.value.code == dp.ERR_INVALID_ARG and "not symmetric" in str(ex.value)
    torch.cuda.synchronize()
    assert bool((e_atom == 7.0).all()) and bool((F == 7.0).all()) and float(et[0]) == 7.0
    ea, F, et = model.compute_energy_forces(pos, species, s.cell, s.pbc, spec.r_c, rp, nj, ns, e)
    torch.cuda.synchronize()
    assert np.isfinite(ea.cpu().numpy()).all() and abs(float(et[0]) - float(ea.sum())) < 1e-9
