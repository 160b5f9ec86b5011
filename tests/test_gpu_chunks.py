"""Dynamics split over several calls.  A displacement-triggered call whose
model still holds the skin list of the previous call (same atom count, cell
and list radius) starts with the displacement check instead of a rebuild.
Every valid list gives the same edges in the same order, so a chunked NVE
or NVT run is bit-identical to one call, with the same rebuilds, and
positions changed between calls are caught by the check."""
import numpy as np
import pytest
import torch

import synth

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


def new_model(dp, name="full"):
    spec, w = synth.model_weights(name)
    return dp.Model(synth.pack_blob(spec, w))


def start(dp, model, s, dev, temperature=600.0):
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    vel = torch.tensor(synth.maxwell_boltzmann(s, temperature), dtype=torch.float64, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 6.5)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    return pos, species, vel, F


def run_chunks(dp, model, s, state, chunks, skin=0.5):
    pos, species, vel, F = state
    eps, eks, nreb = [], [], 0
    for k in chunks:
        ep, ek, nr = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, skin,
                                       1.0, k, 0, F)
        eps.append(ep.clone())
        eks.append(ek.clone())
        nreb += nr
    torch.cuda.synchronize()
    return (pos.cpu().numpy(), vel.cpu().numpy(), F.cpu().numpy(),
            torch.cat(eps).cpu().numpy(), torch.cat(eks).cpu().numpy(), nreb)


@pytest.mark.parametrize("chunks", [(20, 20), (7, 1, 13, 19)])
def test_chunked_nve_equals_one_call(dev, dp, chunks):
    s = synth.make_workload("fcc4000_full")[0]
    model = new_model(dp)
    one = run_chunks(dp, model, s, start(dp, model, s, dev), [sum(chunks)])
    many = run_chunks(dp, model, s, start(dp, model, s, dev), list(chunks))
    assert one[5] >= 2 and many[5] == one[5]
    for a, b in zip(one[:5], many[:5]):
        assert np.array_equal(a, b)


def test_moved_atoms_between_calls_trigger_a_rebuild(dev, dp):
    s = synth.make_workload("fcc4000_full")[0]
    model = new_model(dp)
    pos, species, vel, F = start(dp, model, s, dev)
    run_chunks(dp, model, s, (pos, species, vel, F), [15])
    pos[5, 0] += 0.6                   # beyond half the 0.5 A skin
    pos_b, vel_b, F_b = pos.clone(), vel.clone(), F.clone()
    carried = run_chunks(dp, model, s, (pos, species, vel, F), [10])
    fresh_model = new_model(dp)        # no list to carry over
    fresh = run_chunks(dp, fresh_model, s, (pos_b, species, vel_b, F_b), [10])
    assert carried[5] == fresh[5] >= 1
    for a, b in zip(carried[:5], fresh[:5]):
        assert np.array_equal(a, b)


def test_chunked_nvt_equals_one_call(dev, dp):
    """NVT split over calls: every step boundary, inside a call or between
    calls, applies the chain's closing velocity scale, then takes the opening
    half step from the kinetic energy of the scaled velocities, so the run
    is bit-identical to a single call, with the same rebuilds."""
    s = synth.make_workload("fcc4000_full")[0]
    model = new_model(dp)

    def nvt(chunks):
        pos, species, vel, F = start(dp, model, s, dev)
        chain = torch.zeros(6, dtype=torch.float64, device=dev)
        eps, nreb = [], 0
        for k in chunks:
            ep, ek, eth, _, nr = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc,
                                                6.0, 0.5, 1.0, k, 0, F, 300.0, 100.0, chain)
            eps.append((ep + ek + eth).clone())
            nreb += nr
        torch.cuda.synchronize()
        return pos.cpu().numpy(), torch.cat(eps).cpu().numpy(), chain.cpu().numpy(), nreb

    one = nvt([30])
    many = nvt([10, 10, 10])
    assert one[3] >= 2 and many[3] == one[3]
    for a, b in zip(one[:3], many[:3]):
        assert np.array_equal(a, b)
