"""Open and partly open systems on the GPU path versus the oracle, through
the C ABI: neighbour lists bit-identical, E_i within 1e-5 eV, F within
1e-4 eV/A, inversion symmetry of an isolated cluster, and dynamics."""
import numpy as np
import pytest
import torch

import synth
from oracle import md
from oracle import model as om
from oracle import neighbors as onb

pytestmark = pytest.mark.gpu

E_TOL = 1e-5
F_TOL = 1e-4


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return torch.device("cuda", 0)


@pytest.fixture(scope="module")
def dp():
    import paper_2608_19041_amd as m
    m.library()          # fails loudly if the library is missing
    return m


_models = {}


def gpu_model(dp, name):
    if name not in _models:
        spec, w = synth.model_weights(name)
        _models[name] = (dp.Model(synth.pack_blob(spec, w)), om.Oracle(spec, w))
    return _models[name]


def gpu_rows(row_ptr, nbr_j, nbr_shift, dp):
    rp = row_ptr.cpu().numpy()
    j = nbr_j.cpu().numpy().astype(np.int64)
    n = dp.unpack_shift(nbr_shift.cpu().numpy())
    i = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    return i, j, n


def assert_rows_equal(gpu, ref):
    gi, gj, gn = gpu
    ri, rj, rn = ref
    assert len(gi) == len(ri)
    assert np.array_equal(gi, ri) and np.array_equal(gj, rj) and np.array_equal(gn, rn)


# Single-species copper with a 2.2 A closest approach keeps site energies
# within a few eV, the range the fp32 tolerances are set for; random packings
# with closer contacts reach tens of eV per site.
def cluster(n=40, seed=3, box=11.0):
    return synth.random_cluster(n, seed=seed, box=box, d_min=2.2, n_species=1, types=(28,))


def slab(n=30, seed=4):
    """Periodic in x and y, open in z, atoms spread over 14 A in z."""
    rng = np.random.Generator(np.random.PCG64(seed))
    s = synth.random_periodic(n, seed=seed, cell=np.diag([8.0, 8.5, 14.0]), d_min=2.2,
                              n_species=1, types=(28,))
    s.pos[:, 2] += rng.normal(0.0, 2.0)          # off-centre in the open direction
    # the cell's z length is nominal: nothing along an open axis uses it
    return synth.System("slab", s.pos, s.species, np.diag([8.0, 8.5, 14.0]),
                        np.array([1, 1, 0], np.int32), s.mass_by_type, {})


@pytest.mark.parametrize("kind", ["cluster", "cluster_null_cell", "slab"])
def test_neighbors_open(dev, dp, kind):
    s = slab() if kind == "slab" else cluster()
    cell = None if kind == "cluster_null_cell" else s.cell
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    for r in (4.5, 7.0):
        rp, nj, ns, e = dp.build_neighbors(pos, cell, s.pbc, r)
        ref = onb.neighbor_list(s.pos, s.cell if kind == "slab" else np.diag([1.0, 1.0, 1.0]),
                                s.pbc, r)
        assert_rows_equal(gpu_rows(rp, nj, ns, dp), ref)
        if kind != "slab":
            assert (gpu_rows(rp, nj, ns, dp)[2] == 0).all()


def evaluate(dp, model, s, dev, cell):
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, cell, s.pbc, 7.0)
    ea, F, et = model.compute_energy_forces(pos, species, cell, s.pbc, 6.0, rp, nj, ns, e)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), F.cpu().numpy()


@pytest.mark.parametrize("name", ["small", "full"])
@pytest.mark.parametrize("kind", ["cluster", "slab"])
def test_energy_forces_open(dev, dp, name, kind):
    model, oracle = gpu_model(dp, name)
    s = slab() if kind == "slab" else cluster()
    ea, F = evaluate(dp, model, s, dev, s.cell)
    ref_e, ref_f = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc)
    assert np.abs(ea - ref_e).max() < E_TOL
    assert np.abs(F - ref_f).max() < F_TOL
    assert np.abs(F.sum(0)).max() < 1e-9


def test_isolated_cluster_inversion(dev, dp):
    """E is invariant and F odd under r -> -r for an isolated cluster (no cell)."""
    model, _ = gpu_model(dp, "full")
    s = cluster()
    ea, F = evaluate(dp, model, s, dev, None)
    inv = synth.System("inv", -s.pos, s.species, s.cell, s.pbc, s.mass_by_type, {})
    ea2, F2 = evaluate(dp, model, inv, dev, None)
    assert np.abs(ea - ea2).max() < E_TOL
    assert np.abs(F + F2).max() < F_TOL


def test_open_cluster_dynamics(dev, dp):
    """20 velocity-Verlet steps of a hot open cluster with a 0.3 A skin
    (rebuilds follow the cluster's extent) against the oracle."""
    model, oracle = gpu_model(dp, "small")
    s = cluster(n=30, seed=8, box=9.0)
    v0 = synth.maxwell_boltzmann(s, 900.0)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    vel = torch.tensor(v0, dtype=torch.float64, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, None, None, 6.3)
    _, F, _ = model.compute_energy_forces(pos, species, None, None, 6.0, rp, nj, ns, e)
    ep, ek, nreb = model.verlet_step(pos, vel, species, s.mass_by_type, None, None, 6.0, 0.3, 1.0,
                                     20, 0, F)
    torch.cuda.synchronize()
    rep, rek, rpos, _ = md.nve(oracle, s.pos, v0, s.species, s.cell, s.pbc,
                               s.mass_by_type[s.species], 1.0, 20)
    assert nreb >= 2
    assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
    assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
    assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n


def test_open_axes_need_a_diagonal_cell(dev, dp):
    s = slab()
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    sheared = np.array([[8.0, 0.0, 0.0], [1.0, 8.5, 0.0], [0.0, 0.0, 10.0]])
    with pytest.raises(dp.DPA4CError) as ei:
        dp.build_neighbors(pos, sheared, [1, 1, 0], 7.0)
    assert ei.value.code == -2
