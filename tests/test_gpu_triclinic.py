"""Triclinic periodic cells on the GPU path versus the oracle, through the C
ABI: neighbour lists bit-identical, E_i within 1e-5 eV, F within 1e-4 eV/A,
the virial, and velocity-Verlet and NVT dynamics."""
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
        _models[name] = (dp.Model(synth.pack_blob(spec, w)), om.Oracle(spec, w), spec)
    return _models[name]


def on_dev(s, dev):
    return (torch.tensor(s.pos, dtype=torch.float64, device=dev),
            torch.tensor(s.species, dtype=torch.int32, device=dev))


def gpu_rows(row_ptr, nbr_j, nbr_shift, dp):
    rp = row_ptr.cpu().numpy()
    j = nbr_j.cpu().numpy().astype(np.int64)
    n = dp.unpack_shift(nbr_shift.cpu().numpy())
    i = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    return i, j, n


def assert_rows_equal(gpu, ref, centres=None):
    gi, gj, gn = gpu
    if centres is not None:
        keep = np.isin(gi, centres)
        gi, gj, gn = gi[keep], gj[keep], gn[keep]
    ri, rj, rn = ref
    assert len(gi) == len(ri)
    assert np.array_equal(gi, ri) and np.array_equal(gj, rj) and np.array_equal(gn, rn)


def random_lattice(rng, skew):
    """Rows h_0, h_1, h_2: lengths 3-9 A, off-diagonal shear up to ``skew``
    of the lengths, random sign of the determinant."""
    L = rng.uniform(3.0, 9.0, size=3)
    h = np.diag(L) + rng.uniform(-skew, skew, size=(3, 3)) * L[:, None]
    if rng.integers(0, 2):
        h[[0, 1]] = h[[1, 0]]           # left-handed
    return h


TINY = [(n, skew) for n, skew in [(1, 0.3), (2, 0.5), (3, 0.2), (5, 0.7), (7, 0.4), (12, 0.6),
                                  (9, 0.9), (4, 0.05)]]


@pytest.mark.parametrize("case", range(len(TINY)))
def test_neighbors_tiny_triclinic_cells(dev, dp, case):
    n, skew = TINY[case]
    rng = np.random.Generator(np.random.PCG64(100 + case))
    cell = random_lattice(rng, skew)
    s = synth.random_periodic(n, seed=case, cell=cell, d_min=0.5)
    s.pos[0] += np.array([2, -1, 3]) @ cell     # an atom far outside the cell
    pos, _ = on_dev(s, dev)
    for r in (4.0, 6.5):
        rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, r)
        ref = onb.neighbor_list(s.pos, s.cell, s.pbc, r)
        assert e == len(ref[0])
        assert_rows_equal(gpu_rows(rp, nj, ns, dp), ref)


def fcc_primitive(reps, jitter, seed=0, a=3.615):
    """FCC copper in its rhombohedral primitive cell (60 degree angles),
    reps^3 primitive cells, one atom each."""
    prim = 0.5 * a * np.array([[0.0, 1.0, 1.0], [1.0, 0.0, 1.0], [1.0, 1.0, 0.0]])
    g = np.stack(np.meshgrid(*[np.arange(reps)] * 3, indexing="ij"), -1).reshape(-1, 3)
    pos = g.astype(np.float64) @ prim
    rng = np.random.Generator(np.random.PCG64(seed))
    pos = pos + rng.normal(0.0, jitter, size=pos.shape)
    return synth.System(f"fcc_prim_{reps}", pos, np.full(len(pos), 28, np.int32), reps * prim,
                        np.ones(3, np.int32), synth._mass_table({28: 63.5}), {})


def test_perfect_fcc_in_a_rhombohedral_cell(dev, dp):
    """16^3 primitive cells of perfect FCC: every atom has the 78 neighbours
    of the conventional-cell crystal within 6 A, the list equals the oracle's,
    and E_i equals that of the same crystal in its cubic cell."""
    model, _, _ = gpu_model(dp, "full")
    s = fcc_primitive(16, 0.0)
    pos, species = on_dev(s, dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 6.0)
    counts = np.diff(rp.cpu().numpy())
    assert (counts == 78).all()
    ref = onb.neighbor_list(s.pos, s.cell, s.pbc, 6.0)
    assert_rows_equal(gpu_rows(rp, nj, ns, dp), ref)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    ea, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    cubic = synth.fcc_copper(8, 0.0, seed=0)
    cpos, csp = on_dev(cubic, dev)
    crp, cnj, cns, ce = dp.build_neighbors(cpos, cubic.cell, cubic.pbc, 7.0)
    cea, cF, _ = model.compute_energy_forces(cpos, csp, cubic.cell, cubic.pbc, 6.0, crp, cnj, cns,
                                             ce)
    ea, cea = ea.cpu().numpy(), cea.cpu().numpy()
    assert np.abs(ea - cea[0]).max() < E_TOL
    assert np.abs(F.cpu().numpy()).max() < F_TOL


def evaluate(dp, model, s, dev):
    pos, species = on_dev(s, dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    ea, F, et, vir, _ = model.compute_energy_forces_virial(pos, species, s.cell, s.pbc, 6.0, rp,
                                                           nj, ns, e)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), F.cpu().numpy(), et.item(), vir.cpu().numpy()


@pytest.mark.parametrize("name", ["small", "full"])
def test_energy_forces_virial_triclinic_cell(dev, dp, name):
    model, oracle, _ = gpu_model(dp, name)
    cell = np.array([[8.3, 0.0, 0.0], [1.2, 8.9, 0.0], [0.7, -0.9, 9.4]])
    s = synth.random_periodic(20, seed=5, cell=cell, d_min=1.6)
    ea, F, et, vir = evaluate(dp, model, s, dev)
    ref_e, ref_f, ref_vir, _ = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc, virial=True)
    assert np.abs(ea - ref_e).max() < E_TOL
    assert np.abs(F - ref_f).max() < F_TOL
    assert abs(et - ref_e.sum()) < E_TOL * s.n
    assert np.abs(vir - ref_vir).max() < E_TOL * s.n


def test_jittered_rhombohedral_crystal_sampled(dev, dp):
    """4096-atom jittered FCC in the rhombohedral cell: sampled E_i and forces."""
    model, oracle, _ = gpu_model(dp, "full")
    s = fcc_primitive(16, 0.08, seed=4)
    ea, F, et, vir = evaluate(dp, model, s, dev)
    rng = np.random.Generator(np.random.PCG64(3))
    ks = np.sort(rng.choice(s.n, 4, replace=False)).astype(np.int64)
    _, ej, _ = onb.neighbor_list(s.pos, s.cell, s.pbc, 6.0, centres=ks)
    centres = np.unique(np.concatenate([ks, ej]))
    ref_e, ref_f = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc, centres=centres)
    assert np.abs(ea[centres] - ref_e).max() < E_TOL
    assert np.abs(F[ks] - ref_f[ks]).max() < F_TOL


def test_triclinic_dynamics_match_oracle(dev, dp):
    """A 64-atom jittered rhombohedral FCC cell (r_c reaches several images):
    20 velocity-Verlet steps with a 0.3 A skin (rebuilds and replays) and 10
    NVT steps, each against the oracle's integrators."""
    model, oracle, _ = gpu_model(dp, "small")
    s = fcc_primitive(4, 0.05, seed=2)
    v0 = synth.maxwell_boltzmann(s, 600.0)
    m = s.mass_by_type[s.species]
    for ensemble in ("nve", "nvt"):
        pos, species = on_dev(s, dev)
        vel = torch.tensor(v0, dtype=torch.float64, device=dev)
        rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 6.3)
        _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
        if ensemble == "nve":
            ep, ek, nreb = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0,
                                             0.3, 1.0, 20, 0, F)
            rep, rek, rpos, _ = md.nve(oracle, s.pos, v0, s.species, s.cell, s.pbc, m, 1.0, 20)
            assert nreb >= 2
        else:
            chain = torch.zeros(6, dtype=torch.float64, device=dev)
            ep, ek, eth, _, _ = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc,
                                               6.0, 0.3, 1.0, 10, 0, F, 300.0, 20.0, chain)
            rep, rek, reth, rpos, _, _ = md.nvt(oracle, s.pos, v0, s.species, s.cell, s.pbc, m,
                                                1.0, 10, 300.0, 20.0)
            assert np.abs(eth.cpu().numpy() - reth[1:]).max() < E_TOL * s.n
        torch.cuda.synchronize()
        assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
        assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
        assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n


def test_singular_and_sheared_open_cells_are_rejected(dev, dp):
    model, _, _ = gpu_model(dp, "small")
    s = synth.fcc_copper(3, 0.05, seed=0)
    pos, species = on_dev(s, dev)
    flat = np.array([[10.0, 0.0, 0.0], [5.0, 5.0, 0.0], [15.0, 5.0, 0.0]])
    with pytest.raises(dp.DPA4CError) as ei:
        dp.build_neighbors(pos, flat, s.pbc, 7.0)
    assert ei.value.code == -1
    # an open axis is supported only with a diagonal cell
    sheared = s.cell.copy()
    sheared[1, 0] = 1.0
    with pytest.raises(dp.DPA4CError) as ei:
        dp.build_neighbors(pos, sheared, [1, 1, 0], 7.0)
    assert ei.value.code == -2
