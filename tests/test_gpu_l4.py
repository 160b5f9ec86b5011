"""Harmonics up to degree four on the GPU (the Plus widths with L = 4: nine
coupling triples, S = 232, D_out = 557 as in Supplementary Table S2) versus
the oracle, through the C ABI."""
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
def l4(dev):
    import paper_2608_19041_amd as dp
    dp.library()          # fails loudly if the library is missing
    spec, w = synth.model_weights("plus_l4")
    return dp, dp.Model(synth.pack_blob(spec, w)), om.Oracle(spec, w)


def evaluate(dp, model, s, dev, list_radius=7.0):
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, list_radius)
    ea, F, et = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), F.cpu().numpy(), et.item()


def test_widths(l4):
    _, model, _ = l4
    assert model.info["L"] == 4 and model.info["S"] == 232 and model.info["D_out"] == 557


def test_stages_degree_four(dev, l4):
    """Node state (with the degree-four block) and the descriptor, whose
    degree-four entries are G4 and the (1,3,4), (2,2,4), (2,4,4), (3,3,4),
    (4,4,4) bispectrum blocks."""
    dp, model, oracle = l4
    s = synth.fcc_copper(3, 0.08, seed=3)
    evaluate(dp, model, s, dev)
    node, desc, cnt = model.debug_stages(s.n)
    ref = oracle.stages(s.pos, s.species, s.cell, s.pbc)
    node = node.cpu().numpy().astype(np.float64)
    C0 = oracle.C0
    y_ref = ref["X_flat"].copy()
    y_ref[:, :C0] *= ref["M0"][:, None]
    y_ref[:, C0:] *= ref["M1"][:, None]
    assert y_ref.shape[1] == 232                        # S

    scale = np.abs(y_ref).max()
    assert np.abs(node[:, 2:] - y_ref).max() < 2e-5 * scale
    assert np.abs(node[:, 2 + 223:] - y_ref[:, 223:]).max() < 2e-5 * scale   # the degree-four block
    d = desc.cpu().numpy().astype(np.float64)
    assert d.shape[1] == 557
    assert np.abs(d - ref["D"]).max() < 1e-4 * max(1.0, np.abs(ref["D"]).max())


@pytest.mark.parametrize("structure", ["fcc108", "periodic24", "triclinic20"])
def test_energy_forces_degree_four(dev, l4, structure):
    dp, model, oracle = l4
    if structure == "fcc108":
        s = synth.fcc_copper(3, 0.08, seed=3)
    elif structure == "periodic24":
        s = synth.random_periodic(24, seed=11, cell=np.diag([8.3, 8.9, 9.4]), d_min=1.6)
    else:
        cell = np.array([[8.3, 0.0, 0.0], [1.2, 8.9, 0.0], [0.7, -0.9, 9.4]])
        s = synth.random_periodic(20, seed=5, cell=cell, d_min=1.6)
    ea, F, et = evaluate(dp, model, s, dev)
    ref_e, ref_f = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc)
    assert np.abs(ea - ref_e).max() < E_TOL
    assert np.abs(F - ref_f).max() < F_TOL
    assert abs(et - ref_e.sum()) < E_TOL * s.n


def test_config2_shape_sampled(dev, l4):
    dp, model, oracle = l4
    s = synth.make_workload("fcc4000_full")[0]
    ea, F, et = evaluate(dp, model, s, dev)
    rng = np.random.Generator(np.random.PCG64(21))
    ks = np.sort(rng.choice(s.n, 4, replace=False)).astype(np.int64)
    _, ej, _ = onb.neighbor_list(s.pos, s.cell, s.pbc, 6.0, centres=ks)
    centres = np.unique(np.concatenate([ks, ej]))
    ref_e, ref_f = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc, centres=centres)
    assert np.abs(ea[centres] - ref_e).max() < E_TOL
    assert np.abs(F[ks] - ref_f[ks]).max() < F_TOL


def test_verlet_degree_four(dev, l4):
    dp, model, oracle = l4
    s = synth.make_workload("fcc108_small")[0]
    v0 = synth.maxwell_boltzmann(s, 300.0)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    vel = torch.tensor(v0, dtype=torch.float64, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    ep, ek, _ = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 1.0, 1.0,
                                  20, 0, F)
    torch.cuda.synchronize()
    rep, rek, rpos, _ = md.nve(oracle, s.pos, v0, s.species, s.cell, s.pbc,
                               s.mass_by_type[s.species], 1.0, 20)
    assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
    assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
    assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n
