"""Virial and Nose-Hoover-chain NVT on the GPU versus the float64 oracle,
through the C ABI.

Virial tolerances: the per-centre terms W_i = -sum_j g_ij (x) r_ij add about
80 edge products of float32 gradients and float32 edge vectors; their error
is a few 1e-6 relative per product, so W_i is held to 2e-4 eV per component
and the total Xi to 1e-5 eV per atom (the energy tolerance) times N.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import md
from oracle import model as om
from oracle import neighbors as onb

pytestmark = pytest.mark.gpu

E_TOL = 1e-5
W_TOL = 2e-4
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


def gpu_virial(dp, model, s, dev):
    pos, species = on_dev(s, dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    ea, F, et, vir, w = model.compute_energy_forces_virial(pos, species, s.cell, s.pbc, 6.0, rp,
                                                           nj, ns, e, atom_virial=True)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), F.cpu().numpy(), vir.cpu().numpy(), w.cpu().numpy()


@pytest.mark.parametrize("name,structure", [
    ("small", "fcc108"), ("small", "periodic24"), ("full", "fcc108"), ("full", "periodic24")])
def test_virial_matches_oracle(dev, dp, name, structure):
    model, oracle, _ = gpu_model(dp, name)
    if structure == "fcc108":
        s = synth.fcc_copper(3, 0.08, seed=3)
    else:
        s = synth.random_periodic(24, seed=11, cell=np.diag([8.3, 8.9, 9.4]), d_min=1.6)
    ea, F, vir, w = gpu_virial(dp, model, s, dev)
    ref_e, ref_f, ref_vir, ref_w = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc,
                                                        virial=True)
    assert np.abs(ea - ref_e).max() < E_TOL
    assert np.abs(w - ref_w).max() < W_TOL
    assert np.abs(vir - ref_vir).max() < E_TOL * s.n
    # the per-centre terms sum to the total in the library's own fixed order
    assert np.abs(w.sum(0) - vir).max() < 1e-9 * max(1.0, np.abs(vir).max())


def test_virial_config2_full_size(dev, dp):
    """4000-atom FCC, full model: every W_i and the total against the oracle."""
    model, oracle, _ = gpu_model(dp, "full")
    s = synth.make_workload("fcc4000_full")[0]
    ea, F, vir, w = gpu_virial(dp, model, s, dev)
    ref_e, ref_f, ref_vir, ref_w = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc,
                                                        virial=True)
    assert np.abs(w - ref_w).max() < W_TOL
    assert np.abs(vir - ref_vir).max() < E_TOL * s.n
    assert np.abs(vir - vir.T).max() < E_TOL * s.n


def eight_species_bcc():
    """A BCC cell of eight species, more than the library folds into per-pair
    tables, so the edge kernels take the separable radial table."""
    s = synth.bcc_hea(3, 0.06, seed=7)
    types = np.array(sorted(set(s.meta["types"]) | {0, 7, 28}), dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(3))
    s.species = types[rng.integers(0, len(types), size=s.n)].astype(np.int32)
    return s


@pytest.mark.parametrize("name", ["small", "full"])
@pytest.mark.parametrize("tables", ["folded", "separable"])
def test_virial_leaves_energies_and_forces_bit_identical(dev, dp, name, tables):
    """Asking for the virial changes no bit of E_i or F: NVE and NVT evaluate
    the same gradients (one species: pair-folded tables; eight species: the
    separable table and the pair cache)."""
    model, _, _ = gpu_model(dp, name)
    s = synth.fcc_copper(3, 0.08, seed=3) if tables == "folded" else eight_species_bcc()
    pos, species = on_dev(s, dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    ea, F, et = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    ea2, F2, et2, vir, w = model.compute_energy_forces_virial(pos, species, s.cell, s.pbc, 6.0,
                                                              rp, nj, ns, e, atom_virial=True)
    torch.cuda.synchronize()
    assert torch.equal(ea, ea2) and torch.equal(F, F2) and torch.equal(et, et2)
    assert np.abs(vir.cpu().numpy()).max() > 0.0


def start_state(dp, model, s, dev, temperature, list_radius=7.0):
    v0 = synth.maxwell_boltzmann(s, temperature)
    pos, species = on_dev(s, dev)
    vel = torch.tensor(v0, dtype=torch.float64, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, list_radius)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    return v0, pos, species, vel, F


def test_nvt_matches_oracle_dynamics(dev, dp):
    """Config 1 from 600 K under a 300 K chain with a 20 fs damping time:
    20 steps on the GPU against the oracle's integrator, then the virial of
    the last step against the oracle at the final positions."""
    model, oracle, _ = gpu_model(dp, "small")
    s = synth.make_workload("fcc108_small")[0]
    v0, pos, species, vel, F = start_state(dp, model, s, dev, 600.0)
    chain = torch.zeros(6, dtype=torch.float64, device=dev)
    ep, ek, eth, vir, nreb = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0,
                                            1.0, 1.0, 20, 0, F, 300.0, 20.0, chain, virial=True)
    torch.cuda.synchronize()
    rep, rek, reth, rpos, rvel, rchain = md.nvt(oracle, s.pos, v0, s.species, s.cell, s.pbc,
                                                s.mass_by_type[s.species], 1.0, 20, 300.0, 20.0)
    assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
    assert np.abs(vel.cpu().numpy() - rvel).max() < 1e-6
    assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
    assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n
    assert np.abs(eth.cpu().numpy() - reth[1:]).max() < E_TOL * s.n
    c = chain.cpu().numpy()
    assert np.allclose(c[:3], rchain.xi, rtol=1e-5, atol=1e-8)
    assert np.allclose(c[3:], rchain.v, rtol=1e-5, atol=1e-8)
    # the chain did work: the kinetic energy fell well below its start
    assert rek[-1] < 0.9 * rek[0]
    _, _, ref_vir, _ = oracle.energy_forces(rpos, s.species, s.cell, s.pbc, virial=True)
    assert np.abs(vir[-1].cpu().numpy() - ref_vir).max() < E_TOL * s.n


def test_nvt_with_frequent_rebuilds_matches_oracle(dev, dp):
    """A 0.15 A skin makes batches roll back and replay, with the chain state
    restored; the trajectory still follows the oracle."""
    model, oracle, _ = gpu_model(dp, "small")
    s = synth.make_workload("fcc108_small")[0]
    v0, pos, species, vel, F = start_state(dp, model, s, dev, 600.0, list_radius=6.2)
    chain = torch.zeros(6, dtype=torch.float64, device=dev)
    ep, ek, eth, _, nreb = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0,
                                          0.15, 1.0, 30, 0, F, 300.0, 20.0, chain)
    torch.cuda.synchronize()
    assert nreb >= 3
    rep, rek, reth, rpos, rvel, _ = md.nvt(oracle, s.pos, v0, s.species, s.cell, s.pbc,
                                           s.mass_by_type[s.species], 1.0, 30, 300.0, 20.0)
    assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
    assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
    assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n
    assert np.abs(eth.cpu().numpy() - reth[1:]).max() < E_TOL * s.n


def test_nvt_conserves_the_extended_energy(dev, dp):
    """1000 steps of config 1 at 300 K with the paper's 0.1 ps damping time:
    the drift of E_pot + E_kin + E_thermostat stays below 1e-5 eV/atom/ps,
    the target for NVE."""
    model, _, _ = gpu_model(dp, "small")
    s = synth.make_workload("fcc108_small")[0]
    _, pos, species, vel, F = start_state(dp, model, s, dev, 300.0)
    chain = torch.zeros(6, dtype=torch.float64, device=dev)
    ep, ek, eth, _, _ = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 1.0,
                                       1.0, 1000, 0, F, 300.0, 100.0, chain)
    h = (ep + ek + eth).cpu().numpy()
    assert abs(md.drift_ev_per_atom_ps(h, 1.0, s.n)) < 1e-5
    assert np.abs(eth.cpu().numpy()).max() > 1e-3    # the thermostat exchanged energy


def test_decoupled_chain_reproduces_nve_bit_for_bit(dev, dp):
    """A 1e12 fs damping time leaves every scale factor at exactly 1, so the
    NVT path reproduces verlet_step bit for bit (positions, velocities,
    forces, both energies), including across rebuilds."""
    model, _, _ = gpu_model(dp, "full")
    s = synth.make_workload("fcc4000_full")[0]
    outs = []
    for mode in ("nve", "nvt"):
        _, pos, species, vel, F = start_state(dp, model, s, dev, 600.0)
        if mode == "nve":
            ep, ek, nreb = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0,
                                             0.5, 1.0, 40, 0, F)
        else:
            chain = torch.zeros(6, dtype=torch.float64, device=dev)
            ep, ek, _, _, nreb = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc,
                                                6.0, 0.5, 1.0, 40, 0, F, 300.0, 1e12, chain)
        torch.cuda.synchronize()
        outs.append((pos.cpu().numpy(), vel.cpu().numpy(), F.cpu().numpy(), ep.cpu().numpy(),
                     ek.cpu().numpy(), nreb))
    a, b = outs
    assert a[5] == b[5] and a[5] >= 2
    diff = {name: (int((x != y).sum()), float(np.abs(x - y).max()))
            for name, x, y in zip(("pos", "vel", "forces", "e_pot", "e_kin"), a[:5], b[:5])}
    assert all(c == 0 for c, _ in diff.values()), diff


def test_nvt_is_bit_reproducible(dev, dp):
    model, _, _ = gpu_model(dp, "full")
    s = synth.make_workload("fcc4000_full")[0]
    outs = []
    for _ in range(2):
        _, pos, species, vel, F = start_state(dp, model, s, dev, 600.0)
        chain = torch.zeros(6, dtype=torch.float64, device=dev)
        ep, ek, eth, vir, nreb = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc,
                                                6.0, 0.5, 1.0, 40, 0, F, 300.0, 100.0, chain,
                                                virial=True)
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (pos, vel, F, ep, ek, eth, vir, chain)] + [nreb])
    a, b = outs
    assert a[-1] == b[-1] and a[-1] >= 2
    for x, y in zip(a[:-1], b[:-1]):
        assert np.array_equal(x, y)


def test_nvt_rejects_bad_parameters(dev, dp):
    model, _, _ = gpu_model(dp, "small")
    s = synth.make_workload("fcc108_small")[0]
    _, pos, species, vel, F = start_state(dp, model, s, dev, 300.0)
    for kw in ({"temperature": -1.0, "t_damp_fs": 100.0, "chain": torch.zeros(6, dtype=torch.float64, device=dev)},
               {"temperature": 300.0, "t_damp_fs": 0.0, "chain": torch.zeros(6, dtype=torch.float64, device=dev)},
               {"temperature": 300.0, "t_damp_fs": 100.0, "chain": torch.zeros(18, dtype=torch.float64, device=dev)}):
        with pytest.raises(dp.DPA4CError) as ei:
            model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0, 1.0, 1.0, 5, 0, F,
                           **kw)
        assert ei.value.code == -1


def test_diamond_nvt_matches_oracle(dev, dp):
    """The benchmark's diamond carbon (3^3 conventional cells, 216 atoms, 158
    neighbours each) with the carbon-calibrated full model: 10 NVT steps at
    300 K with the 0.1 ps damping time against the oracle."""
    model, oracle, _ = gpu_model(dp, "full_carbon")
    s = synth.diamond_carbon(3, 0.03, seed=0)
    v0, pos, species, vel, F = start_state(dp, model, s, dev, 300.0)
    chain = torch.zeros(6, dtype=torch.float64, device=dev)
    ep, ek, eth, vir, _ = model.nvt_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, 6.0,
                                         1.0, 1.0, 10, 0, F, 300.0, 100.0, chain, virial=True)
    torch.cuda.synchronize()
    rep, rek, reth, rpos, rvel, _ = md.nvt(oracle, s.pos, v0, s.species, s.cell, s.pbc,
                                           s.mass_by_type[s.species], 1.0, 10, 300.0, 100.0)
    assert np.abs(pos.cpu().numpy() - rpos).max() < 1e-6
    assert np.abs(ep.cpu().numpy() - rep[1:]).max() < E_TOL * s.n
    assert np.abs(ek.cpu().numpy() - rek[1:]).max() < E_TOL * s.n
    assert np.abs(eth.cpu().numpy() - reth[1:]).max() < E_TOL * s.n
    _, _, ref_vir, _ = oracle.energy_forces(rpos, s.species, s.cell, s.pbc, virial=True)
    assert np.abs(vir[-1].cpu().numpy() - ref_vir).max() < E_TOL * s.n


def test_diamond1m_sampled_full_size(dev, dp):
    """The 1,000,000-atom diamond-carbon workload of the NVT benchmark at full
    size, carbon-calibrated full model: E_i and the per-centre virial terms W_i
    of sampled centres and the forces of sampled atoms, each against the
    oracle evaluated on exactly the centres it needs; the total virial is
    symmetric (rotation invariance) to the energy tolerance."""
    model, oracle, _ = gpu_model(dp, "full_carbon")
    s = synth.make_workload("diamond1m_nvt_full")[0]
    pos, species = on_dev(s, dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, 7.0)
    ea, F, et, vir, w = model.compute_energy_forces_virial(pos, species, s.cell, s.pbc, 6.0, rp,
                                                           nj, ns, e, atom_virial=True)
    torch.cuda.synchronize()
    ea, F, vir, w = ea.cpu().numpy(), F.cpu().numpy(), vir.cpu().numpy(), w.cpu().numpy()
    del rp, nj, ns
    rng = np.random.Generator(np.random.PCG64(23))
    ks = np.unique(np.concatenate([[0, s.n - 1], rng.choice(s.n, 1, replace=False)])).astype(np.int64)
    _, ej, _ = onb.neighbor_list(s.pos, s.cell, s.pbc, 6.0, centres=ks)
    centres = np.unique(np.concatenate([ks, ej]))
    ref_e, ref_f, _, ref_w = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc,
                                                  centres=centres, virial=True)
    assert np.abs(ea[centres] - ref_e).max() < E_TOL
    assert np.abs(w[centres] - ref_w).max() < W_TOL
    assert np.abs(F[ks] - ref_f[ks]).max() < F_TOL
    assert np.abs(vir - vir.T).max() < E_TOL * s.n
