"""Pins of the oracle potential (no GPU): finite differences, invariances,
aggregation identities and energy conservation."""
import math

import numpy as np
import pytest
import torch

import synth
from conftest import golden
from oracle import md
from oracle import model as om
from oracle import neighbors as nb

S1 = {k: float(v) for k, v in golden("table_s1_verification.txt")}


def oracle_for(name):
    spec, w = synth.model_weights(name)
    return om.Oracle(spec, w)


def two_element_cell(seed=11, n=24):
    # 24-atom periodic cell of two elements, as in Table S1
    return synth.random_periodic(n, seed=seed, cell=np.diag([8.3, 8.9, 9.4]), d_min=1.6)


def random_rotation(seed):
    g = np.random.Generator(np.random.PCG64(seed))
    q, r = np.linalg.qr(g.normal(size=(3, 3)))
    q = q * np.sign(np.diag(r))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


@pytest.fixture(scope="module")
def small():
    return oracle_for("small")


@pytest.fixture(scope="module")
def full():
    return oracle_for("full")


@pytest.mark.parametrize("which", ["small", "full"])
def test_forces_match_central_differences(which, request):
    o = request.getfixturevalue(which)
    s = two_element_cell()
    edges = nb.neighbor_list(s.pos, s.cell, s.pbc, o.r_c)
    e, F = o.energy_forces(s.pos, s.species, s.cell, s.pbc, edges=edges)
    h = 1e-4
    g = np.random.Generator(np.random.PCG64(3))
    atoms = g.choice(s.n, size=4, replace=False)
    fd = np.zeros((len(atoms), 3))
    for a, k in enumerate(atoms):
        for c in range(3):
            p = s.pos.copy()
            p[k, c] += h
            ep, _ = o.energy_forces(p, s.species, s.cell, s.pbc, edges=edges)
            p[k, c] -= 2 * h
            em, _ = o.energy_forces(p, s.species, s.cell, s.pbc, edges=edges)
            fd[a, c] = -(ep.sum() - em.sum()) / (2 * h)
    rel = np.abs(fd - F[atoms]).max() / np.abs(F[atoms]).max()
    assert rel < 1e-6


@pytest.mark.parametrize("which", ["small", "full"])
def test_total_force_vanishes(which, request):
    o = request.getfixturevalue(which)
    s = two_element_cell(seed=12)
    _, F = o.energy_forces(s.pos, s.species, s.cell, s.pbc)
    assert np.abs(F.sum(0)).max() < 1e-12 * max(1.0, np.abs(F).sum())


@pytest.mark.parametrize("which", ["small", "full"])
def test_rotation_translation_permutation(which, request):
    o = request.getfixturevalue(which)
    s = two_element_cell(seed=13)
    ref = o.stages(s.pos, s.species, s.cell, s.pbc)
    e0, F0 = o.energy_forces(s.pos, s.species, s.cell, s.pbc)
    scale = max(1.0, np.abs(ref["D"]).max())
    # proper rotation, applied to atoms and cell
    R = random_rotation(1)
    rot = o.stages(s.pos @ R.T, s.species, s.cell @ R.T, s.pbc)
    assert np.abs(rot["D"] - ref["D"]).max() <= 50 * S1["rotation_24_atom_periodic"] * scale
    assert np.abs(rot["E"] - ref["E"]).max() <= 1e-13
    _, Fr = o.energy_forces(s.pos @ R.T, s.species, s.cell @ R.T, s.pbc)
    assert np.abs(Fr - F0 @ R.T).max() < 1e-12                 # equivariant forces
    # translation
    tr = o.stages(s.pos + np.array([0.37, -1.91, 2.44]), s.species, s.cell, s.pbc)
    assert np.abs(tr["D"] - ref["D"]).max() <= 50 * S1["translation_24_atom_periodic"] * scale
    # relabelling among atoms of the same element
    g = np.random.Generator(np.random.PCG64(2))
    perm = np.arange(s.n)
    for t in np.unique(s.species):
        idx = np.nonzero(s.species == t)[0]
        perm[idx] = g.permutation(idx)
    inv = np.argsort(perm)                                      # r'_{perm[k]} = r_k
    pp = o.stages(s.pos[inv], s.species[inv], s.cell, s.pbc)
    assert np.abs(pp["D"][perm] - ref["D"]).max() <= 50 * S1["permutation_24_atom_periodic"] * scale
    assert np.abs(pp["E"][perm] - ref["E"]).max() <= 1e-13


@pytest.mark.parametrize("which", ["small", "full"])
def test_inversion_isolated_cluster_is_exact(which, request):
    o = request.getfixturevalue(which)
    s = synth.random_cluster(12, seed=14)
    a = o.stages(s.pos, s.species, s.cell, s.pbc)
    b = o.stages(-s.pos, s.species, -s.cell, s.pbc)
    assert np.abs(a["D"] - b["D"]).max() <= S1["inversion_12_atom_cluster"]


@pytest.mark.parametrize("which", ["small", "full"])
def test_single_aggregation_equals_per_degree_sums(which, request):
    """Eq. (payload)/(moments): the one vectorised segment sum equals plain
    per-edge loops run separately for every degree."""
    o = request.getfixturevalue(which)
    s = two_element_cell(seed=15, n=8)
    ei, ej, en = nb.neighbor_list(s.pos, s.cell, s.pbc, o.r_c)
    st = o.stages(s.pos, s.species, s.cell, s.pbc)
    r = s.pos[ej] + en @ s.cell - s.pos[ei]
    rt = torch.tensor(r)
    rho, u = om.edge_geometry(rt)
    chi = om.envelope(rho, o.r_c)
    f = om.bessel_basis(rho, o.w["omega"])
    h = om.swiglu(f, o.w["W_in"])
    g = h @ o.w["W_out"]
    q = h @ o.w["W_mode"] if o.R else None
    worst = 0.0
    for l in range(o.L + 1):
        B = om.harmonics(u, l)
        Cl = o.C[l]
        for i in range(s.n):
            acc = np.zeros((2 * l + 1, Cl))
            s2 = 0.0
            for e in np.nonzero(ei == i)[0]:
                gam, bet, U = o.pair_coefficients(s.species[i], s.species[ej[e]])
                psi = (gam * g[e] + bet).numpy()
                if o.R:
                    psi = psi + (U @ q[e]).numpy()
                wl = chi[e].item() if l == 0 else chi[e].item() ** 2
                acc += wl * np.outer(B[e].numpy(), psi[:Cl])
                s2 += wl * wl
            M = math.sqrt(0.25 + s2)
            off = o.S - sum((2 * k + 1) * o.C[k] for k in range(l, o.L + 1))
            got = st["X_flat"][i, off:off + (2 * l + 1) * Cl].reshape(2 * l + 1, Cl)
            worst = max(worst, np.abs(got - acc / M).max() / max(1.0, np.abs(acc / M).max()))
    assert worst <= 20 * S1["single_aggregation_vs_per_degree"]


def test_aggregation_is_order_independent(small):
    s = two_element_cell(seed=16)
    ei, ej, en = nb.neighbor_list(s.pos, s.cell, s.pbc, small.r_c)
    g = np.random.Generator(np.random.PCG64(4))
    perm = np.argsort(ei * 10000 + g.permutation(len(ei)) % 10000, kind="stable")
    a = small.stages(s.pos, s.species, s.cell, s.pbc, edges=(ei, ej, en))
    b = small.stages(s.pos, s.species, s.cell, s.pbc, edges=(ei[perm], ej[perm], en[perm]))
    assert np.abs(a["D"] - b["D"]).max() < 1e-12


def test_isolated_atom_features():
    """No neighbours: M0 = M1 = 1/2 (Eq. (masses) floor) and every aggregated
    feature vanishes, so D_tilde = [X0, 0, 1/2, 1/2, 0 ...]."""
    o = oracle_for("small")
    pos = np.array([[0.0, 0.0, 0.0], [20.0, 0.0, 0.0]])
    st = o.stages(pos, np.array([28, 28], np.int32), np.diag([40.0, 40, 40]), np.zeros(3, np.int32))
    C0 = o.C0
    assert np.all(st["Dt"][:, C0:2 * C0] == 0)
    assert np.all(st["Dt"][:, 2 * C0:2 * C0 + 2] == 0.5)
    assert np.all(st["Dt"][:, 2 * C0 + 2:] == 0)
    assert np.allclose(st["Dt"][0, :C0], o.w["type_embed"][28].numpy())


def test_dimer_readout_closed_form():
    """One neighbour along u: X_1 = chi^2 psi_c u / M1 per channel, so the
    degree-one Gram block is chi^4 psi psi^T-shaped (rank one) and the
    degree-two features are proportional to B_2(u)."""
    o = oracle_for("small")
    d = np.array([1.1, -0.7, 1.9])
    pos = np.array([[0.0, 0.0, 0.0], d])
    st = o.stages(pos, np.array([28, 7], np.int32), np.diag([40.0, 40, 40]), np.zeros(3, np.int32))
    C0, C1, C2 = o.C[0], o.C[1], o.C[2]
    X1 = st["X_flat"][0, C0:C0 + 3 * C1].reshape(3, C1)
    rho = math.sqrt(d @ d + 1e-14)
    u = d / rho
    # every channel column of X_1 is parallel to u
    assert np.abs(np.cross(X1.T, u)).max() < 1e-14
    X2 = st["X_flat"][0, C0 + 3 * C1:C0 + 3 * C1 + 5 * C2].reshape(5, C2)
    B2 = om.harmonics(torch.tensor(u[None]), 2).numpy()[0]
    ratio = X2 / B2[:, None]
    assert np.abs(ratio - ratio[0]).max() < 1e-12
    chi = om.envelope(torch.tensor([rho], dtype=torch.float64), o.r_c).item()
    assert math.isclose(st["M1"][0], math.sqrt(0.25 + chi ** 4), rel_tol=1e-15)


@pytest.mark.slow
def test_nve_energy_conservation_config1(small):
    """100 velocity-Verlet steps of the 108-atom cell at 1 fs: drift below
    1e-5 eV/atom/ps (the stated NVE target)."""
    s = synth.fcc_copper(3, 0.05, seed=0)
    v = synth.maxwell_boltzmann(s, 300.0)
    ep, ek, _, _ = md.nve(small, s.pos, v, s.species, s.cell, s.pbc,
                          s.mass_by_type[s.species], 1.0, 100)
    et = ep + ek
    assert abs(md.drift_ev_per_atom_ps(et, 1.0, s.n)) < 1e-5
    assert (et.max() - et.min()) / s.n < 1e-5


def triclinic_cell_system(seed=5, n=20):
    cell = np.array([[8.3, 0.0, 0.0], [1.2, 8.9, 0.0], [0.7, -0.9, 9.4]])
    return synth.random_periodic(n, seed=seed, cell=cell, d_min=1.6)


@pytest.mark.parametrize("which", ["small", "full"])
def test_virial_is_minus_the_strain_derivative_of_the_energy(which, request):
    # Eq. (forces): Xi = -sum g (x) r.  Independently, under a homogeneous
    # deformation x -> (I + eps) x of positions and cell every edge vector
    # becomes (I + eps) r, so dE/d eps_ab = sum_e g_a r_b = -Xi_ab; checked by
    # central differences with the neighbour list held fixed, on a triclinic
    # cell so that every component is distinct.
    o = request.getfixturevalue(which)
    s = triclinic_cell_system()
    edges = nb.neighbor_list(s.pos, s.cell, s.pbc, o.r_c)
    e, F, Xi, W = o.energy_forces(s.pos, s.species, s.cell, s.pbc, edges=edges, virial=True)
    assert np.allclose(W.sum(axis=0), Xi, rtol=0, atol=1e-12)
    h = 1e-5
    fd = np.zeros((3, 3))
    for a in range(3):
        for b in range(3):
            es = []
            for sgn in (1.0, -1.0):
                A = np.eye(3)
                A[a, b] += sgn * h
                st = o.stages(s.pos @ A.T, s.species, s.cell @ A.T, s.pbc, edges=edges)
                es.append(st["E"].sum())
            fd[a, b] = -(es[0] - es[1]) / (2 * h)
    scale = np.abs(Xi).max()
    assert np.abs(fd - Xi).max() < 1e-7 * scale, (fd, Xi)
    # rotation invariance makes the virial symmetric
    assert np.abs(Xi - Xi.T).max() < 1e-12 * scale
