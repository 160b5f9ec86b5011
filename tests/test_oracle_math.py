"""Pins of the oracle's closed-form pieces against the paper's printed values
and against independent mathematics (no GPU)."""
import itertools
import math

import numpy as np
import pytest
import torch

import synth
from conftest import golden
from oracle import model as om

F64 = torch.float64
S1 = {k: float(v) for k, v in golden("table_s1_verification.txt")}


def rand_u(n, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    return torch.tensor(g.normal(size=(n, 3)), dtype=F64)


# -- widths: Table S2 and Table S3 -------------------------------------------
@pytest.mark.parametrize("row", golden("table_s2_widths.txt"))
def test_widths_table_s2(row):
    C0, C1, C2, K1, K2 = map(int, row[:5])
    S = list(map(int, row[5:8]))
    D = list(map(int, row[8:11]))
    for i, L in enumerate((2, 3, 4)):
        C = om.degree_channels(C0, L)
        K = om.probe_ranks(C0, L)
        assert (C[1], C[2], K[1], K[2]) == (C1, C2, K1, K2)
        assert all(c == 1 for c in C[3:])
        assert om.feature_width(C0, L) == S[i]
        assert om.descriptor_width(C0, L) == D[i]
        assert synth.descriptor_width(C0, L) == D[i]


@pytest.mark.parametrize("row", golden("table_s3_variants.txt"))
def test_variants_table_s3(row):
    name = row[0]
    C0, L, R, S, D, F, nl, nrbf, count = map(int, row[1:])
    spec = synth.MODELS[name]
    assert (spec.C0, spec.L, spec.R, spec.F, spec.n_layers, spec.n_rbf) == (C0, L, R, F, nl, nrbf)
    assert om.feature_width(C0, L) == S
    assert om.descriptor_width(C0, L) == D
    # the blob layout (type table with padding row, trainable omega,
    # bias-free gated nets, biased MLP) reproduces the printed count exactly
    assert synth.trainable_count(spec) == count


def test_triples_eq_triples():
    # the paper lists the L = 4 set explicitly (Eq. (triples) and text)
    assert om.admissible_triples(4) == [(1, 1, 2), (1, 2, 3), (1, 3, 4), (2, 2, 2), (2, 2, 4),
                                        (2, 3, 3), (2, 4, 4), (3, 3, 4), (4, 4, 4)]
    assert om.admissible_triples(2) == [(1, 1, 2), (2, 2, 2)]
    assert om.admissible_triples(3) == [(1, 1, 2), (1, 2, 3), (2, 2, 2), (2, 3, 3)]


def test_bispectrum_count_formula():
    # Eq. (bispectrum-count): distinct / two equal / three equal degrees
    for C0, L in itertools.product((8, 16, 32, 64, 128), (2, 3, 4)):
        K = om.probe_ranks(C0, L)
        for t in om.admissible_triples(L):
            k = [K[l] for l in t]
            if t[0] == t[1] == t[2]:
                want = k[0] * (k[0] + 1) * (k[0] + 2) // 6
            elif t[0] == t[1]:
                want = k[0] * (k[0] + 1) // 2 * k[2]
            elif t[1] == t[2]:
                want = k[1] * (k[1] + 1) // 2 * k[0]
            else:
                want = k[0] * k[1] * k[2]
            ent = om.bispectrum_entries(t, K)
            assert len(ent) == want
            # family weights: the squared weights add up to the full tensor size
            assert math.isclose(sum(w * w for _, w in ent), k[0] * k[1] * k[2])


# -- harmonics ---------------------------------------------------------------
@pytest.mark.parametrize("l", range(5))
def test_addition_theorem(l):
    u, v = rand_u(500, 1), rand_u(500, 2)
    lhs = (om.harmonics(u, l) * om.harmonics(v, l)).sum(1)
    nu, nv = u.norm(dim=1), v.norm(dim=1)
    c = ((u * v).sum(1) / (nu * nv)).numpy()
    P = np.polynomial.legendre.legval(c, [0] * l + [1])
    rhs = (nu * nv).numpy() ** l * P
    assert np.abs(lhs.numpy() - rhs).max() <= S1["addition_theorem"] * max(1.0, np.abs(rhs).max())


@pytest.mark.parametrize("l", range(5))
def test_parity(l):
    u = rand_u(200, 3)
    assert torch.equal(om.harmonics(-u, l), (-1) ** l * om.harmonics(u, l))


def test_degree_two_is_the_paper_formula():
    # Eq. (harmonics) degree two, retyped element by element
    u = rand_u(50, 4)
    x, y, z = u.T
    s = x * x + y * y + z * z
    r3 = math.sqrt(3)
    want = torch.stack([r3 * x * y, r3 * y * z, (3 * z * z - s) / 2, r3 * x * z, r3 / 2 * (x * x - y * y)], 1)
    assert torch.allclose(om.harmonics(u, 2), want, atol=0, rtol=1e-15)


def test_stf_isometry_and_quadrupolar_form():
    g = np.random.Generator(np.random.PCG64(5))
    z1 = torch.tensor(g.normal(size=(100, 5)), dtype=F64)
    z2 = torch.tensor(g.normal(size=(100, 5)), dtype=F64)
    Q1, Q2 = om.stf(z1), om.stf(z2)
    assert torch.allclose(Q1, Q1.transpose(1, 2), atol=0)
    assert (Q1.diagonal(dim1=1, dim2=2).sum(1).abs().max() < 1e-14)
    frob = (Q1 * Q2).sum((1, 2))
    assert (frob - (z1 * z2).sum(1)).abs().max() <= S1["stf_isometry"] * 10
    u = rand_u(100, 6)
    Q = om.stf(om.harmonics(u, 2))
    s = (u * u).sum(1)
    want = math.sqrt(1.5) * (u[:, :, None] * u[:, None, :] - s[:, None, None] / 3 * torch.eye(3, dtype=F64))
    assert (Q - want).abs().max() <= S1["quadrupolar_form"]


# -- Gaunt tensors: quadrature versus exact monomial moments -------------------
def _monomial_coeffs(l):
    """Coefficients of B_l (with s = x^2+y^2+z^2) in the degree-l monomial basis,
    recovered by solving a linear system on random points."""
    mons = [(a, b, l - a - b) for a in range(l + 1) for b in range(l + 1 - a)]
    u = rand_u(4 * len(mons) + 8, 7)
    A = torch.stack([u[:, 0] ** a * u[:, 1] ** b * u[:, 2] ** c for a, b, c in mons], 1)
    coef = torch.linalg.lstsq(A, om.harmonics(u, l)).solution       # [n_mon, 2l+1]
    return mons, coef.numpy()


def _sphere_moment(a, b, c):
    # integral over the unit sphere of x^a y^b z^c
    if a % 2 or b % 2 or c % 2:
        return 0.0
    return 2.0 * math.gamma((a + 1) / 2) * math.gamma((b + 1) / 2) * math.gamma((c + 1) / 2) / \
        math.gamma((a + b + c + 3) / 2)


@pytest.mark.parametrize("t", om.admissible_triples(4))
def test_gaunt_quadrature_equals_exact_moments(t):
    got = om.gaunt_integral(*t)
    m1, c1 = _monomial_coeffs(t[0])
    m2, c2 = _monomial_coeffs(t[1])
    m3, c3 = _monomial_coeffs(t[2])
    want = np.zeros(got.shape)
    for (p1, k1), (p2, k2), (p3, k3) in itertools.product(enumerate(m1), enumerate(m2), enumerate(m3)):
        mom = _sphere_moment(k1[0] + k2[0] + k3[0], k1[1] + k2[1] + k3[1], k1[2] + k2[2] + k3[2])
        if mom:
            want += mom * np.einsum("a,b,c->abc", c1[p1], c2[p2], c3[p3])
    assert np.abs(got - want).max() < 1e-12
    assert np.linalg.norm(got) > 0.1


def test_closed_forms_against_gaunt():
    # Eq. (closed-forms) with C = -I/||I||_F (reading R1)
    g = np.random.Generator(np.random.PCG64(8))
    C112 = om.coupling_tensor(1, 1, 2)
    C222 = om.coupling_tensor(2, 2, 2)
    worst = 0.0
    for _ in range(50):
        v1, v2 = g.normal(size=3), g.normal(size=3)
        z = g.normal(size=(3, 5))
        Q = [om.stf(torch.tensor(zz)).numpy() for zz in z]
        j112 = np.einsum("abc,a,b,c->", C112, v1, v2, z[0])
        worst = max(worst, abs(j112 - (-1 / math.sqrt(5)) * v1 @ Q[0] @ v2))
        j222 = np.einsum("abc,a,b,c->", C222, z[0], z[1], z[2])
        worst = max(worst, abs(j222 - (-math.sqrt(12 / 35)) * np.trace(Q[0] @ Q[1] @ Q[2])))
    assert worst <= S1["closed_forms_vs_gaunt"]


def test_coupling_symmetry_equal_degrees():
    # the coupling is symmetric under swaps of equal-degree axes (used by
    # the non-decreasing representative rule of Eq. (bispectrum))
    C = om.coupling_tensor(1, 1, 2)
    assert np.abs(C - C.transpose(1, 0, 2)).max() < 1e-15
    C = om.coupling_tensor(2, 3, 3)
    assert np.abs(C - C.transpose(0, 2, 1)).max() < 1e-15
    C = om.coupling_tensor(2, 2, 2)
    for p in itertools.permutations(range(3)):
        assert np.abs(C - C.transpose(p)).max() < 1e-15


# -- envelope and basis --------------------------------------------------------
def test_envelope_identities():
    rc = 6.0
    rho = torch.linspace(0.0, rc * 1.2, 2001, dtype=F64)
    chi = om.envelope(rho, rc)
    x = torch.clamp(rho / rc, max=1.0)
    expanded = 1 - 56 * x ** 5 + 140 * x ** 6 - 120 * x ** 7 + 35 * x ** 8
    # the expanded form cancels terms of size ~100 near x = 1
    assert (chi - expanded).abs().max() < 1e-13
    assert om.envelope(torch.tensor([0.0], dtype=F64), rc).item() == 1.0
    assert om.envelope(torch.tensor([rc], dtype=F64), rc).item() == 0.0
    assert (chi[rho >= rc] == 0).all()
    # C^3 at the cutoff: derivatives 1..3 vanish from the left, the 4th does not
    r = torch.tensor([rc - 1e-12], dtype=F64, requires_grad=True)
    d = om.envelope(r, rc)
    ders = []
    for k in range(4):
        (d,) = torch.autograd.grad(d.sum(), r, create_graph=True)
        ders.append(d.item())
    assert all(abs(v) < 1e-8 for v in ders[:3])
    assert abs(ders[3]) > 1e-3


def test_bessel_basis_limit():
    # Eq. (bessel-basis): f_n -> omega_n as rho -> 0
    omega = torch.tensor([1.0, 3.0, 8.0], dtype=F64)
    f = om.bessel_basis(torch.tensor([1e-7], dtype=F64), omega)
    assert torch.allclose(f[0], omega, rtol=1e-12)
    rho = torch.tensor([0.7], dtype=F64)
    assert torch.allclose(om.bessel_basis(rho, omega)[0], torch.sin(omega * 0.7) / 0.7, rtol=0)
