"""Pins of the oracle's readout, pair modulation, gated units and MLP (no GPU).

Each test fixes a part of the oracle by something the paper or the
mathematics states, not by the oracle's own formula:

- the Gram half-vectorisation preserves the Frobenius norm (Eq. (gram));
- the channel alignment of a single-neighbour environment has a closed form
  (Eq. (alignment) applied to a rank-one feature block);
- the retained bispectrum entries equal the closed forms of
  Eq. (closed-forms), scaled by the square root of their family size, and
  keep the norm of the full symmetric tensor (Eq. (bispectrum));
- the quartic invariant equals its second form v^T Q^2 v (Eq. (quartic));
- hand-set pair-network weights give the modulation of Eq. (pairfilm) in
  closed form, with the gate and value branches of Eq. (swiglu);
- hand-set MLP weights give the residual chain of Eq. (fitting) in closed
  form.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import model as om

RTOL = 1e-12


def silu(z):
    """The paper's SiLU, z / (1 + exp(-z)), written out on floats."""
    return z / (1.0 + math.exp(-z))


def oracle_with(name, **overrides):
    """The oracle of a workload model with some weight arrays replaced."""
    spec, w = synth.model_weights(name)
    w = {k: np.array(v, dtype=np.float64) for k, v in w.items()}
    for k, v in overrides.items():
        w[k] = np.asarray(v, dtype=np.float64)
    return om.Oracle(spec, w), spec, w


def zero_align(name):
    spec, w = synth.model_weights(name)
    return {f"W_align{l}": np.zeros_like(w[f"W_align{l}"]) for l in (1, 2)}


def env(seed=21, n=10):
    return synth.random_periodic(n, seed=seed, cell=np.diag([7.6, 8.1, 8.7]), d_min=1.7)


def split_x(o, x_flat):
    """Node features X_l as (2l+1) x C_l blocks from the flat degree -> m ->
    channel layout."""
    out, off = [], 0
    for l in range(o.L + 1):
        k = (2 * l + 1) * o.C[l]
        out.append(x_flat[off:off + k].reshape(2 * l + 1, o.C[l]))
        off += k
    return out


def bis_count(triple, K):
    """Eq. (bispectrum-count)."""
    l1, l2, l3 = triple
    if l1 == l2 == l3:
        k = K[l1]
        return k * (k + 1) * (k + 2) // 6
    if l1 == l2 or l2 == l3:
        rep = l2
        other = l3 if l1 == l2 else l1
        return K[rep] * (K[rep] + 1) // 2 * K[other]
    return K[l1] * K[l2] * K[l3]


def blocks_of(o, dt):
    """Split one descriptor row into the blocks of Eq. (descriptor), with the
    widths of Eqs. (dim-out) and (bispectrum-count)."""
    C0, L = o.C0, o.L
    out, off = {}, 0
    for name, k in (("X0i", C0), ("X0", C0), ("M0", 1), ("M1", 1)):
        out[name] = dt[off:off + k]
        off += k
    for l in range(1, L + 1):
        k = o.C[l] * (o.C[l] + 1) // 2
        out[("vech", l)] = dt[off:off + k]
        off += k
    trip = [t for t in sorted(
        (a, b, c) for a in range(1, L + 1) for b in range(a, L + 1) for c in range(b, L + 1)
        if c <= a + b and (a + b + c) % 2 == 0)]
    for t in trip:
        k = bis_count(t, o.K)
        out[("J", t)] = dt[off:off + k]
        off += k
    out["Pi"] = dt[off:off + o.K[1] * o.K[2]]
    off += o.K[1] * o.K[2]
    assert off == len(dt) == o.D_out
    return out


def stf_matrix(z):
    """Eq. (stf): the symmetric trace-free matrix of a packed degree-two
    vector in the order of B_2 (xy, yz, z^2, xz, x^2 - y^2), the linear map
    with STF[B_2(u)] = sqrt(3/2) (u u^T - |u|^2 I / 3), written entry by entry
    (checked against that definition below)."""
    a, b, c, d, e = z
    r2, r6 = math.sqrt(2.0), math.sqrt(6.0)
    return np.array([[-c / r6 + e / r2, a / r2, d / r2],
                     [a / r2, -c / r6 - e / r2, b / r2],
                     [d / r2, b / r2, 2 * c / r6]])


def test_stf_helper_matches_its_definition():
    rng = np.random.Generator(np.random.PCG64(6))
    u = rng.normal(size=(20, 3))
    B2 = om.harmonics(torch.tensor(u), 2).numpy()
    for k in range(len(u)):
        want = math.sqrt(1.5) * (np.outer(u[k], u[k]) - (u[k] @ u[k]) / 3.0 * np.eye(3))
        assert np.allclose(stf_matrix(B2[k]), want, rtol=0, atol=1e-13 * (u[k] @ u[k]))


@pytest.mark.parametrize("name", ["small", "full"])
def test_gram_half_vectorisation_preserves_frobenius_norm(name):
    """Eq. (gram): with the off-diagonal entries scaled by sqrt 2 the vech
    block has the Frobenius norm of G = X^T X, which is sum_k sigma_k^4 over
    the singular values of X (alignment switched off so that X~ = X); the
    diagonal entries are the channel powers |X[:, c]|^2."""
    o, _, _ = oracle_with(name, **zero_align(name))
    s = env()
    st = o.stages(s.pos, s.species, s.cell, s.pbc)
    for i in range(s.n):
        X = split_x(o, st["X_flat"][i])
        b = blocks_of(o, st["Dt"][i])
        for l in range(1, o.L + 1):
            v = b[("vech", l)]
            sig = np.linalg.svd(X[l], compute_uv=False)
            want = float((sig ** 4).sum())
            assert abs(float(v @ v) - want) <= RTOL * want
            C = o.C[l]
            diag_pos = [c * C - c * (c - 1) // 2 for c in range(C)]   # row-major upper triangle
            assert np.allclose(v[diag_pos], (X[l] ** 2).sum(0), rtol=RTOL, atol=0)


@pytest.mark.parametrize("name", ["small", "full"])
def test_alignment_of_a_single_neighbour_has_a_closed_form(name):
    """One neighbour along u: X_l = B_l(u) a^T is rank one, so Eq. (alignment)
    gives X~_l = B_l(u) b^T with b = (I + W_l)^T a, and the Gram block is
    |B_l(u)|^2 b b^T.  The test sets W_l to a non-symmetric random matrix of
    order one, so that dropping W_l or transposing it changes every entry."""
    _, spec, w0 = oracle_with(name)
    rng = np.random.Generator(np.random.PCG64(7))
    Ws = {f"W_align{l}": 0.7 * rng.normal(size=w0[f"W_align{l}"].shape) for l in (1, 2)}
    o, _, _ = oracle_with(name, **Ws)
    d = np.array([1.1, -0.7, 1.9])
    pos = np.array([[0.0, 0.0, 0.0], d])
    st = o.stages(pos, np.array([28, 7], np.int32), np.diag([40.0, 40, 40]), np.zeros(3, np.int32))
    X = split_x(o, st["X_flat"][0])
    b = blocks_of(o, st["Dt"][0])
    u = torch.tensor((d / math.sqrt(d @ d + om.EPS ** 2))[None])
    for l in range(1, o.L + 1):
        B = om.harmonics(u, l).numpy()[0]
        nb = float(B @ B)
        a = X[l].T @ B / nb                      # X_l = B a^T
        assert np.abs(X[l] - np.outer(B, a)).max() <= 1e-13 * np.abs(X[l]).max()
        bb = (np.eye(o.C[l]) + Ws[f"W_align{l}"]).T @ a if l <= 2 else a
        C = o.C[l]
        want = np.array([nb * bb[c] * bb[e] * (1.0 if c == e else math.sqrt(2.0))
                         for c in range(C) for e in range(c, C)])
        assert np.allclose(b[("vech", l)], want, rtol=1e-11, atol=1e-14 * np.abs(want).max())


def probes(o, w, X):
    """Eq. (probes) with the alignment switched off: v_k = (X_1 A_1)[:, k],
    Q_eta = STF((X_2 A_2)[:, eta])."""
    Z1 = X[1] if o.K[1] == o.C[1] else X[1] @ w["A1"]
    Z2 = X[2] @ w["A2"]
    v = [Z1[:, k] for k in range(Z1.shape[1])]
    Q = [stf_matrix(Z2[:, e]) for e in range(Z2.shape[1])]
    return v, Q


def distinct_perms(idx):
    return math.factorial(len(idx)) // math.prod(math.factorial(idx.count(x)) for x in set(idx))


@pytest.mark.parametrize("name", ["small", "full"])
def test_bispectrum_blocks_equal_the_closed_forms_with_family_weights(name):
    """Eq. (closed-forms): J112 = -v1^T Q v2 / sqrt 5 and
    J222 = -sqrt(12/35) tr(Q1 Q2 Q3).  The descriptor keeps the non-decreasing
    representative on equal-degree axes, row-major, scaled by sqrt(number of
    distinct permutations) (Eq. (bispectrum)), so the retained block has the
    norm of the full symmetric tensor."""
    o, _, w = oracle_with(name, **zero_align(name))
    s = env(seed=22)
    st = o.stages(s.pos, s.species, s.cell, s.pbc)
    for i in range(s.n):
        X = split_x(o, st["X_flat"][i])
        b = blocks_of(o, st["Dt"][i])
        v, Q = probes(o, w, X)
        K1, K2 = len(v), len(Q)
        full112 = np.array([[[-(v[a] @ Q[e] @ v[c]) / math.sqrt(5.0) for e in range(K2)]
                             for c in range(K1)] for a in range(K1)])
        want = [full112[a, c, e] * math.sqrt(distinct_perms([a, c]))
                for a in range(K1) for c in range(a, K1) for e in range(K2)]
        got = b[("J", (1, 1, 2))]
        scale = np.abs(full112).max()
        assert np.allclose(got, want, rtol=0, atol=1e-12 * scale)
        assert abs(float(got @ got) - float((full112 ** 2).sum())) <= 1e-11 * scale ** 2
        full222 = np.array([[[-math.sqrt(12.0 / 35.0) * np.trace(Q[a] @ Q[c] @ Q[e])
                              for e in range(K2)] for c in range(K2)] for a in range(K2)])
        want = [full222[a, c, e] * math.sqrt(distinct_perms([a, c, e]))
                for a in range(K2) for c in range(a, K2) for e in range(c, K2)]
        got = b[("J", (2, 2, 2))]
        scale = np.abs(full222).max()
        assert np.allclose(got, want, rtol=0, atol=1e-12 * scale)
        assert abs(float(got @ got) - float((full222 ** 2).sum())) <= 1e-11 * scale ** 2


@pytest.mark.parametrize("name", ["small", "full"])
def test_quartic_block_equals_v_q_squared_v(name):
    """Eq. (quartic): Pi[eta, k] = |Q_eta v_k|^2 = v_k^T Q_eta^2 v_k, eta-major."""
    o, _, w = oracle_with(name, **zero_align(name))
    s = env(seed=23)
    st = o.stages(s.pos, s.species, s.cell, s.pbc)
    for i in range(s.n):
        X = split_x(o, st["X_flat"][i])
        v, Q = probes(o, w, X)
        want = np.array([v[k] @ Q[e] @ Q[e] @ v[k] for e in range(len(Q)) for k in range(len(v))])
        got = blocks_of(o, st["Dt"][i])["Pi"]
        assert np.allclose(got, want, rtol=1e-11, atol=0)


def test_swiglu_gate_and_value_branches():
    """Eq. (swiglu): the first H columns of xW are the gate, the last H the
    value; SiLU(2) * 3 versus the swapped SiLU(3) * 2."""
    x = torch.tensor([[1.0, 0.5]], dtype=torch.float64)
    W = torch.tensor([[2.0, -1.0, 3.0, 0.25], [0.0, 4.0, -2.0, 2.0]], dtype=torch.float64)
    got = om.swiglu(x, W)[0].tolist()
    want = [silu(2.0) * 2.0, silu(1.0) * 1.25]
    assert got == pytest.approx(want, rel=1e-15)


@pytest.mark.parametrize("name", ["small", "full"])
def test_pair_modulation_closed_form(name):
    """Eq. (pairfilm) with hand-set weights.  W_p,out = 0 gives gamma = 1,
    beta = X0_a + X0_b and U = 0.  Then one hidden unit k with gate weight 1
    on the first entry of X0_a and value weight 1 on the first entry of X0_b
    gives p = 0.1 SiLU(X0_a[0]) X0_b[0] (times the W_p,out row) for the
    ordered pair (a, b), and s_0, t_0 and the mode entries U[0, 0], U[0, 1]
    (channel-major reshape) follow in closed form."""
    _, spec, w0 = oracle_with(name)
    C0, R = spec.C0, spec.R
    Hp = w0["Wp_in"].shape[1] // 2
    o, _, w = oracle_with(name, Wp_out=np.zeros_like(w0["Wp_out"]))
    X0 = w["type_embed"]
    for a, b in ((28, 7), (7, 28), (3, 3)):
        g, bt, U = (t.numpy() for t in o.pair_coefficients(a, b))
        assert np.all(g == 1.0) and np.all(U == 0.0)
        assert np.array_equal(bt, X0[a] + X0[b])
    k = 5
    Wp_in = np.zeros_like(w0["Wp_in"])
    Wp_in[0, k] = 1.0            # gate of unit k reads X0_a[0]
    Wp_in[C0, Hp + k] = 1.0      # value of unit k reads X0_b[0]
    Wp_out = np.zeros_like(w0["Wp_out"])
    Wp_out[k, 0] = 1.0           # s_0
    Wp_out[k, C0 + 3] = -2.0     # t_3
    if R:
        Wp_out[k, 2 * C0 + 0] = 1.5      # w -> U[0, 0]
        Wp_out[k, 2 * C0 + 1] = -0.5     # w -> U[0, 1] (channel-major)
    o, _, w = oracle_with(name, Wp_in=Wp_in, Wp_out=Wp_out)
    for a, b in ((28, 7), (7, 28)):
        p = 0.1 * silu(X0[a][0]) * X0[b][0]
        g, bt, U = (t.numpy() for t in o.pair_coefficients(a, b))
        assert g[0] == pytest.approx(1.0 + math.tanh(p), rel=1e-14)
        assert np.all(g[1:] == 1.0)
        want_b = X0[a] + X0[b]
        want_b[3] += math.tanh(-2.0 * p)
        assert np.allclose(bt, want_b, rtol=1e-14, atol=1e-15)
        if R:
            want_u = np.zeros((C0, R))
            want_u[0, 0], want_u[0, 1] = math.tanh(1.5 * p), math.tanh(-0.5 * p)
            assert np.allclose(U, want_u, rtol=1e-14, atol=0)


@pytest.mark.parametrize("name", ["small", "full"])
def test_edge_amplitude_with_only_the_shift(name):
    """Eqs. (radial-map), (pairfilm), (amplitude): with W_out = 0, W_mode = 0 and
    W_p,out = 0 every edge carries psi = X0_a + X0_b.  For a dimer the scalar
    block is X_0 = chi(rho) psi / M0 with M0 = sqrt(1/4 + chi^2)
    (Eqs. (payload), (masses), (moments))."""
    _, spec, w0 = oracle_with(name)
    o, _, w = oracle_with(name, W_out=np.zeros_like(w0["W_out"]),
                          W_mode=np.zeros_like(w0["W_mode"]), Wp_out=np.zeros_like(w0["Wp_out"]))
    d = np.array([0.4, 2.2, -1.3])
    pos = np.array([[0.0, 0.0, 0.0], d])
    st = o.stages(pos, np.array([28, 7], np.int32), np.diag([40.0, 40, 40]), np.zeros(3, np.int32))
    rho = math.sqrt(d @ d + om.EPS ** 2)
    chi = om.envelope(torch.tensor([rho], dtype=torch.float64), spec.r_c).item()
    X0 = w["type_embed"]
    for i, (a, b) in enumerate(((28, 7), (7, 28))):
        want = chi * (X0[a] + X0[b]) / math.sqrt(0.25 + chi * chi)
        got = st["X_flat"][i][:o.C0]
        assert np.allclose(got, want, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("name", ["small", "full"])
def test_mlp_residual_chain_closed_form(name):
    """Eq. (fitting) with Theta_tau = 0: h1 = SiLU(b1) (no residual, since
    D_out differs from the width), h_tau = SiLU(b_tau) + h_(tau-1), so
    E_i = (SiLU(b1) + SiLU(b2) + SiLU(b3)) . w_head + b_head + E_ref[a_i]
    (Eq. (atomic-energy))."""
    _, spec, w0 = oracle_with(name)
    rng = np.random.Generator(np.random.PCG64(9))
    F = spec.F
    over = {f"Theta{t}": np.zeros_like(w0[f"Theta{t}"]) for t in range(1, spec.n_layers + 1)}
    for t in range(1, spec.n_layers + 1):
        over[f"b{t}"] = rng.normal(size=F)
    over["w_head"] = rng.normal(size=F)
    over["b_head"] = np.array([0.3])
    E_ref = np.zeros(119)
    E_ref[28], E_ref[7] = -1.25, 0.5
    over["E_ref"] = E_ref
    o, _, w = oracle_with(name, **over)
    assert w0["Theta1"].shape[0] != F
    s = env(seed=24, n=6)
    sp = np.where(np.arange(s.n) % 2 == 0, 28, 7).astype(np.int32)
    st = o.stages(s.pos, sp, s.cell, s.pbc)
    h = sum(np.array([silu(x) for x in over[f"b{t}"]]) for t in range(1, spec.n_layers + 1))
    base = float(h @ over["w_head"]) + 0.3
    want = base + E_ref[sp]
    assert np.allclose(st["E"], want, rtol=1e-14, atol=1e-13)


def test_calibration_is_elementwise_affine():
    """Eq. (calibration): D = (D~ - mu) / sigma entry by entry."""
    _, spec, w0 = oracle_with("small")
    rng = np.random.Generator(np.random.PCG64(10))
    mu = rng.normal(size=w0["mu"].shape)
    sigma = rng.uniform(0.5, 2.0, size=w0["sigma"].shape)
    o, _, _ = oracle_with("small", mu=mu, sigma=sigma)
    s = env(seed=25, n=6)
    st = o.stages(s.pos, s.species, s.cell, s.pbc)
    assert np.allclose(st["D"] * sigma + mu, st["Dt"], rtol=1e-14, atol=1e-14)
