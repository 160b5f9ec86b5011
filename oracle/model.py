"""DPA4C oracle: the potential as the paper's Methods define it, in float64.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module; the GPU path
never does, and this module imports nothing from the GPU path.

Plain, slow and direct: every quantity is computed from its defining
equation with dense torch CPU ops in float64, in the order of Methods
"One message-passing layer" and "Nonlinear readout and atomic energy".
Forces are the negative gradient of the energy (Eq. (forces)), obtained with
torch autograd through those same operations.

Numbered readings of the paper used here (the paper leaves these open):
  R1  Gaunt sign: C = -I/||I||_F for every triple (Eq. (gaunt) leaves the
      sign to a convention; this one reproduces both closed forms of
      Eq. (closed-forms)).
  R2  vech order: upper triangle, row-major over c <= c'.  Bispectrum order:
      triples in lexicographic order, entries row-major over (k1, k2, k3)
      restricted to non-decreasing indices on equal-degree axes, each scaled
      by sqrt(number of distinct permutations).  Quartic order: eta-major.
  R3  SwiGLU split: gate = first H columns, value = last H columns.  Pair
      output split [s, t, w] in that order, w reshaped channel-major (C0, R).
  R4  Harmonics use the exact s = |u|^2 (the compressed kernel may use 1).
  R5  The padding type is the last row of the type table (index 118).
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import torch

from . import neighbors as _nbr

F64 = torch.float64
EPS = 1.0e-7        # Eq. (edge-geometry)
PAIR_SCALE = 0.1    # Eq. (pairfilm) fixed output scale


# ---------------------------------------------------------------------------
# structural widths
# ---------------------------------------------------------------------------
def degree_channels(C0: int, L: int) -> list[int]:
    """Eq. (degree-channels): [C_0, C_1, ..., C_L]."""
    C1 = max(4, 2 ** math.ceil(0.5 * math.log2(C0)))
    C2 = max(4, C1 // 2)
    return ([C0, C1, C2] + [1] * L)[: L + 1]


def probe_ranks(C0: int, L: int) -> list[int]:
    """Eq. (probe-ranks): [None, K_1, ..., K_L]."""
    C = degree_channels(C0, L)
    return ([None, C[2], 2] + [1] * L)[: L + 1]


def feature_width(C0: int, L: int) -> int:
    """Eq. (moment-width): S = sum_l (2l+1) C_l."""
    return sum((2 * l + 1) * c for l, c in enumerate(degree_channels(C0, L)))


def admissible_triples(L: int) -> list[tuple[int, int, int]]:
    """Eq. (triples) in lexicographic order."""
    out = []
    for l1, l2, l3 in itertools.product(range(1, L + 1), repeat=3):
        if l1 <= l2 <= l3 and l3 <= l1 + l2 and (l1 + l2 + l3) % 2 == 0:
            out.append((l1, l2, l3))
    return sorted(out)


def bispectrum_entries(triple, ranks) -> list[tuple[tuple[int, int, int], float]]:
    """Retained (k1, k2, k3) of one triple with their sqrt(family size) weights.

    Eq. (bispectrum) and the text after it: on axes of equal degree only the
    non-decreasing representative is kept, rescaled by the square root of the
    number of distinct index permutations it stands for (reading R2).
    """
    ks = [ranks[l] for l in triple]
    out = []
    for idx in itertools.product(*(range(k) for k in ks)):
        ok = True
        weight = 1
        for deg in set(triple):
            axes = [a for a in range(3) if triple[a] == deg]
            sub = [idx[a] for a in axes]
            if any(sub[t] > sub[t + 1] for t in range(len(sub) - 1)):
                ok = False
                break
            counts = {}
            for v in sub:
                counts[v] = counts.get(v, 0) + 1
            fam = math.factorial(len(sub))
            for c in counts.values():
                fam //= math.factorial(c)
            weight *= fam
        if ok:
            out.append((idx, math.sqrt(weight)))
    return out


def descriptor_width(C0: int, L: int) -> int:
    """Eq. (dim-out)."""
    C = degree_channels(C0, L)
    K = probe_ranks(C0, L)
    d_bis = sum(len(bispectrum_entries(t, K)) for t in admissible_triples(L))
    return 2 * C0 + 2 + sum(C[l] * (C[l] + 1) // 2 for l in range(1, L + 1)) + d_bis + K[1] * K[2]


# ---------------------------------------------------------------------------
# edge functions
# ---------------------------------------------------------------------------
def edge_geometry(r: torch.Tensor):
    """Eq. (edge-geometry): rho = sqrt(|r|^2 + eps^2), u = r / rho."""
    rho = torch.sqrt((r * r).sum(-1) + EPS * EPS)
    return rho, r / rho[:, None]


def envelope(rho: torch.Tensor, r_c: float) -> torch.Tensor:
    """Eq. (envelope): t^4 (1 + 4x + 10x^2 + 20x^3 + 35x^4)."""
    t = torch.clamp(1.0 - rho / r_c, 0.0, 1.0)
    x = 1.0 - t
    return t ** 4 * (1.0 + 4.0 * x + 10.0 * x ** 2 + 20.0 * x ** 3 + 35.0 * x ** 4)


def bessel_basis(rho: torch.Tensor, omega: torch.Tensor) -> torch.Tensor:
    """Eq. (bessel-basis): f_n = sin(omega_n rho) / rho."""
    return torch.sin(rho[:, None] * omega[None, :]) / rho[:, None]


def silu(z: torch.Tensor) -> torch.Tensor:
    """SiLU(z) = z / (1 + exp(-z)), written as z * sigmoid(z) so that its
    autograd derivative stays finite for large |z|."""
    return z * torch.sigmoid(z)


def swiglu(x: torch.Tensor, W: torch.Tensor) -> torch.Tensor:
    """Eq. (swiglu): SiLU(x_g) * x_v with [x_g, x_v] = x W (reading R3)."""
    y = x @ W
    h = W.shape[1] // 2
    return silu(y[:, :h]) * y[:, h:]


def harmonics(u: torch.Tensor, l: int) -> torch.Tensor:
    """Real Cartesian harmonics B_l(u), Eq. (harmonics) and Supplementary
    Note "Real solid harmonics of degrees three and four" (reading R4)."""
    x, y, z = u[:, 0], u[:, 1], u[:, 2]
    s = x * x + y * y + z * z
    if l == 0:
        return torch.ones_like(x)[:, None]
    if l == 1:
        return torch.stack([x, y, z], -1)
    if l == 2:
        r3 = math.sqrt(3.0)
        return torch.stack([r3 * x * y, r3 * y * z, 0.5 * (3 * z * z - s), r3 * x * z,
                            0.5 * r3 * (x * x - y * y)], -1)
    if l == 3:
        return torch.stack([
            math.sqrt(5 / 8) * y * (3 * x * x - y * y),
            math.sqrt(15) * x * y * z,
            math.sqrt(3 / 8) * y * (5 * z * z - s),
            0.5 * z * (5 * z * z - 3 * s),
            math.sqrt(3 / 8) * x * (5 * z * z - s),
            0.5 * math.sqrt(15) * z * (x * x - y * y),
            math.sqrt(5 / 8) * x * (x * x - 3 * y * y)], -1)
    if l == 4:
        return torch.stack([
            0.5 * math.sqrt(35) * x * y * (x * x - y * y),
            0.25 * math.sqrt(70) * y * z * (3 * x * x - y * y),
            0.5 * math.sqrt(5) * x * y * (7 * z * z - s),
            0.25 * math.sqrt(10) * y * z * (7 * z * z - 3 * s),
            0.125 * (35 * z ** 4 - 30 * z * z * s + 3 * s * s),
            0.25 * math.sqrt(10) * x * z * (7 * z * z - 3 * s),
            0.25 * math.sqrt(5) * (x * x - y * y) * (7 * z * z - s),
            0.25 * math.sqrt(70) * x * z * (x * x - 3 * y * y),
            0.125 * math.sqrt(35) * (x ** 4 - 6 * x * x * y * y + y ** 4)], -1)
    raise ValueError(l)


def stf_basis() -> torch.Tensor:
    """Matrices E_m with STF(z) = sum_m z_m E_m, Eq. (stf), in B_2 order
    (xy, yz, z^2, xz, x^2 - y^2).  Orthonormal in the Frobenius product."""
    E = torch.zeros(5, 3, 3, dtype=F64)
    s2 = 1.0 / math.sqrt(2.0)
    E[0, 0, 1] = E[0, 1, 0] = s2
    E[1, 1, 2] = E[1, 2, 1] = s2
    E[2] = torch.diag(torch.tensor([-1.0, -1.0, 2.0], dtype=F64)) / math.sqrt(6.0)
    E[3, 0, 2] = E[3, 2, 0] = s2
    E[4] = torch.diag(torch.tensor([1.0, -1.0, 0.0], dtype=F64)) * s2
    return E


def stf(z: torch.Tensor) -> torch.Tensor:
    """Packed degree-two vectors [..., 5] -> symmetric trace-free [..., 3, 3]."""
    return torch.einsum("...m,mab->...ab", z, stf_basis())


def gaunt_integral(l1: int, l2: int, l3: int) -> np.ndarray:
    """I_{m1 m2 m3} = integral over the unit sphere of B B B, Eq. (gaunt).

    The integrand is a polynomial of degree <= 12 on the sphere; a product
    rule (Gauss-Legendre in cos(theta), uniform in phi) with 10 x 26 nodes
    integrates it exactly.
    """
    zg, wg = np.polynomial.legendre.leggauss(10)
    nphi = 26
    phi = 2.0 * math.pi * np.arange(nphi) / nphi
    Z, P = np.meshgrid(zg, phi, indexing="ij")
    W = np.repeat(wg[:, None], nphi, axis=1) * (2.0 * math.pi / nphi)
    st = np.sqrt(1.0 - Z * Z)
    u = torch.tensor(np.stack([st * np.cos(P), st * np.sin(P), Z], -1).reshape(-1, 3), dtype=F64)
    w = torch.tensor(W.reshape(-1), dtype=F64)
    B1, B2, B3 = harmonics(u, l1), harmonics(u, l2), harmonics(u, l3)
    return torch.einsum("p,pa,pb,pc->abc", w, B1, B2, B3).numpy()


def coupling_tensor(l1: int, l2: int, l3: int) -> np.ndarray:
    """Eq. (gaunt): C = -I / ||I||_F (reading R1)."""
    I = gaunt_integral(l1, l2, l3)
    return -I / np.linalg.norm(I)


# ---------------------------------------------------------------------------
# the model
# ---------------------------------------------------------------------------
class Oracle:
    """DPA4C in float64.  ``weights`` is a dict of float32 numpy arrays (the
    random-init parameters) and ``spec`` holds C0, L, R, n_rbf, F, n_layers,
    r_c.  float32 parameters are promoted exactly to float64."""

    def __init__(self, spec, weights: dict):
        self.spec = spec
        self.C0, self.L, self.R = spec.C0, spec.L, spec.R
        self.r_c = float(spec.r_c)
        self.C = degree_channels(self.C0, self.L)
        self.K = probe_ranks(self.C0, self.L)
        self.S = feature_width(self.C0, self.L)
        self.D_out = descriptor_width(self.C0, self.L)
        self.w = {k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in weights.items()}
        if self.w["mu"].shape[0] != self.D_out:
            raise ValueError("calibration width does not match Eq. (dim-out)")
        self.triples = admissible_triples(self.L)
        self.coupling = {t: torch.tensor(coupling_tensor(*t)) for t in self.triples}
        self.bis = {t: bispectrum_entries(t, self.K) for t in self.triples}
        self._pair_cache: dict[tuple[int, int], tuple] = {}

    # -- Eq. (pairfilm): one evaluation per ordered type pair ---------------
    def pair_coefficients(self, a: int, b: int):
        key = (int(a), int(b))
        if key not in self._pair_cache:
            X0 = self.w["type_embed"]
            z = torch.cat([X0[a], X0[b]])[None, :]
            p = PAIR_SCALE * (swiglu(z, self.w["Wp_in"]) @ self.w["Wp_out"])[0]
            C0, R = self.C0, self.R
            s, t, w = p[:C0], p[C0:2 * C0], p[2 * C0:]
            gamma = 1.0 + torch.tanh(s)
            beta = X0[a] + X0[b] + torch.tanh(t)
            U = torch.tanh(w).reshape(C0, R)
            self._pair_cache[key] = (gamma, beta, U)
        return self._pair_cache[key]

    def pair_tables(self, species_i: np.ndarray, species_j: np.ndarray):
        """gamma, beta, U gathered per edge from the per-pair evaluations."""
        if len(species_i) == 0:
            z = torch.zeros(0, self.C0, dtype=F64)
            return z, z, torch.zeros(0, self.C0, self.R, dtype=F64)
        pairs = np.stack([species_i, species_j], 1)
        uniq, inv = np.unique(pairs, axis=0, return_inverse=True)
        inv = torch.as_tensor(inv.reshape(-1), dtype=torch.long)
        g, bt, U = zip(*(self.pair_coefficients(a, b) for a, b in uniq))
        return torch.stack(g)[inv], torch.stack(bt)[inv], torch.stack(U)[inv]

    # -- one message-passing layer -----------------------------------------
    def aggregate(self, r: torch.Tensor, centre: torch.Tensor, n_centres: int,
                  species_i: np.ndarray, species_j: np.ndarray) -> dict:
        """Eqs. (edge-geometry) .. (moments) for the given edges.

        r        [E, 3] edge displacements r_ij = r_j - r_i
        centre   [E] local index of the centre i of every edge
        Returns S0 = sum chi^2, S1 = sum chi^4, M0, M1 and X_l [n, 2l+1, C_l].
        """
        w = self.w
        rho, u = edge_geometry(r)
        chi = envelope(rho, self.r_c)
        f = bessel_basis(rho, w["omega"])
        h = swiglu(f, w["W_in"])                                    # Eq. (radial-map)
        g = h @ w["W_out"]
        gamma, beta, U = self.pair_tables(species_i, species_j)
        psi = gamma * g + beta                                      # Eq. (amplitude)
        if self.R > 0:
            q = h @ w["W_mode"]                                     # Eq. (radial-modes)
            psi = psi + torch.einsum("ecm,em->ec", U, q)
        chi_l = [chi] + [chi * chi] * self.L                        # Eq. (degree-weight)
        zeros = lambda *s: torch.zeros(*s, dtype=F64)
        S0 = zeros(n_centres).index_add(0, centre, chi_l[0] ** 2)   # payload entries 0, 1
        S1 = zeros(n_centres).index_add(0, centre, chi_l[1] ** 2)
        M0 = torch.sqrt(0.25 + S0)                                  # Eq. (masses)
        M1 = torch.sqrt(0.25 + S1)
        X = []
        for l in range(self.L + 1):
            B = harmonics(u, l)                                     # [E, 2l+1]
            Cl = self.C[l]
            msg = chi_l[l][:, None, None] * B[:, :, None] * psi[:, None, :Cl]
            Y = zeros(n_centres, 2 * l + 1, Cl).index_add(0, centre, msg)
            X.append(Y / (M0 if l == 0 else M1)[:, None, None])    # Eq. (moments)
        return {"S0": S0, "S1": S1, "M0": M0, "M1": M1, "X": X, "rho": rho, "chi": chi}

    # -- nonlinear readout --------------------------------------------------
    def descriptor(self, agg: dict, species_c: np.ndarray):
        """Eqs. (alignment) .. (calibration).  Returns (D_tilde, D)."""
        w = self.w
        X = agg["X"]
        n = X[0].shape[0]
        Xt = [X[0]]
        for l in range(1, self.L + 1):                              # Eq. (alignment)
            if l <= 2:
                M = torch.eye(self.C[l], dtype=F64) + w[f"W_align{l}"]
                Xt.append(X[l] @ M)
            else:
                Xt.append(X[l])
        blocks = [w["type_embed"][torch.as_tensor(species_c, dtype=torch.long)],
                  X[0][:, 0, :], agg["M0"][:, None], agg["M1"][:, None]]
        for l in range(1, self.L + 1):                              # Eq. (gram)
            G = torch.einsum("nmc,nmd->ncd", Xt[l], Xt[l])
            C = self.C[l]
            iu, ju = np.triu_indices(C)
            scale = torch.tensor(np.where(iu == ju, 1.0, math.sqrt(2.0)), dtype=F64)
            blocks.append(G[:, iu, ju] * scale)
        Z = [None]
        for l in range(1, self.L + 1):                              # Eq. (probes)
            if self.K[l] == self.C[l]:
                Z.append(Xt[l])
            else:
                Z.append(Xt[l] @ w[f"A{l}"])
        for t in self.triples:                                      # Eq. (bispectrum)
            Cc = self.coupling[t]
            J = torch.einsum("abc,nai,nbj,nck->nijk", Cc, Z[t[0]], Z[t[1]], Z[t[2]])
            idx = self.bis[t]
            sel = torch.stack([J[:, a, b, c] for (a, b, c), _ in idx], 1)
            wts = torch.tensor([wt for _, wt in idx], dtype=F64)
            blocks.append(sel * wts)
        Q = stf(Z[2].transpose(1, 2))                               # [n, K2, 3, 3]
        Qv = torch.einsum("nhab,nbk->nhka", Q, Z[1])                # [n, K2, K1, 3]
        blocks.append((Qv * Qv).sum(-1).reshape(n, -1))            # Eq. (quartic)
        Dt = torch.cat(blocks, 1)                                   # Eq. (descriptor)
        if Dt.shape[1] != self.D_out:
            raise AssertionError("descriptor width mismatch")
        D = (Dt - w["mu"]) / w["sigma"]                             # Eq. (calibration)
        return Dt, D

    def mlp_energy(self, D: torch.Tensor, species_c: np.ndarray) -> torch.Tensor:
        """Eqs. (atomic-energy), (fitting) with phi = SiLU."""
        w = self.w
        h = D
        for tau in range(1, self.spec.n_layers + 1):
            out = silu(h @ w[f"Theta{tau}"] + w[f"b{tau}"])
            h = out + h if out.shape[1] == h.shape[1] else out
        E = h @ w["w_head"] + w["b_head"][0]
        return E + w["E_ref"][torch.as_tensor(species_c, dtype=torch.long)]

    # -- energies and forces -------------------------------------------------
    def atomic_energies(self, pos_t, species, cell, edges, centres):
        """E_i for ``centres`` (int64 array, sorted) given all edges of those
        centres.  ``pos_t`` is a float64 tensor (may require grad)."""
        ei, ej, en = edges
        cell_t = torch.as_tensor(cell, dtype=F64)
        local = np.searchsorted(centres, ei)
        r = pos_t[torch.as_tensor(ej)] + torch.as_tensor(en, dtype=F64) @ cell_t \
            - pos_t[torch.as_tensor(ei)]
        if r.requires_grad:
            r.retain_grad()                    # dE/dr_ij, for the virial
        agg = self.aggregate(r, torch.as_tensor(local, dtype=torch.long), len(centres),
                             species[ei], species[ej])
        Dt, D = self.descriptor(agg, species[centres])
        return self.mlp_energy(D, species[centres]), {"agg": agg, "Dt": Dt, "D": D, "r": r}

    def energy_forces(self, pos, species, cell, pbc, centres=None, chunk: int = 256,
                      edges=None, virial: bool = False):
        """Per-atom energies of ``centres`` (all atoms if None) and the forces
        F = -dE/dr of their sum, E = sum over those centres of E_i.

        With ``centres`` = all atoms this is the full energy and force of
        Eq. (forces).  The sum is split over chunks of centres, each chunk
        differentiated separately; E_i of different centres are independent
        (Eq. (energy-decomposition)), so the split is exact.

        With ``virial`` also returns the virial of Eq. (forces),
        Xi = -sum_i sum_{j in N_i} dE/dr_ij (x) r_ij (eV, [a][b] = -sum g_a r_b),
        and the per-centre terms W_i = -sum_{j in N_i} dE/dr_ij (x) r_ij, whose
        sum over all centres is Xi.
        """
        pos = np.asarray(pos, dtype=np.float64)
        n = pos.shape[0]
        if centres is None:
            centres = np.arange(n, dtype=np.int64)
        centres = np.asarray(centres, dtype=np.int64)
        if edges is None:
            edges = _nbr.neighbor_list(pos, cell, pbc, self.r_c, centres=centres)
        ei, ej, en = edges
        pos_t = torch.tensor(pos, dtype=F64, requires_grad=True)
        e_out = np.empty(len(centres))
        starts = np.searchsorted(ei, centres)
        ends = np.searchsorted(ei, centres, side="right")
        w_atom = np.zeros((len(centres), 3, 3))
        for c0 in range(0, len(centres), chunk):
            cs = centres[c0:c0 + chunk]
            a, b = starts[c0], ends[min(c0 + chunk, len(centres)) - 1]
            E, aux = self.atomic_energies(pos_t, species, cell, (ei[a:b], ej[a:b], en[a:b]), cs)
            E.sum().backward()
            e_out[c0:c0 + chunk] = E.detach().numpy()
            if virial and b > a:
                g = aux["r"].grad.numpy()                       # dE/dr_ij
                r = aux["r"].detach().numpy()
                local = np.searchsorted(cs, ei[a:b])
                np.add.at(w_atom[c0:c0 + chunk], local, -g[:, :, None] * r[:, None, :])
        forces = -pos_t.grad.numpy()
        if virial:
            return e_out, forces, w_atom.sum(axis=0), w_atom
        return e_out, forces

    def stages(self, pos, species, cell, pbc, centres=None, edges=None):
        """Intermediate quantities for stage-by-stage comparison: node state
        [S0, S1, X flat], D_tilde, D and E_i (no gradients)."""
        pos = np.asarray(pos, dtype=np.float64)
        if centres is None:
            centres = np.arange(pos.shape[0], dtype=np.int64)
        if edges is None:
            edges = _nbr.neighbor_list(pos, cell, pbc, self.r_c, centres=centres)
        with torch.no_grad():
            E, aux = self.atomic_energies(torch.tensor(pos, dtype=F64), species, cell, edges,
                                          np.asarray(centres, np.int64))
        agg = aux["agg"]
        flat = torch.cat([x.reshape(x.shape[0], -1) for x in agg["X"]], 1)
        return {"S0": agg["S0"].numpy(), "S1": agg["S1"].numpy(),
                "M0": agg["M0"].numpy(), "M1": agg["M1"].numpy(),
                "X_flat": flat.numpy(), "Dt": aux["Dt"].numpy(), "D": aux["D"].numpy(),
                "E": E.numpy()}
