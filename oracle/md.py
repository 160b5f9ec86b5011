"""Velocity-Verlet NVE dynamics and Nose-Hoover-chain NVT dynamics on the
oracle potential (test infrastructure).

Units: Angstrom, fs, eV, atomic mass units, K.  The neighbour list is
rebuilt from scratch at every step, so no skin is involved.
"""
from __future__ import annotations

import numpy as np

# 1 u (A/fs)^2 in eV, from CODATA 2018 values of the atomic mass unit and the
# elementary charge
_MVV2E = 1.66053906660e-27 * 1.0e10 / 1.602176634e-19


def kinetic_energy(vel, masses) -> float:
    return float(0.5 * _MVV2E * (masses[:, None] * vel * vel).sum())


def nve(oracle, pos, vel, species, cell, pbc, masses, dt: float, steps: int):
    """Returns (E_pot [steps+1], E_kin [steps+1], final pos, final vel)."""
    pos = np.array(pos, dtype=np.float64)
    vel = np.array(vel, dtype=np.float64)
    inv_m = 1.0 / (masses * _MVV2E)                  # (eV/A)/u -> A/fs^2
    e_atom, F = oracle.energy_forces(pos, species, cell, pbc)
    ep, ek = [e_atom.sum()], [kinetic_energy(vel, masses)]
    for _ in range(steps):
        vel += 0.5 * dt * F * inv_m[:, None]
        pos += dt * vel
        e_atom, F = oracle.energy_forces(pos, species, cell, pbc)
        vel += 0.5 * dt * F * inv_m[:, None]
        ep.append(e_atom.sum())
        ek.append(kinetic_energy(vel, masses))
    return np.array(ep), np.array(ek), pos, vel


def drift_ev_per_atom_ps(e_total, dt_fs: float, n_atoms: int) -> float:
    """Least-squares slope of E_total/N against time, in eV/atom/ps."""
    t = np.arange(len(e_total)) * dt_fs * 1e-3
    return float(np.polyfit(t, np.asarray(e_total) / n_atoms, 1)[0])


# Boltzmann constant in eV/K (CODATA 2018, exact in the 2019 SI)
KB_EV = 8.617333262e-5


class NoseHooverChain:
    """Nose-Hoover chain of length M (Martyna, Klein and Tuckerman, J. Chem.
    Phys. 97, 2635 (1992)) for N_f degrees of freedom at temperature T, with
    masses Q_1 = N_f kT tau^2 and Q_k = kT tau^2 for k > 1 (tau = the damping
    time), propagated over half a time step by the Trotter factorisation of
    Martyna, Tuckerman, Tobias and Klein, Mol. Phys. 87, 1117 (1996), with a
    single pass and no Suzuki-Yoshida weights.

    The chain forces are G_1 = (2 K - N_f kT)/Q_1 and
    G_k = (Q_{k-1} v_{k-1}^2 - kT)/Q_k; a half step updates the thermostat
    velocities from the end of the chain inwards, scales the particle
    velocities by exp(-dt/2 v_1), advances the positions xi_k by dt/2 v_k and
    updates the thermostat velocities outwards again.  The conserved energy
    of the extended system is E_pot + K + energy().
    """

    def __init__(self, n_dof: int, temperature: float, t_damp: float, length: int = 3):
        self.kT = KB_EV * temperature
        self.nf = float(n_dof)
        tau2 = t_damp * t_damp
        self.Q = np.array([self.nf * self.kT * tau2] + [self.kT * tau2] * (length - 1))
        self.xi = np.zeros(length)
        self.v = np.zeros(length)

    def _force(self, k: int, kinetic: float) -> float:
        if k == 0:
            return (2.0 * kinetic - self.nf * self.kT) / self.Q[0]
        return (self.Q[k - 1] * self.v[k - 1] ** 2 - self.kT) / self.Q[k]

    def _update(self, k: int, kinetic: float, dt: float):
        # v_k over dt/4, damped by the next link over dt/8 on both sides
        M = len(self.Q)
        if k == M - 1:
            self.v[k] += 0.25 * dt * self._force(k, kinetic)
        else:
            f = np.exp(-0.125 * dt * self.v[k + 1])
            self.v[k] = (self.v[k] * f + 0.25 * dt * self._force(k, kinetic)) * f

    def half_step(self, kinetic: float, dt: float) -> float:
        """Propagates the chain by dt/2 for particle kinetic energy
        ``kinetic`` (eV); returns the factor to scale all velocities by."""
        M = len(self.Q)
        for k in range(M - 1, -1, -1):
            self._update(k, kinetic, dt)
        s = float(np.exp(-0.5 * dt * self.v[0]))
        kinetic *= s * s
        self.xi += 0.5 * dt * self.v
        for k in range(M):
            self._update(k, kinetic, dt)
        return s

    def energy(self) -> float:
        """Thermostat energy: sum Q_k v_k^2 / 2 + N_f kT xi_1 + kT sum_{k>1} xi_k."""
        return float(0.5 * (self.Q * self.v * self.v).sum() + self.nf * self.kT * self.xi[0]
                     + self.kT * self.xi[1:].sum())


def nvt(oracle, pos, vel, species, cell, pbc, masses, dt: float, steps: int,
        temperature: float, t_damp: float, length: int = 3):
    """Nose-Hoover-chain NVT velocity Verlet: per step a chain half step,
    v += dt/2 F/m, r += dt v, F = F(r), v += dt/2 F/m and a chain half step,
    with N_f = 3N - 3.  Returns (E_pot, E_kin, E_thermostat) [steps+1] after
    each step, the final pos and vel and the chain."""
    pos = np.array(pos, dtype=np.float64)
    vel = np.array(vel, dtype=np.float64)
    inv_m = 1.0 / (masses * _MVV2E)
    chain = NoseHooverChain(3 * len(pos) - 3, temperature, t_damp, length)
    e_atom, F = oracle.energy_forces(pos, species, cell, pbc)
    ep, ek, eth = [e_atom.sum()], [kinetic_energy(vel, masses)], [chain.energy()]
    for _ in range(steps):
        vel *= chain.half_step(kinetic_energy(vel, masses), dt)
        vel += 0.5 * dt * F * inv_m[:, None]
        pos += dt * vel
        e_atom, F = oracle.energy_forces(pos, species, cell, pbc)
        vel += 0.5 * dt * F * inv_m[:, None]
        vel *= chain.half_step(kinetic_energy(vel, masses), dt)
        ep.append(e_atom.sum())
        ek.append(kinetic_energy(vel, masses))
        eth.append(chain.energy())
    return np.array(ep), np.array(ek), np.array(eth), pos, vel, chain
