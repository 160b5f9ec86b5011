"""Velocity-Verlet NVE dynamics on the oracle potential (test infrastructure).

Units: Angstrom, fs, eV, atomic mass units.  The neighbour list is rebuilt
from scratch at every step, so no skin is involved.
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
