"""Pins of the oracle's Nose-Hoover-chain integrator (no GPU):
second-order conservation of the extended energy, thermalisation of a free
gas, and reduction to velocity Verlet when the chain is decoupled."""
import numpy as np
import pytest

import synth
from oracle import md
from oracle import model as om


class FreeParticles:
    """No potential: the chain alone changes the kinetic energy."""

    def energy_forces(self, pos, species, cell, pbc):
        return np.zeros(len(pos)), np.zeros_like(pos)


def free_gas(n=64, seed=4, sigma=0.02):
    g = np.random.Generator(np.random.PCG64(seed))
    return np.zeros((n, 3)), g.normal(size=(n, 3)) * sigma, np.full(n, 12.0)


def extended_energy_error(dt, t_total=400.0, t_damp=20.0):
    pos, vel, m = free_gas()
    steps = int(round(t_total / dt))
    ep, ek, eth, *_ = md.nvt(FreeParticles(), pos, vel, np.zeros(len(m), np.int32), None, None,
                             m, dt, steps, 300.0, t_damp)
    h = ep + ek + eth
    return np.abs(h - h[0]).max(), ek


def test_extended_energy_error_is_second_order_in_the_time_step():
    # The Trotter splitting is second order, so the deviation of
    # E_pot + K + E_thermostat shrinks four-fold per halving of dt; a wrong
    # chain force, mass or thermostat energy leaves an O(1) error instead.
    # The gas starts near 5,000 K and is cooled to 300 K, so the chain
    # exchanges far more energy than the error.
    e1, ek = extended_energy_error(1.0)
    e2, _ = extended_energy_error(0.5)
    e4, _ = extended_energy_error(0.25)
    assert ek[0] - ek[-1] > 30.0
    assert 3.6 < e1 / e2 < 4.4 and 3.6 < e2 / e4 < 4.4, (e1, e2, e4)
    assert e4 < 1e-3 * (ek[0] - ek[-1])


def test_free_gas_thermalises_to_the_target():
    pos, vel, m = free_gas(n=200, seed=7)
    steps = 3000
    ep, ek, eth, *_ = md.nvt(FreeParticles(), pos, vel, np.zeros(len(m), np.int32), None, None,
                             m, 1.0, steps, 300.0, 20.0)
    nf = 3 * len(m) - 3
    t_mean = 2.0 * ek[steps // 2:].mean() / (nf * md.KB_EV)
    assert abs(t_mean - 300.0) < 15.0, t_mean


def test_decoupled_chain_is_velocity_verlet():
    # With a damping time of 1e12 fs the chain masses are so large that its
    # velocities stay below 1e-20 /fs: every scale factor is exactly 1.0 and
    # the trajectory is the NVE one, bit for bit.
    spec, w = synth.model_weights("small")
    o = om.Oracle(spec, w)
    s = synth.random_periodic(16, seed=3, cell=np.diag([7.9, 8.2, 8.6]), d_min=1.7)
    g = np.random.Generator(np.random.PCG64(9))
    masses = np.full(s.n, 58.7)
    vel = g.normal(size=(s.n, 3)) * 0.005
    ep0, ek0, p0, v0 = md.nve(o, s.pos, vel, s.species, s.cell, s.pbc, masses, 1.0, 4)
    ep1, ek1, eth, p1, v1, chain = md.nvt(o, s.pos, vel, s.species, s.cell, s.pbc, masses, 1.0, 4,
                                          300.0, 1e12)
    assert np.array_equal(p0, p1) and np.array_equal(v0, v1)
    assert np.array_equal(ep0, ep1) and np.array_equal(ek0, ek1)
    assert np.abs(chain.v).max() < 1e-20


@pytest.mark.slow
def test_extended_energy_is_conserved_on_the_potential():
    # with the small model on a 16-atom cell, driven from 600 K towards
    # 300 K: the extended energy moves far less than the energy exchanged
    spec, w = synth.model_weights("small")
    o = om.Oracle(spec, w)
    s = synth.random_periodic(16, seed=3, cell=np.diag([7.9, 8.2, 8.6]), d_min=1.7)
    masses = np.full(s.n, 58.7)
    g = np.random.Generator(np.random.PCG64(9))
    vel = g.normal(size=(s.n, 3)) * np.sqrt(md.KB_EV * 600.0 / (masses[:, None] * md._MVV2E))
    ep, ek, eth, *_ = md.nvt(o, s.pos, vel, s.species, s.cell, s.pbc, masses, 0.5, 120, 300.0, 10.0)
    h = ep + ek + eth
    assert np.abs(h - h[0]).max() < 0.02 * np.abs(eth).max(), (np.abs(h - h[0]).max(), eth)
