"""Fix the calibration vectors and the head scale of the random-init models.

Writes ``synth/calibration.json``; run as ``python -m oracle.calibrate
[model ...]`` (default: every model of ``synth.MODELS``; named models are
recomputed and merged into the existing file).

Eq. (calibration) holds fixed statistics estimated from sample frames.  With
no training frames available, the sample is frame 0 of the synthetic
workloads that use each model:

* entries of the initial feature X0 of the centre: mu = 0, sigma = 1
  (passed through unchanged);
* the two normalising scales M0, M1: mu = mean, sigma = centred standard
  deviation, floored at 0.1 |mean| (near-perfect crystals have almost no
  spread);
* every other entry: mu = 0, sigma = root mean square, floored at 1e-6.

The sample frames are the workload crystals rattled by 0.25 A (and the
water-like liquid as generated): on the near-perfect production crystals the
degree-1 and degree-2 features nearly vanish by cubic symmetry, and statistics
taken there would blow the symmetry-breaking invariants up by orders of
magnitude.

The head weight vector is then rescaled so that the RMS force on sampled
atoms is 0.3 eV/A (a gentle random potential that keeps NVE stable).
"""
from __future__ import annotations

import json
import os

import numpy as np

import synth
from oracle.model import Oracle
from oracle import neighbors as nbr

TARGET_RMS_FORCE = 0.3
OUT = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "synth", "calibration.json")


RATTLE = 0.25   # A; jitter of the calibration crystals


def _frames(model_name: str):
    """Calibration sample: the workload structures with the crystals rattled
    by N(0, 0.25 A) instead of their small production jitter, so that the
    symmetry-breaking invariants (which vanish on a perfect cubic lattice)
    are sampled at a realistic spread and not amplified by a tiny sigma."""
    if model_name == "small":
        return [synth.fcc_copper(3, RATTLE, seed=101)]
    if model_name == "full_carbon":
        return [synth.diamond_carbon(4, RATTLE, seed=104)]
    return [synth.fcc_copper(10, RATTLE, seed=102), synth.bcc_hea(25, RATTLE, seed=103),
            synth.make_workload("water24000_full")[0]]


def calibrate(model_name: str, n_centres: int = 200, n_force: int = 12, seed: int = 7):
    spec = synth.MODELS[model_name]
    w = synth.random_weights(spec)
    oracle = Oracle(spec, w)
    C0 = spec.C0
    rng = np.random.Generator(np.random.PCG64(seed))
    frames = _frames(model_name)
    samples = []
    dts = []
    for s in frames:
        cs = np.sort(rng.choice(s.n, size=min(n_centres, s.n), replace=False)).astype(np.int64)
        samples.append(cs)
        dts.append(oracle.stages(s.pos, s.species, s.cell, s.pbc, centres=cs)["Dt"])
    Dt = np.concatenate(dts, 0)
    mu = np.zeros(Dt.shape[1])
    sigma = np.sqrt((Dt * Dt).mean(0))
    sigma = np.maximum(sigma, 1e-6)
    mu[:C0] = 0.0
    sigma[:C0] = 1.0
    for k in (2 * C0, 2 * C0 + 1):
        mu[k] = Dt[:, k].mean()
        sigma[k] = max(Dt[:, k].std(), 0.1 * abs(mu[k]))
    w["mu"] = mu.astype(np.float32)
    w["sigma"] = sigma.astype(np.float32)
    oracle = Oracle(spec, w)
    fsq = []
    for s in frames:
        ks = np.sort(rng.choice(s.n, size=min(n_force, s.n), replace=False)).astype(np.int64)
        ei, ej, _ = nbr.neighbor_list(s.pos, s.cell, s.pbc, spec.r_c, centres=ks)
        centres = np.unique(np.concatenate([ks, ej]))
        _, F = oracle.energy_forces(s.pos, s.species, s.cell, s.pbc, centres=centres)
        fsq.append((F[ks] ** 2).sum(1))
    rms = float(np.sqrt(np.concatenate(fsq).mean() / 3.0))
    return {"mu": w["mu"].tolist(), "sigma": w["sigma"].tolist(),
            "head_scale": TARGET_RMS_FORCE / rms, "rms_force_unscaled": rms,
            "frames": [s.name for s in frames]}


def main(names=None):
    import sys
    names = names or sys.argv[1:] or list(synth.MODELS)
    out = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            out = json.load(f)
    for name in names:
        out[name] = calibrate(name)
        v = out[name]
        print(name, "head_scale", v["head_scale"], "rms_force_unscaled", v["rms_force_unscaled"],
              flush=True)
    with open(OUT, "w") as f:
        json.dump({k: out[k] for k in synth.MODELS if k in out}, f)


if __name__ == "__main__":
    main()
