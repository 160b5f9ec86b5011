"""Oracle for the DPA4C energy-and-force path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 CPU implementation of the potential exactly as the
paper's Methods define it (neighbour set, edge geometry, envelope, Bessel
basis, radial map, ordered-pair modulation, Cartesian harmonics, one
aggregation, Gram / bispectrum / quartic invariants, calibration, MLP), of
the virial of Eq. (forces), and of velocity-Verlet (NVE) and Nose-Hoover-chain
(NVT) dynamics over it.  Forces are the autograd gradient of the float64
energy.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call, link or execute anything in this directory.
The GPU library shares no code with it: no headers, kernels, helpers, tables
or constant generators.  Both sides read the same seeded inputs from the
``synth`` package, which contains no arithmetic of the method.

Parity status: every function is pinned by a test in ``tests/test_oracle_*``
against something other than itself (printed tables, closed forms,
invariances, finite differences, brute force).  The absolute values of E_i
for given random weights are "parity unpinned" beyond those properties: the
paper prints no worked example.
"""
