"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module holds no arithmetic of the potential itself.  It draws random
numbers and lays them out:

* atomic structures shaped like the paper's crystal scans (FCC copper, BCC
  alloy) and a disordered water-like liquid,
* Maxwell-Boltzmann velocities,
* random-init model parameters with the array shapes of the paper's
  parameter inventory (Methods, Eqs. init-features .. fitting; Table S3), and
  the binary weight blob that the C-ABI library reads.

Every generator takes an explicit seed and uses numpy's PCG64.
Units are LAMMPS "metal": Angstrom, eV, fs, atomic mass units.
"""
from __future__ import annotations

import dataclasses
import math
import struct

import numpy as np

# ---------------------------------------------------------------------------
# physical constants (CODATA 2018); unit conversions for metal units with fs
# ---------------------------------------------------------------------------
KB_EV = 8.617333262e-5                     # Boltzmann constant, eV/K
AMU_KG = 1.66053906660e-27
EV_J = 1.602176634e-19
# 1 u * (Angstrom/fs)^2 expressed in eV
MVV2E = AMU_KG * 1.0e10 / EV_J             # = 103.6427 eV
# acceleration conversion: (eV/Angstrom)/u -> Angstrom/fs^2
FTM2V = 1.0 / MVV2E

N_TYPES = 118                               # the paper's 118-element type map
PAD_TYPE = N_TYPES                          # index of the zero padding type

# standard atomic weights of Z = 1..118 (IUPAC abridged; mass numbers of the
# most stable isotope for elements without a standard weight)
ATOMIC_MASS = np.array([
    1.008, 4.0026, 6.94, 9.0122, 10.81, 12.011, 14.007, 15.999, 18.998, 20.180,
    22.990, 24.305, 26.982, 28.085, 30.974, 32.06, 35.45, 39.948, 39.098, 40.078,
    44.956, 47.867, 50.942, 51.996, 54.938, 55.845, 58.933, 58.693, 63.546, 65.38,
    69.723, 72.630, 74.922, 78.971, 79.904, 83.798, 85.468, 87.62, 88.906, 91.224,
    92.906, 95.95, 97.0, 101.07, 102.91, 106.42, 107.87, 112.41, 114.82, 118.71,
    121.76, 127.60, 126.90, 131.29, 132.91, 137.33, 138.91, 140.12, 140.91, 144.24,
    145.0, 150.36, 151.96, 157.25, 158.93, 162.50, 164.93, 167.26, 168.93, 173.05,
    174.97, 178.49, 180.95, 183.84, 186.21, 190.23, 192.22, 195.08, 196.97, 200.59,
    204.38, 207.2, 208.98, 209.0, 210.0, 222.0, 223.0, 226.0, 227.0, 232.04,
    231.04, 238.03, 237.0, 244.0, 243.0, 247.0, 247.0, 251.0, 252.0, 257.0,
    258.0, 259.0, 262.0, 267.0, 270.0, 269.0, 270.0, 270.0, 278.0, 281.0,
    281.0, 285.0, 286.0, 289.0, 289.0, 293.0, 293.0, 294.0])
assert ATOMIC_MASS.shape == (N_TYPES,)


# ---------------------------------------------------------------------------
# structures
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class System:
    """One periodic (or open) configuration."""
    name: str
    pos: np.ndarray          # float64 [N, 3], Angstrom
    species: np.ndarray      # int32 [N], type index 0..117 (element Z-1)
    cell: np.ndarray         # float64 [3, 3], rows are lattice vectors
    pbc: np.ndarray          # int32 [3]
    mass_by_type: np.ndarray  # float64 [119], u (padding type gets 1.0)
    meta: dict

    @property
    def n(self) -> int:
        return int(self.pos.shape[0])


def _mass_table(overrides: dict | None = None) -> np.ndarray:
    m = np.ones(N_TYPES + 1)
    m[:N_TYPES] = ATOMIC_MASS
    for t, v in (overrides or {}).items():
        m[t] = v
    return m


def lattice(kind: str, a: float, reps: tuple[int, int, int]) -> tuple[np.ndarray, np.ndarray]:
    """Perfect cubic lattice: positions [reps.prod()*basis, 3] and the cell."""
    basis = {
        "fcc": [(0, 0, 0), (0.5, 0.5, 0), (0.5, 0, 0.5), (0, 0.5, 0.5)],
        "bcc": [(0, 0, 0), (0.5, 0.5, 0.5)],
        "diamond": [(0, 0, 0), (0.5, 0.5, 0), (0.5, 0, 0.5), (0, 0.5, 0.5),
                    (0.25, 0.25, 0.25), (0.75, 0.75, 0.25), (0.75, 0.25, 0.75),
                    (0.25, 0.75, 0.75)],
        "sc": [(0, 0, 0)],
    }[kind]
    basis = np.asarray(basis, dtype=np.float64)
    nx, ny, nz = reps
    cells = np.stack(np.meshgrid(np.arange(nx), np.arange(ny), np.arange(nz),
                                 indexing="ij"), axis=-1).reshape(-1, 3)
    frac = (cells[:, None, :] + basis[None, :, :]).reshape(-1, 3)
    pos = frac * a
    cell = np.diag([nx * a, ny * a, nz * a]).astype(np.float64)
    return pos, cell


def _reps3(reps) -> tuple[int, int, int]:
    if np.ndim(reps) == 0:
        return (int(reps),) * 3
    nx, ny, nz = (int(r) for r in reps)
    return nx, ny, nz


def near_cubic_reps(atoms: int, per_cell: int) -> tuple[int, int, int]:
    """Replication counts whose edges differ by at most one and whose product
    of cells is nearest to atoms / per_cell (ties go to the smaller one): the
    supercell rule of the paper's single-GPU capacity scans (Supplementary
    Note on the computational-reference benchmark), which reproduces the
    realised sizes of its scan tables, e.g. 2,370,192 = 8 * 66 * 67 * 67
    for 2,359,296 requested diamond atoms."""
    want = max(atoms / per_cell, 1.0)
    k = max(int(round(want ** (1.0 / 3.0))), 1)
    best = None
    for base in (k - 1, k, k + 1):
        if base < 1:
            continue
        for up in range(4):   # how many edges are base + 1
            r = (base,) * (3 - up) + (base + 1,) * up
            p = r[0] * r[1] * r[2]
            key = (abs(p - want), p)
            if best is None or key < best[0]:
                best = (key, r)
    return best[1]


def fcc_copper(reps, jitter: float, seed: int = 0, a: float = 3.615,
               name: str | None = None) -> System:
    """FCC copper supercell (4-atom conventional cell); ``reps`` is an edge
    count or a triple of them."""
    pos, cell = lattice("fcc", a, _reps3(reps))
    rng = np.random.Generator(np.random.PCG64(seed))
    pos = pos + rng.normal(0.0, jitter, size=pos.shape)
    species = np.full(pos.shape[0], 28, dtype=np.int32)       # Cu, Z = 29
    return System(name or f"fcc_cu_{reps}", pos, species, cell,
                  np.ones(3, np.int32), _mass_table({28: 63.5}),
                  {"lattice": "fcc", "a": a, "reps": reps, "jitter": jitter,
                   "seed": seed})


def diamond_carbon(reps, jitter: float, seed: int = 0, a: float = 3.567) -> System:
    """Diamond-carbon supercell (8-atom conventional cell, lattice constant
    3.567 A) with Gaussian coordinate perturbations: the structure of the
    paper's whole-step MD benchmark.  ``reps`` is an edge count or a triple."""
    pos, cell = lattice("diamond", a, _reps3(reps))
    rng = np.random.Generator(np.random.PCG64(seed))
    pos = pos + rng.normal(0.0, jitter, size=pos.shape)
    species = np.full(pos.shape[0], 5, dtype=np.int32)        # C, Z = 6
    return System(f"diamond_c_{reps}", pos, species, cell, np.ones(3, np.int32),
                  _mass_table(), {"lattice": "diamond", "a": a, "reps": reps,
                                  "jitter": jitter, "seed": seed})


def bcc_hea(reps: int = 25, jitter: float = 0.06, seed: int = 0,
            species_seed: int = 1, a: float = 2.87) -> System:
    """BCC high-entropy alloy: every site takes one of 5 types uniformly."""
    pos, cell = lattice("bcc", a, (reps, reps, reps))
    rng = np.random.Generator(np.random.PCG64(seed))
    pos = pos + rng.normal(0.0, jitter, size=pos.shape)
    srng = np.random.Generator(np.random.PCG64(species_seed))
    types = np.sort(srng.choice(N_TYPES, size=5, replace=False)).astype(np.int32)
    species = types[srng.integers(0, 5, size=pos.shape[0])].astype(np.int32)
    return System(f"bcc_hea_{reps}", pos, species, cell, np.ones(3, np.int32),
                  _mass_table(), {"lattice": "bcc", "a": a, "reps": reps,
                                  "jitter": jitter, "types": types.tolist(),
                                  "seed": seed, "species_seed": species_seed})


def water_box(n_mol: int = 8000, density_g_cm3: float = 1.0, seed: int = 2,
              d_min: float = 2.6, r_oh: float = 0.96, angle_deg: float = 104.5) -> System:
    """Disordered water-like liquid.

    Molecule centres (the O atoms) come from random sequential addition with
    minimum periodic O-O distance ``d_min``, accelerated with a cubic grid;
    each molecule gets a uniform random rotation (normalised 4-Gaussian
    quaternion).  Masses are 16 (O) and 1 (H).
    """
    mol_mass = 16.0 + 2.0 * 1.0
    volume = n_mol * mol_mass / 6.02214076e23 / density_g_cm3 * 1.0e24  # A^3
    box = volume ** (1.0 / 3.0)
    rng = np.random.Generator(np.random.PCG64(seed))
    # grid of cubes with side <= d_min/sqrt(3): each holds at most one centre
    ng = int(math.ceil(box / (d_min / math.sqrt(3.0))))
    gsz = box / ng
    reach = int(math.ceil(d_min / gsz))
    occ = np.full((ng, ng, ng), -1, dtype=np.int64)
    offs = np.stack(np.meshgrid(*(np.arange(-reach, reach + 1),) * 3,
                                indexing="ij"), -1).reshape(-1, 3)
    centres = np.empty((n_mol, 3))
    placed = 0
    attempts = 0
    d2 = d_min * d_min
    batch = 64
    while placed < n_mol:
        if attempts > 400 * n_mol:
            raise RuntimeError("random sequential addition did not converge")
        cand = rng.uniform(0.0, box, size=(batch, 3))
        attempts += batch
        g = np.minimum((cand / gsz).astype(np.int64), ng - 1)
        nb = (g[:, None, :] + offs[None, :, :]) % ng               # [M, K, 3]
        idx = occ[nb[..., 0], nb[..., 1], nb[..., 2]]              # [M, K]
        d = centres[np.maximum(idx, 0)] - cand[:, None, :]
        d -= box * np.round(d / box)
        clash = ((d * d).sum(-1) < d2) & (idx >= 0)
        survivors = np.nonzero(~clash.any(1))[0]
        # survivors are re-checked one at a time, in proposal order, against
        # the grid as it fills: identical to one-at-a-time sequential addition
        n_acc = 0
        for c in survivors:
            if placed == n_mol:
                break
            nbc = nb[c]
            ids = occ[nbc[:, 0], nbc[:, 1], nbc[:, 2]]
            ids = ids[ids >= 0]
            e = centres[ids] - cand[c]
            e -= box * np.round(e / box)
            if ids.size and ((e * e).sum(-1) < d2).any():
                continue
            centres[placed] = cand[c]
            gi = g[c]
            occ[gi[0], gi[1], gi[2]] = placed
            placed += 1
            n_acc += 1
        rate = max(n_acc, 1) / batch
        batch = int(min(8192, max(64, 32 / rate)))
    half = math.radians(angle_deg) / 2.0
    h1 = np.array([math.sin(half), 0.0, math.cos(half)]) * r_oh
    h2 = np.array([-math.sin(half), 0.0, math.cos(half)]) * r_oh
    q = rng.normal(size=(n_mol, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    w, x, y, z = q.T
    rot = np.stack([
        np.stack([1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)], -1),
        np.stack([2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)], -1),
        np.stack([2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)], -1),
    ], axis=1)                                                  # [n, 3, 3]
    pos = np.empty((3 * n_mol, 3))
    pos[0::3] = centres
    pos[1::3] = centres + rot @ h1
    pos[2::3] = centres + rot @ h2
    species = np.empty(3 * n_mol, dtype=np.int32)
    species[0::3] = 7          # O, Z = 8
    species[1::3] = 0          # H, Z = 1
    species[2::3] = 0
    cell = np.diag([box, box, box])
    return System(f"water_{n_mol}", pos, species, cell, np.ones(3, np.int32),
                  _mass_table({7: 16.0, 0: 1.0}),
                  {"n_mol": n_mol, "box": box, "seed": seed, "d_min": d_min,
                   "rsa_attempts": attempts})


def random_cluster(n: int, seed: int, n_species: int = 2, box: float = 8.0,
                   d_min: float = 1.2, types: tuple[int, ...] = (28, 13)) -> System:
    """Small open cluster (no periodicity) for inversion / symmetry checks."""
    rng = np.random.Generator(np.random.PCG64(seed))
    pts: list[np.ndarray] = []
    while len(pts) < n:
        p = rng.uniform(0.0, box, size=3)
        if all(np.linalg.norm(p - q) >= d_min for q in pts):
            pts.append(p)
    pos = np.asarray(pts)
    species = np.asarray(types, dtype=np.int32)[rng.integers(0, n_species, size=n)]
    return System(f"cluster_{n}", pos, species, np.diag([box, box, box]),
                  np.zeros(3, np.int32), _mass_table(), {"seed": seed})


def random_periodic(n: int, seed: int, cell: np.ndarray, n_species: int = 2,
                    d_min: float = 1.2, types: tuple[int, ...] = (28, 13)) -> System:
    """Small random periodic cell (orthorhombic or triclinic ``cell``)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    cell = np.asarray(cell, dtype=np.float64)
    inv = np.linalg.inv(cell)
    pts: list[np.ndarray] = []
    while len(pts) < n:
        p = rng.uniform(0.0, 1.0, size=3) @ cell
        good = True
        for q in pts:
            f = (p - q) @ inv
            f -= np.round(f)
            if np.linalg.norm(f @ cell) < d_min:
                good = False
                break
        if good:
            pts.append(p)
    pos = np.asarray(pts)
    species = np.asarray(types, dtype=np.int32)[rng.integers(0, n_species, size=n)]
    return System(f"periodic_{n}", pos, species, cell, np.ones(3, np.int32),
                  _mass_table(), {"seed": seed})


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------
WORKLOADS = {
    # name: (structure builder, model name, temperature K, dt fs, steps, rebuild_every)
    "fcc108_small": (lambda: fcc_copper(3, 0.05, seed=0), "small", 300.0, 1.0, 100, 0),
    "fcc4000_full": (lambda: fcc_copper(10, 0.08, seed=0), "full", 600.0, 1.0, 1000, 0),
    "bcc_hea31250_full": (lambda: bcc_hea(25, 0.06, seed=0), "full", 1000.0, 1.0, 500, 10),
    "water24000_full": (lambda: water_box(8000, 1.0, seed=2), "full", 300.0, 0.5, 500, 0),
    "fcc1m_full": (lambda: fcc_copper(63, 0.08, seed=0), "full", 300.0, 1.0, 200, 20),
    # the paper's whole-step benchmark shape: diamond carbon, sigma 0.03 A,
    # NVT at 300 K, 1 fs, 1 A skin checked every step (50^3 cells, 1,000,000 atoms)
    "diamond1m_nvt_full": (lambda: diamond_carbon(50, 0.03, seed=0), "full_carbon", 300.0, 1.0,
                           200, 0),
}

# thermostat of the NVT workloads: (damping time fs, chain length); the
# benchmark listing's 0.1 ps damping and a chain of three
NVT_WORKLOADS = {
    "diamond1m_nvt_full": (100.0, 3),
}


def make_workload(name: str) -> tuple[System, str, float, float, int, int]:
    build, model, temp, dt, steps, every = WORKLOADS[name]
    return build(), model, temp, dt, steps, every


def maxwell_boltzmann(system: System, temperature: float, seed: int = 12345) -> np.ndarray:
    """Velocities (Angstrom/fs) at exactly ``temperature`` with zero momentum.

    Per-component Gaussian with variance kT/m, centre-of-mass motion removed,
    then rescaled so that the kinetic temperature with 3N-3 degrees of
    freedom equals ``temperature``.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    m = system.mass_by_type[system.species]
    sigma = np.sqrt(KB_EV * temperature / (m * MVV2E))
    v = rng.normal(size=(system.n, 3)) * sigma[:, None]
    p = (m[:, None] * v).sum(0)
    v -= p / m.sum()
    ke = 0.5 * MVV2E * (m[:, None] * v * v).sum()
    dof = 3 * system.n - 3
    t_now = 2.0 * ke / (dof * KB_EV)
    if t_now > 0:
        v *= math.sqrt(temperature / t_now)
    return v


# ---------------------------------------------------------------------------
# model hyper-parameters and random-init parameters
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ModelSpec:
    C0: int
    L: int
    R: int
    n_rbf: int
    F: int           # MLP hidden width
    n_layers: int    # MLP hidden layers (Lambda)
    r_c: float = 6.0
    delta: float = 0.002   # radial-table spacing used by the compressed path
    n_types: int = N_TYPES


MODELS = {
    # DPA4C-Mini structure with 8 radial functions (config 1)
    "small": ModelSpec(C0=32, L=2, R=0, n_rbf=8, F=192, n_layers=3),
    # DPA4C-Plus structure (configs 2-5)
    "full": ModelSpec(C0=128, L=3, R=4, n_rbf=16, F=384, n_layers=3),
    # the five variants of Table S3 (16 radial functions)
    "nano": ModelSpec(C0=8, L=2, R=0, n_rbf=16, F=96, n_layers=3),
    "mini": ModelSpec(C0=32, L=2, R=0, n_rbf=16, F=192, n_layers=3),
    "neo": ModelSpec(C0=64, L=2, R=0, n_rbf=16, F=256, n_layers=3),
    "air": ModelSpec(C0=64, L=3, R=4, n_rbf=16, F=256, n_layers=3),
    "plus": ModelSpec(C0=128, L=3, R=4, n_rbf=16, F=384, n_layers=3),
    # the full model with its calibration taken on diamond carbon
    "full_carbon": ModelSpec(C0=128, L=3, R=4, n_rbf=16, F=384, n_layers=3),
    # the Plus widths with harmonics up to degree four (nine coupling triples)
    "plus_l4": ModelSpec(C0=128, L=4, R=4, n_rbf=16, F=384, n_layers=3),
}


def array_shapes(spec: ModelSpec) -> list[tuple[str, tuple[int, ...]]]:
    """Names and shapes of every stored array, in blob order.

    The widths follow Eqs. (degree-channels), (probe-ranks), (dim-out) and the
    hidden widths of Eqs. (radial-map) and (pairfilm).  This is layout only;
    the arithmetic that uses the arrays lives elsewhere.
    """
    C0, L, R = spec.C0, spec.L, spec.R
    C1 = max(4, 1 << math.ceil(0.5 * math.log2(C0)))
    C2 = max(4, C1 // 2)
    K1, K2 = C2, 2
    H = 8 * math.ceil(C0 / 3)
    Hp = 8 * math.ceil(2 * C0 / 3)
    Cl = [C0, C1, C2] + [1] * max(0, L - 2)
    Kl = [None, K1, K2] + [1] * max(0, L - 2)
    d_out = descriptor_width(C0, L)
    shapes = [
        ("type_embed", (spec.n_types + 1, C0)),
        ("omega", (spec.n_rbf,)),
        ("W_in", (spec.n_rbf, 2 * H)),
        ("W_out", (H, C0)),
        ("W_mode", (H, R)),
        ("Wp_in", (2 * C0, 2 * Hp)),
        ("Wp_out", (Hp, C0 * (2 + R))),
        ("W_align1", (C1, C1)),
        ("W_align2", (C2, C2)),
    ]
    if Kl[1] != Cl[1]:
        shapes.append(("A1", (C1, K1)))
    shapes.append(("A2", (C2, K2)))
    fan = d_out
    for tau in range(1, spec.n_layers + 1):
        shapes.append((f"Theta{tau}", (fan, spec.F)))
        shapes.append((f"b{tau}", (spec.F,)))
        fan = spec.F
    shapes += [("w_head", (spec.F,)), ("b_head", (1,)),
               ("E_ref", (spec.n_types + 1,)),
               ("mu", (d_out,)), ("sigma", (d_out,))]
    return shapes


def descriptor_width(C0: int, L: int) -> int:
    """Counting of Eq. (dim-out) with Eq. (bispectrum-count); layout only."""
    C1 = max(4, 1 << math.ceil(0.5 * math.log2(C0)))
    C2 = max(4, C1 // 2)
    Cl = [C0, C1, C2] + [1] * max(0, L - 2)
    Kl = [0, C2, 2] + [1] * max(0, L - 2)
    n = 2 * C0 + 2 + sum(Cl[l] * (Cl[l] + 1) // 2 for l in range(1, L + 1))
    for l1 in range(1, L + 1):
        for l2 in range(l1, L + 1):
            for l3 in range(l2, L + 1):
                if l3 > l1 + l2 or (l1 + l2 + l3) % 2:
                    continue
                if l1 == l2 == l3:
                    k = Kl[l1]
                    n += k * (k + 1) * (k + 2) // 6
                elif l1 == l2:
                    n += Kl[l1] * (Kl[l1] + 1) // 2 * Kl[l3]
                elif l2 == l3:
                    n += Kl[l2] * (Kl[l2] + 1) // 2 * Kl[l1]
                else:
                    n += Kl[l1] * Kl[l2] * Kl[l3]
    return n + Kl[1] * Kl[2]


TRAINABLE_EXCLUDED = ("E_ref", "mu", "sigma")


def random_weights(spec: ModelSpec, seed: int = 2608) -> dict[str, np.ndarray]:
    """Random-init parameters (float32).

    Distributions: type table N(0,1); every matrix N(0, 1/fan_in); the
    channel-alignment maps N(0, 0.1^2/C); MLP biases N(0, 0.1^2); the head
    vector half-normal |N(0, 1/F)|; radial frequencies omega_n = n*pi/r_c;
    E_ref uniform in [-1, 0) eV.  The
    calibration vectors start at mu = 0, sigma = 1 and the head is unscaled;
    a calibration step fixes them later.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    out: dict[str, np.ndarray] = {}
    for name, shape in array_shapes(spec):
        if name == "type_embed":
            a = rng.normal(size=shape)
            a[-1] = 0.0                               # zero padding type
        elif name == "omega":
            a = np.arange(1, shape[0] + 1) * math.pi / spec.r_c
        elif name in ("W_align1", "W_align2"):
            a = rng.normal(size=shape) * 0.1 / math.sqrt(shape[0])
        elif name.startswith("b") and name != "b_head":
            a = rng.normal(size=shape) * 0.1
        elif name == "b_head":
            a = np.zeros(shape)
        elif name == "E_ref":
            a = rng.uniform(-1.0, 0.0, size=shape)
        elif name == "mu":
            a = np.zeros(shape)
        elif name == "sigma":
            a = np.ones(shape)
        elif name == "w_head":
            # half-normal: a nonnegative head over SiLU units (SiLU >= -0.279)
            # makes every atomic energy bounded below, so a random potential
            # cannot release unbounded energy into the dynamics
            a = np.abs(rng.normal(size=shape)) / math.sqrt(shape[0])
        else:
            a = rng.normal(size=shape) / math.sqrt(shape[0])
        out[name] = np.ascontiguousarray(a, dtype=np.float32)
    return out


def trainable_count(spec: ModelSpec) -> int:
    return int(sum(int(np.prod(s)) for n, s in array_shapes(spec)
                   if n not in TRAINABLE_EXCLUDED))


BLOB_MAGIC = b"DPA4CW01"
BLOB_HEADER = struct.Struct("<8s8i2d")     # 8 + 32 + 16 = 56 bytes, padded to 64
BLOB_HEADER_BYTES = 64


def pack_blob(spec: ModelSpec, weights: dict[str, np.ndarray]) -> bytes:
    """Binary weight blob: 64-byte header followed by float32 arrays in the
    order of :func:`array_shapes` (each C-contiguous, row-major)."""
    head = BLOB_HEADER.pack(BLOB_MAGIC, 1, spec.C0, spec.L, spec.R, spec.n_rbf,
                            spec.F, spec.n_layers, spec.n_types, spec.r_c, spec.delta)
    parts = [head.ljust(BLOB_HEADER_BYTES, b"\0")]
    for name, shape in array_shapes(spec):
        a = np.ascontiguousarray(weights[name], dtype=np.float32)
        if a.shape != shape:
            raise ValueError(f"{name}: shape {a.shape} != {shape}")
        parts.append(a.tobytes())
    return b"".join(parts)


def unpack_blob(blob: bytes) -> tuple[ModelSpec, dict[str, np.ndarray]]:
    magic, ver, C0, L, R, n_rbf, F, nl, nt, rc, delta = BLOB_HEADER.unpack_from(blob, 0)
    if magic != BLOB_MAGIC or ver != 1:
        raise ValueError("not a weight blob")
    spec = ModelSpec(C0, L, R, n_rbf, F, nl, rc, delta, nt)
    off = BLOB_HEADER_BYTES
    out = {}
    for name, shape in array_shapes(spec):
        n = int(np.prod(shape))
        out[name] = np.frombuffer(blob, dtype=np.float32, count=n, offset=off).reshape(shape).copy()
        off += 4 * n
    if off != len(blob):
        raise ValueError("blob size mismatch")
    return spec, out


_CALIB = None


def model_weights(name: str) -> tuple[ModelSpec, dict[str, np.ndarray]]:
    """Random-init parameters of a named model with its stored calibration
    (mu, sigma and head scale from ``calibration.json``) applied."""
    import json
    import os
    global _CALIB
    spec = MODELS[name]
    w = random_weights(spec)
    if _CALIB is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calibration.json")
        with open(path) as f:
            _CALIB = json.load(f)
    c = _CALIB[name]
    w["mu"] = np.asarray(c["mu"], dtype=np.float32)
    w["sigma"] = np.asarray(c["sigma"], dtype=np.float32)
    w["w_head"] = (w["w_head"].astype(np.float64) * c["head_scale"]).astype(np.float32)
    return spec, w
