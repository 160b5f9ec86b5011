"""Pins of the oracle neighbour list (no GPU)."""
import numpy as np
import pytest

import synth
from oracle import neighbors as nb


def as_tuples(ei, ej, en):
    return [tuple([int(a), int(b)] + [int(x) for x in n]) for a, b, n in zip(ei, ej, en)]


@pytest.mark.parametrize("case", ["ortho", "triclinic", "open", "small_box"])
def test_c_brute_force_matches_python_definition(case):
    if case == "ortho":
        s = synth.random_periodic(7, seed=1, cell=np.diag([7.0, 8.0, 9.5]))
    elif case == "triclinic":
        s = synth.random_periodic(6, seed=2, cell=np.array([[7.0, 0.0, 0.0], [2.1, 7.5, 0.0],
                                                            [-1.3, 1.7, 8.2]]))
    elif case == "small_box":
        # box shorter than the cutoff: several images of every atom
        s = synth.random_periodic(3, seed=3, cell=np.diag([4.1, 4.4, 5.0]))
    else:
        s = synth.random_cluster(9, seed=4)
    r = 6.0
    c = as_tuples(*nb.neighbor_list(s.pos, s.cell, s.pbc, r))
    py = nb.neighbor_list_python(s.pos, s.cell, s.pbc, r, n_image=3)
    assert c == py
    assert len(c) > 0


@pytest.mark.parametrize("kind,a,count", [("fcc", 3.615, 78), ("diamond", 3.567, 158),
                                          ("bcc", 2.87, 64)])
def test_perfect_crystal_counts(kind, a, count):
    # FCC Cu 78 and diamond C 158 neighbours at 6 A are printed in Supplementary
    # Note "Single-GPU crystal scans"; BCC at 2.87 A follows from its shells
    pos, cell = synth.lattice(kind, a, (3, 3, 3))
    ei, ej, en = nb.neighbor_list(pos, cell, np.ones(3, np.int32), 6.0)
    assert np.all(np.bincount(ei, minlength=len(pos)) == count)


def test_config1_multiple_images_and_symmetry():
    s = synth.fcc_copper(3, 0.05, seed=0)
    ei, ej, en = nb.neighbor_list(s.pos, s.cell, s.pbc, 6.0)
    # box 10.845 A < 2 r_c: some atoms see several images of the same j
    pairs = set()
    dup = False
    for a, b in zip(ei, ej):
        dup |= (a, b) in pairs
        pairs.add((a, b))
    assert dup
    # both orientations are stored: (i, j, n) <-> (j, i, -n)
    fwd = set(as_tuples(ei, ej, en))
    assert all((j, i, -x, -y, -z) in fwd for (i, j, x, y, z) in fwd)
    # canonical order
    keys = list(zip(ei, ej, en[:, 0], en[:, 1], en[:, 2]))
    assert keys == sorted(keys)
    # no self edge at n = 0
    assert not np.any((ei == ej) & np.all(en == 0, axis=1))


def test_centre_subset_equals_rows_of_full_list():
    s = synth.fcc_copper(4, 0.08, seed=5)
    full = as_tuples(*nb.neighbor_list(s.pos, s.cell, s.pbc, 7.0))
    cs = np.array([0, 17, 100, 255])
    sub = as_tuples(*nb.neighbor_list(s.pos, s.cell, s.pbc, 7.0, centres=cs))
    assert sub == [t for t in full if t[0] in set(cs.tolist())]


def test_unwrapped_positions_give_shifted_images():
    # moving an atom by a lattice vector changes only its image labels
    s = synth.random_periodic(5, seed=6, cell=np.diag([6.5, 7.0, 7.5]))
    p2 = s.pos.copy()
    p2[2] += s.cell[0] * 2 - s.cell[2]
    e1 = as_tuples(*nb.neighbor_list(s.pos, s.cell, s.pbc, 6.0))
    e2 = as_tuples(*nb.neighbor_list(p2, s.cell, s.pbc, 6.0))
    assert len(e1) == len(e2)
    shift = np.array([2, 0, -1])
    fix = []
    for i, j, x, y, z in e2:
        n = np.array([x, y, z])
        if j == 2:
            n = n + shift
        if i == 2:
            n = n - shift
        fix.append((i, j) + tuple(int(v) for v in n))
    assert sorted(fix) == e1
