"""The capacity protocol of the paper's single-GPU crystal scans (Methods,
single-GPU crystal scans; Supplementary Note on the computational-reference
benchmark): near-cubic supercells whose edge counts differ by at most one,
doubling from 128 requested atoms to the first out-of-memory failure, then
three bisections.  Pinned to the realised sizes printed in the diamond-carbon
and FCC-copper V100 scan tables (Supplementary Tables of the V100 scans):
given a memory boundary between a row's largest completed and first failed
system, the protocol must land on exactly that row's bracket."""
import pytest

import bench
import synth

# (atoms per cell, largest completed, first failed) of the table rows
BRACKETS = [
    (8, 2_097_152, 2_370_192),     # diamond carbon, every DPA4C variant
    (8, 1_968_624, 2_097_152),     # diamond carbon, NEP89
    (4, 4_203_216, 4_719_120),     # FCC copper, Nano to Air
    (4, 3_920_400, 4_203_216),     # FCC copper, Plus
]
# realised sizes of the tables' other columns (atoms at saturated throughput)
SIZES = [(8, 64_000), (8, 32_768), (8, 130_000), (8, 524_800),
         (4, 1_048_576), (4, 262_400), (4, 65_000), (4, 520_200)]


def realised(req, per_cell):
    r = synth.near_cubic_reps(req, per_cell)
    assert max(r) - min(r) <= 1
    return per_cell * r[0] * r[1] * r[2]


@pytest.mark.parametrize("per_cell,ok_atoms,fail_atoms", BRACKETS)
def test_scan_lands_on_the_printed_bracket(per_cell, ok_atoms, fail_atoms):
    limit = (ok_atoms + fail_atoms) / 2      # any boundary inside the bracket

    def point(req):
        n = realised(req, per_cell)
        return {"requested": req, "atoms": n, "status": "ok" if n <= limit else "oom"}

    points, ok, fail = bench.scan_bracket(point, 128, 3)
    assert ok["atoms"] == ok_atoms and fail["atoms"] == fail_atoms
    assert points[0]["requested"] == 128
    # doubling until the first failure, then exactly three bisections
    n_double = next(k for k, p in enumerate(points) if p["status"] == "oom") + 1
    assert len(points) == n_double + 3
    assert all(points[k + 1]["requested"] == 2 * points[k]["requested"] for k in range(n_double - 1))


@pytest.mark.parametrize("per_cell,atoms", SIZES)
def test_printed_sizes_are_realised_doubling_points(per_cell, atoms):
    # the sizes where throughput saturates are realisations of doubling
    # requests 128 * 2^k
    assert any(realised(128 * 2 ** k, per_cell) == atoms for k in range(20))


def test_first_point_out_of_memory_gives_no_bracket():
    points, ok, fail = bench.scan_bracket(
        lambda req: {"requested": req, "atoms": req, "status": "oom"}, 128, 3)
    assert ok is None and len(points) == 1
