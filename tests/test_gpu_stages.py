"""Stage-level parity of the GPU path with the continuous float64 oracle,
through the C ABI, at the precision class of the paper's own check.

Supplementary Table S1 reports the tabulated (Delta = 0.002 A) against the
continuous feature vector, both in single precision, as a maximum deviation
relative to the largest feature-vector entry: 1.3e-7 to 1.8e-7 on three
profiles.  Here the reference is the float64 continuous model, so the GPU's
deviation also holds the float32 rounding of its inputs: the edge vector is
the float64 difference stored in float32 (6e-8 relative per component), and
the envelope amplifies that near the cutoff (d ln chi / d rho is -4 / (r_c t)
for the t^4 factor), most of all in the standardised M1 entry, whose sum of
chi^4 then carries ~7e-7 relative error (measured on the small and full
profiles: M1 holds the largest deviation, 1.3-1.8e-6 of the largest entry,
while the float32 node state stays at ~3e-7).
The node state and the descriptor are therefore held to STAGE_FACTOR = 15
times the largest bound of Table S1 (read from the golden file), against
1e-4 before.

Also: the Plus profile's stages on both table paths, the pair-folded tables
against the separable ones on the same systems, and every E_i and force of
a 5-species alloy cell on the folded tables.
"""
import numpy as np
import pytest
import torch

import synth
from conftest import golden
from oracle import model as om

pytestmark = pytest.mark.gpu

E_TOL = 1e-5
F_TOL = 1e-4
S1 = {k: float(v) for k, v in golden("table_s1_verification.txt")}
TAB_BOUND = max(v for k, v in S1.items() if k.startswith("tabulated_vs_continuous"))
STAGE_FACTOR = 15.0      # the multiple of the paper's bound the GPU stages are held to


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


def run(dp, model, s, dev, r_list=7.0, noalloc=False):
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, r_list)
    if noalloc:
        ea = torch.empty(s.n, dtype=torch.float64, device=dev)
        F = torch.empty(s.n, 3, dtype=torch.float64, device=dev)
        et = torch.empty(1, dtype=torch.float64, device=dev)
        model.compute_energy_forces_noalloc(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e,
                                            ea, F, et)
    else:
        ea, F, et = model.compute_energy_forces(pos, species, s.cell, s.pbc, 6.0, rp, nj, ns, e)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), F.cpu().numpy()


def many_species_bcc():
    s = synth.bcc_hea(3, 0.06, seed=7)
    types = np.array(sorted(set(s.meta["types"]) | {0, 7, 28}), dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(3))
    s.species = types[rng.integers(0, len(types), size=s.n)].astype(np.int32)
    return s


def stage_deviations(dp, dev, name, s):
    spec, w = synth.model_weights(name)
    model = dp.Model(synth.pack_blob(spec, w))
    run(dp, model, s, dev)
    node, desc, cnt = model.debug_stages(s.n)
    ref = om.Oracle(spec, w).stages(s.pos, s.species, s.cell, s.pbc)
    node = node.cpu().numpy().astype(np.float64)
    C0 = spec.C0
    y = ref["X_flat"].copy()
    y[:, :C0] *= ref["M0"][:, None]
    y[:, C0:] *= ref["M1"][:, None]
    full = np.concatenate([ref["S0"][:, None], ref["S1"][:, None], y], 1)
    d = desc.cpu().numpy().astype(np.float64)
    dev_node = np.abs(node - full).max() / np.abs(full).max()
    dev_desc = np.abs(d - ref["D"]).max() / np.abs(ref["D"]).max()
    return dev_node, dev_desc


CASES = [("small", "fcc108"), ("full", "fcc108"), ("full", "hea54"), ("full", "bcc8species"),
         ("nano", "fcc108"), ("air", "fcc108"), ("plus_l4", "fcc108")]


def system_of(key):
    if key == "fcc108":
        return synth.fcc_copper(3, 0.08, seed=3)
    if key == "hea54":
        return synth.bcc_hea(3, 0.06, seed=7)
    return many_species_bcc()


@pytest.mark.parametrize("name,key", CASES)
def test_feature_vector_at_the_tabulation_class(dev, dp, name, key):
    """max |D_gpu - D_oracle| / max |D_oracle| and the same for the node
    state, within STAGE_FACTOR times the largest tabulated-against-continuous
    deviation of Table S1."""
    s = system_of(key)
    dn, dd = stage_deviations(dp, dev, name, s)
    print(f"{name} {key} ({len(np.unique(s.species))} species): node state {dn:.2e}, "
          f"descriptor {dd:.2e} relative (bound {STAGE_FACTOR * TAB_BOUND:.1e})", flush=True)
    assert dn <= STAGE_FACTOR * TAB_BOUND
    assert dd <= STAGE_FACTOR * TAB_BOUND


@pytest.mark.parametrize("key", ["fcc108", "hea54"])
def test_folded_tables_equal_separable_tables(dev, dp, key):
    """The same system on the pair-folded tables (c0, c1 in float32, c2, c3
    in scaled float16, c4 and c5 not stored, their bound being below float32
    resolution for this model) and on the separable float32 tables of the
    full quintic (a fresh model's first call without allocation has no
    folded tables): E_i and F agree to float32 rounding, and each is within
    the stated tolerance of the oracle."""
    spec, w = synth.model_weights("full")
    blob = synth.pack_blob(spec, w)
    s = system_of(key)
    folded = dp.Model(blob)
    assert folded.info["fold_words"] == 3
    e_f, f_f = run(dp, folded, s, dev)
    e_s, f_s = run(dp, dp.Model(blob), s, dev, noalloc=True)
    ref_e, ref_f = om.Oracle(spec, w).energy_forces(s.pos, s.species, s.cell, s.pbc)
    de, df = np.abs(e_f - e_s).max(), np.abs(f_f - f_s).max()
    print(f"{key}: folded - separable max|dE_i| {de:.2e} (|E_i| <= {np.abs(ref_e).max():.1f}), "
          f"max|dF| {df:.2e} (|F| <= {np.abs(ref_f).max():.2f}); oracle: folded "
          f"{np.abs(e_f - ref_e).max():.2e} / {np.abs(f_f - ref_f).max():.2e}, separable "
          f"{np.abs(e_s - ref_e).max():.2e} / {np.abs(f_s - ref_f).max():.2e}", flush=True)
    assert de <= 2e-7 * max(1.0, np.abs(ref_e).max())
    assert df <= 2e-6 * max(1.0, np.abs(ref_f).max())
    for e, f in ((e_f, f_f), (e_s, f_s)):
        assert np.abs(e - ref_e).max() < E_TOL and np.abs(f - ref_f).max() < F_TOL


def test_five_species_alloy_cell_on_folded_tables(dev, dp):
    """Every E_i and force of a 54-atom cell of the 5-species alloy with the
    full model, which folds its 25 ordered pairs."""
    spec, w = synth.model_weights("full")
    s = synth.bcc_hea(3, 0.06, seed=7)
    assert len(np.unique(s.species)) == 5
    e, f = run(dp, dp.Model(synth.pack_blob(spec, w)), s, dev)
    ref_e, ref_f = om.Oracle(spec, w).energy_forces(s.pos, s.species, s.cell, s.pbc)
    assert np.abs(e - ref_e).max() < E_TOL
    assert np.abs(f - ref_f).max() < F_TOL
