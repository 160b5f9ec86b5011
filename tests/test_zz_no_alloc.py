"""The entry point without device allocation against compute_energy_forces,
through the C ABI: two calls in a row, the second with a smaller input, on
the same model, and on a fresh model whose first call is the no-allocation
one (separable tables).  Device memory in use does not change across the
no-allocation calls, and an input beyond the scratch is refused."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

E_TOL = 1e-5
F_TOL = 1e-4


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


def inputs(dp, s, dev, r_list):
    pos = torch.tensor(s.pos, dtype=torch.float64, device=dev)
    species = torch.tensor(s.species, dtype=torch.int32, device=dev)
    rp, nj, ns, e = dp.build_neighbors(pos, s.cell, s.pbc, r_list)
    return pos, species, rp, nj, ns, e


def systems():
    big = synth.make_workload("fcc4000_full")[0]
    small = synth.random_periodic(24, seed=11, cell=np.diag([8.3, 8.9, 9.4]), d_min=1.6)
    return big, small


@pytest.mark.parametrize("warm", [True, False])
def test_noalloc_equals_compute_energy_forces(dev, dp, warm):
    spec, w = synth.model_weights("full")
    blob = synth.pack_blob(spec, w)
    ref_model = dp.Model(blob)
    model = ref_model if warm else dp.Model(blob)
    for s in systems():      # two calls in a row, the second smaller
        pos, species, rp, nj, ns, e = inputs(dp, s, dev, spec.r_c + 1.0)
        ref_e, ref_f, ref_t = ref_model.compute_energy_forces(pos, species, s.cell, s.pbc,
                                                              spec.r_c, rp, nj, ns, e)
        ea = torch.empty(s.n, dtype=torch.float64, device=dev)
        F = torch.empty(s.n, 3, dtype=torch.float64, device=dev)
        et = torch.empty(1, dtype=torch.float64, device=dev)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info(dev)[0]
        model.compute_energy_forces_noalloc(pos, species, s.cell, s.pbc, spec.r_c, rp, nj, ns, e,
                                            ea, F, et)
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info(dev)[0] == free0
        de = float((ea - ref_e).abs().max())
        df = float((F - ref_f).abs().max())
        print(f"{s.name}: {s.n} atoms, {e} entries, warm={warm}: max|dE_i| {de:.2e}, "
              f"max|dF| {df:.2e}", flush=True)
        assert de < E_TOL and df < F_TOL
        assert abs(float(et[0] - ref_t[0])) < E_TOL * s.n
        if warm:    # the same tables and kernels: the same bits
            assert de == 0.0 and df == 0.0


def test_noalloc_refuses_inputs_beyond_its_scratch(dev, dp):
    spec, w = synth.model_weights("full")
    model = dp.Model(synth.pack_blob(spec, w))
    s = systems()[1]
    pos, species, rp, nj, ns, e = inputs(dp, s, dev, spec.r_c + 1.0)
    ea = torch.empty(s.n, dtype=torch.float64, device=dev)
    F = torch.empty(s.n, 3, dtype=torch.float64, device=dev)
    et = torch.empty(1, dtype=torch.float64, device=dev)
    with pytest.raises(dp.DPA4CError) as ex:
        model.compute_energy_forces_noalloc(pos, species, s.cell, s.pbc, spec.r_c, rp, nj, ns,
                                            1 << 24, ea, F, et)
    assert ex.value.code == dp.ERR_INVALID_ARG and "scratch" in str(ex.value)
