"""The FP64 debug precision (MACE_FP64) through the C ABI against the FP64
oracle: energies, every per-atom energy and force, and the stress within
1e-10 relative (FP64 rounding of two differently ordered evaluations of the
same function; the FP32 arms sit at 1e-6..1e-5). Covers hidden l <= 2 (every
edge-product path and output irrep), the stress inputs (every correlation
order of Eq. 27 contributing), a batch of non-periodic molecules of ten
species, an atom without neighbours, run-to-run determinism, and the settings
an FP64 handle refuses."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (STRESS, STRESS_GAINS, assert_parity, lib_blob, oracle_blob, oracle_stress,  # noqa: E402
                        run_gpu, run_oracle, stress_error)
from paper_2510_23621_amd.graph import MaceGraph  # noqa: E402

TOL64 = 1e-10


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _check(params, sysm, seed=0, gains=None, label="", stress=False):
    bo, bl = oracle_blob(params, seed, gains), lib_blob(params, seed, gains)
    assert np.array_equal(bo, bl)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl, prec=B.MACE_FP64, stress=stress)
    assert gpu["n_edges"] == len(ref["graph"].sender)
    err = assert_parity(gpu, ref, B.MACE_FP64, label)
    if stress:
        sref = oracle_stress(params, sysm, bo)
        serr = stress_error(gpu["stress"], sref)
        print(f"[fp64] {label} stress rel {serr:.3e}", flush=True)
        assert serr <= TOL64
    return err


def test_cfg0_nominal_fp64():
    _check(model_params(0), make_system(0, seed=0), label="cfg0 nominal", stress=True)


def test_cfg0_stress_inputs_fp64():
    _check(model_params(0, **STRESS), make_system(0, seed=1), gains=STRESS_GAINS, label="cfg0 stress")


@pytest.mark.parametrize("K,hl", [(64, 1), (32, 2)])
def test_small_water_hidden_l_fp64(K, hl):
    params = model_params(0, K=K, hidden_lmax=hl, **STRESS)
    _check(params, synth.water_box(34, seed=7, box=10.0), seed=3, gains=STRESS_GAINS,
           label=f"water102 K={K} l={hl}", stress=True)


def test_per_layer_hidden_l_fp64():
    """Three layers with hidden l_max 2 then 1 (one per layer)."""
    params = model_params(0, K=32, n_layers=3, hidden_lmax=(2, 1), **STRESS)
    _check(params, synth.water_box(34, seed=7, box=10.0), seed=3, gains=STRESS_GAINS,
           label="water102 K=32 l=(2, 1)", stress=True)


def test_molecule_batch_fp64():
    params = model_params(4, K=32, **STRESS)
    sysm = synth.molecule_batch(6, seed=5)
    _check(params, sysm, seed=2, gains=STRESS_GAINS, label="6 molecules, 10 species", stress=True)


def test_isolated_atom_and_determinism_fp64():
    params = model_params(0, K=32, **STRESS)
    base = make_system(0, seed=4)
    pos = np.vstack([base.positions, [[50.0, 50.0, 50.0]]])
    sysm = synth.System(pos, np.append(base.species, 1).astype(np.int32), None,
                        np.zeros(len(pos), np.int32), 1)
    bl = lib_blob(params, 1, STRESS_GAINS)
    ref = run_oracle(params, sysm, oracle_blob(params, 1, STRESS_GAINS))
    outs = run_gpu(params, sysm, bl, prec=B.MACE_FP64, repeats=2)
    assert_parity(outs[0], ref, B.MACE_FP64, "cluster + isolated atom")
    assert np.array_equal(outs[0]["forces"], outs[1]["forces"]) and np.array_equal(outs[0]["eps"], outs[1]["eps"])
    assert np.all(outs[0]["forces"][-1] == 0.0)


def test_fp64_handle_settings():
    params = model_params(0)
    sysm = make_system(0, seed=0)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells)
    g = MaceGraph(B.make_desc(**params), lib_blob(params, 0), sysm.species, np.stack([snd, rcv]), sh, sysm.cells,
                  None, 1, B.MACE_FP64)
    assert B.mace_layer0_form(g.handle, -1) == B.MACE_L0_EDGE
    with pytest.raises(B.MaceError):
        B.mace_layer0_form(g.handle, B.MACE_L0_FACTORED)
    with pytest.raises(B.MaceError):
        B.mace_block_rounding(g.handle, B.MACE_BLOCK_EDGE_PRODUCT, 1)
    with pytest.raises(B.MaceError):
        B.mace_fp32_products(g.handle, B.MACE_PRODUCTS_FP32)
    eps, E, F = g.energy_forces(torch.from_numpy(sysm.positions).cuda())
    assert eps.dtype == torch.float64 and F.dtype == torch.float64
    g.close()
