"""Parity at the workloads' full sizes, in the configuration bench.py times.

* 1536-atom water (K=128, 0e+1o): every per-atom energy and force against
  the FP64 oracle, FP32 and BF16-linear.
* 4608- and 36,864-atom water: per-atom energies of sampled atoms against
  the oracle evaluated on a cluster cut of radius 2 r_c + margin around the
  atom (eps_i depends only on atoms within 2 r_c: layer 1 sums h^(1) of
  neighbours, which sum their own neighbours), plus properties that hold at
  any size: sum F = 0, rotation covariance of the whole periodic box (forces
  and stress), determinism, BF16-linear vs FP32.
* 1536-atom water also checks the stress against the oracle.
* 512-molecule batch: sampled molecules are whole graphs, so their energy
  and forces are compared exactly.
"""
import numpy as np
import pytest
import torch

import synth
from synth.configs import CONFIGS, make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (TOL, assert_parity, cluster_cut, errors, lib_blob, oracle_blob, oracle_stress,  # noqa: E402
                        run_gpu, run_oracle, stress_error)
from oracle import so3  # noqa: E402

PER_ATOM_TOL = {B.MACE_FP32: 2e-5, B.MACE_BF16_LINEAR: 5e-2}


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _per_atom_check(gpu_eps, ref_eps, atoms, scale, prec, label):
    err = np.abs(gpu_eps[atoms] - ref_eps) / scale
    print(f"[fullsize] {label} per-atom max rel err {err.max():.3e} (n={len(atoms)})", flush=True)
    assert err.max() <= PER_ATOM_TOL[prec], (label, err)


def _rotate(system, R):
    cells = None if system.cells is None else system.cells @ R.T
    return synth.System(system.positions @ R.T, system.species, cells, system.graph_of_atom, system.n_graphs)


# ------------------------------------------------------------------ 1536 atoms, complete

@pytest.fixture(scope="module")
def cfg1():
    params = model_params(1)
    sysm = make_system(1, seed=0)
    blob = oracle_blob(params, 0)
    assert np.array_equal(blob, lib_blob(params, 0))
    ref = run_oracle(params, sysm, blob)
    return params, sysm, blob, ref


def test_cfg1_full_fp32(cfg1):
    params, sysm, blob, ref = cfg1
    gpu = run_gpu(params, sysm, blob, stress=True)
    assert gpu["n_edges"] == len(ref["graph"].sender)
    assert_parity(gpu, ref, B.MACE_FP32, "water1536 full")
    sref = oracle_stress(params, sysm, blob)
    err = stress_error(gpu["stress"], sref)
    print(f"[fullsize] water1536 stress rel {err:.3e} (pressure {-np.trace(sref[0]) / 3:.4e})", flush=True)
    assert err <= TOL[B.MACE_FP32]["forces"]


def test_cfg1_full_bf16(cfg1):
    params, sysm, blob, ref = cfg1
    gpu = run_gpu(params, sysm, blob, prec=B.MACE_BF16_LINEAR)
    assert_parity(gpu, ref, B.MACE_BF16_LINEAR, "water1536 full bf16")


# ------------------------------------------------------------------ larger periodic boxes

@pytest.mark.parametrize("cfg", [2, 3])
def test_large_water_sampled_and_properties(cfg):
    params = model_params(cfg)
    sysm = make_system(cfg, seed=0)
    blob = lib_blob(params, 0)
    g32 = run_gpu(params, sysm, blob)
    N = sysm.n_atoms
    F = g32["forces"]
    print(f"[fullsize] water{N}: {g32['n_edges']} edges", flush=True)
    # sum of forces vanishes (translation invariance)
    assert np.abs(F.sum(0)).max() <= 1e-5 * np.abs(F).max() * np.sqrt(N)
    # sampled per-atom energies against the oracle on cluster cuts
    rng = np.random.default_rng(cfg)
    atoms = rng.choice(N, size=3, replace=False)
    rc = params["r_cut"]
    ref = []
    for i in atoms:
        cl, _ = cluster_cut(sysm, int(i), 2 * rc + 0.5)
        out = run_oracle(params, cl, oracle_blob(params, 0), forces=False)
        ref.append(out["eps"][0])
    scale = np.abs(g32["eps"]).mean()
    _per_atom_check(g32["eps"], np.array(ref), atoms, scale, B.MACE_FP32, f"water{N}")
    # rotation covariance of the whole box (GPU against GPU)
    R = so3.random_rotation(np.random.default_rng(100 + cfg))
    rot = _rotate(sysm, R)
    g_rot = run_gpu(params, rot, blob, stress=True)
    e_err = np.abs(g_rot["energy"] - g32["energy"]).max() / np.abs(g32["eps"]).sum()
    f_err = np.linalg.norm(g_rot["forces"] - F @ R.T) / np.linalg.norm(F)
    # stress is a rank-2 tensor: sigma(x R^T) = R sigma R^T
    s32 = run_gpu(params, sysm, blob, stress=True)["stress"]
    s_err = stress_error(g_rot["stress"], R @ s32 @ R.T)
    print(f"[fullsize] water{N} rotation: energy {e_err:.2e} forces {f_err:.2e} stress {s_err:.2e}", flush=True)
    assert e_err <= 2 * TOL[B.MACE_FP32]["energy"] and f_err <= 2 * TOL[B.MACE_FP32]["forces"]
    assert s_err <= 2 * TOL[B.MACE_FP32]["forces"]
    # BF16-linear against FP32 at full size
    g16 = run_gpu(params, sysm, blob, prec=B.MACE_BF16_LINEAR)
    err = errors(g16, g32)
    print(f"[fullsize] water{N} bf16 vs fp32 {err}", flush=True)
    assert err["energy"] <= TOL[B.MACE_BF16_LINEAR]["energy"] and err["forces"] <= TOL[B.MACE_BF16_LINEAR]["forces"]
    # determinism at full size
    again = run_gpu(params, sysm, blob)
    assert np.array_equal(again["forces"], F) and np.array_equal(again["eps"], g32["eps"])


# ------------------------------------------------------------------ 512-molecule batch

@pytest.mark.parametrize("prec", [B.MACE_BF16_LINEAR, B.MACE_FP32])
def test_molecule_batch_sampled_graphs(prec):
    params = model_params(4)
    sysm = make_system(4, seed=0)
    blob = lib_blob(params, 0)
    gpu = run_gpu(params, sysm, blob, prec=prec)
    assert gpu["energy"].shape == (512,)
    rng = np.random.default_rng(4)
    for g in rng.choice(512, size=4, replace=False):
        idx = np.nonzero(sysm.graph_of_atom == g)[0]
        sub = synth.System(sysm.positions[idx], sysm.species[idx], None, np.zeros(len(idx), np.int32), 1)
        ref = run_oracle(params, sub, oracle_blob(params, 0))
        part = dict(eps=gpu["eps"][idx], energy=gpu["energy"][g:g + 1], forces=gpu["forces"][idx])
        assert_parity(part, ref, prec, f"molecule graph {g} ({len(idx)} atoms)")
