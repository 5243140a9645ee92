"""Parity at the workloads' full sizes, in the configuration bench.py times.

* 1536-atom water (K=128, 0e+1o): every per-atom energy and force against
  the FP64 oracle, FP32 and BF16-linear; the stress against the oracle.
* 1536-atom water with the stress inputs (c_norm 1, last radial layer x4),
  where every correlation order of Eq. 27 contributes (the oracle-side share
  of each order is asserted by a CPU test): every atom, FP32.
* 4608- and 36,864-atom water: every per-atom energy and force against FP64
  oracle references written by tests/golden/make_fullsize_refs.py (the
  oracle's two-pass chunked VJP), FP32 and BF16-linear; the inputs'
  fingerprint is checked first. Plus properties that hold at any size:
  sum F = 0, rotation covariance of the whole periodic box (forces and
  stress), determinism.
* 512-molecule batch: sampled molecules are whole graphs, so their energy
  and forces are compared exactly.
"""
import os
import sys

import numpy as np
import pytest
import torch

import synth
from synth.configs import CONFIGS, make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (TOL, assert_parity, errors, lib_blob, oracle_blob, oracle_stress,  # noqa: E402
                        run_gpu, run_oracle, stress_error)
from oracle import mace, so3  # noqa: E402
from paper_2510_23621_amd.graph import MaceGraph  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
sys.path.insert(0, GOLDEN)
import make_fullsize_refs as refs  # noqa: E402


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _rotate(system, R):
    cells = None if system.cells is None else system.cells @ R.T
    return synth.System(system.positions @ R.T, system.species, cells, system.graph_of_atom, system.n_graphs)


def _stored_ref(name):
    """(params, system, blob, ref) of a stored FP64 reference, after checking
    that the library's neighbour list and the seeded inputs reproduce the
    fingerprint the reference was written for."""
    params, sysm, blob = refs.workload(name)
    z = np.load(refs.ref_path(name))
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells, sysm.graph_of_atom,
                                        sysm.n_graphs)
    assert len(snd) == int(z["n_edges"])
    assert refs.fingerprint(sysm, blob, snd, rcv, sh) == str(z["fingerprint"]), name
    ref = dict(eps=z["eps"], energy=z["energy"], forces=z["forces"])
    return params, sysm, blob, ref


# ------------------------------------------------------------------ 1536 atoms, complete

@pytest.fixture(scope="module")
def cfg1():
    params = model_params(1)
    sysm = make_system(1, seed=0)
    blob = oracle_blob(params, 0)
    assert np.array_equal(blob, lib_blob(params, 0))
    ref = mace.energy_forces_chunked(mace.ModelDesc(**params), blob, sysm)
    return params, sysm, blob, ref


def test_cfg1_full_fp32(cfg1):
    params, sysm, blob, ref = cfg1
    gpu = run_gpu(params, sysm, blob, stress=True)
    assert gpu["n_edges"] == len(ref["graph"].sender)
    # the chunked oracle against the whole-graph one is pinned on the CPU
    assert_parity(gpu, ref, B.MACE_FP32, "water1536 full")
    sref = oracle_stress(params, sysm, blob)
    err = stress_error(gpu["stress"], sref)
    print(f"[fullsize] water1536 stress rel {err:.3e} (pressure {-np.trace(sref[0]) / 3:.4e})", flush=True)
    assert err <= TOL[B.MACE_FP32]["forces"]


def test_cfg1_full_bf16(cfg1):
    params, sysm, blob, ref = cfg1
    gpu = run_gpu(params, sysm, blob, prec=B.MACE_BF16_LINEAR)
    assert_parity(gpu, ref, B.MACE_BF16_LINEAR, "water1536 full bf16")


# ------------------------------------------------------------------ stress inputs, every order of Eq. 27

def test_cfg1_full_stress_inputs_fp32():
    params, sysm, blob, ref = _stored_ref("water1536_k128_l1_stress")
    gpu = run_gpu(params, sysm, blob)
    assert_parity(gpu, ref, B.MACE_FP32, "water1536 stress inputs full")


# ------------------------------------------------------------------ larger periodic boxes, every atom

@pytest.mark.parametrize("prec", [B.MACE_FP32, B.MACE_BF16_LINEAR, B.MACE_FP16_LINEAR, B.MACE_BF16_RADIAL])
@pytest.mark.parametrize("name", ["water4608_k128_l1", "water36864_k128_l2"])
def test_large_water_every_atom_vs_fp64(name, prec):
    """Every atom against the stored FP64 reference, in every precision mode
    (at 36,864 atoms the waves of the l_h = 2 backward walk about 36
    receivers each: in the BF16-radial mode with the next tile's R product
    pipelined across them)."""
    params, sysm, blob, ref = _stored_ref(name)
    gpu = run_gpu(params, sysm, blob, prec=prec)
    print(f"[fullsize] {name}: {gpu['n_edges']} edges", flush=True)
    assert_parity(gpu, ref, prec, f"{name} every atom")


@pytest.mark.parametrize("prec", [B.MACE_BF16_LINEAR, B.MACE_FP16_LINEAR])
def test_large_water_16bit_linear_layouts_bitwise(prec):
    """On the 36,864-atom box the 16-bit modes fuse the first layer's linears
    and give the wide linear blocks eight node tiles; energies and forces
    equal those of the plain layout (three launches, four tiles) bit for bit."""
    params = model_params(3)
    sysm = make_system(3, seed=0)
    blob = lib_blob(params, 0)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells)
    g = MaceGraph(B.make_desc(**params), blob, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                  sh, sysm.cells, None, 1, prec)
    pos = torch.from_numpy(sysm.positions.astype(np.float32)).cuda()
    outs = []
    for layout in (3, 0):
        assert B.mace_debug_fused_linears(g.handle, layout) == layout
        eps, E, F = g.energy_forces(pos)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy() for t in (eps, E, F)])
    g.close()
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("cfg", [2, 3])
def test_large_water_properties(cfg):
    params = model_params(cfg)
    sysm = make_system(cfg, seed=0)
    blob = lib_blob(params, 0)
    g32 = run_gpu(params, sysm, blob)
    N = sysm.n_atoms
    F = g32["forces"]
    # sum of forces vanishes (translation invariance)
    assert np.abs(F.sum(0)).max() <= 1e-5 * np.abs(F).max() * np.sqrt(N)
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
