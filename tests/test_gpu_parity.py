"""Parity of the HIP path (through the C ABI) against the FP64 oracle on the
same seeded inputs: energies within 1e-6 (FP32) / 5e-3 (BF16-linear) of
sum_i |eps_i|, forces within 1e-5 / 2e-2 relative RMS.  Sizes span several
node tiles and ragged tails; edge cases: empty neighbourhoods, isolated
atoms, a batch of graphs, determinism.
"""
import numpy as np
import pytest
import torch

import synth
from synth.configs import CONFIGS, make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (  # noqa: E402
    STRESS, STRESS_GAINS, TOL, assert_parity, errors, lib_blob, oracle_blob, oracle_stress, run_gpu, run_oracle,
    stress_error)


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _case(cfg, seed=0, gains=None, **kw):
    params = model_params(cfg, **kw)
    blob_o = oracle_blob(params, seed, gains)
    blob_l = lib_blob(params, seed, gains)
    assert np.array_equal(blob_o, blob_l)
    return params, blob_o, blob_l


def test_cfg0_nominal_fp32():
    params, bo, bl = _case(0)
    sysm = make_system(0, seed=0)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert gpu["n_edges"] == len(ref["graph"].sender)
    assert_parity(gpu, ref, B.MACE_FP32, "cfg0 nominal")


def test_cfg0_stress_fp32():
    params, bo, bl = _case(0, gains=STRESS_GAINS, **STRESS)
    sysm = make_system(0, seed=1)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert_parity(gpu, ref, B.MACE_FP32, "cfg0 stress")


@pytest.mark.parametrize("K,hl", [(64, 1), (96, 1), (128, 1), (128, 2), (32, 2)])
def test_small_water_variants_fp32(K, hl):
    """34 molecules = 102 atoms: species tiles of 16 are ragged (34 O, 68 H)."""
    params = model_params(0, K=K, hidden_lmax=hl, **STRESS)
    bo = oracle_blob(params, 3, STRESS_GAINS)
    bl = lib_blob(params, 3, STRESS_GAINS)
    sysm = synth.water_box(34, seed=7, box=10.0)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert_parity(gpu, ref, B.MACE_FP32, f"water102 K={K} l={hl}")


def test_many_layers_fp32():
    """Six interaction layers: more than the four layers one launch of the
    edge prologue (geometry plus the radial hidden layers) takes, so the
    chunked launches are exercised; five linear readouts below the last layer,
    more than one readout launch takes, so the node energies are built over two
    launches; the backward accumulates dE/dY and dE/de over six layers."""
    params = model_params(0, K=32, hidden_lmax=1, n_layers=6, **STRESS)
    bo = oracle_blob(params, 5, STRESS_GAINS)
    bl = lib_blob(params, 5, STRESS_GAINS)
    sysm = synth.water_box(12, seed=11, box=7.5)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert_parity(gpu, ref, B.MACE_FP32, "water36 six layers")


def test_molecule_batch_fp32_and_bf16():
    params = model_params(4, K=64, **STRESS)
    bo = oracle_blob(params, 4, STRESS_GAINS)
    bl = lib_blob(params, 4, STRESS_GAINS)
    sysm = synth.molecule_batch(12, seed=2)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert gpu["energy"].shape == (12,)
    assert_parity(gpu, ref, B.MACE_FP32, "molecules12")
    gpu16 = run_gpu(params, sysm, bl, prec=B.MACE_BF16_LINEAR)
    assert_parity(gpu16, ref, B.MACE_BF16_LINEAR, "molecules12 bf16 vs fp64")


def test_bf16_linear_vs_fp64_and_fp32():
    params, bo, bl = _case(0, gains=STRESS_GAINS, **STRESS)
    sysm = make_system(0, seed=2)
    ref = run_oracle(params, sysm, bo)
    g32 = run_gpu(params, sysm, bl)
    g16 = run_gpu(params, sysm, bl, prec=B.MACE_BF16_LINEAR)
    assert_parity(g16, ref, B.MACE_BF16_LINEAR, "cfg0 bf16 vs fp64")
    assert_parity(g16, g32, B.MACE_BF16_LINEAR, "cfg0 bf16 vs gpu fp32")
    # the oracle's own BF16 emulation lands in the same band
    ref16 = run_oracle(params, sysm, bo, bf16=True)
    err = errors(g16, ref16)
    print("[parity] bf16 gpu vs bf16-emulating oracle", err, flush=True)
    assert err["energy"] < 5e-3


@pytest.mark.parametrize("hl", [(2, 1), (2, 0), (1, 1, 0)])
def test_per_layer_hidden_lmax_fp32(hl):
    """One hidden l_max per layer: the edge product of each layer runs at its
    own l_h (2 then 1, 2 then 0, ...), with the residual species linear on the
    irreps a layer shares with its input."""
    params = model_params(0, K=32, n_layers=len(hl) + 1, hidden_lmax=hl, **STRESS)
    bo = oracle_blob(params, 4, STRESS_GAINS)
    bl = lib_blob(params, 4, STRESS_GAINS)
    assert np.array_equal(bo, bl)
    sysm = synth.water_box(34, seed=7, box=10.0)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert_parity(gpu, ref, B.MACE_FP32, f"hidden l_max per layer {hl}")


def test_isolated_atoms_and_empty_neighbourhoods():
    """Atoms with no neighbour (and a graph with no edge at all) get the
    species-only energy and zero force."""
    params = model_params(4, K=32, **STRESS)
    bo = oracle_blob(params, 5, STRESS_GAINS)
    bl = lib_blob(params, 5, STRESS_GAINS)
    pos = np.array([[0.0, 0, 0], [1.2, 0.1, 0], [30.0, 0, 0], [60.0, 1.0, 2.0], [200.0, 0, 0]])
    sysm = synth.System(pos, np.array([0, 1, 2, 3, 4], np.int32), None, np.array([0, 0, 0, 1, 2], np.int32), 3)
    ref = run_oracle(params, sysm, bo)
    gpu = run_gpu(params, sysm, bl)
    assert_parity(gpu, ref, B.MACE_FP32, "isolated")
    assert np.all(gpu["forces"][2:] == 0.0)
    lone = synth.System(pos[4:], np.array([3], np.int32), None, np.zeros(1, np.int32), 1)
    ref1 = run_oracle(params, lone, bo)
    gpu1 = run_gpu(params, lone, bl)
    assert gpu1["n_edges"] == 0
    assert abs(gpu1["energy"][0] - ref1["energy"][0]) <= 1e-6 * max(1e-30, abs(ref1["energy"][0]))


def test_deterministic_bitwise():
    params, bo, bl = _case(0, gains=STRESS_GAINS, **STRESS)
    sysm = make_system(0, seed=3)
    outs = run_gpu(params, sysm, bl, repeats=3)
    for o in outs[1:]:
        assert np.array_equal(o["eps"], outs[0]["eps"])
        assert np.array_equal(o["energy"], outs[0]["energy"])
        assert np.array_equal(o["forces"], outs[0]["forces"])
    e_only = run_gpu(params, sysm, bl, forces=False)
    assert np.array_equal(e_only["eps"], outs[0]["eps"])


def test_forces_sum_to_zero_on_gpu():
    params, bo, bl = _case(1, gains=STRESS_GAINS, **STRESS)
    sysm = make_system(1, seed=0)
    gpu = run_gpu(params, sysm, bl)
    F = gpu["forces"]
    assert np.abs(F.sum(0)).max() <= 1e-4 * np.abs(F).max() * np.sqrt(len(F))


@pytest.mark.parametrize("case", ["water96_nominal", "water96_stress_inputs", "molecules12"])
def test_stress_against_oracle(case):
    """Per-graph stress sigma = (1/V) dE/d(epsilon) (the oracle by autograd
    through a homogeneous strain) at the force tolerance; a batch of
    molecules (no cell, V = 1) checks the per-graph segmentation. FP32 is
    compared with the FP64 oracle; BF16-linear with the oracle's BF16
    emulation (a pressure is a small residual of large edge terms, so the
    model's own BF16 deviation from FP64 can exceed the force tolerance)."""
    if case == "molecules12":
        params = model_params(4, K=64, **STRESS)
        sysm = synth.molecule_batch(12, seed=2)
        gains = STRESS_GAINS
    else:
        params = model_params(0) if case == "water96_nominal" else model_params(0, **STRESS)
        sysm = make_system(0, seed=0)
        gains = None if case == "water96_nominal" else STRESS_GAINS
    bo = oracle_blob(params, 6, gains)
    bl = lib_blob(params, 6, gains)
    ref64 = oracle_stress(params, sysm, bo)
    ref16 = oracle_stress(params, sysm, bo, bf16=True)
    for prec, ref in ((B.MACE_FP32, ref64), (B.MACE_BF16_LINEAR, ref16)):
        gpu = run_gpu(params, sysm, bl, prec=prec, stress=True)
        err = stress_error(gpu["stress"], ref)
        print(f"[parity] stress {case} prec={prec} rel {err:.3e} (vs FP64 {stress_error(gpu['stress'], ref64):.3e}) "
              f"|sigma| {np.abs(ref64).max():.3e}", flush=True)
        assert gpu["stress"].shape == ref.shape
        assert err <= TOL[prec]["forces"], (case, prec, err)
    again = run_gpu(params, sysm, bl, stress=True)
    assert np.array_equal(again["stress"], run_gpu(params, sysm, bl, stress=True)["stress"])


@pytest.mark.parametrize("case", ["water96_stress_inputs", "molecules12_k64"])
def test_fp16_linear_vs_fp64_and_emulation(case):
    """FP16-linear mode (binary16 inputs and weights of every channel-mixing
    linear, FP32 accumulation): against the FP64 oracle at the 16-bit
    tolerances, and against the oracle's FP16 emulation."""
    if case == "molecules12_k64":
        params = model_params(4, K=64, **STRESS)
        sysm = synth.molecule_batch(12, seed=2)
    else:
        params = model_params(0, **STRESS)
        sysm = make_system(0, seed=0)
    bo = oracle_blob(params, 7, STRESS_GAINS)
    bl = lib_blob(params, 7, STRESS_GAINS)
    ref = run_oracle(params, sysm, bo)
    g16 = run_gpu(params, sysm, bl, prec=B.MACE_FP16_LINEAR)
    assert_parity(g16, ref, B.MACE_FP16_LINEAR, f"{case} fp16 vs fp64")
    emu = run_oracle(params, sysm, bo, fp16=True)
    err = errors(g16, emu)
    print(f"[parity] {case} fp16 gpu vs fp16-emulating oracle {err}", flush=True)
    assert err["energy"] <= 5e-4 and err["forces"] <= 5e-3, err
    # binary16 keeps three more significand bits than bfloat16
    gb = run_gpu(params, sysm, bl, prec=B.MACE_BF16_LINEAR)
    assert errors(g16, ref)["forces"] < errors(gb, ref)["forces"]


@pytest.mark.parametrize("case", ["water96_stress_inputs", "water102_k128_l2", "molecules12_k64"])
def test_bf16_radial_vs_fp64_and_emulation(case):
    """BF16-radial mode (BF16-linear, and the wide last radial layer on BF16
    MFMA in both directions): against the FP64 oracle at the 16-bit
    tolerances, and against the oracle's emulation (which does not round dE/dR
    in the backward product, hence the looser force bound)."""
    if case == "molecules12_k64":
        params = model_params(4, K=64, **STRESS)
        sysm = synth.molecule_batch(12, seed=2)
    elif case == "water102_k128_l2":
        params = model_params(0, K=128, hidden_lmax=2, **STRESS)
        sysm = synth.water_box(34, seed=7, box=10.0)
    else:
        params = model_params(0, **STRESS)
        sysm = make_system(0, seed=0)
    bo = oracle_blob(params, 8, STRESS_GAINS)
    bl = lib_blob(params, 8, STRESS_GAINS)
    ref = run_oracle(params, sysm, bo)
    gr = run_gpu(params, sysm, bl, prec=B.MACE_BF16_RADIAL, stress=True)
    assert_parity(gr, ref, B.MACE_BF16_RADIAL, f"{case} bf16-radial vs fp64")
    emu = run_oracle(params, sysm, bo, bf16_radial=True)
    err = errors(gr, emu)
    print(f"[parity] {case} bf16-radial gpu vs emulating oracle {err}", flush=True)
    assert err["energy"] <= 1e-3 and err["forces"] <= 1e-2, err
    if case == "water96_stress_inputs":
        se = stress_error(gr["stress"], oracle_stress(params, sysm, bo, bf16_radial=True))
        print(f"[parity] {case} bf16-radial stress vs emulating oracle {se:.3e}", flush=True)
        assert se <= 2e-2, se


def test_bf16_radial_waves_over_several_receivers():
    """The l_h = 2 backward of the BF16-radial mode forms the next tile's R
    product inside the current contraction, also across the receivers that
    one wave walks: 336 atoms at K = 128 give each wave two or three
    receivers, and six isolated atoms (empty receivers) sit where a wave's
    first receiver, and the receiver after a non-empty one, are empty."""
    params = model_params(0, K=128, hidden_lmax=2, **STRESS)
    w = synth.water_box(110, seed=3, box=15.0)
    pos, spec = w.positions.copy(), w.species.copy()
    isolated = [40, 41, 170, 171, 300, 301]
    for k, at in enumerate(isolated):
        pos = np.insert(pos, at, [500.0 + 60.0 * k, 7.0, -3.0], axis=0)
        spec = np.insert(spec, at, k % 2)
    sysm = synth.System(pos, spec.astype(np.int32), None, np.zeros(len(pos), np.int32), 1)
    bo = oracle_blob(params, 8, STRESS_GAINS)
    bl = lib_blob(params, 8, STRESS_GAINS)
    ref = run_oracle(params, sysm, bo)
    gr = run_gpu(params, sysm, bl, prec=B.MACE_BF16_RADIAL)
    assert gr["n_edges"] == len(ref["graph"].sender)
    assert_parity(gr, ref, B.MACE_BF16_RADIAL, "bf16-radial, several receivers per wave")
    assert np.all(gr["forces"][isolated] == 0.0)
    emu = run_oracle(params, sysm, bo, bf16_radial=True)
    err = errors(gr, emu)
    print(f"[parity] bf16-radial, several receivers per wave, vs emulating oracle {err}", flush=True)
    assert err["energy"] <= 1e-3 and err["forces"] <= 1e-2, err


def test_device_status_word_flags_bad_positions():
    """Device-detected errors: a NaN coordinate sets flag 1 (MACE_ENONFINITE),
    two atoms joined by an edge moved onto each other set flag 2
    (MACE_ERANGE); the check resets the word and a later good call reads
    clean, with the same outputs as before."""
    from paper_2510_23621_amd.graph import MaceGraph
    params = model_params(0)
    sysm = make_system(0, seed=0)
    bl = lib_blob(params, 8)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells)
    g = MaceGraph(B.make_desc(**params), bl, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                  sh, sysm.cells, None, 1, B.MACE_FP32)
    pos = torch.from_numpy(sysm.positions.astype(np.float32)).cuda()
    _, E0, F0 = g.energy_forces(pos)
    assert g.check() == (0, 0)
    bad = pos.clone()
    bad[5, 1] = float("nan")
    g.energy_forces(bad)
    code, flags = g.check()
    print(f"[status] nan position -> {code} {flags}", flush=True)
    assert flags & 1 and code == -5
    assert g.check() == (0, 0)
    # move the sender of an edge without periodic shift onto its receiver: d = 0
    e0 = int(np.flatnonzero((sh == 0).all(axis=1))[0])
    bad = pos.clone()
    bad[int(snd[e0])] = bad[int(rcv[e0])]
    g.energy(bad)
    code, flags = g.check()
    print(f"[status] coincident atoms -> {code} {flags}", flush=True)
    assert flags == 2 and code == -2
    _, E1, F1 = g.energy_forces(pos)
    assert g.check() == (0, 0)
    assert torch.equal(E0, E1) and torch.equal(F0, F1)
    g.close()

