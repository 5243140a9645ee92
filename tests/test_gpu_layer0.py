"""The first interaction layer in both of its forms, through the C ABI: the
per-edge product (as every later layer) and the factorised one (the sum over
a receiver's edges of a3 (x) Y per sender species, then one node-level
contraction).  Both are checked against the FP64 oracle and, in the 16-bit
modes, against the oracle's emulation of the mode, and against each other;
the automatic choice follows the documented rule."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (  # noqa: E402
    STRESS, STRESS_GAINS, assert_parity, errors, lib_blob, oracle_blob, oracle_stress, run_gpu, run_oracle,
    stress_error)
from paper_2510_23621_amd.graph import MaceGraph  # noqa: E402

EMULATION = {B.MACE_BF16_LINEAR: dict(bf16=True), B.MACE_FP16_LINEAR: dict(fp16=True),
             B.MACE_BF16_RADIAL: dict(bf16_radial=True)}
# GPU vs the oracle's emulation of the mode (energy, forces), as in the mode tests
EMU_TOL = {B.MACE_BF16_LINEAR: (1e-3, 1e-2), B.MACE_FP16_LINEAR: (5e-4, 5e-3), B.MACE_BF16_RADIAL: (1e-3, 1e-2)}


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _water(K, hl, seed):
    params = model_params(0, K=K, hidden_lmax=hl, **STRESS)
    return params, oracle_blob(params, seed, STRESS_GAINS), lib_blob(params, seed, STRESS_GAINS)


@pytest.mark.parametrize("prec", [B.MACE_FP32, B.MACE_BF16_LINEAR, B.MACE_FP16_LINEAR, B.MACE_BF16_RADIAL])
@pytest.mark.parametrize("K,hl", [(64, 1), (128, 1), (32, 0)])
def test_both_forms_against_oracle(prec, K, hl):
    """96-atom periodic water, two species, every correlation order
    contributing: each form against FP64 (and the mode's emulation), and the
    two forms against each other."""
    params, bo, bl = _water(K, hl, 5)
    sysm = make_system(0, seed=2)
    ref = run_oracle(params, sysm, bo)
    emu = run_oracle(params, sysm, bo, **EMULATION[prec]) if prec in EMULATION else None
    out = {}
    for form in (B.MACE_L0_EDGE, B.MACE_L0_FACTORED):
        g = run_gpu(params, sysm, bl, prec, stress=True, l0_form=form)
        assert g["l0_form"] == form
        if emu is None:
            assert_parity(g, ref, prec, f"layer-0 form {form} K={K} hl={hl}")
        else:
            # with these O(1) inputs the 16-bit rounding itself can move the
            # result past the nominal bounds; the GPU may be no further from
            # FP64 than twice the mode's emulation is (or the nominal bound),
            # and the emulation check below is the tight one
            err, own = errors(g, ref), errors(emu, ref)
            print(f"[parity] layer-0 form {form} K={K} hl={hl} prec={prec} vs fp64 {err} (emulation {own})",
                  flush=True)
            for q, nominal in (("energy", 5e-3), ("forces", 2e-2)):
                assert err[q] <= max(nominal, 2 * own[q]), (q, err, own)
        se = stress_error(g["stress"], oracle_stress(params, sysm, bo, **(EMULATION.get(prec, {}))))
        print(f"[parity] layer-0 form {form} prec={prec} stress {se:.3e}", flush=True)
        assert se <= (1e-5 if prec == B.MACE_FP32 else 2e-2), se
        if emu is not None:
            err = errors(g, emu)
            print(f"[parity] layer-0 form {form} prec={prec} vs emulation {err}", flush=True)
            assert err["energy"] <= EMU_TOL[prec][0] and err["forces"] <= EMU_TOL[prec][1], err
        out[form] = g
    err = errors(out[B.MACE_L0_FACTORED], out[B.MACE_L0_EDGE])
    print(f"[parity] factorised vs per-edge prec={prec} {err}", flush=True)
    if prec == B.MACE_FP32:
        assert err["energy"] <= 1e-6 and err["forces"] <= 1e-5, err
    else:   # the two forms may round a 16-bit linear input to neighbouring values
        assert err["energy"] <= 1e-3 and err["forces"] <= 1e-2, err


def test_factorised_form_ragged_and_isolated():
    """Ragged species tiles (102 atoms), a receiver without neighbours and a
    one-species graph, in the factorised form."""
    params, bo, bl = _water(96, 1, 9)
    sysm = synth.water_box(34, seed=7, box=10.0)
    # move one atom far from every other (a receiver and sender of no edge)
    pos = sysm.positions.copy()
    sysm = synth.System(pos, sysm.species, None, np.zeros(len(pos), np.int32), 1)
    sysm.positions[0] = np.array([40.0, 40.0, 40.0])
    ref = run_oracle(params, sysm, bo)
    g = run_gpu(params, sysm, bl, B.MACE_FP32, l0_form=B.MACE_L0_FACTORED)
    assert_parity(g, ref, B.MACE_FP32, "factorised, isolated atom")
    one = synth.System(pos[:40].copy(), np.zeros(40, np.int32), None, np.zeros(40, np.int32), 1)
    ref1 = run_oracle(params, one, bo)
    g1 = run_gpu(params, one, bl, B.MACE_FP32, l0_form=B.MACE_L0_FACTORED)
    assert_parity(g1, ref1, B.MACE_FP32, "factorised, one species present")


def test_automatic_choice_and_rejection():
    """Setup picks the factorised form for dense water (E >= 3 S N) and the
    per-edge form for ten species; the factorised form is refused for S > 4."""
    params, _, bl = _water(64, 1, 1)
    sysm = make_system(0, seed=0)
    g = run_gpu(params, sysm, bl)
    assert g["l0_form"] == B.MACE_L0_FACTORED
    mparams = model_params(4, K=64, **STRESS)
    msys = synth.molecule_batch(6, seed=1)
    mblob = lib_blob(mparams, 2, STRESS_GAINS)
    snd, rcv, _ = B.mace_neighbor_list(msys.positions, mparams["r_cut"], None, msys.graph_of_atom, msys.n_graphs)
    mg = MaceGraph(B.make_desc(**mparams), mblob, msys.species.astype(np.int32),
                   np.stack([snd, rcv]).astype(np.int32), None, None, msys.graph_of_atom.astype(np.int32),
                   msys.n_graphs, B.MACE_FP32)
    assert B.mace_layer0_form(mg.handle, -1) == B.MACE_L0_EDGE
    with pytest.raises(B.MaceError) as ex:
        B.mace_layer0_form(mg.handle, B.MACE_L0_FACTORED)
    assert ex.value.code == -7
    assert B.mace_layer0_form(mg.handle, B.MACE_L0_EDGE) == B.MACE_L0_EDGE
    mg.close()


def test_factorised_form_deterministic():
    params, _, bl = _water(128, 1, 4)
    sysm = make_system(0, seed=1)
    outs = run_gpu(params, sysm, bl, B.MACE_FP32, repeats=3, l0_form=B.MACE_L0_FACTORED)
    for o in outs[1:]:
        assert np.array_equal(o["eps"], outs[0]["eps"]) and np.array_equal(o["forces"], outs[0]["forces"])


@pytest.mark.parametrize("prec", [B.MACE_BF16_LINEAR, B.MACE_FP16_LINEAR, B.MACE_BF16_RADIAL])
def test_fused_first_layer_linears_bitwise(prec):
    """In the 16-bit modes at K = 128 with two species the factorised first
    layer's three linears (and their transposes) run as one launch each way;
    energies, forces and stress equal those of the separate launches bit for
    bit, on a 1,536-atom box (24 node quads of mixed species) and on a
    96-atom one."""
    for cfg, seed in ((1, 0), (0, 3)):
        params = model_params(cfg, K=128, hidden_lmax=1, **STRESS)
        sysm = make_system(cfg, seed=seed)
        bl = lib_blob(params, seed, STRESS_GAINS)
        snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells)
        g = MaceGraph(B.make_desc(**params), bl, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                      sh, sysm.cells, None, 1, prec)
        assert B.mace_layer0_form(g.handle, -1) == B.MACE_L0_FACTORED
        pos = torch.from_numpy(sysm.positions.astype(np.float32)).cuda()
        outs = []
        for fuse in (3, 0, 3):
            assert B.mace_debug_fused_linears(g.handle, fuse) == (fuse & 1)   # no eight-tile blocks at these sizes
            eps, E, F, S = g.energy_forces_stress(pos)
            torch.cuda.synchronize()
            outs.append([t.cpu().numpy() for t in (eps, E, F, S)])
        for a, b in zip(outs[0], outs[1]):
            assert np.array_equal(a, b), f"cfg {cfg}: fused and separate first-layer linears differ"
        for a, b in zip(outs[0], outs[2]):
            assert np.array_equal(a, b)
        g.close()


def test_fused_first_layer_linears_only_where_shapes_allow():
    """FP32 composes the first layer's linears on the host (nothing to fuse);
    K = 64 and the per-edge first layer keep separate launches."""
    sysm = make_system(0, seed=0)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, 5.0, sysm.cells)
    for K, prec, form, want in ((128, B.MACE_FP32, None, 0), (64, B.MACE_BF16_LINEAR, None, 0),
                                (128, B.MACE_BF16_LINEAR, B.MACE_L0_EDGE, 0), (128, B.MACE_FP16_LINEAR, None, 1)):
        # (bit 1, eight node tiles per block, needs at least 256 four-tile blocks: not at 96 atoms)
        params = model_params(0, K=K, hidden_lmax=1)
        g = MaceGraph(B.make_desc(**params), lib_blob(params, 0), sysm.species.astype(np.int32),
                      np.stack([snd, rcv]).astype(np.int32), sh, sysm.cells, None, 1, prec)
        if form is not None:
            B.mace_layer0_form(g.handle, form)
        assert B.mace_debug_fused_linears(g.handle) == want, (K, prec, form)
        g.close()
    with pytest.raises(B.MaceError):
        B.mace_debug_fused_linears(None, 0)
