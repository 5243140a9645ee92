"""Per-block precision study on the GPU (the paper's per-block low-precision
experiments, run on the whole model through the C ABI): the operands of the
edge product, of the symmetric contraction or of the radial MLP rounded to bfloat16 or binary16
(FP32 arithmetic), each against the oracle's emulation of the same rounding
and against FP64.  The printed deviations from FP64 are the study's result."""
import numpy as np
import pytest
import torch

from synth.configs import make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import errors, lib_blob, oracle_blob, run_gpu, run_oracle  # noqa: E402

BLOCKS = {B.MACE_BLOCK_EDGE_PRODUCT: "tp_round", B.MACE_BLOCK_SYMMETRIC_CONTRACTION: "symcon_round",
          B.MACE_BLOCK_RADIAL_MLP: "radial_round"}
FORMATS = {1: "bf16", 2: "fp16"}
# GPU (FP32 arithmetic on rounded FP32 values) against the FP64 emulation: the
# same roundings up to a value that sits within FP32 rounding of a 16-bit
# rounding boundary (measured: 1e-9 to 3e-7 on energies, up to 2e-6 for the
# radial MLP's binary16 arm, 5e-7 on forces)
EMU_TOL = {1: (1e-5, 1e-4), 2: (1e-5, 1e-4)}


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def case():
    params = model_params(0, K=64, hidden_lmax=1)
    return params, oracle_blob(params, 3), lib_blob(params, 3), make_system(0, seed=6)


@pytest.mark.parametrize("block", list(BLOCKS))
def test_block_rounding_against_emulation_and_fp64(case, block):
    params, bo, bl, sysm = case
    ref = run_oracle(params, sysm, bo)
    dev = {}
    for fmt, name in FORMATS.items():
        g = run_gpu(params, sysm, bl, B.MACE_FP32, rounding={block: fmt})
        emu = run_oracle(params, sysm, bo, **{BLOCKS[block]: name})
        e_emu, e_64, own = errors(g, emu), errors(g, ref), errors(emu, ref)
        print(f"[study] {BLOCKS[block]}={name}: gpu vs fp64 {e_64}; emulation vs fp64 {own}; gpu vs emulation "
              f"{e_emu}", flush=True)
        assert e_emu["energy"] <= EMU_TOL[fmt][0] and e_emu["forces"] <= EMU_TOL[fmt][1], e_emu
        # the GPU is as far from FP64 as the emulation says the rounding moves it
        assert e_64["forces"] <= 2 * own["forces"] + 1e-5, (e_64, own)
        dev[name] = e_64["forces"]
    assert dev["fp16"] < dev["bf16"], dev
    plain = run_gpu(params, sysm, bl, B.MACE_FP32)
    assert errors(plain, ref)["forces"] < dev["fp16"]


def test_block_rounding_setting_and_combination(case):
    """The setting is per handle and queryable; it combines with the
    BF16-linear mode (against the emulation of both), and switching it back
    off restores the FP32 results bit for bit."""
    params, bo, bl, sysm = case
    base = run_gpu(params, sysm, bl, B.MACE_FP32)
    both = run_gpu(params, sysm, bl, B.MACE_BF16_LINEAR, rounding={B.MACE_BLOCK_EDGE_PRODUCT: 1,
                                                                  B.MACE_BLOCK_SYMMETRIC_CONTRACTION: 1})
    emu = run_oracle(params, sysm, bo, bf16=True, tp_round="bf16", symcon_round="bf16")
    err = errors(both, emu)
    print(f"[study] bf16-linear + both blocks bf16: gpu vs emulation {err}", flush=True)
    assert err["energy"] <= 2e-3 and err["forces"] <= 2e-2, err
    off = run_gpu(params, sysm, bl, B.MACE_FP32, rounding={B.MACE_BLOCK_EDGE_PRODUCT: 0,
                                                          B.MACE_BLOCK_SYMMETRIC_CONTRACTION: 0})
    assert np.array_equal(off["forces"], base["forces"]) and np.array_equal(off["eps"], base["eps"])
    from paper_2510_23621_amd.graph import MaceGraph
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells, None, 1)
    g = MaceGraph(B.make_desc(**params), bl, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                  sh, sysm.cells, None, 1, B.MACE_FP32)
    assert B.mace_block_rounding(g.handle, B.MACE_BLOCK_EDGE_PRODUCT) == 0
    assert B.mace_block_rounding(g.handle, B.MACE_BLOCK_EDGE_PRODUCT, 2) == 2
    assert B.mace_block_rounding(g.handle, B.MACE_BLOCK_SYMMETRIC_CONTRACTION) == 0
    assert B.mace_block_rounding(g.handle, B.MACE_BLOCK_RADIAL_MLP, 1) == 1
    assert B.mace_block_rounding(g.handle, B.MACE_BLOCK_RADIAL_MLP) == 1
    with pytest.raises(B.MaceError):
        B.mace_block_rounding(g.handle, 7, 1)
    with pytest.raises(B.MaceError):
        B.mace_block_rounding(g.handle, B.MACE_BLOCK_EDGE_PRODUCT, 3)
    g.close()


def test_study_table_on_one_case(case):
    """Every precision arm on the same case, against FP64 (the study's table):
    each 16-bit arm is further from FP64 than FP32 and within the 16-bit
    tolerances."""
    params, bo, bl, sysm = case
    ref = run_oracle(params, sysm, bo)
    arms = [("fp32", B.MACE_FP32, None), ("bf16 linears", B.MACE_BF16_LINEAR, None),
            ("fp16 linears", B.MACE_FP16_LINEAR, None), ("bf16 linears + radial", B.MACE_BF16_RADIAL, None)]
    for blk, key in BLOCKS.items():
        for fmt, name in FORMATS.items():
            arms.append((f"{key[:-6]} {name}", B.MACE_FP32, {blk: fmt}))
    base = None
    for label, prec, rounding in arms:
        err = errors(run_gpu(params, sysm, bl, prec, rounding=rounding), ref)
        print(f"[study-table] {label:24s} energy {err['energy']:.2e} eps_l2 {err['eps_l2']:.2e} "
              f"forces {err['forces']:.2e}", flush=True)
        if base is None:
            base = err
            continue
        assert base["forces"] < err["forces"] <= 2e-2 and err["energy"] <= 5e-3, (label, err)
