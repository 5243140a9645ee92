"""The last radial layer on split-BF16 operands (each FP32 operand as three
bfloat16 parts, six partial products, FP32 accumulation) against the same
layer on FP32 MFMA and against the FP64 oracle, in the FP32 and the
16-bit-linear modes, for hidden l <= 0, 1, 2 (the three edge-product kernels)."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")
from gpu_common import (  # noqa: E402
    STRESS, STRESS_GAINS, assert_parity, errors, lib_blob, oracle_blob, run_gpu, run_oracle)


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("K,hl", [(32, 0), (128, 1), (64, 2)])
def test_split_bf16_matches_fp32_and_oracle(K, hl):
    params = model_params(0, K=K, hidden_lmax=hl, **STRESS)
    bo, bl = oracle_blob(params, 6, STRESS_GAINS), lib_blob(params, 6, STRESS_GAINS)
    sysm = synth.water_box(34, seed=5, box=10.0)
    ref = run_oracle(params, sysm, bo)
    # both forms of layer 0, so that layer 0's edge product (P = 4) runs too
    for form in (B.MACE_L0_EDGE, B.MACE_L0_FACTORED):
        plain = run_gpu(params, sysm, bl, B.MACE_FP32, l0_form=form, radial=B.MACE_PRODUCTS_FP32)
        split = run_gpu(params, sysm, bl, B.MACE_FP32, l0_form=form, radial=B.MACE_PRODUCTS_SPLIT_BF16)
        assert_parity(plain, ref, B.MACE_FP32, f"radial fp32 K={K} hl={hl} form={form}")
        assert_parity(split, ref, B.MACE_FP32, f"radial split-bf16 K={K} hl={hl} form={form}")
        err = errors(split, plain)
        print(f"[parity] split-bf16 vs fp32 radial K={K} hl={hl} form={form} {err}", flush=True)
        assert err["energy"] <= 1e-6 and err["forces"] <= 1e-5, err


def test_split_bf16_default_and_modes():
    params = model_params(0, K=64, hidden_lmax=1, **STRESS)
    bl = lib_blob(params, 2, STRESS_GAINS)
    bo = oracle_blob(params, 2, STRESS_GAINS)
    sysm = make_system(0, seed=4)
    snd, rcv, sh = B.mace_neighbor_list(sysm.positions, params["r_cut"], sysm.cells, None, 1)
    from paper_2510_23621_amd.graph import MaceGraph
    for prec, want in ((B.MACE_FP32, 2), (B.MACE_BF16_LINEAR, 2), (B.MACE_FP16_LINEAR, 2), (B.MACE_BF16_RADIAL, 1)):
        g = MaceGraph(B.make_desc(**params), bl, sysm.species.astype(np.int32), np.stack([snd, rcv]).astype(np.int32),
                      sh, sysm.cells, None, 1, prec)
        assert B.mace_fp32_products(g.handle, -1) == want
        if prec == B.MACE_BF16_RADIAL:
            with pytest.raises(B.MaceError):
                B.mace_fp32_products(g.handle, B.MACE_PRODUCTS_FP32)
        g.close()
    # 16-bit-linear mode with the split radial layer against the mode's emulation
    emu = run_oracle(params, sysm, bo, bf16=True)
    for radial in (B.MACE_PRODUCTS_FP32, B.MACE_PRODUCTS_SPLIT_BF16):
        g = run_gpu(params, sysm, bl, B.MACE_BF16_LINEAR, l0_form=B.MACE_L0_EDGE, radial=radial)
        err = errors(g, emu)
        print(f"[parity] bf16-linear radial={radial} vs emulation {err}", flush=True)
        assert err["energy"] <= 1e-3 and err["forces"] <= 1e-2, err
