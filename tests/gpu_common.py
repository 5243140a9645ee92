"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and the oracle on the same seeded inputs, and compare with the documented
metrics (energy error relative to sum_i |eps_i|, per-atom relative L2,
force relative RMS)."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import mace
from paper_2510_23621_amd import binding as B
from paper_2510_23621_amd.graph import MaceGraph

STRESS = dict(c_norm=1.0)
STRESS_GAINS = {".radial.3": 4.0}

TOL = {B.MACE_FP32: dict(energy=1e-6, forces=1e-5), B.MACE_BF16_LINEAR: dict(energy=5e-3, forces=2e-2),
       B.MACE_FP16_LINEAR: dict(energy=5e-3, forces=2e-2), B.MACE_BF16_RADIAL: dict(energy=5e-3, forces=2e-2)}


def lib_blob(params: dict, seed: int, gains=None) -> np.ndarray:
    lay, _ = B.mace_weight_layout(B.make_desc(**params))
    return synth.weight_blob([(name, (n,), f) for name, n, f in lay], seed, gains)


def oracle_blob(params: dict, seed: int, gains=None) -> np.ndarray:
    return synth.weight_blob(mace.weight_layout(mace.ModelDesc(**params)), seed, gains)


def run_gpu(params: dict, system, blob: np.ndarray, prec=B.MACE_FP32, forces=True, repeats=1, stress=False,
            l0_form=None, radial=None, rounding=None):
    desc = B.make_desc(**params)
    snd, rcv, sh = B.mace_neighbor_list(system.positions, params["r_cut"], system.cells, system.graph_of_atom,
                                        system.n_graphs)
    ei = np.stack([snd, rcv]).astype(np.int32)
    periodic = system.cells is not None
    g = MaceGraph(desc, blob, system.species.astype(np.int32), ei, sh if periodic else None,
                  system.cells if periodic else None,
                  system.graph_of_atom.astype(np.int32) if system.n_graphs > 1 else None, system.n_graphs, prec)
    form = B.mace_layer0_form(g.handle, -1 if l0_form is None else l0_form)
    if radial is not None:
        B.mace_fp32_products(g.handle, radial)
    for blk, fmt in (rounding or {}).items():
        B.mace_block_rounding(g.handle, blk, fmt)
    pos = torch.from_numpy(system.positions.astype(np.float32)).cuda()
    outs = []
    for _ in range(repeats):
        S = None
        if stress:
            eps, E, F, S = g.energy_forces_stress(pos)
        elif forces:
            eps, E, F = g.energy_forces(pos)
        else:
            (eps, E), F = g.energy(pos), None
        torch.cuda.synchronize()
        outs.append(dict(eps=eps.cpu().numpy().astype(np.float64), energy=E.cpu().numpy(),
                         forces=None if F is None else F.cpu().numpy().astype(np.float64), n_edges=len(snd),
                         stress=None if S is None else S.cpu().numpy(), l0_form=form))
    g.close()
    return outs if repeats > 1 else outs[0]


def run_oracle(params: dict, system, blob: np.ndarray, bf16=False, forces=True, fp16=False, bf16_radial=False,
               tp_round=None, symcon_round=None, radial_round=None):
    return mace.energy_forces(mace.ModelDesc(**params), blob, system, bf16_linear=bf16 or bf16_radial,
                              forces=forces, fp16_linear=fp16, bf16_radial=bf16_radial, tp_round=tp_round,
                              symcon_round=symcon_round, radial_round=radial_round)


def oracle_stress(params: dict, system, blob: np.ndarray, bf16=False, fp16=False, bf16_radial=False):
    return mace.stress(mace.ModelDesc(**params), blob, system, bf16_linear=bf16 or bf16_radial, fp16_linear=fp16,
                       bf16_radial=bf16_radial)


def stress_error(gpu_stress: np.ndarray, ref_stress: np.ndarray) -> float:
    """Relative Frobenius error over all graphs (the stress tolerance is the force one)."""
    return float(np.linalg.norm(gpu_stress - ref_stress) / max(np.linalg.norm(ref_stress), 1e-300))


def errors(gpu: dict, ref: dict) -> dict:
    eps_g, eps_r = gpu["eps"], ref["eps"]
    scale = np.abs(eps_r).sum()
    out = dict(
        energy=float(np.abs(gpu["energy"] - ref["energy"]).max() / max(scale, 1e-300)),
        eps_l2=float(np.linalg.norm(eps_g - eps_r) / max(np.linalg.norm(eps_r), 1e-300)),
    )
    if gpu.get("forces") is not None and ref.get("forces") is not None:
        out["forces"] = float(np.linalg.norm(gpu["forces"] - ref["forces"]) /
                              max(np.linalg.norm(ref["forces"]), 1e-300))
    return out


def assert_parity(gpu: dict, ref: dict, prec, label=""):
    err = errors(gpu, ref)
    tol = TOL[prec]
    print(f"[parity] {label} prec={prec} {err}", flush=True)
    assert err["energy"] <= tol["energy"], (label, err)
    if "forces" in err:
        assert err["forces"] <= tol["forces"], (label, err)
    return err


def cluster_cut(system, i, radius):
    """Non-periodic system of every image of every atom within `radius` of
    atom i (atom i first, at its own position)."""
    x0 = system.positions[i]
    if system.cells is None:
        g = system.graph_of_atom[i]
        idx = np.nonzero(system.graph_of_atom == g)[0]
        d = np.linalg.norm(system.positions[idx] - x0, axis=1)
        keep = idx[d < radius]
        keep = np.concatenate([[i], keep[keep != i]])
        return synth.System(system.positions[keep], system.species[keep], None, np.zeros(len(keep), np.int32), 1), keep
    cell = system.cells[0]
    L = np.linalg.norm(cell, axis=1).min()
    n = int(np.ceil(radius / L)) + 1
    pos, spec, src = [x0[None]], [system.species[i:i + 1]], [np.array([i])]
    for a in range(-n, n + 1):
        for b in range(-n, n + 1):
            for c in range(-n, n + 1):
                shift = a * cell[0] + b * cell[1] + c * cell[2]
                p = system.positions + shift
                d = np.linalg.norm(p - x0, axis=1)
                sel = d < radius
                if a == 0 and b == 0 and c == 0:
                    sel[i] = False
                pos.append(p[sel])
                spec.append(system.species[sel])
                src.append(np.nonzero(sel)[0])
    P = np.vstack(pos)
    return synth.System(P, np.concatenate(spec), None, np.zeros(len(P), np.int32), 1), np.concatenate(src)
