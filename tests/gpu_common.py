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
       B.MACE_FP16_LINEAR: dict(energy=5e-3, forces=2e-2), B.MACE_BF16_RADIAL: dict(energy=5e-3, forces=2e-2),
       B.MACE_FP64: dict(energy=1e-10, forces=1e-10)}

# Per-atom bounds, asserted beside the aggregate ones: the worst atom energy
# relative to the mean |eps_i|, and the worst per-atom force error relative to
# the largest force. They catch a wrong atom (an O(1) error) that the
# aggregates average away. Set from the unit roundoff u of the format that
# rounds (FP32 2^-24, bfloat16 2^-8) times the depth of the computation an
# atom's energy goes through: FP32 300 u = 1.8e-5; 16-bit linears
# (and the bfloat16 radial layer) 25 u_bf16 = 0.1.
PER_ATOM_TOL = {B.MACE_FP64: dict(energy=1e-10, forces=1e-10),
                B.MACE_FP32: dict(energy=2e-5, forces=2e-5),
                B.MACE_BF16_LINEAR: dict(energy=0.1, forces=0.1),
                B.MACE_FP16_LINEAR: dict(energy=0.1, forces=0.1),
                B.MACE_BF16_RADIAL: dict(energy=0.1, forces=0.1)}


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
    if l0_form is not None:
        B.mace_layer0_form(g.handle, l0_form)
    if radial is not None:
        B.mace_fp32_products(g.handle, radial)
    for blk, fmt in (rounding or {}).items():
        B.mace_block_rounding(g.handle, blk, fmt)
    form = B.mace_layer0_form(g.handle, -1)   # the form the calls below run
    pos = torch.from_numpy(system.positions.astype(np.float64 if prec == B.MACE_FP64 else np.float32)).cuda()
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
    """energy: max over graphs |E_g - E_g^ref| / sum_i |eps_i^ref|;
    eps_l2: ||eps - eps^ref||_2 / ||eps^ref||_2;
    eps_max: max_i |eps_i - eps_i^ref| / mean_i |eps_i^ref| (worst atom);
    rae_e: |sum E - sum E^ref| / |sum E^ref| (the paper's RAE_E, reported only:
    it is unbounded where the total energy of random weights is near zero);
    forces: ||F - F^ref||_F / ||F^ref||_F (the paper's RAE_F);
    f_max: max_a ||f_a - f_a^ref|| / max_a ||f_a^ref|| (worst atom)."""
    eps_g, eps_r = gpu["eps"], ref["eps"]
    scale = np.abs(eps_r).sum()
    de = np.abs(eps_g - eps_r)
    out = dict(
        energy=float(np.abs(gpu["energy"] - ref["energy"]).max() / max(scale, 1e-300)),
        eps_l2=float(np.linalg.norm(eps_g - eps_r) / max(np.linalg.norm(eps_r), 1e-300)),
        eps_max=float(de.max() / max(np.abs(eps_r).mean(), 1e-300)) if len(de) else 0.0,
        rae_e=float(abs(np.sum(gpu["energy"]) - np.sum(ref["energy"])) / max(abs(np.sum(ref["energy"])), 1e-300)),
    )
    if gpu.get("forces") is not None and ref.get("forces") is not None:
        dF = gpu["forces"] - ref["forces"]
        out["forces"] = float(np.linalg.norm(dF) / max(np.linalg.norm(ref["forces"]), 1e-300))
        fmax = np.linalg.norm(ref["forces"], axis=1).max() if len(dF) else 0.0
        out["f_max"] = float(np.linalg.norm(dF, axis=1).max() / max(fmax, 1e-300)) if len(dF) else 0.0
    return out


def assert_parity(gpu: dict, ref: dict, prec, label="", per_atom=True):
    """Aggregate bounds (TOL) and, unless per_atom is False, the per-atom
    bounds (PER_ATOM_TOL)."""
    err = errors(gpu, ref)
    tol = TOL[prec]
    print(f"[parity] {label} prec={prec} " + " ".join(f"{k}={v:.3e}" for k, v in err.items()), flush=True)
    assert err["energy"] <= tol["energy"], (label, err)
    if "forces" in err:
        assert err["forces"] <= tol["forces"], (label, err)
    if per_atom:
        pt = PER_ATOM_TOL[prec]
        assert err["eps_max"] <= pt["energy"], (label, "per-atom energy", err)
        if "f_max" in err:
            assert err["f_max"] <= pt["forces"], (label, "per-atom force", err)
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
