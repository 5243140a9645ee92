"""Pins for the oracle's large-graph routes (CPU).

* The two-pass chunked vector-Jacobian product equals the whole-graph
  autograd evaluation (energies and forces within 1e-12 relative) for every
  model shape of the workloads (hidden 0e, 0e+1o, 0e+1o+2e), in FP64 and in
  the BF16-linear emulation, with chunks small enough that every receiver's
  edges and the node set span several chunks. It is exact up to summation
  order because the neighbour sum of Eq. 26 is linear in the edge messages
  and every step after it acts node by node.
* The stress inputs (c_norm 1, last radial layer x4) make every correlation
  order of Eq. 27 contribute: each order's share of |B| is at least 1e-3 at
  every layer and output irrep, for the full-size 1536-atom case and for
  the small cases the GPU parity tests run with those inputs. At the nominal
  inputs the higher orders are negligible (asserted too, so that no test
  claims them).
* The stored FP64 references of the full-size GPU tests carry the
  fingerprint of the inputs they were written for.
"""
import os
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import mace
from synth.configs import make_system, model_params

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
import make_fullsize_refs as refs  # noqa: E402

STRESS = dict(c_norm=1.0)
STRESS_GAINS = {".radial.3": 4.0}


def _rel(a, b):
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


@pytest.mark.parametrize("cfg,stress,bf16", [(0, True, False), (0, False, True), (1, False, False),
                                             (1, True, True), (3, True, False), (3, False, True)])
def test_chunked_vjp_equals_whole_graph_autograd(cfg, stress, bf16):
    torch.set_num_threads(min(8, os.cpu_count() or 1))
    params = model_params(cfg, **(STRESS if stress else {}))
    d = mace.ModelDesc(**params)
    # the workload's model on a 96-atom box (the full boxes take minutes each)
    sysm = make_system(0, seed=1) if cfg == 0 else synth.water_box(32, seed=3)
    blob = synth.weight_blob(mace.weight_layout(d), 2, STRESS_GAINS if stress else None)
    g = mace.build_graph(sysm, d)
    whole = mace.energy_forces(d, blob, sysm, graph=g, bf16_linear=bf16)
    chunk = mace.energy_forces_chunked(d, blob, sysm, graph=g, bf16_linear=bf16, edge_chunk=613, node_chunk=7)
    assert len(g.sender) > 7 * 613
    assert _rel(chunk["eps"], whole["eps"]) <= 1e-12
    assert _rel(chunk["energy"], whole["energy"]) <= 1e-12
    assert _rel(chunk["forces"], whole["forces"]) <= 1e-12


def test_chunked_vjp_matches_finite_differences():
    """Independent of the whole-graph route: central differences of the
    chunked oracle's own energy."""
    params = model_params(3, **STRESS)
    d = mace.ModelDesc(**params)
    sysm = synth.water_box(8, seed=5, box=6.5)
    blob = synth.weight_blob(mace.weight_layout(d), 4, STRESS_GAINS)
    g = mace.build_graph(sysm, d)
    out = mace.energy_forces_chunked(d, blob, sysm, graph=g, edge_chunk=97, node_chunk=5)
    h = 1e-5
    for a, c in ((0, 0), (5, 2), (17, 1)):
        vals = []
        for sgn in (1, -1):
            p = sysm.positions.copy()
            p[a, c] += sgn * h
            s2 = synth.System(p, sysm.species, sysm.cells, sysm.graph_of_atom, 1)
            vals.append(mace.energy_forces(d, blob, s2, graph=g, forces=False)["energy"].sum())
        fd = -(vals[0] - vals[1]) / (2 * h)
        assert abs(fd - out["forces"][a, c]) <= 1e-6 * max(1.0, np.abs(out["forces"]).max())


def _assert_shares(shares, floor, label):
    for t, per_l in shares.items():
        for L, per_nu in per_l.items():
            for nu, v in per_nu.items():
                assert v >= floor, (label, t, L, nu, v)


def test_stress_inputs_exercise_every_correlation_order_full_size():
    torch.set_num_threads(min(8, os.cpu_count() or 1))
    params, sysm, blob = refs.workload("water1536_k128_l1_stress")
    shares = mace.contraction_order_shares(mace.ModelDesc(**params), blob, sysm)
    print("[shares] water1536 stress inputs", shares)
    _assert_shares(shares, 1e-3, "water1536 stress inputs")


@pytest.mark.parametrize("K,hl,system", [(32, 0, "cfg0"), (64, 1, "cfg0"), (128, 2, "water102"), (32, 2, "water102")])
def test_stress_inputs_exercise_every_correlation_order_small(K, hl, system):
    params = model_params(0, K=K, hidden_lmax=hl, **STRESS)
    sysm = make_system(0, seed=2) if system == "cfg0" else synth.water_box(34, seed=7, box=10.0)
    blob = synth.weight_blob(mace.weight_layout(mace.ModelDesc(**params)), 3, STRESS_GAINS)
    shares = mace.contraction_order_shares(mace.ModelDesc(**params), blob, sysm)
    _assert_shares(shares, 1e-3, f"{system} K={K} l={hl}")


def test_nominal_inputs_leave_higher_orders_negligible():
    """Why the stress inputs exist: at c_norm = 52.5 and N(0,1)/sqrt(fan_in)
    weights the nu = 3 term is below 1e-3 of |B| at the second layer."""
    params = model_params(0)
    sysm = make_system(0, seed=0)
    blob = synth.weight_blob(mace.weight_layout(mace.ModelDesc(**params)), 0)
    shares = mace.contraction_order_shares(mace.ModelDesc(**params), blob, sysm)
    assert shares[1][0][3] < 1e-3


@pytest.mark.parametrize("name", sorted(refs.REFS))
def test_stored_reference_matches_its_inputs(name):
    path = refs.ref_path(name)
    if not os.path.exists(path):
        pytest.skip(f"{os.path.basename(path)} not generated")
    from oracle.neighbors import neighbor_list
    params, sysm, blob = refs.workload(name)
    z = np.load(path)
    if sysm.n_atoms > 5000:
        # the brute-force list of the largest box takes minutes: check the
        # seeded inputs and sizes, the edge list is checked on the GPU side
        assert z["eps"].shape == (sysm.n_atoms,) and z["forces"].shape == (sysm.n_atoms, 3)
        return
    s, r, S = neighbor_list(sysm.positions, params["r_cut"], sysm.cells, sysm.graph_of_atom)
    assert refs.fingerprint(sysm, blob, s, r, S) == str(z["fingerprint"])
    assert z["eps"].shape == (sysm.n_atoms,) and np.isfinite(z["forces"]).all()
    # sum of forces vanishes (translation invariance of the stored forces)
    assert np.abs(z["forces"].sum(0)).max() <= 1e-9 * np.abs(z["forces"]).max() * sysm.n_atoms
