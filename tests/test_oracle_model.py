"""Pins for the oracle's radial basis, neighbour list and whole model (CPU).

Whole-model pins: E(3) invariance (rotation, translation, permutation,
inversion), forces = -central finite differences, sum F = 0, zero torque for
an isolated cluster, F = 0 on a perfect lattice, supercell identity, batch
independence, locality, cutoff continuity; brute-force per-edge loops for the
edge product and neighbour sum; brute force for the product basis; the
parameter counts printed in the appendix table.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import synth
from oracle import mace, so3
from oracle.neighbors import neighbor_list
from synth.configs import make_system, model_params

HERE = os.path.dirname(os.path.abspath(__file__))
STRESS = dict(c_norm=1.0)
STRESS_GAINS = {".radial.3": 4.0}


def _desc(cfg=0, **kw):
    return mace.ModelDesc(**model_params(cfg, **kw))


def _small_desc(hidden_lmax=1, K=8, S=2, rc=3.0, **kw):
    base = dict(n_species=S, K=K, hidden_lmax=hidden_lmax, r_cut=rc, c_norm=1.0)
    base.update(kw)
    return mace.ModelDesc(**base)


def _cluster(n, seed, S=2, box=None, radius=2.5):
    rng = np.random.default_rng(seed)
    pts = []
    while len(pts) < n:
        p = rng.uniform(-radius, radius, 3)
        if pts and np.min(np.linalg.norm(np.asarray(pts) - p, axis=1)) < 0.9:
            continue
        pts.append(p)
    pos = np.asarray(pts).astype(np.float32).astype(np.float64)
    spec = rng.integers(0, S, n).astype(np.int32)
    cells = None if box is None else np.diag([box] * 3)[None].astype(np.float64)
    if box is not None:
        pos = np.mod(pos, box)
    return synth.System(pos, spec, cells, np.zeros(n, np.int32), 1)


def _energy(d, blob, system, **kw):
    return mace.energy_forces(d, blob, system, forces=False, **kw)["energy"].sum()


# ------------------------------------------------------------------ radial

def test_bessel_closed_form_and_envelope():
    rc, p = 5.0, 5
    r = torch.tensor([0.7, 1.3, 2.9, 4.99], dtype=torch.float64)
    e = mace.bessel_basis(r, rc, 8, p).numpy()
    for i, rv in enumerate(r.numpy()):
        x = rv / rc
        u = 1 - 21 * x ** 5 + 35 * x ** 6 - 15 * x ** 7
        for n in range(1, 9):
            ref = math.sqrt(2 / rc) * math.sin(n * math.pi * rv / rc) / rv * u
            assert abs(e[i, n - 1] - ref) < 1e-14
    # u(1) = u'(1) = u''(1) = 0, u(0) = 1
    x = torch.tensor([1.0 - 1e-12], dtype=torch.float64, requires_grad=True)
    import sympy as sp
    X = sp.symbols("x")
    u = 1 - sp.Rational(21) * X ** 5 + 35 * X ** 6 - 15 * X ** 7
    assert u.subs(X, 1) == 0 and sp.diff(u, X).subs(X, 1) == 0 and sp.diff(u, X, 2).subs(X, 1) == 0
    assert float(mace.envelope(torch.tensor([0.0], dtype=torch.float64), p)) == 1.0
    assert float(mace.envelope(torch.tensor([1.0, 1.5], dtype=torch.float64), p).abs().sum()) == 0.0


# ------------------------------------------------------------------ neighbours

def _nl_pure_python(pos, rc, cell, nimg):
    out = []
    for i in range(len(pos)):
        for j in range(len(pos)):
            for S in itertools.product(range(-nimg, nimg + 1), repeat=3):
                sv = [((S[0] * cell[0][c]) + (S[1] * cell[1][c])) + (S[2] * cell[2][c]) for c in range(3)]
                d = [(pos[j][c] - pos[i][c]) + sv[c] for c in range(3)]
                r2 = (d[0] * d[0] + d[1] * d[1]) + d[2] * d[2]
                if 0.0 < r2 < rc * rc:
                    out.append((i, j, S[0], S[1], S[2]))
    return sorted(out)


def test_neighbor_list_brute_force_small_box():
    sysm = make_system(0, seed=3)
    pos = sysm.positions[:18]
    cell = sysm.cells[0]
    s, r, S = neighbor_list(pos, 5.0, sysm.cells, np.zeros(18, np.int32))
    got = sorted(zip(r.tolist(), s.tolist(), *S.T.tolist()))
    ref = _nl_pure_python(pos.tolist(), 5.0, cell.tolist(), 2)
    assert got == ref
    assert len(got) > 0


def test_neighbor_list_symmetry_and_density():
    sysm = make_system(0, seed=0)
    s, r, S = neighbor_list(sysm.positions, 5.0, sysm.cells, sysm.graph_of_atom)
    fwd = set(zip(s.tolist(), r.tolist(), map(tuple, S.tolist())))
    for a, b, sh in fwd:
        assert (b, a, tuple(-x for x in sh)) in fwd
    # rc = 5 > L/2: some pairs appear under several images
    pairs = list(zip(s.tolist(), r.tolist()))
    assert len(pairs) > len(set(pairs))
    deg = len(s) / sysm.n_atoms
    assert 40 < deg < 65       # 0.1 atoms/A^3 * 4/3 pi 125 = 52.5 expected


def test_neighbor_list_graphs_disjoint():
    sysm = synth.molecule_batch(3, seed=1)
    s, r, S = neighbor_list(sysm.positions, 5.0, None, sysm.graph_of_atom)
    assert np.all(sysm.graph_of_atom[s] == sysm.graph_of_atom[r])
    assert np.all(S == 0)
    assert np.all(np.diff(r) >= 0)


# ------------------------------------------------------------------ layout

def test_param_counts_match_appendix_table():
    gold = json.load(open(os.path.join(HERE, "golden", "param_counts_appendix.json")))
    m = gold["model"]
    d = mace.ModelDesc(n_species=m["n_species"], K=m["K"], hidden_lmax=m["hidden_lmax"],
                       r_cut=6.0, c_norm=1.0, n_layers=m["n_layers"])
    lay = {n: (shape, int(np.prod(shape))) for n, shape, _ in mace.weight_layout(d)}
    c = gold["counts"]

    def tot(prefix):
        return sum(v[1] for k, v in lay.items() if k.startswith(prefix))
    assert lay["embed"][1] == c["embed"]
    for t in (0, 1):
        assert tot(f"{t}.up.") == c[f"{t}.up"]
        assert len(mace.tp_paths(d, t)) == c[f"{t}.paths"]
        assert sum(2 * lo + 1 for (_, _, lo) in mace.tp_paths(d, t)) == c[f"{t}.mid"]
        widths = [lay[f"{t}.radial.0"][0][0]] + [lay[f"{t}.radial.{i}"][0][1] for i in range(4)]
        assert widths == c[f"{t}.radial_widths"]
        assert tot(f"{t}.linear.") == c[f"{t}.linear"]
        assert tot(f"{t}.skip.") == c[f"{t}.skip"]
        assert tot(f"{t}.prod.") == c[f"{t}.prod"]
        assert tot(f"{t}.readout") == c[f"{t}.readout"]


# ------------------------------------------------------------------ brute force pieces

def _edge_sum_loops(d, W, g, Y, Rall, ht, t):
    paths = mace.tp_paths(d, t)
    N = int(g.receiver.max()) + 1
    out = [np.zeros((N, 2 * lo + 1, d.K)) for (_, _, lo) in paths]
    for e in range(len(g.sender)):
        j, i = int(g.sender[e]), int(g.receiver[e])
        for p, (lh, ly, lo) in enumerate(paths):
            C = so3.real_cg(lh, ly, lo)
            for k in range(d.K):
                for m1 in range(2 * lh + 1):
                    for m2 in range(2 * ly + 1):
                        for m3 in range(2 * lo + 1):
                            out[p][i, m3, k] += (C[m1, m2, m3] * ht[lh][j, m1, k]
                                                 * Y[e, ly * ly + m2] * Rall[e, p, k])
    return [o / d.c_norm for o in out]


def test_edge_product_matches_loops():
    d = _small_desc(hidden_lmax=1, K=3, rc=3.5, c_norm=1.7)
    sysm = _cluster(5, seed=5, radius=1.6)
    W = mace.unpack_weights(d, synth.weight_blob(mace.weight_layout(d), 1, STRESS_GAINS))
    g = mace.build_graph(sysm, d)
    pos = torch.tensor(sysm.positions)
    eps, inter = mace.node_energies(d, W, g, pos, return_intermediates=True)
    t = 1
    paths = mace.tp_paths(d, t)
    h1 = inter["0.h"]
    ht = {l: (h1[l] @ W[f"{t}.up.{l}"]).numpy() for l in (0, 1)}
    Rall = mace.radial_mlp(inter["rbf"], W, t, 3).reshape(-1, len(paths), d.K).numpy()
    At = _edge_sum_loops(d, W, g, inter["Y"].numpy(), Rall, ht, t)
    # oracle A for layer 1 = sum_p At[p] @ W_linear[p] (no species linear at t >= 1)
    A = np.zeros((sysm.n_atoms, 16, d.K))
    for p, (_, _, lo) in enumerate(paths):
        A[:, lo * lo:lo * lo + 2 * lo + 1] += At[p] @ W[f"{t}.linear.{p}"].numpy()
    np.testing.assert_allclose(inter["1.A"].numpy(), A, rtol=1e-12, atol=1e-12)


def test_symmetric_contraction_brute_force():
    rng = np.random.default_rng(0)
    K, S = 2, 2
    A = torch.from_numpy(rng.standard_normal((3, 16, K)))
    z = torch.tensor([0, 1, 1])
    for L in (0, 1, 2):
        W = {}
        for nu in (1, 2, 3):
            W[f"0.symc.{L}.{nu}"] = torch.from_numpy(rng.standard_normal((S, so3.n_eta(nu, L), K)))
        B = mace.symmetric_contraction(A, W, 0, L, z, 3).numpy()
        ref = np.zeros_like(B)
        for n in range(3):
            for k in range(K):
                a = A[n, :, k].numpy()
                for nu in (1, 2, 3):
                    _, us = so3.u_basis(nu, L)
                    for eta, U in enumerate(us):
                        w = W[f"0.symc.{L}.{nu}"][z[n], eta, k].item()
                        for idx in itertools.product(range(16), repeat=nu):
                            prod = 1.0
                            for q in idx:
                                prod *= a[q]
                            ref[n, :, k] += w * U[(slice(None),) + idx] * prod
        np.testing.assert_allclose(B, ref, rtol=1e-11, atol=1e-12)


# ------------------------------------------------------------------ whole model

@pytest.fixture(scope="module")
def cfg0():
    d = _desc(0, **STRESS)
    blob = synth.weight_blob(mace.weight_layout(d), 0, STRESS_GAINS)
    sysm = make_system(0, seed=0)
    return d, blob, sysm


def _rotated(sysm, R, t=np.zeros(3), invert=False):
    M = -R if invert else R
    pos = sysm.positions @ M.T + t
    cells = None if sysm.cells is None else sysm.cells @ M.T
    return synth.System(pos, sysm.species, cells, sysm.graph_of_atom, sysm.n_graphs)


def test_invariance_rotation_translation_inversion(cfg0):
    d, blob, sysm = cfg0
    ref = mace.energy_forces(d, blob, sysm, forces=True)
    R = so3.random_rotation(np.random.default_rng(11))
    for inv in (False, True):
        rs = _rotated(sysm, R, t=np.array([0.3, -1.1, 2.0]), invert=inv)
        out = mace.energy_forces(d, blob, rs, forces=True)
        M = -R if inv else R
        np.testing.assert_allclose(out["eps"], ref["eps"], rtol=1e-9, atol=1e-10 * np.abs(ref["eps"]).max())
        np.testing.assert_allclose(out["forces"], ref["forces"] @ M.T, atol=1e-9 * np.abs(ref["forces"]).max())


def test_invariance_permutation(cfg0):
    d, blob, sysm = cfg0
    ref = mace.energy_forces(d, blob, sysm, forces=True)
    perm = np.random.default_rng(2).permutation(sysm.n_atoms)
    ps = synth.System(sysm.positions[perm], sysm.species[perm], sysm.cells, sysm.graph_of_atom, 1)
    out = mace.energy_forces(d, blob, ps, forces=True)
    np.testing.assert_allclose(out["eps"], ref["eps"][perm], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(out["forces"], ref["forces"][perm], rtol=1e-8, atol=1e-11)


def test_forces_finite_difference_and_sum():
    d = _small_desc(hidden_lmax=1, K=4, rc=3.0)
    sysm = _cluster(6, seed=9, radius=1.8)
    blob = synth.weight_blob(mace.weight_layout(d), 3, STRESS_GAINS)
    out = mace.energy_forces(d, blob, sysm)
    F = out["forces"]
    h = 1e-5
    for a in range(sysm.n_atoms):
        for c in range(3):
            sp, sm = [synth.System(sysm.positions.copy(), sysm.species, None, sysm.graph_of_atom, 1) for _ in range(2)]
            sp.positions[a, c] += h
            sm.positions[a, c] -= h
            fd = -(_energy(d, blob, sp) - _energy(d, blob, sm)) / (2 * h)
            assert abs(fd - F[a, c]) < 1e-6 * max(1.0, np.abs(F).max()), (a, c, fd, F[a, c])
    np.testing.assert_allclose(F.sum(0), 0, atol=1e-12 * max(1, np.abs(F).max()))
    torque = np.cross(sysm.positions, F).sum(0)
    np.testing.assert_allclose(torque, 0, atol=1e-11 * max(1, np.abs(F).max()))


def test_forces_periodic_fd(cfg0):
    d, blob, sysm = cfg0
    out = mace.energy_forces(d, blob, sysm)
    F = out["forces"]
    h = 1e-5
    for a, c in [(0, 0), (1, 2), (50, 1)]:
        sp = synth.System(sysm.positions.copy(), sysm.species, sysm.cells, sysm.graph_of_atom, 1)
        sm = synth.System(sysm.positions.copy(), sysm.species, sysm.cells, sysm.graph_of_atom, 1)
        sp.positions[a, c] += h
        sm.positions[a, c] -= h
        fd = -(_energy(d, blob, sp) - _energy(d, blob, sm)) / (2 * h)
        assert abs(fd - F[a, c]) < 1e-6 * np.abs(F).max()
    np.testing.assert_allclose(F.sum(0), 0, atol=1e-10 * np.abs(F).max())


def test_zero_force_perfect_lattice():
    d = _small_desc(hidden_lmax=1, K=4, S=1, rc=3.1)
    a = 2.0
    n = 3
    pos = np.array([(i, j, k) for i in range(n) for j in range(n) for k in range(n)], float) * a
    sysm = synth.System(pos, np.zeros(len(pos), np.int32), np.diag([a * n] * 3)[None], np.zeros(len(pos), np.int32), 1)
    out = mace.energy_forces(d, synth.weight_blob(mace.weight_layout(d), 4, STRESS_GAINS), sysm)
    assert np.abs(out["forces"]).max() < 1e-10 * max(1.0, np.abs(out["eps"]).max())
    np.testing.assert_allclose(out["eps"], out["eps"][0], rtol=1e-10)


def test_supercell_identity():
    d = _small_desc(hidden_lmax=1, K=4, rc=3.2)
    box = 4.0
    base = _cluster(6, seed=13, box=box, radius=1.9)
    blob = synth.weight_blob(mace.weight_layout(d), 5, STRESS_GAINS)
    e1 = _energy(d, blob, base)
    reps = [np.array(s) for s in itertools.product(range(2), repeat=3)]
    pos = np.vstack([base.positions + box * s for s in reps])
    big = synth.System(pos, np.tile(base.species, 8), np.diag([2 * box] * 3)[None], np.zeros(len(pos), np.int32), 1)
    e8 = _energy(d, blob, big)
    assert abs(e8 - 8 * e1) < 1e-10 * max(1.0, abs(e8))


def test_batch_independence_and_locality():
    d = _small_desc(hidden_lmax=1, K=4, S=3, rc=3.0)
    blob = synth.weight_blob(mace.weight_layout(d), 6, STRESS_GAINS)
    mols = [_cluster(5 + i, seed=20 + i, S=3, radius=1.8) for i in range(3)]
    singles = [mace.energy_forces(d, blob, m, forces=False)["energy"][0] for m in mols]
    pos = np.vstack([m.positions + np.array([10.0 * i, 0, 0]) for i, m in enumerate(mols)])
    gid = np.concatenate([np.full(m.n_atoms, i, np.int32) for i, m in enumerate(mols)])
    batch = synth.System(pos, np.concatenate([m.species for m in mols]), None, gid, 3)
    eb = mace.energy_forces(d, blob, batch, forces=False)["energy"]
    np.testing.assert_allclose(eb, singles, rtol=1e-12, atol=1e-14)
    # locality: atoms of a far-away cluster move, the first cluster's eps stay
    sysm = synth.System(pos, batch.species, None, np.zeros(len(pos), np.int32), 1)
    e_a = mace.energy_forces(d, blob, sysm, forces=False)["eps"]
    moved = sysm.positions.copy()
    moved[mols[0].n_atoms + mols[1].n_atoms:] += 0.37
    e_b = mace.energy_forces(d, blob, synth.System(moved, batch.species, None, sysm.graph_of_atom, 1), forces=False)["eps"]
    n0 = mols[0].n_atoms
    np.testing.assert_array_equal(e_a[:n0], e_b[:n0])


def test_cutoff_continuity():
    """Only the pair (atom 0, moving atom) crosses r_c: beyond it the energy is
    constant, and the approach to r_c is smooth (envelope and basis vanish)."""
    d = _small_desc(hidden_lmax=1, K=4, rc=3.0)
    blob = synth.weight_blob(mace.weight_layout(d), 7, STRESS_GAINS)
    base = np.array([[0.0, 0, 0], [1.1, 0.3, 0], [0.2, 1.2, 0.1]])

    def e_at(x):
        pos = np.vstack([base, [-x, 0, 0]])
        sysm = synth.System(pos, np.array([0, 1, 0, 1], np.int32), None, np.zeros(4, np.int32), 1)
        return _energy(d, blob, sysm)
    far = e_at(3.5)
    assert e_at(3.0001) == far
    assert abs(e_at(2.9999) - far) < 1e-9 * max(1.0, abs(far))
    assert abs(e_at(2.9) - far) > 1e-9 * max(1.0, abs(far))


# ------------------------------------------------------------------ planted mistakes

def test_planted_cg_sign_error_breaks_invariance(monkeypatch, cfg0):
    """A plausible oracle bug (one CG path with a flipped sign on part of its
    entries) must be caught by the rotation-invariance pin."""
    d, blob, sysm = cfg0
    orig = so3.real_cg

    def bad(l1, l2, l3):
        c = orig(l1, l2, l3)
        if (l1, l2, l3) == (0, 2, 2):
            c[:, :2, :] *= -1
        return c
    monkeypatch.setattr(so3, "real_cg", bad)
    ref = mace.energy_forces(d, blob, sysm, forces=False)["eps"]
    R = so3.random_rotation(np.random.default_rng(11))
    out = mace.energy_forces(d, blob, _rotated(sysm, R), forces=False)["eps"]
    assert np.abs(out - ref).max() > 1e-6 * np.abs(ref).max()


def test_planted_transposed_harmonic_breaks_invariance(monkeypatch, cfg0):
    d, blob, sysm = cfg0
    orig = so3.sh_all

    def bad(u, lmax):
        y = orig(u, lmax)
        return torch.cat([y[:, :1], y[:, [3, 2, 1]], y[:, 4:]], dim=1)   # l=1 as (x,z,y)
    monkeypatch.setattr(so3, "sh_all", bad)
    ref = mace.energy_forces(d, blob, sysm, forces=False)["eps"]
    R = so3.random_rotation(np.random.default_rng(12))
    out = mace.energy_forces(d, blob, _rotated(sysm, R), forces=False)["eps"]
    assert np.abs(out - ref).max() > 1e-6 * np.abs(ref).max()


def test_no_edges_energy_constant_zero_force():
    """Force equation: with no atom pair inside the cutoff E does not depend
    on positions, so F = 0 exactly."""
    d = _small_desc(hidden_lmax=1, K=4, rc=2.0)
    blob = synth.weight_blob(mace.weight_layout(d), 8, STRESS_GAINS)
    sysm = synth.System(np.array([[0.0, 0, 0], [5.0, 0, 0]]), np.array([0, 1], np.int32), None,
                        np.zeros(2, np.int32), 1)
    out = mace.energy_forces(d, blob, sysm)
    assert np.all(out["forces"] == 0.0)
    moved = synth.System(sysm.positions + 1.0, sysm.species, None, sysm.graph_of_atom, 1)
    assert _energy(d, blob, moved) == out["energy"][0]


# ------------------------------------------------------------------ stress

def _strained(system, eps):
    M = np.eye(3) + eps
    cells = None if system.cells is None else np.asarray(system.cells) @ M
    return synth.System(np.asarray(system.positions) @ M, system.species, cells, system.graph_of_atom,
                        system.n_graphs)


def test_stress_matches_strain_finite_differences():
    """sigma = (1/V) dE/d(epsilon) against central differences of E under a
    small homogeneous strain (positions and cell, neighbour list rebuilt)."""
    d = _small_desc(hidden_lmax=1, K=6, rc=3.2)
    blob = synth.weight_blob(mace.weight_layout(d), 11, {".radial.3": 4.0})
    system = _cluster(14, seed=5, box=6.3)
    sig = mace.stress(d, blob, system)[0]
    V = abs(np.linalg.det(system.cells[0]))
    h = 1e-5
    for a, b in [(0, 0), (1, 2), (2, 1), (2, 2), (0, 1)]:
        e = np.zeros((3, 3))
        e[a, b] = h
        fd = (_energy(d, blob, _strained(system, e)) - _energy(d, blob, _strained(system, -e))) / (2 * h * V)
        assert abs(fd - sig[a, b]) <= 1e-6 * np.abs(sig).max() + 1e-12, (a, b, fd, sig[a, b])
    # rotation invariance makes dE/d(epsilon) symmetric
    assert np.abs(sig - sig.T).max() <= 1e-10 * np.abs(sig).max()


def test_stress_of_isolated_cluster_is_the_position_force_moment():
    """Without a cell every atom moves with the strain, so dE/d(epsilon)_ab =
    sum_i x_ia dE/dx_ib = -sum_i x_ia F_ib (V = 1)."""
    d = _small_desc(hidden_lmax=1, K=6, rc=3.2)
    blob = synth.weight_blob(mace.weight_layout(d), 12, {".radial.3": 4.0})
    system = _cluster(10, seed=9)
    out = mace.energy_forces(d, blob, system)
    ref = -np.asarray(system.positions).T @ out["forces"]
    sig = mace.stress(d, blob, system)[0]
    assert np.abs(sig - ref).max() <= 1e-10 * np.abs(ref).max()


def test_stress_is_intensive_under_supercell():
    """Doubling a periodic cell along x doubles E and V: sigma is unchanged."""
    d = _small_desc(hidden_lmax=1, K=6, rc=3.2)
    blob = synth.weight_blob(mace.weight_layout(d), 13, {".radial.3": 4.0})
    system = _cluster(12, seed=3, box=6.5)
    cell = system.cells[0]
    pos2 = np.concatenate([system.positions, system.positions + cell[0]])
    sup = synth.System(pos2, np.concatenate([system.species, system.species]),
                       (np.diag([2.0, 1.0, 1.0]) @ cell)[None], np.zeros(24, np.int32), 1)
    s1 = mace.stress(d, blob, system)[0]
    s2 = mace.stress(d, blob, sup)[0]
    assert np.abs(s1 - s2).max() <= 1e-9 * np.abs(s1).max()


# ------------------------------------------------------------------ 16-bit linears

def test_fp16_rounding_is_ieee_binary16_nearest_even():
    """The FP16-linear emulation rounds to IEEE binary16 (10 fraction bits),
    ties to even, overflow to infinity: values fixed by the format itself."""
    u = 2.0 ** -10                                   # ulp of binary16 at 1
    x = torch.tensor([1 + u / 2, 1 + 1.5 * u, 1 + 0.75 * u, 65504.0, 65519.0, 65520.0, -70000.0,
                      2.0 ** -24, 2.0 ** -26, 3 * 2.0 ** -25], dtype=torch.float64)
    want = [1.0, 1 + 2 * u, 1 + u, 65504.0, 65504.0, math.inf, -math.inf, 2.0 ** -24, 0.0, 2 * 2.0 ** -24]
    got = mace._round_fp16(x).tolist()
    assert got == want, got


def test_bf16_rounding_is_bfloat16_nearest_even():
    u = 2.0 ** -7                                    # ulp of bfloat16 at 1
    x = torch.tensor([1 + u / 2, 1 + 1.5 * u, 1 + 0.25 * u, 3.0e38], dtype=torch.float64)
    got = mace._round_bf16(x).tolist()
    assert got[:3] == [1.0, 1 + 2 * u, 1.0], got
    assert got[3] == float(np.float32(3.0e38)) or abs(got[3] / 3.0e38 - 1) < 2 ** -8


def test_16bit_linear_modes_stay_close_to_fp64():
    """Rounding the linears' inputs and weights moves energies and forces by
    about the format's precision: FP16 (11 significant bits) less than BF16 (8)."""
    d = _desc(0)
    blob = synth.weight_blob(mace.weight_layout(d), 4)
    system = make_system(0, seed=0)
    ref = mace.energy_forces(d, blob, system)
    dev = {}
    for name, kw in (("bf16", dict(bf16_linear=True)), ("fp16", dict(fp16_linear=True))):
        out = mace.energy_forces(d, blob, system, graph=ref["graph"], **kw)
        dev[name] = (abs(out["energy"] - ref["energy"]).max() / np.abs(ref["eps"]).sum(),
                     np.linalg.norm(out["forces"] - ref["forces"]) / np.linalg.norm(ref["forces"]))
    assert dev["fp16"][1] < dev["bf16"][1] and dev["fp16"][1] < 2e-3 and dev["bf16"][1] < 2e-2, dev
    assert dev["fp16"][0] < dev["bf16"][0] + 1e-9, dev


def test_bf16_radial_mode_rounds_the_last_radial_product():
    """R13: BF16-radial changes the result relative to BF16-linear (the
    rounding of the last radial product takes effect) but stays within the
    16-bit force tolerance of FP64 (the rounding itself is pinned by the
    bfloat16 nearest-even values above)."""
    d = _desc(0)
    blob = synth.weight_blob(mace.weight_layout(d), 4)
    system = make_system(0, seed=0)
    ref = mace.energy_forces(d, blob, system)
    lin = mace.energy_forces(d, blob, system, graph=ref["graph"], bf16_linear=True)
    rad = mace.energy_forces(d, blob, system, graph=ref["graph"], bf16_linear=True, bf16_radial=True)
    assert not np.array_equal(lin["forces"], rad["forces"])
    fdev = np.linalg.norm(rad["forces"] - ref["forces"]) / np.linalg.norm(ref["forces"])
    assert fdev < 2e-2, fdev


# ------------------------------------------------------- per-block precision study

def _np_round16(x, fmt):
    """Round to nearest even through FP32, written with numpy only: bfloat16
    by the 16-bit truncation of the FP32 pattern with a nearest-even bias,
    binary16 by numpy's half type."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    if fmt == "fp16":
        return x32.astype(np.float16).astype(np.float64)
    u = x32.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_edge_product_rounding_rounds_features_harmonics_and_radial_weights(fmt):
    """The edge-product rounding of the precision study rounds exactly the
    sender features, the harmonics and the radial weights (brute-force loops
    on independently rounded operands), not the CG constants."""
    d = _small_desc(hidden_lmax=1, K=3, rc=3.5, c_norm=1.7)
    sysm = _cluster(5, seed=5, radius=1.6)
    W = mace.unpack_weights(d, synth.weight_blob(mace.weight_layout(d), 1, STRESS_GAINS))
    g = mace.build_graph(sysm, d)
    pos = torch.tensor(sysm.positions)
    _, ref = mace.node_energies(d, W, g, pos, return_intermediates=True)
    _, inter = mace.node_energies(d, W, g, pos, return_intermediates=True, tp_round=fmt)
    # layer 0 of the rounded run: A from rounded table, harmonics and radial weights
    t = 0
    paths = mace.tp_paths(d, t)
    ht = {0: _np_round16((W["embed"][g.species][:, None, :] @ W["0.up.0"]).numpy(), fmt)}
    Rall = _np_round16(mace.radial_mlp(inter["rbf"], W, t, 3).reshape(-1, len(paths), d.K).numpy(), fmt)
    At = _edge_sum_loops(d, W, g, _np_round16(inter["Y"].numpy(), fmt), Rall, ht, t)
    A = [sum(At[p] @ W[f"0.linear.{p}"].numpy() for p, (_, _, lo) in enumerate(paths) if lo == l) for l in range(4)]
    z = g.species.numpy()
    A = np.concatenate([np.einsum("nck,nkj->ncj", A[l], W[f"0.skip.{l}"].numpy()[z]) for l in range(4)], axis=1)
    np.testing.assert_allclose(inter["0.A"].numpy(), A, rtol=1e-12, atol=1e-12)
    assert not np.allclose(inter["0.A"].numpy(), ref["0.A"].numpy(), rtol=1e-7, atol=0)


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_symmetric_contraction_rounding_rounds_a_and_weights(fmt):
    """The contraction's rounding rounds A and the weights W (not U): the
    unrounded contraction of independently rounded A and W."""
    rng = np.random.default_rng(1)
    K, S = 3, 2
    A = torch.from_numpy(rng.standard_normal((4, 16, K)))
    z = torch.tensor([0, 1, 1, 0])
    for L in (0, 1, 2):
        W = {f"0.symc.{L}.{nu}": torch.from_numpy(rng.standard_normal((S, so3.n_eta(nu, L), K))) for nu in (1, 2, 3)}
        Wr = {k: torch.from_numpy(_np_round16(v.numpy(), fmt)) for k, v in W.items()}
        got = mace.symmetric_contraction(A, W, 0, L, z, 3, rnd=mace._rounding(fmt)).numpy()
        want = mace.symmetric_contraction(torch.from_numpy(_np_round16(A.numpy(), fmt)), Wr, 0, L, z, 3).numpy()
        np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_radial_mlp_rounding_rounds_every_layers_input_and_weights(fmt):
    """The radial-MLP rounding of the precision study rounds the input of
    every layer (the basis, then each SiLU output) and every layer's weights:
    a numpy MLP on independently rounded operands; leaving out any one of
    those roundings gives a different result."""
    d = _desc(0)
    W = mace.unpack_weights(d, synth.weight_blob(mace.weight_layout(d), 2))
    rng = np.random.default_rng(7)
    e = rng.uniform(-0.5, 1.5, (40, d.n_bessel))
    t, nh = 0, len(d.radial_hidden)
    got = mace.radial_mlp(torch.from_numpy(e), W, t, nh, rnd=mace._rounding(fmt)).numpy()

    def np_mlp(skip=None):
        r = lambda x, tag: x if tag == skip else _np_round16(x, fmt)  # noqa: E731
        h = e
        for i in range(nh + 1):
            z = r(h, ("in", i)) @ r(W[f"{t}.radial.{i}"].numpy(), ("w", i))
            h = z / (1.0 + np.exp(-z)) if i < nh else z
        return h
    np.testing.assert_allclose(got, np_mlp(), rtol=1e-12, atol=1e-13)
    for skip in [("in", i) for i in range(nh + 1)] + [("w", i) for i in range(nh + 1)]:
        assert not np.allclose(got, np_mlp(skip), rtol=1e-9, atol=0), skip


def test_block_rounding_moves_the_result_by_about_the_format_precision():
    """Rounding the edge product's, the contraction's or the radial MLP's operands moves
    energies and forces away from FP64 by about the format's precision:
    binary16 (11 significant bits) less than bfloat16 (8)."""
    d = _desc(0)
    blob = synth.weight_blob(mace.weight_layout(d), 4)
    system = make_system(0, seed=0)
    ref = mace.energy_forces(d, blob, system)
    for key in ("tp_round", "symcon_round", "radial_round"):
        dev = {}
        for fmt in ("bf16", "fp16"):
            out = mace.energy_forces(d, blob, system, graph=ref["graph"], **{key: fmt})
            dev[fmt] = np.linalg.norm(out["forces"] - ref["forces"]) / np.linalg.norm(ref["forces"])
        assert 0 < dev["fp16"] < dev["bf16"] < 5e-2, (key, dev)


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_block_rounding_value_is_the_rounding_and_gradient_passes_through(fmt):
    x = torch.tensor(np.random.default_rng(3).standard_normal(64) * 3.0, requires_grad=True)
    w = torch.tensor(np.random.default_rng(4).standard_normal(64))
    y = mace._rounding(fmt)(x)
    np.testing.assert_array_equal(y.detach().numpy(), _np_round16(x.detach().numpy(), fmt))
    (g,) = torch.autograd.grad((w * y).sum(), x)
    np.testing.assert_array_equal(g.numpy(), w.numpy())
