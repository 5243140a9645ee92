"""CPU-side checks of the HIP library (no GPU calls): the library loads and
exports every entry point of include/mace.h; its weight layout, CG tables,
coupling-tree selection and neighbour list agree with the oracle; its
harmonics/radial closed forms (the same functions the kernels inline,
evaluated on the host) agree with the oracle's; argument errors return the
documented status codes.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import synth
from oracle import mace, so3
from oracle.neighbors import neighbor_list as oracle_nl
from synth.configs import CONFIGS, make_system, model_params

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
B = pytest.importorskip("paper_2510_23621_amd.binding")


def _lib_available():
    return os.path.exists(B.LIB_PATH)


pytestmark = pytest.mark.skipif(not _lib_available(), reason="libmace_amd.so not built")


def _desc_pair(cfg, **kw):
    p = model_params(cfg, **kw)
    return mace.ModelDesc(**p), B.make_desc(**p)


def test_exports_every_header_symbol():
    hdr = open(os.path.join(ROOT, "include", "mace.h")).read()
    names = set(re.findall(r"\b(mace_[a-z0-9_]+)\s*\(", hdr))
    assert names, "no declarations found"
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert set(B.EXPORTED) == names


@pytest.mark.parametrize("cfg", [0, 1, 3, 4])
def test_weight_layout_matches_oracle(cfg):
    od, ld = _desc_pair(cfg)
    lay_o = [(name, int(np.prod(s)), f) for name, s, f in mace.weight_layout(od)]
    lay_l, tot = B.mace_weight_layout(ld)
    assert lay_l == lay_o
    assert tot == sum(n for _, n, _ in lay_o)


@pytest.mark.parametrize("layers,hl", [(3, (2, 1)), (4, (2, 2, 0)), (3, (1, 1))])
def test_weight_layout_per_layer_lmax_matches_oracle(layers, hl):
    """One hidden l_max per layer (non-increasing) in the descriptor."""
    od, ld = _desc_pair(0, K=32, n_layers=layers, hidden_lmax=hl)
    lay_o = [(name, int(np.prod(s)), f) for name, s, f in mace.weight_layout(od)]
    lay_l, tot = B.mace_weight_layout(ld)
    assert lay_l == lay_o
    assert tot == sum(n for _, n, _ in lay_o)


def test_per_layer_lmax_refused_when_rising_or_too_many_layers():
    with pytest.raises(B.MaceError) as e:
        B.mace_weight_layout(B.make_desc(**model_params(0, K=32, n_layers=3, hidden_lmax=(1, 2))))
    assert e.value.code == -7   # MACE_EUNSUPPORTED: a layer's output l not among its inputs
    with pytest.raises(B.MaceError) as e:
        B.mace_weight_layout(B.make_desc(**model_params(0, K=32, n_layers=3, hidden_lmax=(3, 1))))
    assert e.value.code == -7
    with pytest.raises(ValueError):
        B.make_desc(**model_params(0, K=32, n_layers=9, hidden_lmax=1))


def test_weight_blob_identical_from_both_layouts():
    od, ld = _desc_pair(1)
    blob_o = synth.weight_blob(mace.weight_layout(od), 5, {".radial.3": 4.0})
    lay_l, _ = B.mace_weight_layout(ld)
    blob_l = synth.weight_blob([(name, (n,), f) for name, n, f in lay_l], 5, {".radial.3": 4.0})
    assert np.array_equal(blob_o, blob_l)


def _all_paths():
    out = []
    for l1 in range(4):
        for l2 in range(4):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                out.append((l1, l2, l3))
    return out + [(3, 3, 6), (2, 3, 5), (3, 3, 5), (4, 3, 1), (5, 3, 2), (4, 2, 2)]


@pytest.mark.parametrize("l1,l2,l3", _all_paths())
def test_real_cg_matches_oracle(l1, l2, l3):
    np.testing.assert_allclose(B.mace_debug_real_cg(l1, l2, l3), so3.real_cg(l1, l2, l3), atol=1e-12)


@pytest.mark.parametrize("L,parity", [(0, 1), (1, -1), (2, 1), (3, -1), (1, 1), (2, -1)])
def test_trees_match_oracle(L, parity):
    for nu in (1, 2, 3):
        trees, scales = B.mace_debug_trees(nu, L, parity)
        o_trees, o_us = so3.u_basis(nu, L, parity)
        assert len(trees) == len(o_trees)
        for t, s, ot in zip(trees, scales, o_trees):
            assert tuple(int(x) for x in t[:len(ot)]) == (ot if nu != 3 else (ot[0], ot[1], ot[2], ot[3]))
            # scale = 1/||Sym T||: U_eta = scale * Sym(T)
            S = so3.symmetrise(so3.tree_tensor(ot, L))
            assert abs(s - 1.0 / np.linalg.norm(S)) < 1e-12


@pytest.mark.parametrize("cfg,seed", [(0, 0), (0, 1), (1, 0), (4, 0)])
def test_neighbor_list_bit_exact(cfg, seed):
    sysm = make_system(cfg, seed=seed)
    if cfg == 4:   # a slice of the batch keeps the oracle fast
        keep = sysm.graph_of_atom < 40
        sysm = synth.System(sysm.positions[keep], sysm.species[keep], None, sysm.graph_of_atom[keep], 40)
    rc = CONFIGS[cfg]["model"]["r_cut"]
    s_o, r_o, S_o = oracle_nl(sysm.positions, rc, sysm.cells, sysm.graph_of_atom)
    s_l, r_l, S_l = B.mace_neighbor_list(sysm.positions, rc, sysm.cells, sysm.graph_of_atom, sysm.n_graphs)
    assert np.array_equal(s_o, s_l) and np.array_equal(r_o, r_l) and np.array_equal(S_o, S_l)


def test_neighbor_list_empty_and_isolated():
    pos = np.array([[0.0, 0, 0], [10.0, 0, 0]])
    s, r, S = B.mace_neighbor_list(pos, 5.0)
    assert len(s) == 0


def test_edge_feature_closed_forms_match_oracle():
    rng = np.random.default_rng(0)
    vec = rng.normal(size=(500, 3)).astype(np.float32)
    vec *= (rng.uniform(0.5, 4.9, size=(500, 1)) / np.linalg.norm(vec, axis=1, keepdims=True)).astype(np.float32)
    Y, rbf = B.mace_debug_edge_features(vec, 5.0, 5, 8)
    v64 = torch.from_numpy(vec.astype(np.float64))
    r = v64.norm(dim=1)
    Yo = so3.sh_all(v64 / r[:, None], 3).numpy()
    ro = mace.bessel_basis(r, 5.0, 8, 5).numpy()
    np.testing.assert_allclose(Y, Yo, rtol=2e-6, atol=2e-6)
    np.testing.assert_allclose(rbf, ro, rtol=1e-5, atol=1e-6)


def test_status_codes_without_gpu():
    d = B.make_desc(2, 48, 0, 5.0, 1.0)      # K = 48 is not implemented
    assert B.mace_workspace_bytes(d, 10, 10, 1) == 0
    lay = B.lib().mace_weight_layout(ctypes.byref(d), 0, None, None, None, 0, None, None)
    assert lay == -7
    good = B.make_desc(2, 32, 0, 5.0, 1.0)
    h = ctypes.c_void_p()
    # null weights -> EINVAL before any device call
    code = B.lib().mace_graph_setup(ctypes.byref(good), None, 0, 10, None, 0, None, None, None, None, 1, 0,
                                    None, 0, None, ctypes.byref(h))
    assert code == -1
    assert B.mace_status_string(-3).startswith("workspace")


def test_device_neighbor_workspace_size_without_gpu():
    """The device list's workspace size is a host computation: positive for
    valid input, 0 for a non-positive cutoff, a singular cell or offsets
    that do not cover the atoms; larger with more periodic images."""
    cell = np.eye(3)[None] * 10.0
    n1 = B.mace_neighbor_workspace_bytes(100, 5.0, cell)
    assert n1 > 0
    assert B.mace_neighbor_workspace_bytes(100, 5.0, None) > 0
    assert B.mace_neighbor_workspace_bytes(100, 12.0, cell) > n1     # more images per atom
    assert B.mace_neighbor_workspace_bytes(100, 0.0, cell) == 0
    assert B.mace_neighbor_workspace_bytes(100, 5.0, np.zeros((1, 3, 3))) == 0
    assert B.mace_neighbor_workspace_bytes(100, 5.0, None, np.array([0, 50, 90], np.int32), 2) == 0
    assert B.mace_neighbor_workspace_bytes(100, 5.0, None, np.array([0, 50, 100], np.int32), 2) > 0
