"""Device neighbour list against the host list (itself bit-exact against the
oracle's brute-force list): identical (sender, receiver, shift) arrays."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import CONFIGS, make_system

pytestmark = pytest.mark.gpu
B = pytest.importorskip("paper_2510_23621_amd.binding")


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _offsets(sysm):
    if sysm.n_graphs == 1:
        return None
    return np.concatenate([[0], np.cumsum(np.bincount(sysm.graph_of_atom, minlength=sysm.n_graphs))]).astype(np.int32)


def _compare(label, pos, rc, cells, graph_of_atom, n_graphs, offsets):
    s_h, r_h, S_h = B.mace_neighbor_list(pos, rc, cells, graph_of_atom, n_graphs)
    dpos = torch.from_numpy(np.ascontiguousarray(pos, dtype=np.float64)).cuda()
    s_d, r_d, S_d = B.mace_neighbor_list_device(dpos, rc, cells, offsets, n_graphs)
    torch.cuda.synchronize()
    s_d, r_d, S_d = s_d.cpu().numpy(), r_d.cpu().numpy(), S_d.cpu().numpy()
    print(f"[neighbors] {label}: host {len(s_h)} device {len(s_d)} edges", flush=True)
    assert np.array_equal(r_h, r_d) and np.array_equal(s_h, s_d) and np.array_equal(S_h, S_d)
    return len(s_h)


@pytest.mark.parametrize("cfg", [0, 1, 3, 4])
def test_device_list_equals_host_list(cfg):
    sysm = make_system(cfg, seed=0)
    rc = CONFIGS[cfg]["model"]["r_cut"]
    E = _compare(f"cfg{cfg}", sysm.positions, rc, sysm.cells, sysm.graph_of_atom if sysm.n_graphs > 1 else None,
                 sysm.n_graphs, _offsets(sysm))
    assert E > 0


def test_unwrapped_positions_and_triclinic_cell():
    """Atoms moved by random lattice vectors (positions outside the cell) in
    a skewed cell: the shifts change, the edge set stays exact."""
    rng = np.random.default_rng(5)
    cell = np.array([[9.0, 0.0, 0.0], [3.1, 8.2, 0.0], [-1.7, 2.3, 7.6]])
    frac = rng.uniform(0, 1, size=(150, 3))
    pos = frac @ cell + rng.integers(-3, 4, size=(150, 3)) @ cell
    _compare("triclinic unwrapped", pos, 5.0, cell[None], None, 1, None)


def test_small_cell_many_images():
    """A 3 A cell with a 5 A cutoff: every pair appears under many shifts,
    and an atom meets its own images."""
    rng = np.random.default_rng(6)
    cell = np.eye(3) * 3.0
    pos = rng.uniform(0, 3.0, size=(4, 3))
    E = _compare("3 A cell", pos, 5.0, cell[None], None, 1, None)
    assert E > 4 * 50


def test_dense_images_long_segments():
    """A 2.2 A cell with a 7 A cutoff: about 400 edges per receiver, beyond
    the segment length the device list sorts through LDS."""
    rng = np.random.default_rng(8)
    cell = np.eye(3) * 2.2
    pos = rng.uniform(0, 2.2, size=(3, 3))
    E = _compare("2.2 A cell, 7 A cutoff", pos, 7.0, cell[None], None, 1, None)
    assert E > 3 * 300


def test_mixed_batch_and_no_edges():
    """Empty graphs and graphs without any pair in range inside a batch."""
    a = np.array([[0.0, 0, 0], [1.0, 0, 0], [0, 1.2, 0]])
    b = np.array([[0.0, 0, 0], [20.0, 0, 0]])
    pos = np.concatenate([a, b, a + 100.0])
    goa = np.array([0, 0, 0, 2, 2, 3, 3, 3], np.int32)   # graph 1 is empty
    offsets = np.array([0, 3, 3, 5, 8], np.int32)
    _compare("batch with an empty graph", pos, 5.0, None, goa, 4, offsets)
    far = np.array([[0.0, 0, 0], [10.0, 0, 0]])
    assert _compare("no pair in range", far, 5.0, None, None, 1, None) == 0


def test_capacity_and_bad_positions():
    sysm = make_system(0, seed=1)
    dpos = torch.from_numpy(sysm.positions).cuda()
    s, r, S = B.mace_neighbor_list_device(dpos, 5.0, sysm.cells)
    E = len(s)
    with pytest.raises(B.MaceError) as ex:
        B.mace_neighbor_list_device(dpos, 5.0, sysm.cells, max_edges=E - 1)
    assert ex.value.code == -3
    bad = dpos.clone()
    bad[3, 0] = float("nan")
    with pytest.raises(B.MaceError) as ex:
        B.mace_neighbor_list_device(bad, 5.0, sysm.cells)
    assert ex.value.code == -5
