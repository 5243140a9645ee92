"""The allocation-free device neighbour list (mace_neighbor_list_device_noalloc)
against the workspace entry point it varies (mace_neighbor_list_device):
element for element on two calls in a row, the second with a smaller input
(the static scratch keeps the first call's contents, so whatever must start
at zero has to be cleared by the call itself), then a size beyond the scratch
limit, refused on the host before anything is enqueued."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import make_system, model_params

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2510_23621_amd.binding")


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _goff(system):
    if system.n_graphs == 1:
        return None
    return np.concatenate([[0], np.cumsum(np.bincount(system.graph_of_atom, minlength=system.n_graphs))]).astype(
        np.int32)


def _both(system, r_cut):
    pos = torch.from_numpy(np.ascontiguousarray(system.positions, dtype=np.float64)).cuda()
    goff = _goff(system)
    ref = B.mace_neighbor_list_device(pos, r_cut, system.cells, goff, system.n_graphs)
    out = B.mace_neighbor_list_device_noalloc(pos, r_cut, system.cells, goff, system.n_graphs)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in ref], [t.cpu().numpy() for t in out]


def test_noalloc_equals_workspace_list_two_calls_second_smaller():
    cases = [(make_system(1, seed=0), model_params(1)["r_cut"]),     # 1,536 atoms
             (make_system(0, seed=3), model_params(0)["r_cut"])]     # then 96 atoms
    for system, rc in cases:
        print(f"[noalloc] {system.n_atoms} atoms, r_cut {rc}", flush=True)
        ref, out = _both(system, rc)
        assert len(ref[0]) > 0
        for a, b in zip(ref, out):
            assert np.array_equal(a, b)


def test_noalloc_molecule_batch_then_largest_box():
    """Many graphs (offsets), then the 36,864-atom box that fills most of the scratch."""
    for cfg in (4, 3):
        system = make_system(cfg, seed=0)
        rc = model_params(cfg)["r_cut"]
        need = B.mace_neighbor_workspace_bytes(system.n_atoms, rc, system.cells, _goff(system), system.n_graphs)
        assert 0 < need <= B.MACE_NEIGHBOR_SCRATCH_BYTES
        print(f"[noalloc] cfg {cfg}: {system.n_atoms} atoms, {need / 2**20:.1f} MiB of scratch", flush=True)
        ref, out = _both(system, rc)
        for a, b in zip(ref, out):
            assert np.array_equal(a, b)


def test_noalloc_refuses_sizes_beyond_the_scratch():
    n = 50_000
    box = 80.0
    cells = np.diag([box] * 3)[None].astype(np.float64)
    need = B.mace_neighbor_workspace_bytes(n, 5.0, cells, None, 1)
    assert need > B.MACE_NEIGHBOR_SCRATCH_BYTES   # the host plan alone decides; nothing is launched
    pos = torch.from_numpy(np.random.default_rng(0).uniform(0, box, (n, 3))).cuda()
    with pytest.raises(B.MaceError) as exc:
        B.mace_neighbor_list_device_noalloc(pos, 5.0, cells, None, 1, max_edges=0)
    assert exc.value.code == -3
    # the entry point still works afterwards
    system = synth.water_box(16, seed=2, box=8.0)
    ref, out = _both(system, 4.0)
    for a, b in zip(ref, out):
        assert np.array_equal(a, b)
