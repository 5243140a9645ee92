"""One graph bound to the library: torch allocates the workspace and the
outputs on the device, the library's kernels do all the work."""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B


class MaceGraph:
    def __init__(self, desc, weights, species, edge_index, unit_shifts=None, cells=None, graph_of_atom=None,
                 n_graphs: int = 1, prec: int = B.MACE_FP32, device="cuda", stream=None):
        """weights: float32 [n]; species: int32 [N]; edge_index: int32 [2, E]
        (senders, receivers; receivers nondecreasing); unit_shifts int32 [E, 3]
        or None; cells float64 [G, 3, 3] or None; graph_of_atom int32 [N] or
        None.  numpy arrays are copied to the device first."""
        dev = torch.device(device)

        def t(x, dt):
            if x is None:
                return None
            if isinstance(x, np.ndarray):
                x = torch.from_numpy(np.ascontiguousarray(x))
            return x.to(device=dev, dtype=dt).contiguous()
        self.desc = desc
        self.n_atoms = int(species.shape[0])
        self.n_edges = int(edge_index.shape[1])
        self.n_graphs = int(n_graphs)
        self.prec = prec
        self._w = t(weights, torch.float32)
        sp = t(species, torch.int32)
        ei = t(edge_index, torch.int32)
        us = t(unit_shifts, torch.int32)
        cl = t(cells, torch.float64)
        ga = t(graph_of_atom, torch.int32)
        nbytes = B.mace_workspace_bytes(desc, self.n_atoms, self.n_edges, self.n_graphs, prec)
        if nbytes == 0:
            raise B.MaceError(-1, "mace_workspace_bytes")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.handle = B.mace_graph_setup(desc, self._w, self.n_atoms, sp, self.n_edges, ei, us, cl, ga,
                                         self.n_graphs, prec, self.workspace, stream)
        self.device = dev

    @property
    def dtype(self):
        """dtype of positions, node energies and forces (FP64 in the debug precision)."""
        return torch.float64 if self.prec == B.MACE_FP64 else torch.float32

    def outputs(self, forces: bool):
        eps = torch.empty(self.n_atoms, dtype=self.dtype, device=self.device)
        E = torch.empty(self.n_graphs, dtype=torch.float64, device=self.device)
        F = torch.empty(self.n_atoms, 3, dtype=self.dtype, device=self.device) if forces else None
        return eps, E, F

    def energy(self, positions, stream=None):
        pos = positions.to(device=self.device, dtype=self.dtype).contiguous()
        eps, E, _ = self.outputs(False)
        B.mace_forward_energy(self.handle, pos, eps, E, stream)
        return eps, E

    def energy_forces(self, positions, stream=None):
        pos = positions.to(device=self.device, dtype=self.dtype).contiguous()
        eps, E, F = self.outputs(True)
        B.mace_forces(self.handle, pos, eps, E, F, stream)
        return eps, E, F

    def energy_forces_stress(self, positions, stream=None):
        pos = positions.to(device=self.device, dtype=self.dtype).contiguous()
        eps, E, F = self.outputs(True)
        S = torch.empty(self.n_graphs, 3, 3, dtype=torch.float64, device=self.device)
        B.mace_forces_stress(self.handle, pos, eps, E, F, S, stream)
        return eps, E, F, S

    def check(self, stream=None):
        """(status, flags) of the device checks since setup or the last check."""
        return B.mace_graph_check(self.handle, stream)

    def close(self):
        if getattr(self, "handle", None):
            B.mace_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
