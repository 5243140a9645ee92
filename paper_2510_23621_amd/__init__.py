"""MI355X (gfx950) MACE layer library: energies and forces through a C ABI.

The kernels live in ``libmace_amd.so`` (built in-tree by ``build.build()``);
``binding`` exposes its entry points under their C names and ``MaceGraph``
wraps one graph's workspace and handle.  There is no CPU fallback: loading
the binding raises when the library is missing.
"""
from .binding import (MACE_BF16_LINEAR, MACE_FP32, MaceError, make_desc, mace_forces, mace_forward_energy,
                      mace_graph_destroy, mace_graph_setup, mace_neighbor_list, mace_status_string,
                      mace_weight_layout, mace_workspace_bytes)
from .graph import MaceGraph

__all__ = ["MACE_BF16_LINEAR", "MACE_FP32", "MaceError", "MaceGraph", "make_desc", "mace_forces",
           "mace_forward_energy", "mace_graph_destroy", "mace_graph_setup", "mace_neighbor_list",
           "mace_status_string", "mace_weight_layout", "mace_workspace_bytes"]
