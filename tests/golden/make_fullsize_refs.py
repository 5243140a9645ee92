"""Write the FP64 oracle references of the full-size parity tests.

Calls only ``oracle/`` and ``synth/``: per-atom energies, per-graph energies
and forces of the seeded periodic-water workloads, evaluated by the oracle's
two-pass chunked vector-Jacobian product (exact up to summation order: the
neighbour sum of Eq. 26 is linear in the edge messages, and every later step
acts node by node). The file also stores a fingerprint of the inputs
(positions, species, weights, edge list) so that a test can check that it
compares the same problem.

    python tests/golden/make_fullsize_refs.py water4608_k128_l1 water36864_k128_l2 water1536_k128_l1_stress

Each workload takes minutes (4,608 atoms) to about an hour (36,864 atoms) of
CPU time.
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# workload -> (config index, model overrides, weight gains). The stress inputs
# (c_norm 1, last radial layer x4) make every correlation order of Eq. 27
# contribute at full size.
REFS = {
    "water4608_k128_l1": (2, {}, None),
    "water36864_k128_l2": (3, {}, None),
    "water1536_k128_l1_stress": (1, {"c_norm": 1.0}, {".radial.3": 4.0}),
}


def ref_path(name: str) -> str:
    return os.path.join(HERE, f"{name}_fp64.npz")


def fingerprint(system, blob, sender, receiver, shifts) -> str:
    """sha256 over the inputs both sides see (positions as float32, species,
    the float32 weight blob, the edge list)."""
    h = hashlib.sha256()
    for a in (np.asarray(system.positions, np.float32), np.asarray(system.species, np.int32),
              np.asarray(blob, np.float32), np.asarray(sender, np.int32), np.asarray(receiver, np.int32),
              np.asarray(shifts, np.int32)):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def workload(name: str):
    """(params, system, blob) of a named reference workload."""
    import synth
    from oracle import mace
    from synth.configs import make_system, model_params
    cfg, over, gains = REFS[name]
    params = model_params(cfg, **over)
    system = make_system(cfg, seed=0)
    blob = synth.weight_blob(mace.weight_layout(mace.ModelDesc(**params)), 0, gains)
    return params, system, blob


def make(name: str) -> str:
    import torch

    from oracle import mace
    from oracle.neighbors import neighbor_list
    torch.set_num_threads(os.cpu_count() or 1)
    params, system, blob = workload(name)
    d = mace.ModelDesc(**params)
    t0 = time.time()
    graph = mace.build_graph(system, d)
    s, r, S = neighbor_list(system.positions, d.r_cut, system.cells, system.graph_of_atom)
    out = mace.energy_forces_chunked(d, blob, system, graph=graph)
    secs = time.time() - t0
    np.savez(ref_path(name), eps=out["eps"], energy=out["energy"], forces=out["forces"],
             n_edges=np.int64(len(s)), fingerprint=np.array(fingerprint(system, blob, s, r, S)),
             oracle_seconds=np.float64(secs), threads=np.int64(torch.get_num_threads()))
    print(f"{name}: {system.n_atoms} atoms, {len(s)} edges, {secs:.0f} s on {torch.get_num_threads()} threads",
          flush=True)
    return ref_path(name)


if __name__ == "__main__":
    for n in sys.argv[1:] or list(REFS):
        make(n)
