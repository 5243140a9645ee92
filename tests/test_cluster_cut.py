"""The cluster cut used by the full-size parity tests reproduces the
oracle's periodic per-atom energy (eps_i depends only on atoms within
2 r_c), checked on the 96-atom periodic box (CPU)."""
import numpy as np

import synth
from oracle import mace
from synth.configs import make_system, model_params

from gpu_common import cluster_cut


def test_cluster_cut_matches_periodic_eps():
    params = model_params(0, c_norm=1.0)
    d = mace.ModelDesc(**params)
    blob = synth.weight_blob(mace.weight_layout(d), 0, {".radial.3": 4.0})
    sysm = make_system(0, seed=0)
    full = mace.energy_forces(d, blob, sysm, forces=False)["eps"]
    for i in (0, 41):
        cl, _ = cluster_cut(sysm, i, 2 * params["r_cut"] + 0.5)
        eps = mace.energy_forces(d, blob, cl, forces=False)["eps"]
        assert abs(eps[0] - full[i]) <= 1e-10 * np.abs(full).max(), (i, eps[0], full[i])
