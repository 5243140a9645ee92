"""Named workloads: geometry recipe + model hyper-parameters (plain data).

The systems mirror the paper's benchmark shapes (128 channels, cutoff
5-6 A, correlation 3, 8 Bessel functions, 3x64 radial MLP, two interaction
layers; periodic liquid water at 1 g/cm^3 and batches of small molecules).
``c_norm`` is the mean neighbour count at the workload's density (the model
constant dividing the neighbour sum).
"""
from __future__ import annotations

from . import molecule_batch, water_box

CONFIGS = {
    0: dict(name="water96_k32", system=("water", 32, 9.85),
            model=dict(n_species=2, K=32, hidden_lmax=0, r_cut=5.0, c_norm=52.5)),
    1: dict(name="water1536_k128_l1", system=("water", 512, None),
            model=dict(n_species=2, K=128, hidden_lmax=1, r_cut=5.0, c_norm=52.5)),
    2: dict(name="water4608_k128_l1", system=("water", 1536, None),
            model=dict(n_species=2, K=128, hidden_lmax=1, r_cut=5.0, c_norm=52.5)),
    3: dict(name="water36864_k128_l2", system=("water", 12288, None),
            model=dict(n_species=2, K=128, hidden_lmax=2, r_cut=6.0, c_norm=90.7)),
    4: dict(name="molecules512_k128_l1", system=("molecules", 512, None),
            model=dict(n_species=10, K=128, hidden_lmax=1, r_cut=5.0, c_norm=22.0)),
}


def make_system(cfg: int, seed: int = 0):
    kind, n, box = CONFIGS[cfg]["system"]
    if kind == "water":
        return water_box(n, seed=seed, box=box)
    return molecule_batch(n, seed=seed)


def model_params(cfg: int, **overrides) -> dict:
    p = dict(CONFIGS[cfg]["model"])
    p.update(overrides)
    return p
