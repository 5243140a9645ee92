"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module only draws random numbers and lays out geometry; it holds none
of the MACE arithmetic (no spherical harmonics, couplings, radial basis,
neighbour search or model evaluation).  Both sides of every parity check
take their inputs from here and nothing else.

Workloads stand in for the paper's benchmark systems (periodic water boxes at
liquid density and batches of small molecules, see the experimental set-up
and the MD case-study sections): the shapes and statistics follow those
systems, the coordinates are random.

* ``water_box``   -- O on a jittered cubic lattice, H at 0.96 A / 104.5 deg,
  random orientation, N(0, 0.05 A) noise, wrapped into the periodic box.
* ``molecule_batch`` -- independent non-periodic clusters of 20..60 atoms,
  uniform in a sphere at 0.1 atoms/A^3 with a 0.9 A minimum distance.
* ``weight_blob`` -- N(0,1)/sqrt(fan_in) float32 weights for a layout given
  by the caller as a list of (name, shape, fan_in).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

WATER_MOLAR_MASS = 18.015  # g/mol
AVOGADRO = 6.02214076e23
OH_BOND = 0.96  # Angstrom
HOH_ANGLE = math.radians(104.5)


def _streams(seed: int):
    """Two independent generators: geometry and weights."""
    geo, wts = np.random.SeedSequence(seed).spawn(2)
    return np.random.default_rng(geo), np.random.default_rng(wts)


def geometry_rng(seed: int) -> np.random.Generator:
    return _streams(seed)[0]


def weight_rng(seed: int) -> np.random.Generator:
    return _streams(seed)[1]


@dataclass
class System:
    """A batch of one or more graphs.

    positions: [N,3] float64 holding float32-representable values (the GPU
    path computes in float32 and both sides must see identical inputs).
    species:   [N] int32 in 0..S-1.
    cells:     [G,3,3] float64 rows = lattice vectors, or None (no PBC).
    graph_of_atom: [N] int32, nondecreasing.
    """
    positions: np.ndarray
    species: np.ndarray
    cells: np.ndarray | None
    graph_of_atom: np.ndarray
    n_graphs: int
    name: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def n_atoms(self) -> int:
        return int(self.positions.shape[0])


def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Uniform random rotation from a uniform unit quaternion."""
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def _min_image_dist(a: np.ndarray, b: np.ndarray, L: float) -> np.ndarray:
    d = a[:, None, :] - b[None, :, :]
    d -= L * np.round(d / L)
    return np.sqrt((d * d).sum(-1))


def water_box_length(n_molecules: int, density_g_cm3: float = 1.0) -> float:
    """Cubic box edge (A) holding n water molecules at the given density."""
    grams = n_molecules * WATER_MOLAR_MASS / AVOGADRO
    vol_cm3 = grams / density_g_cm3
    return (vol_cm3 * 1e24) ** (1.0 / 3.0)


def water_box(n_molecules: int, seed: int, box: float | None = None,
              noise: float = 0.05, min_dist: float = 1.0) -> System:
    """Periodic water: species O=0, H=1, ordered O,H,H per molecule."""
    rng = geometry_rng(seed)
    L = float(box) if box is not None else water_box_length(n_molecules)
    m = int(math.ceil(n_molecules ** (1.0 / 3.0) - 1e-12))
    spacing = L / m
    sites = np.array([(i, j, k) for i in range(m) for j in range(m) for k in range(m)], dtype=np.float64)
    chosen = rng.permutation(len(sites))[:n_molecules]
    oxy = (sites[chosen] + 0.5) * spacing
    oxy += rng.uniform(-0.1, 0.1, size=oxy.shape) * spacing
    half = HOH_ANGLE / 2
    h_local = OH_BOND * np.array([[math.sin(half), 0.0, math.cos(half)],
                                  [-math.sin(half), 0.0, math.cos(half)]])
    mols = np.zeros((n_molecules, 3, 3))
    for a in range(n_molecules):
        for _attempt in range(200):
            R = _random_rotation(rng)
            hs = oxy[a] + h_local @ R.T
            cand = np.vstack([oxy[a][None], hs])
            if a == 0:
                break
            prev = mols[:a].reshape(-1, 3)
            if _min_image_dist(cand, prev, L).min() >= min_dist:
                break
        mols[a] = cand
    pos = mols.reshape(-1, 3)
    pos = pos + rng.normal(0.0, noise, size=pos.shape)
    pos = np.mod(pos, L)
    pos = pos.astype(np.float32).astype(np.float64)
    species = np.tile(np.array([0, 1, 1], dtype=np.int32), n_molecules)
    cell = np.diag([L, L, L]).astype(np.float64)[None]
    return System(positions=pos, species=species, cells=cell,
                  graph_of_atom=np.zeros(len(pos), dtype=np.int32), n_graphs=1,
                  name=f"water{n_molecules}", meta={"box": L, "seed": seed})


def molecule_batch(n_graphs: int, seed: int, n_min: int = 20, n_max: int = 60,
                   n_species: int = 10, density: float = 0.1,
                   min_dist: float = 0.9, spacing: float = 100.0) -> System:
    """Independent non-periodic clusters; graph g is translated by g*spacing
    along x so that no two graphs overlap (edges never cross graphs anyway)."""
    rng = geometry_rng(seed)
    pos_all, spec_all, gid_all = [], [], []
    for g in range(n_graphs):
        n = int(rng.integers(n_min, n_max + 1))
        radius = (3.0 * n / (4.0 * math.pi * density)) ** (1.0 / 3.0)
        pts = []
        while len(pts) < n:
            p = rng.uniform(-radius, radius, size=3)
            if p @ p > radius * radius:
                continue
            if pts and np.min(np.linalg.norm(np.asarray(pts) - p, axis=1)) < min_dist:
                continue
            pts.append(p)
        pts = np.asarray(pts) + np.array([g * spacing, 0.0, 0.0])
        pos_all.append(pts)
        spec_all.append(rng.integers(0, n_species, size=n).astype(np.int32))
        gid_all.append(np.full(n, g, dtype=np.int32))
    pos = np.vstack(pos_all).astype(np.float32).astype(np.float64)
    return System(positions=pos, species=np.concatenate(spec_all), cells=None,
                  graph_of_atom=np.concatenate(gid_all), n_graphs=n_graphs,
                  name=f"molecules{n_graphs}", meta={"seed": seed})


def weight_blob(layout, seed: int, gains: dict | None = None) -> np.ndarray:
    """float32 blob: each tensor of ``layout`` (name, shape, fan_in), in order,
    filled with N(0,1)/sqrt(fan_in) from the weight stream of ``seed``.

    ``gains`` optionally maps a substring of a tensor name to an extra factor
    (used by stress inputs that keep activations O(1) under random weights)."""
    rng = weight_rng(seed)
    parts = []
    for name, shape, fan_in in layout:
        n = int(np.prod(shape))
        g = 1.0
        for key, val in (gains or {}).items():
            if key in name:
                g *= float(val)
        parts.append((g * rng.standard_normal(n) / math.sqrt(fan_in)).astype(np.float32))
    if not parts:
        return np.zeros(0, dtype=np.float32)
    return np.concatenate(parts)


def perturb(system: System, seed: int, scale: float) -> System:
    """Same system with float32-representable uniform noise on positions."""
    rng = np.random.default_rng(seed)
    pos = system.positions + rng.uniform(-scale, scale, size=system.positions.shape)
    pos = pos.astype(np.float32).astype(np.float64)
    return System(pos, system.species.copy(), None if system.cells is None else system.cells.copy(),
                  system.graph_of_atom.copy(), system.n_graphs, system.name, dict(system.meta))
