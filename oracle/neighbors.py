"""Brute-force neighbour list (oracle, FP64).

The graph of the problem statement connects atom j (sender) to atom i
(receiver) whenever their distance is below the cutoff, periodic images
included (section "Graph representation of atomic configurations").  The
paper does not fix the details; the oracle's reading:

* edge vector d = (x_j - x_i) + (S_0 a_0 + S_1 a_1 + S_2 a_2) in FP64, for
  integer image shift S and lattice rows a_0..a_2;
* kept iff 0 < (d_x^2 + d_y^2) + d_z^2 < r_c^2 (strict, evaluated in this
  order), so an atom is never its own neighbour without a shift;
* every image is enumerated, so one pair may appear under several shifts
  (the cutoff may exceed half the box);
* atoms of different graphs are never connected; without a cell only S = 0;
* edges sorted by (receiver, sender, S_0, S_1, S_2).
"""
from __future__ import annotations

import math

import numpy as np


def _image_range(cell: np.ndarray, frac_span: np.ndarray, rc: float) -> np.ndarray:
    """Largest |S_a| that can give |d| < rc, per lattice direction."""
    recip = np.linalg.inv(cell).T          # rows b_a with a_i . b_j = delta_ij
    bn = np.linalg.norm(recip, axis=1)
    return np.floor(rc * bn + frac_span).astype(np.int64)


def neighbor_list(positions: np.ndarray, r_cut: float, cells=None, graph_of_atom=None):
    """Return (sender[E], receiver[E], shift[E,3]) int arrays, canonical order."""
    pos = np.asarray(positions, dtype=np.float64)
    n = len(pos)
    gid = np.zeros(n, dtype=np.int64) if graph_of_atom is None else np.asarray(graph_of_atom, dtype=np.int64)
    rc2 = float(r_cut) * float(r_cut)
    out_s, out_r, out_S = [], [], []
    for g in np.unique(gid):
        idx = np.nonzero(gid == g)[0]
        p = pos[idx]
        if cells is not None:
            cell = np.asarray(cells[g], dtype=np.float64)
            frac = p @ np.linalg.inv(cell)
            span = frac.max(axis=0) - frac.min(axis=0) if len(p) else np.zeros(3)
            nr = _image_range(cell, span, r_cut)
            shifts = np.array([(a, b, c)
                               for a in range(-nr[0], nr[0] + 1)
                               for b in range(-nr[1], nr[1] + 1)
                               for c in range(-nr[2], nr[2] + 1)], dtype=np.int64)
            svec = ((shifts[:, 0:1] * cell[0]) + (shifts[:, 1:2] * cell[1])) + (shifts[:, 2:3] * cell[2])
        else:
            shifts = np.zeros((1, 3), dtype=np.int64)
            svec = np.zeros((1, 3))
        for ii in range(len(p)):
            dj = p - p[ii]                                     # x_j - x_i, [n,3]
            d = dj[:, None, :] + svec[None, :, :]              # [n, nS, 3]
            r2 = (d[..., 0] * d[..., 0] + d[..., 1] * d[..., 1]) + d[..., 2] * d[..., 2]
            jj, ss = np.nonzero((r2 < rc2) & (r2 > 0.0))
            out_s.append(idx[jj])
            out_r.append(np.full(len(jj), idx[ii], dtype=np.int64))
            out_S.append(shifts[ss])
    if not out_s:
        return (np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros((0, 3), np.int64))
    s = np.concatenate(out_s)
    r = np.concatenate(out_r)
    S = np.concatenate(out_S).reshape(-1, 3)
    order = np.lexsort((S[:, 2], S[:, 1], S[:, 0], s, r))
    return s[order], r[order], S[order]
