"""Shapes of the kernels' work per layer (paths, mid dimension, CG nonzeros),
from the library's own exported layout and CG tables; used to convert
measured kernel times into bytes/s and flop/s."""
from __future__ import annotations

from . import binding as B


def _paths(lh_max, sh_lmax=3):
    out = []
    for a in range(lh_max + 1):
        for b in range(sh_lmax + 1):
            for c in range(abs(a - b), min(a + b, sh_lmax) + 1):
                if (a + b + c) % 2 == 0:
                    out.append((a, b, c))
    return out


def layer_shapes(params: dict) -> dict:
    T = params.get("n_layers", 2)
    hl = params["hidden_lmax"]
    hl = [hl] * max(T - 1, 0) if isinstance(hl, int) else list(hl)
    layers = []
    for t in range(T):
        lh = 0 if t == 0 else hl[t - 1]
        lo = 0 if t == T - 1 else hl[t]
        paths = _paths(lh)
        nnz = sum(int((B.mace_debug_real_cg(*p) != 0).sum()) for p in paths)
        layers.append(dict(P=len(paths), mid=sum(2 * p[2] + 1 for p in paths), din=(lh + 1) ** 2,
                           dout=(lo + 1) ** 2, nnz=nnz))
    return dict(K=params["K"], n_bessel=params.get("n_bessel", 8), layers=layers)
