"""SO(3) building blocks of the oracle (FP64).

Spherical harmonics Y_lm and Clebsch-Gordan couplings appear in the two-body
edge embedding (Eq. 26); the generalised Clebsch-Gordan tensors C^{LM}_{eta,lm}
of the node-local product basis appear in Eq. 27.  The paper names these
objects but fixes no basis, phase or normalisation; the oracle uses:

* Real spherical harmonics, m = -l..l, m>0 ~ cos(m phi), m<0 ~ sin(|m| phi),
  no Condon-Shortley phase, component normalisation sum_m Y_lm(u)^2 = 2l+1.
  So Y_1 = sqrt(3) (y, z, x).
* Real CG C^{l3}_{l1 l2}[m1, m2, m3]: the rotation-invariant real tensor
  (unique up to scale), scaled so that sum_{m1 m2} C[.,.,m3] C[.,.,m3'] =
  delta_{m3 m3'}, sign chosen so that its first nonzero entry in
  lexicographic (m1, m2, m3) order is positive.  Computed from its definition:
  the common fixed vector of D1 (x) D2 (x) D3 for two generic rotations.
* U tensors: for correlation nu and output L, coupling trees over the 16
  components of A (l = 0..3, natural parity) enumerated in a fixed order,
  symmetrised over the nu factors, kept when linearly independent of the
  trees kept before them, and scaled to unit Frobenius norm.
"""
from __future__ import annotations

import itertools
import math
from functools import lru_cache

import numpy as np
import torch

A_LMAX = 3          # A carries l = 0..3 (natural parity): 16 components


def comp_offset(l: int) -> int:
    """Offset of block l inside a stacked l = 0..lmax component axis."""
    return l * l


# --------------------------------------------------------------------------
# spherical harmonics (Eq. 26: Y_{l m}(r_hat_ji))
# --------------------------------------------------------------------------

@lru_cache(maxsize=None)
def _legendre_derivative_coeffs(l: int, m: int) -> tuple:
    """Coefficients (ascending powers of z) of d^m/dz^m P_l(z), with
    P_l(z) = 1/(2^l l!) d^l/dz^l (z^2 - 1)^l  (Rodrigues' formula)."""
    base = np.polynomial.polynomial.polypow([-1.0, 0.0, 1.0], l)      # (z^2-1)^l
    p = np.polynomial.polynomial.polyder(base, l + m) if l + m > 0 else base
    p = p / (2.0 ** l * math.factorial(l))
    return tuple(float(c) for c in np.atleast_1d(p))


def real_sh(l: int, u: torch.Tensor) -> torch.Tensor:
    """Y_l(u) for unit vectors u [...,3] -> [..., 2l+1] (component normalised).

    Y_lm = sqrt(2l+1) sqrt((l-|m|)!/(l+|m|)!) c_m P_l^(|m|)(z) T_m(x, y)
    with c_0 = 1, c_m = sqrt(2) otherwise, T_m = Re (x+iy)^m for m > 0,
    Im (x+iy)^|m| for m < 0, 1 for m = 0.
    """
    x, y, z = u[..., 0], u[..., 1], u[..., 2]
    re = [torch.ones_like(x)]
    im = [torch.zeros_like(x)]
    for _ in range(l):
        r0, i0 = re[-1], im[-1]
        re.append(r0 * x - i0 * y)
        im.append(r0 * y + i0 * x)
    out = []
    for m in range(-l, l + 1):
        am = abs(m)
        coeffs = _legendre_derivative_coeffs(l, am)
        poly = torch.zeros_like(z)
        for c in reversed(coeffs):
            poly = poly * z + c
        norm = math.sqrt((2 * l + 1) * math.factorial(l - am) / math.factorial(l + am))
        if m != 0:
            norm *= math.sqrt(2.0)
        trig = re[am] if m > 0 else (im[am] if m < 0 else torch.ones_like(x))
        out.append(norm * poly * trig)
    return torch.stack(out, dim=-1)


def sh_all(u: torch.Tensor, lmax: int) -> torch.Tensor:
    """Stack of Y_0..Y_lmax -> [..., (lmax+1)^2]."""
    return torch.cat([real_sh(l, u) for l in range(lmax + 1)], dim=-1)


# --------------------------------------------------------------------------
# Wigner D matrices in this basis (fitted from the harmonics themselves)
# --------------------------------------------------------------------------

def random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


_D_SAMPLES = None


def wigner_d(l: int, R: np.ndarray) -> np.ndarray:
    """D^l(R) with Y_l(R u) = D^l(R) Y_l(u), by least squares over fixed samples."""
    global _D_SAMPLES
    if _D_SAMPLES is None:
        v = np.random.default_rng(12345).standard_normal((256, 3))
        _D_SAMPLES = v / np.linalg.norm(v, axis=1, keepdims=True)
    u = torch.from_numpy(_D_SAMPLES)
    ru = torch.from_numpy(_D_SAMPLES @ R.T)
    Yu = real_sh(l, u).numpy()
    Yr = real_sh(l, ru).numpy()
    X, *_ = np.linalg.lstsq(Yu, Yr, rcond=None)      # Yr = Yu @ X
    return X.T


# --------------------------------------------------------------------------
# real Clebsch-Gordan couplings (Eq. 26: C^{l3 m3}_{l1 m1, l2 m2})
# --------------------------------------------------------------------------

def _fix_sign(t: np.ndarray, tol: float = 1e-9) -> np.ndarray:
    flat = t.reshape(-1)
    nz = np.nonzero(np.abs(flat) > tol)[0]
    if len(nz) and flat[nz[0]] < 0:
        t = -t
    return t


@lru_cache(maxsize=None)
def _real_cg_cached(l1: int, l2: int, l3: int) -> np.ndarray:
    if not (abs(l1 - l2) <= l3 <= l1 + l2):
        raise ValueError(f"triangle violated: {l1} {l2} {l3}")
    rng = np.random.default_rng(7)
    n = (2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1)
    rows = []
    for _ in range(2):
        R = random_rotation(rng)
        K = np.kron(np.kron(wigner_d(l1, R), wigner_d(l2, R)), wigner_d(l3, R))
        rows.append(K - np.eye(n))
    M = np.vstack(rows)
    _, s, vt = np.linalg.svd(M)
    if s[-1] > 1e-8 or (len(s) > 1 and s[-2] < 1e-6):
        raise RuntimeError(f"invariant space of {l1}x{l2}x{l3} is not one-dimensional")
    c = vt[-1].reshape(2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1)
    c = c * math.sqrt((2 * l3 + 1) / np.sum(c * c))
    c[np.abs(c) < 1e-13] = 0.0
    return _fix_sign(c)


def real_cg(l1: int, l2: int, l3: int) -> np.ndarray:
    """C^{l3}_{l1 l2}[m1, m2, m3] in the basis of ``real_sh`` (copy)."""
    return _real_cg_cached(l1, l2, l3).copy()


# --------------------------------------------------------------------------
# generalised CG (U) tensors of the product basis (Eq. 27)
# --------------------------------------------------------------------------

def coupling_trees(nu: int, L: int, parity: int, lmax: int = A_LMAX):
    """Candidate trees, in the fixed enumeration order.

    nu=1: (l1,)                       l1 = L
    nu=2: (l1, l2)            l1<=l2, |l1-l2| <= L <= l1+l2
    nu=3: (l1, l2, l3, l12)   l1<=l2<=l3, l12 ascending, (l1 l2)->l12, (l12 l3)->L
    A-component l has parity (-1)^l, so a tree is kept only if
    (-1)^(l1+..+l_nu) equals the requested parity of L.
    """
    out = []
    ls = range(lmax + 1)
    if nu == 1:
        for l1 in ls:
            if l1 == L and (-1) ** l1 == parity:
                out.append((l1,))
    elif nu == 2:
        for l1, l2 in itertools.product(ls, ls):
            if l1 <= l2 and abs(l1 - l2) <= L <= l1 + l2 and (-1) ** (l1 + l2) == parity:
                out.append((l1, l2))
    elif nu == 3:
        for l1, l2, l3 in itertools.product(ls, ls, ls):
            if not (l1 <= l2 <= l3) or (-1) ** (l1 + l2 + l3) != parity:
                continue
            for l12 in range(abs(l1 - l2), l1 + l2 + 1):
                if abs(l12 - l3) <= L <= l12 + l3:
                    out.append((l1, l2, l3, l12))
    else:
        raise ValueError("correlation order must be 1, 2 or 3")
    return out


def tree_tensor(tree, L: int, lmax: int = A_LMAX) -> np.ndarray:
    """Unsymmetrised tree tensor T[M, a_1..a_nu] over the full A index space."""
    n = (lmax + 1) ** 2
    nu = 1 if len(tree) == 1 else (2 if len(tree) == 2 else 3)
    T = np.zeros((2 * L + 1,) + (n,) * nu)
    if nu == 1:
        l1 = tree[0]
        o = comp_offset(l1)
        for M in range(2 * L + 1):
            T[M, o + M] = 1.0
    elif nu == 2:
        l1, l2 = tree
        C = real_cg(l1, l2, L)
        o1, o2 = comp_offset(l1), comp_offset(l2)
        T[:, o1:o1 + 2 * l1 + 1, o2:o2 + 2 * l2 + 1] = np.transpose(C, (2, 0, 1))
    else:
        l1, l2, l3, l12 = tree
        C1 = real_cg(l1, l2, l12)
        C2 = real_cg(l12, l3, L)
        block = np.einsum("abk,kcM->Mabc", C1, C2)
        o1, o2, o3 = comp_offset(l1), comp_offset(l2), comp_offset(l3)
        T[:, o1:o1 + 2 * l1 + 1, o2:o2 + 2 * l2 + 1, o3:o3 + 2 * l3 + 1] = block
    return T


def symmetrise(T: np.ndarray) -> np.ndarray:
    """Average over permutations of the factor axes (all axes but the first)."""
    nu = T.ndim - 1
    acc = np.zeros_like(T)
    perms = list(itertools.permutations(range(1, nu + 1)))
    for p in perms:
        acc += np.transpose(T, (0,) + p)
    return acc / len(perms)


@lru_cache(maxsize=None)
def _u_basis_cached(nu: int, L: int, parity: int, lmax: int):
    kept_trees, kept, ortho = [], [], []
    for tree in coupling_trees(nu, L, parity, lmax):
        S = symmetrise(tree_tensor(tree, L, lmax))
        v = S.reshape(-1)
        nrm = np.linalg.norm(v)
        if nrm < 1e-12:
            continue
        r = v.copy()
        for q in ortho:
            r -= (q @ r) * q
        if np.linalg.norm(r) <= 1e-8 * nrm:
            continue
        ortho.append(r / np.linalg.norm(r))
        kept_trees.append(tree)
        kept.append(S / nrm)
    return tuple(kept_trees), tuple(kept)


def u_basis(nu: int, L: int, parity: int | None = None, lmax: int = A_LMAX):
    """(trees, [U_eta]) with U_eta[M, a_1..a_nu] symmetric and of unit norm."""
    if parity is None:
        parity = (-1) ** L
    trees, us = _u_basis_cached(nu, L, parity, lmax)
    return list(trees), [u.copy() for u in us]


def n_eta(nu: int, L: int, parity: int | None = None) -> int:
    return len(u_basis(nu, L, parity)[0])
