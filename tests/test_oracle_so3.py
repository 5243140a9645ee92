"""Pins for the oracle's harmonics, CG couplings and U tensors (CPU only).

Each pin ties the oracle to something other than itself: textbook closed
forms, scipy's complex harmonics, sympy's exact Clebsch-Gordan coefficients,
the addition theorem, exact quadrature, rotation invariance, and
character-theory multiplicities computed here from the Weyl integration
formula.
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special as sps
import torch

from oracle import so3


def _unit(n, seed=0):
    v = np.random.default_rng(seed).standard_normal((n, 3))
    return v / np.linalg.norm(v, axis=1, keepdims=True)


def _Q(l):
    """Complex (Condon-Shortley) -> real basis: Y^r_m = sum_mu Q[m, mu] Y^c_mu."""
    Q = np.zeros((2 * l + 1, 2 * l + 1), dtype=complex)
    for m in range(-l, l + 1):
        i = m + l
        if m == 0:
            Q[i, l] = 1.0
        elif m > 0:
            Q[i, l - m] = 1 / math.sqrt(2)
            Q[i, l + m] = (-1) ** m / math.sqrt(2)
        else:
            mu = -m
            Q[i, l - mu] = 1j / math.sqrt(2)
            Q[i, l + mu] = -1j * (-1) ** mu / math.sqrt(2)
    return Q


def test_sh_closed_forms_l1_l2():
    u = _unit(50, 1)
    x, y, z = u.T
    Y1 = so3.real_sh(1, torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(Y1, math.sqrt(3) * np.stack([y, z, x], 1), atol=1e-14)
    Y2 = so3.real_sh(2, torch.from_numpy(u)).numpy()
    s15 = math.sqrt(15)
    ref = np.stack([s15 * x * y, s15 * y * z, math.sqrt(5) / 2 * (3 * z * z - 1),
                    s15 * x * z, s15 / 2 * (x * x - y * y)], 1)
    np.testing.assert_allclose(Y2, ref, atol=1e-13)
    Y0 = so3.real_sh(0, torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(Y0, 1.0)


@pytest.mark.parametrize("l", [0, 1, 2, 3, 4])
def test_sh_matches_scipy_complex(l):
    u = _unit(64, 2)
    theta = np.arccos(np.clip(u[:, 2], -1, 1))
    phi = np.arctan2(u[:, 1], u[:, 0])
    Yc = np.stack([sps.sph_harm_y(l, mu, theta, phi) for mu in range(-l, l + 1)], 1)
    Yr = (Yc @ _Q(l).T) * math.sqrt(4 * math.pi)
    assert np.abs(Yr.imag).max() < 1e-12
    ours = so3.real_sh(l, torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(ours, Yr.real, atol=1e-12)


@pytest.mark.parametrize("l", [0, 1, 2, 3])
def test_sh_addition_theorem(l):
    u, v = _unit(40, 3), _unit(40, 4)
    Yu = so3.real_sh(l, torch.from_numpy(u)).numpy()
    Yv = so3.real_sh(l, torch.from_numpy(v)).numpy()
    lhs = (Yu * Yv).sum(1)
    rhs = (2 * l + 1) * sps.eval_legendre(l, (u * v).sum(1))
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)


def test_sh_quadrature_orthonormal():
    # Gauss-Legendre in cos(theta) x uniform phi: exact for degree <= 6 products
    zs, wz = np.polynomial.legendre.leggauss(8)
    phis = np.arange(16) * 2 * math.pi / 16
    Z, P = np.meshgrid(zs, phis, indexing="ij")
    Wt = np.repeat(wz[:, None], len(phis), 1) / (2 * len(phis))
    s = np.sqrt(1 - Z * Z)
    u = np.stack([s * np.cos(P), s * np.sin(P), Z], -1).reshape(-1, 3)
    Y = so3.sh_all(torch.from_numpy(u), 3).numpy()
    G = (Y * Wt.reshape(-1, 1)).T @ Y
    np.testing.assert_allclose(G, np.eye(16), atol=1e-12)


def _paths():
    out = []
    for l1, l2 in itertools.product(range(4), range(4)):
        for l3 in range(abs(l1 - l2), l1 + l2 + 1):
            out.append((l1, l2, l3))
    return out


@pytest.mark.parametrize("l1,l2,l3", _paths())
def test_cg_orthonormal_and_invariant(l1, l2, l3):
    C = so3.real_cg(l1, l2, l3)
    G = np.einsum("abm,abn->mn", C, C)
    np.testing.assert_allclose(G, np.eye(2 * l3 + 1), atol=1e-12)
    rng = np.random.default_rng(l1 * 100 + l2 * 10 + l3)
    for _ in range(2):
        R = so3.random_rotation(rng)
        D1, D2, D3 = (so3.wigner_d(l, R) for l in (l1, l2, l3))
        rot = np.einsum("abc,ai,bj,ck->ijk", C, D1, D2, D3)
        np.testing.assert_allclose(rot, C, atol=1e-11)


@pytest.mark.parametrize("l1,l2,l3", [p for p in _paths() if p[2] <= 3] + [(3, 3, 6), (2, 3, 5), (3, 3, 4)])
def test_cg_matches_sympy(l1, l2, l3):
    from sympy.physics.wigner import clebsch_gordan
    Cc = np.zeros((2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1))
    for m1 in range(-l1, l1 + 1):
        for m2 in range(-l2, l2 + 1):
            m3 = m1 + m2
            if abs(m3) <= l3:
                Cc[m1 + l1, m2 + l2, m3 + l3] = float(clebsch_gordan(l1, l2, l3, m1, m2, m3))
    Cr = np.einsum("ia,jb,kc,abc->ijk", _Q(l1).conj(), _Q(l2).conj(), _Q(l3), Cc)
    k = np.argmax(np.abs(Cr))
    Cr = Cr / (Cr.reshape(-1)[k] / abs(Cr.reshape(-1)[k]))
    assert np.abs(Cr.imag).max() < 1e-12
    Cr = Cr.real
    ours = so3.real_cg(l1, l2, l3)
    sign = 1.0 if np.sum(Cr * ours) > 0 else -1.0
    np.testing.assert_allclose(ours, sign * Cr, atol=1e-12)
    # sign convention: first nonzero entry positive
    flat = ours.reshape(-1)
    assert flat[np.nonzero(np.abs(flat) > 1e-9)[0][0]] > 0


def test_cg_nnz_table():
    nnz = {(0, 0, 0): 1, (0, 1, 1): 3, (0, 2, 2): 5, (0, 3, 3): 7, (1, 0, 1): 3, (1, 1, 0): 3,
           (1, 1, 2): 11, (1, 2, 1): 11, (1, 2, 3): 21, (1, 3, 2): 21, (2, 0, 2): 5, (2, 1, 1): 11,
           (2, 1, 3): 21, (2, 2, 0): 5, (2, 2, 2): 25, (2, 3, 1): 21, (2, 3, 3): 41}
    for k, v in nnz.items():
        assert int((np.abs(so3.real_cg(*k)) > 1e-12).sum()) == v, k


# ---------------------------------------------------------------- U tensors

def _char(l, theta):
    if abs(theta) < 1e-12:
        return 2 * l + 1
    return math.sin((l + 0.5) * theta) / math.sin(theta / 2)


def _char_A(theta, inv):
    # A = 0e + 1o + 2e + 3o; inversion acts on l as (-1)^l
    return sum(((-1) ** l if inv else 1) * _char(l, theta) for l in range(4))


def _mult(nu, L, parity):
    """Multiplicity of L^parity in Sym^nu(A) by the Weyl integration formula."""
    th = np.linspace(0, math.pi, 4001)[1:]
    wt = (1 - np.cos(th)) / math.pi
    tot = 0.0
    for inv in (False, True):
        vals = []
        for t in th:
            c1 = _char_A(t, inv)
            c2 = _char_A(2 * t, False)           # g^2: inversion squares to identity
            c3 = _char_A(3 * t, inv)
            if nu == 1:
                s = c1
            elif nu == 2:
                s = (c1 * c1 + c2) / 2
            else:
                s = (c1 ** 3 + 3 * c2 * c1 + 2 * c3) / 6
            vals.append(s * _char(L, t) * ((parity if inv else 1)))
        tot += np.trapezoid(np.array(vals) * wt, th)
    return tot / 2


@pytest.mark.parametrize("L,parity", [(0, 1), (1, -1), (2, 1), (3, -1), (1, 1), (2, -1), (3, 1)])
def test_u_multiplicity_character_theory(L, parity):
    for nu in (1, 2, 3):
        expect = round(_mult(nu, L, parity))
        assert abs(_mult(nu, L, parity) - expect) < 1e-3
        assert so3.n_eta(nu, L, parity) == expect, (nu, L, parity)


def test_u_multiplicity_survey_numbers():
    assert [so3.n_eta(nu, 0) for nu in (1, 2, 3)] == [1, 4, 8]
    assert [so3.n_eta(nu, 1) for nu in (1, 2, 3)] == [1, 3, 12]
    assert [so3.n_eta(nu, 2) for nu in (1, 2, 3)] == [1, 5, 14]


@pytest.mark.parametrize("L", [0, 1, 2])
def test_u_symmetric_unit_equivariant(L):
    rng = np.random.default_rng(L)
    R = so3.random_rotation(rng)
    DA = np.zeros((16, 16))
    for l in range(4):
        o = l * l
        DA[o:o + 2 * l + 1, o:o + 2 * l + 1] = so3.wigner_d(l, R)
    DL = so3.wigner_d(L, R)
    A = rng.standard_normal(16)
    for nu in (1, 2, 3):
        _, us = so3.u_basis(nu, L)
        for U in us:
            assert abs(np.linalg.norm(U) - 1) < 1e-12
            for p in itertools.permutations(range(1, nu + 1)):
                np.testing.assert_allclose(np.transpose(U, (0,) + p), U, atol=1e-14)
            def ev(a):
                t = U
                for _ in range(nu):
                    t = t @ a
                return t
            np.testing.assert_allclose(ev(DA @ A), DL @ ev(A), atol=1e-11)


def test_u_nu1_is_identity_selection():
    for L in (0, 1, 2):
        trees, us = so3.u_basis(1, L)
        assert trees == [(L,)]
        A = np.arange(16, dtype=float)
        B = us[0] @ A * math.sqrt(2 * L + 1)
        np.testing.assert_allclose(B, A[L * L:L * L + 2 * L + 1])


def test_u_spans_full_invariant_space():
    """The kept U of (nu=2, L=0) span every symmetric invariant quadratic
    form: each such form is sum_l c_l |A_l|^2, a 4-dim space."""
    _, us = so3.u_basis(2, 0)
    M = np.stack([u.reshape(-1) for u in us])
    for l in range(4):
        q = np.zeros((16, 16))
        o = l * l
        q[o:o + 2 * l + 1, o:o + 2 * l + 1] = np.eye(2 * l + 1)
        coef, res, *_ = np.linalg.lstsq(M.T, q.reshape(-1), rcond=None)
        assert np.linalg.norm(M.T @ coef - q.reshape(-1)) < 1e-12
