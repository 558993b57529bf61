"""Pins of the fp64 oracle against values and facts outside the oracle itself.

* Wigner 3j: exact sympy values; the closed form of G^{l0}_{l1 0 l2 0}
  (Eq. cg-explicit with the triangle coefficient Eq. triangle) in exact integer
  arithmetic; CG orthogonality; the parity zero Eq. parity-zero.
* kappa^-1: values printed in App. A (worked (1,1,1) example) and App. B.
* Eq. Q-CG itself: the curl integral of complex CS harmonics by dense
  brute-force quadrature with finite-difference surface gradients, divided by
  the sympy CG, must be m-independent and equal the closed form (App. B tests).
* Real tables GR/QR: brute-force quadrature of scipy harmonics at lmax <= 3;
  textbook values; {x, y} = z; symmetry, antisymmetry, supports; Jacobi identity.
"""
from __future__ import annotations

import math
import os
import random
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


# ---------------------------------------------------------------- 3j / CG ---

def test_wigner3j_matches_sympy_exact():
    from sympy.physics.wigner import wigner_3j

    rnd = random.Random(7)
    cases = []
    while len(cases) < 250:
        j1, j2 = rnd.randint(0, 22), rnd.randint(0, 22)
        j3 = rnd.randint(abs(j1 - j2), min(j1 + j2, 44))
        m1, m2 = rnd.randint(-j1, j1), rnd.randint(-j2, j2)
        if abs(m1 + m2) > j3:
            continue
        cases.append((j1, j2, j3, m1, m2, -m1 - m2))
    cases += [(j, j, j, 0, 0, 0) for j in range(0, 22, 2)]
    cases += [(j, j, j - 1, -1, 1, 0) for j in range(1, 22)]
    for c in cases:
        exact = float(wigner_3j(*c).evalf(30))
        got = oracle.wigner3j(*c)
        assert abs(got - exact) <= 1e-14 * max(1.0, abs(exact)) + 1e-16, c


def _cg_l0_closed_form_sq(l1, l2, l):
    """(G^{l0}_{l1 0 l2 0})^2 from Eq. cg-explicit and Eq. triangle, exact rational."""
    f = math.factorial
    g2 = l1 + l2 + l
    if g2 % 2:
        return Fraction(0), 1
    g = g2 // 2
    delta = Fraction(f(l1 + l2 - l) * f(l1 - l2 + l) * f(-l1 + l2 + l), f(l1 + l2 + l + 1))
    ratio = Fraction(f(g), f(g - l1) * f(g - l2) * f(g - l))
    sign = -1 if (l1 - l2 + g) % 2 else 1
    return (2 * l + 1) * delta * ratio * ratio, sign


def test_cg_l0_closed_form_and_parity_zero():
    for l1 in range(0, 13):
        for l2 in range(0, 13):
            for l in range(abs(l1 - l2), l1 + l2 + 1):
                sq, sign = _cg_l0_closed_form_sq(l1, l2, l)
                ref = sign * math.sqrt(float(sq))
                got = oracle.cg(l1, 0, l2, 0, l, 0)
                if (l1 + l2 + l) % 2:
                    assert abs(got) < 1e-15, (l1, l2, l)    # Eq. parity-zero
                else:
                    assert abs(got - ref) < 1e-13, (l1, l2, l, got, ref)


def test_cg_orthogonality():
    for l1 in range(0, 5):
        for l2 in range(0, 5):
            ls = range(abs(l1 - l2), l1 + l2 + 1)
            for l in ls:
                for lp in ls:
                    for m in range(-l, l + 1):
                        for mp in range(-lp, lp + 1):
                            s = sum(oracle.cg(l1, m1, l2, m2, l, m) * oracle.cg(l1, m1, l2, m2, lp, mp)
                                    for m1 in range(-l1, l1 + 1) for m2 in range(-l2, l2 + 1))
                            assert abs(s - (1.0 if (l, m) == (lp, mp) else 0.0)) < 1e-13


def test_cg_antisymmetry_on_odd_support():
    # Eq. CG-antisym: G(1<->2) = -G when l1+l2+l is odd
    for l1 in range(1, 5):
        for l2 in range(1, 5):
            for l in range(abs(l1 - l2), l1 + l2 + 1):
                s = (-1) ** (l1 + l2 - l)
                for m1 in range(-l1, l1 + 1):
                    for m2 in range(-l2, l2 + 1):
                        a = oracle.cg(l1, m1, l2, m2, l, m1 + m2) if abs(m1 + m2) <= l else 0.0
                        b = oracle.cg(l2, m2, l1, m1, l, m1 + m2) if abs(m1 + m2) <= l else 0.0
                        assert abs(a - s * b) < 1e-14


# ---------------------------------------------------------------- kappa^-1 ---

def test_kappa_inv_printed_values():
    for l1, l2, l, q, val, digits, *_ in _read_golden("kappa_inv_paper.txt"):
        l1, l2, l, val, digits = int(l1), int(l2), int(l), float(val), int(digits)
        k = oracle.kappa_inv_im(l1, l2, l)
        got = k if q == "im" else abs(k)
        assert abs(got - val) <= 0.6 * 10.0 ** (-digits), (l1, l2, l, got, val)


def test_worked_example_111():
    g = {r[0]: float(r[1]) for r in _read_golden("worked_example_111.txt")}
    assert abs(oracle.curl_conj_im(1, 1, 1, -1, 1, 0) - g["Q10_11_1m1_im"]) < 1e-15
    assert abs(oracle.cg(1, 1, 1, -1, 1, 0) - g["G10_11_1m1"]) < 1e-15
    assert abs(oracle.kappa_inv_im(1, 1, 1) - g["kappa_inv_111_im"]) < 1e-15


def _complex_sh_and_derivs(lmax, n_theta=20, n_phi=40):
    """Complex CS harmonics and their e_theta / e_phi surface derivatives (FD)."""
    from scipy.special import sph_harm_y

    pts, T, P, W = bf.dense_grid(n_theta, n_phi)
    idx = bf.lm_index(lmax)

    def f(q):
        th = np.arccos(np.clip(q[:, 2], -1, 1))
        ph = np.arctan2(q[:, 1], q[:, 0])
        return np.stack([sph_harm_y(l, m, th, ph) for (l, m) in idx], axis=-1)

    Y = f(pts)
    Dt, Dp = bf.surface_derivs(f, pts, T, P)
    return idx, Y, Dt, Dp, W


def test_curl_identity_by_quadrature_complex_basis():
    """App. B checks of Eq. Q-CG / Eq. kappa-inv-closed: the brute-force curl
    integral over CG is m-independent, purely imaginary, equals the closed form,
    and vanishes on the even support."""
    from sympy.physics.quantum.cg import CG

    lmax = 4
    idx, Y, Dt, Dp, W = _complex_sh_and_derivs(lmax)
    pos = {lm: i for i, lm in enumerate(idx)}
    for l1 in range(1, 4):
        for l2 in range(1, 4):
            for l in range(abs(l1 - l2), min(l1 + l2, lmax) + 1):
                ratios = []
                for m1 in range(-l1, l1 + 1):
                    for m2 in range(-l2, l2 + 1):
                        m = m1 + m2
                        if abs(m) > l:
                            continue
                        a, b, c = pos[(l1, m1)], pos[(l2, m2)], pos[(l, m)]
                        integrand = bf.bracket(Dt[:, a], Dp[:, a], Dt[:, b], Dp[:, b])
                        q = np.sum(W * np.conj(Y[:, c]) * integrand)
                        if (l1 + l2 + l) % 2 == 0:
                            assert abs(q) < 1e-8, (l1, l2, l, m1, m2)
                            continue
                        cgv = float(CG(l1, m1, l2, m2, l, m).doit())
                        if abs(cgv) < 1e-12:
                            assert abs(q) < 1e-8
                            continue
                        ratios.append(q / cgv)
                if (l1 + l2 + l) % 2 == 1:
                    ratios = np.array(ratios)
                    assert np.abs(ratios.real).max() < 1e-8
                    assert np.ptp(ratios.imag) < 1e-8
                    assert abs(ratios.imag.mean() - oracle.kappa_inv_im(l1, l2, l)) < 1e-8


def test_oracle_complex_tables_match_quadrature():
    idx, Y, Dt, Dp, W = _complex_sh_and_derivs(3)
    for a, (l1, m1) in enumerate(idx):
        for b, (l2, m2) in enumerate(idx):
            for c, (l, m) in enumerate(idx):
                gq = np.sum(W * Y[:, a] * Y[:, b] * np.conj(Y[:, c]))
                assert abs(gq - oracle.gaunt_conj(l1, m1, l2, m2, l, m)) < 1e-12
                integrand = bf.bracket(Dt[:, a], Dp[:, a], Dt[:, b], Dp[:, b])
                qq = np.sum(W * np.conj(Y[:, c]) * integrand)
                assert abs(qq - 1j * oracle.curl_conj_im(l1, m1, l2, m2, l, m)) < 1e-8


# ---------------------------------------------------------------- real tables ---

@pytest.fixture(scope="module")
def dense_real():
    return bf.sh_and_derivs(3)


def test_real_tables_match_bruteforce(dense_real):
    Y, Dt, Dp, W = dense_real
    G = oracle.dense_table(0, 3)
    Q = oracle.dense_table(1, 3)
    Gq = np.einsum("p,pa,pb,pc->abc", W, Y, Y, Y)
    br = np.einsum("pa,pb->pab", Dt, Dp) - np.einsum("pa,pb->pab", Dp, Dt)
    Qq = np.einsum("p,pab,pc->abc", W, br, Y)
    assert np.abs(G - Gq).max() < 1e-13
    assert np.abs(Q - Qq).max() < 1e-8
    assert np.abs(Q).max() > 0.1 and np.abs(G).max() > 0.1


def test_real_tables_are_real():
    for kind in (0, 1):
        *_, max_im = oracle.real_table(kind, 8)
        assert max_im < 1e-14


def test_real_table_textbook_values():
    c = math.sqrt(3 / (4 * math.pi))
    # {x, y} = z on the unit sphere (Eq. poisson-S2); Y_{1,(-1,0,1)} = c (y, z, x)
    Q = oracle.dense_table(1, 1)
    ky, kz, kx = 1, 2, 3
    eps = {(kx, ky, kz): 1, (ky, kz, kx): 1, (kz, kx, ky): 1,
           (ky, kx, kz): -1, (kz, ky, kx): -1, (kx, kz, ky): -1}
    for a in range(1, 4):
        for b in range(1, 4):
            for d in range(1, 4):
                assert abs(Q[a, b, d] - c * eps.get((a, b, d), 0)) < 1e-15
    assert np.abs(Q[0]).max() == 0 and np.abs(Q[:, 0]).max() == 0 and np.abs(Q[:, :, 0]).max() == 0
    G = oracle.dense_table(0, 4)
    for k in range(25):
        assert abs(G[0, k, k] - 1 / math.sqrt(4 * math.pi)) < 1e-15
    # x*y = sqrt(4pi/15) * Y_{2,-2} * ... : int Y_{1,1} Y_{1,-1} Y_{2,-2} = sqrt(15/pi)/10
    assert abs(G[3, 1, 4] - math.sqrt(15 / math.pi) / 10) < 1e-15


def _degree(k):
    return int(math.isqrt(k))


def test_real_table_symmetry_and_supports():
    lmax = 6
    for kind in (0, 1):
        k1, k2, k3, v, _ = oracle.real_table(kind, lmax)
        d = {(a, b, c): x for a, b, c, x in zip(k1, k2, k3, v)}
        for (a, b, c), x in d.items():
            l1, l2, l = _degree(a), _degree(b), _degree(c)
            assert abs(l1 - l2) <= l <= l1 + l2
            if kind == 0:
                assert (l1 + l2 + l) % 2 == 0                 # Eq. parity-zero
                assert d.get((b, a, c), 0.0) == pytest.approx(x, abs=1e-15)
            else:
                assert (l1 + l2 + l) % 2 == 1                 # App. A step 3
                assert l1 >= 1 and l2 >= 1
                assert d.get((b, a, c), 0.0) == pytest.approx(-x, abs=1e-15)


def test_real_kappa_magnitudes_basis_invariant():
    """App. B, real basis: |kappa^-1| is the same in the real and complex bases.

    For fixed (l1, l2, l) the complex curl block equals kappa^-1 times the CG
    block, whose Frobenius norm is sqrt(2l+1) (one unit column per m). The real
    basis is a unitary change of each index, so the real block QR must have
    Frobenius norm |kappa^-1| sqrt(2l+1)."""
    Q = oracle.dense_table(1, 4, 7)
    for l1 in range(1, 5):
        for l2 in range(1, 5):
            for l in range(abs(l1 - l2), l1 + l2 + 1):
                blk = Q[l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2, l * l:(l + 1) ** 2]
                norm = np.sqrt(np.sum(blk ** 2))
                ref = abs(oracle.kappa_inv_im(l1, l2, l)) * math.sqrt(2 * l + 1)
                assert abs(norm - ref) < 1e-12, (l1, l2, l)


def test_poisson_jacobi_identity():
    """Eq. poisson-structure-constants: the bracket closes into a Lie algebra."""
    Q = oracle.dense_table(1, 3, 4)        # inputs up to l=3, outputs up to l=4 (untruncated)
    n2 = 9                                  # inputs a, b, c with l <= 2
    nb = 16                                 # {Y_b, Y_c} has degree <= 3
    worst = 0.0
    for a in range(n2):
        for b in range(n2):
            for c in range(n2):
                t = (Q[b, c, :nb] @ Q[a, :nb, :] + Q[c, a, :nb] @ Q[b, :nb, :]
                     + Q[a, b, :nb] @ Q[c, :nb, :])
                worst = max(worst, np.abs(t).max())
    assert worst < 1e-13


def test_real_sh_matches_scipy():
    rng = np.random.default_rng(3)
    pts = rng.standard_normal((64, 3))
    pts /= np.linalg.norm(pts, axis=1, keepdims=True)
    pts[0] = [0, 0, 1]
    pts[1] = [0, 0, -1]
    assert np.abs(oracle.real_sh(10, pts) - bf.real_sh_xyz(10, pts)).max() < 1e-13
