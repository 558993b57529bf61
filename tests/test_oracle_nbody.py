"""Pins of the oracle's nu-body on-site product (the grid pointwise product extended to nu
operands followed by one inverse transform; Eq. phi-cg is nu = 2). The oracle evaluates it
as a chain of exact real Gaunt couplings in coefficient space; these tests tie it to facts
that do not depend on that chain:

* nu = 1: the projection of H_1 itself (out = U_out^T U_1^T X_1 per degree).
* nu = 2: the bilinear on-site contraction out_even.
* A constant third operand (only its l = 0 coefficient) reduces nu = 3 to nu = 2 with the
  output weights scaled per rank by H_3[r][0] Y_00.
* Dense-grid quadrature (scipy harmonics on a Gauss-Legendre x Fourier grid fine enough for
  the (nu + 1) lmax integrand) of the nu-fold product.
* Rotation equivariance, inversion parity (natural), invariance under reordering the
  operands with their factors.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.test_oracle_contractions import _parity_diag, _per_k, _rel


def _ops(lmax, nu, n=4, C=3, R=2, seed=31):
    rng = np.random.default_rng(seed)
    X = [inputs.coefficients(rng, n, C, lmax, per_degree=False) for _ in range(nu)]
    U = [inputs.cp_factors(rng, lmax, C, R) for _ in range(nu)]
    Uo = inputs.cp_factors(rng, lmax, C, R)
    return X, U, Uo


def test_nu1_is_projection():
    lmax = 3
    X, U, Uo = _ops(lmax, 1)
    got = oracle.nbody(lmax, X, U, Uo)
    H = np.einsum("knr,ink->irk", _per_k(U[0].astype(np.float64), lmax), X[0].astype(np.float64))
    ref = np.einsum("knr,irk->ink", _per_k(Uo.astype(np.float64), lmax), H)
    assert _rel(got, ref) < 1e-14


def test_nu2_is_bilinear_onsite():
    lmax = 4
    X, U, Uo = _ops(lmax, 2)
    got = oracle.nbody(lmax, X, U, Uo)
    ref = oracle.onsite(lmax, X[0], X[1], U[0], U[1], Uo, Uo)[0]
    assert _rel(got, ref) < 1e-13


def test_constant_operand_reduces_order():
    lmax = 3
    X, U, Uo = _ops(lmax, 3, seed=32)
    X3 = np.zeros_like(X[2])
    X3[:, :, 0] = X[2][:, :, 0]
    got = oracle.nbody(lmax, [X[0], X[1], X3], U, Uo)
    # per node i and rank r, field 3 is the constant H_3[i][r][0] Y_00
    H3 = np.einsum("nr,in->ir", U[2][0].astype(np.float64), X3[:, :, 0].astype(np.float64))
    y00 = 1.0 / np.sqrt(4 * np.pi)
    for i in range(X[0].shape[0]):
        Uo_i = Uo.astype(np.float64) * (H3[i] * y00)[None, None, :]
        ref = oracle.onsite(lmax, X[0][i:i + 1], X[1][i:i + 1], U[0], U[1], Uo_i, Uo_i)[0]
        assert _rel(got[i:i + 1], ref) < 1e-13


@pytest.mark.parametrize("lmax,nu", [(1, 3), (2, 3), (1, 4), (2, 4)])
def test_nbody_dense_quadrature(lmax, nu):
    X, U, Uo = _ops(lmax, nu, seed=33 + nu)
    got = oracle.nbody(lmax, X, U, Uo)
    deg = (nu + 1) * lmax
    x, w = np.polynomial.legendre.leggauss(deg // 2 + 2)
    nphi = deg + 3
    theta = np.arccos(x)
    phi = 2 * np.pi * np.arange(nphi) / nphi
    T, P = np.meshgrid(theta, phi, indexing="ij")
    Y = bf.real_sh_angles(lmax, T.ravel(), P.ravel())            # [points, K]
    W = (w[:, None] * np.full(nphi, 2 * np.pi / nphi)[None, :]).ravel()
    prod = 1.0
    for t in range(nu):
        H = np.einsum("knr,ink->irk", _per_k(U[t].astype(np.float64), lmax),
                      X[t].astype(np.float64))
        prod = prod * np.einsum("irk,pk->irp", H, Y)
    Tq = np.einsum("p,irp,pk->irk", W, prod, Y)
    ref = np.einsum("knr,irk->ink", _per_k(Uo.astype(np.float64), lmax), Tq)
    assert _rel(got, ref) < 1e-12


@pytest.mark.parametrize("nu", [3, 4])
def test_nbody_symmetries(nu):
    lmax = 3
    X, U, Uo = _ops(lmax, nu, seed=40 + nu)
    got = oracle.nbody(lmax, X, U, Uo)
    order = list(range(nu))[::-1]
    perm = oracle.nbody(lmax, [X[t] for t in order], [U[t] for t in order], Uo)
    assert _rel(perm, got) < 1e-13
    Pd = _parity_diag(lmax)
    inv = oracle.nbody(lmax, [x * Pd for x in X], U, Uo)
    assert _rel(inv, got * Pd) < 1e-13
    D = bf.wigner_d_real(lmax, bf.random_rotation(np.random.default_rng(50 + nu)))
    rot = oracle.nbody(lmax, [bf.rotate_coeffs(D, x.astype(np.float64)) for x in X], U, Uo)
    assert _rel(rot, bf.rotate_coeffs(D, got)) < 1e-12
