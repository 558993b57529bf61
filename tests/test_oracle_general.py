"""Pins of the oracle's general parity parameterization: independent factors for the Gaunt
(Category alpha) and curl (Category beta) couplings (Eqs. msgpass-cp-alpha, msgpass-cp-beta),
and on-site operands that each carry a natural- and a parity-flipped slot (the two
parity-bearing factors case, Eq. twoparity-phi with the on-site specialization).

* Without the optional inputs, and with the curl factors equal to the Gaunt ones, the
  results are the single-slot shared-factor ones, exactly.
* With one slot each, out_even does not depend on the curl factors and out_odd equals the
  shared-factor result computed with the curl factors.
* Dense-grid brute force (scipy harmonics, finite-difference surface gradients, numpy
  quadrature) of the on-site sum over the four slot pairs and of message passing with
  independent factors.
* Inversion with each slot multiplied by its own parity; rotation equivariance.
* On-site dispatch check in the manner of App. B: operand 1 restricted to one degree l1 in
  its natural slot, operand 2 only in the slot of absolute parity +1: only output sectors of
  parity (-1)^l1 are non-zero.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.test_oracle_contractions import _grid_fields, _parity_diag, _per_k, _rel


def _onsite_d(lmax, n=3, C=3, R=4, seed=11):
    d = inputs.onsite_inputs(n, lmax, C, R, seed=seed, distinct_out=True)
    rng = np.random.default_rng(seed + 1000)
    K = (lmax + 1) ** 2
    d["A_flip"] = rng.standard_normal((n, C, K)).astype(np.float32)
    d["B_flip"] = rng.standard_normal((n, C, K)).astype(np.float32)
    d["U_A_curl"] = (rng.standard_normal((lmax + 1, C, R)) / np.sqrt(C)).astype(np.float32)
    d["U_B_curl"] = (rng.standard_normal((lmax + 1, C, R)) / np.sqrt(C)).astype(np.float32)
    return d


def _on(lmax, d, **over):
    a = dict(A=d["A"], B=d["B"], U_A=d["U_A"], U_B=d["U_B"], U_out_even=d["U_out_even"],
             U_out_odd=d["U_out_odd"], A_flip=d["A_flip"], B_flip=d["B_flip"],
             U_A_curl=d["U_A_curl"], U_B_curl=d["U_B_curl"])
    a.update(over)
    return oracle.onsite(lmax, **a)


def _brute_onsite_general(lmax, d):
    Y, Dt, Dp, W = bf.sh_and_derivs(lmax)
    f64 = lambda k: d[k].astype(np.float64)
    U = {k: _per_k(f64(k), lmax) for k in ("U_A", "U_B", "U_A_curl", "U_B_curl",
                                           "U_out_even", "U_out_odd")}
    H = lambda Uk, X: np.einsum("knr,ink->irk", U[Uk], f64(X))
    slots1 = {"n": "A", "f": "A_flip"}
    slots2 = {"n": "B", "f": "B_flip"}
    Sn = So = 0.0
    for s1, x1 in slots1.items():
        for s2, x2 in slots2.items():
            a1 = _grid_fields(H("U_A", x1), Y, Dt, Dp)[0]
            a2 = _grid_fields(H("U_B", x2), Y, Dt, Dp)[0]
            _, t1, p1 = _grid_fields(H("U_A_curl", x1), Y, Dt, Dp)
            _, t2, p2 = _grid_fields(H("U_B_curl", x2), Y, Dt, Dp)
            g, c = a1 * a2, bf.bracket(t1, p1, t2, p2)
            if s1 == s2:
                Sn, So = Sn + g, So + c
            else:
                Sn, So = Sn + c, So + g
    Tn = np.einsum("p,irp,pk->irk", W, Sn, Y)
    To = np.einsum("p,irp,pk->irk", W, So, Y)
    return (np.einsum("knr,irk->ink", U["U_out_even"], Tn),
            np.einsum("knr,irk->ink", U["U_out_odd"], To))


def test_onsite_optional_inputs_reduce_to_base():
    lmax = 3
    d = _onsite_d(lmax)
    base = oracle.onsite(lmax, d["A"], d["B"], d["U_A"], d["U_B"], d["U_out_even"],
                         d["U_out_odd"])
    none = _on(lmax, d, A_flip=None, B_flip=None, U_A_curl=None, U_B_curl=None)
    same = _on(lmax, d, A_flip=None, B_flip=None, U_A_curl=d["U_A"], U_B_curl=d["U_B"])
    for o in (none, same):
        assert np.array_equal(o[0], base[0]) and np.array_equal(o[1], base[1])


def test_onsite_independent_factors_route_by_category():
    lmax = 4
    d = _onsite_d(lmax, seed=12)
    ind = _on(lmax, d, A_flip=None, B_flip=None)
    base_g = oracle.onsite(lmax, d["A"], d["B"], d["U_A"], d["U_B"], d["U_out_even"],
                           d["U_out_odd"])
    base_c = oracle.onsite(lmax, d["A"], d["B"], d["U_A_curl"], d["U_B_curl"],
                           d["U_out_even"], d["U_out_odd"])
    assert _rel(ind[0], base_g[0]) < 1e-14
    assert _rel(ind[1], base_c[1]) < 1e-14


@pytest.mark.parametrize("lmax", [1, 2, 3])
def test_onsite_general_matches_dense_bruteforce(lmax):
    d = _onsite_d(lmax, seed=13)
    oe, oo = _on(lmax, d)
    be, bo = _brute_onsite_general(lmax, d)
    assert _rel(oe, be) < 1e-8
    assert _rel(oo, bo) < 1e-8
    assert np.abs(oe).max() > 1e-2 and np.abs(oo).max() > 1e-2


@pytest.mark.parametrize("lmax", [2, 4])
def test_onsite_general_inversion_and_rotation(lmax):
    d = _onsite_d(lmax, n=4, seed=14)
    oe, oo = _on(lmax, d)
    P = _parity_diag(lmax)
    ie, io = _on(lmax, d, A=d["A"] * P, B=d["B"] * P, A_flip=-d["A_flip"] * P,
                 B_flip=-d["B_flip"] * P)
    assert _rel(ie, oe * P) < 1e-13
    assert _rel(io, -oo * P) < 1e-13
    D = bf.wigner_d_real(lmax, bf.random_rotation(np.random.default_rng(21)))
    rot = {k: bf.rotate_coeffs(D, d[k].astype(np.float64)) for k in ("A", "B", "A_flip", "B_flip")}
    re_, ro = _on(lmax, d, **rot)
    assert _rel(re_, bf.rotate_coeffs(D, oe)) < 1e-12
    assert _rel(ro, bf.rotate_coeffs(D, oo)) < 1e-12


@pytest.mark.parametrize("l1", [1, 2])
def test_onsite_dispatch_rule_single_degree(l1):
    lmax = 3
    d = _onsite_d(lmax, n=3, seed=15)
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    A = np.where((lk == l1)[None, None, :], d["A"].astype(np.float64), 0.0)
    even_l = lk % 2 == 0
    X = d["B"].astype(np.float64)
    Bn = np.where(even_l[None, None, :], X, 0.0)    # absolute parity +1: natural at even l2
    Bf = np.where(even_l[None, None, :], 0.0, X)    # ... flipped at odd l2
    oe, oo = _on(lmax, d, A=A, A_flip=None, B=Bn, B_flip=Bf)
    want = (-1) ** l1
    p_even = np.where(even_l, 1, -1)
    scale = max(np.abs(oe).max(), np.abs(oo).max())
    for out, par in ((oe, p_even), (oo, -p_even)):
        assert np.abs(out[:, :, par != want]).max() <= 1e-14 * scale
    assert max(np.abs(oe[:, :, p_even == want]).max(),
               np.abs(oo[:, :, -p_even == want]).max()) > 1e-3 * scale


# ------------------------------------------------------------------ message passing ---

def _mp_d(lmax, seed=5):
    d = inputs.mp_inputs(14, lmax, 3, 2, seed, density=0.1, r_cut=2.5, distinct_out=True,
                         two_slot=True)
    rng = np.random.default_rng(seed + 2000)
    d["U_E_curl"] = (rng.standard_normal((lmax + 1, 3, 2)) / np.sqrt(3)).astype(np.float32)
    d["U_I_curl"] = (rng.standard_normal((lmax + 1, 3, 2)) / np.sqrt(3)).astype(np.float32)
    return d


def _mp(lmax, d, rec, **over):
    a = dict(row_ptr=d["row_ptr"], col=d["col"], edge_unit=d["edge_unit"],
             edge_radial=d["edge_radial"], node_feat=d["node_feat"], U_E=d["U_E"], U_I=d["U_I"],
             U_out_even=d["U_out_even"], U_out_odd=d["U_out_odd"], receivers=rec,
             node_flip=d["node_flip"], U_E_curl=d["U_E_curl"], U_I_curl=d["U_I_curl"])
    a.update(over)
    return oracle.message_pass(lmax, **a)


def test_mp_independent_factors_route_by_category():
    lmax = 3
    d = _mp_d(lmax)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    ind = _mp(lmax, d, rec, node_flip=None)
    base_g = _mp(lmax, d, rec, node_flip=None, U_E_curl=None, U_I_curl=None)
    base_c = _mp(lmax, d, rec, node_flip=None, U_E_curl=None, U_I_curl=None,
                 U_E=d["U_E_curl"], U_I=d["U_I_curl"])
    assert _rel(ind[0], base_g[0]) < 1e-14
    assert _rel(ind[1], base_c[1]) < 1e-14
    same = _mp(lmax, d, rec, U_E_curl=d["U_E"], U_I_curl=d["U_I"])
    shared = _mp(lmax, d, rec, U_E_curl=None, U_I_curl=None)
    assert np.array_equal(same[0], shared[0]) and np.array_equal(same[1], shared[1])


@pytest.mark.parametrize("lmax", [1, 2, 3])
def test_mp_general_matches_dense_bruteforce(lmax):
    d = _mp_d(lmax, seed=6)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    Y, Dt, Dp, W = bf.sh_and_derivs(lmax)
    f64 = lambda k: d[k].astype(np.float64)
    U = {k: _per_k(f64(k), lmax) for k in ("U_E", "U_I", "U_E_curl", "U_I_curl",
                                           "U_out_even", "U_out_odd")}
    Ye = bf.real_sh_xyz(lmax, f64("edge_unit"))
    rad = f64("edge_radial")
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    HEg = np.einsum("knr,enk->erk", U["U_E"], rad[:, :, lk]) * Ye[:, None, :]
    HEc = np.einsum("knr,enk->erk", U["U_E_curl"], rad[:, :, lk]) * Ye[:, None, :]
    HI = {(s, c): np.einsum("knr,ink->irk", U[c], f64(s)) for s in ("node_feat", "node_flip")
          for c in ("U_I", "U_I_curl")}
    rp, col = d["row_ptr"], d["col"]
    bn, bo = [], []
    for i in rec:
        Sn = So = 0.0
        for e in range(rp[i], rp[i + 1]):
            j = col[e]
            ag = _grid_fields(HEg[e], Y, Dt, Dp)[0]
            _, tc, pc = _grid_fields(HEc[e], Y, Dt, Dp)
            an = _grid_fields(HI[("node_feat", "U_I")][j], Y, Dt, Dp)[0]
            af = _grid_fields(HI[("node_flip", "U_I")][j], Y, Dt, Dp)[0]
            _, tn, pn = _grid_fields(HI[("node_feat", "U_I_curl")][j], Y, Dt, Dp)
            _, tf, pf = _grid_fields(HI[("node_flip", "U_I_curl")][j], Y, Dt, Dp)
            Sn = Sn + ag * an + bf.bracket(tc, pc, tf, pf)
            So = So + bf.bracket(tc, pc, tn, pn) + ag * af
        bn.append(np.einsum("knr,rk->nk", U["U_out_even"], np.einsum("p,rp,pk->rk", W, Sn, Y)))
        bo.append(np.einsum("knr,rk->nk", U["U_out_odd"], np.einsum("p,rp,pk->rk", W, So, Y)))
    assert _rel(on, np.array(bn)) < 1e-8
    assert _rel(oo, np.array(bo)) < 1e-8
