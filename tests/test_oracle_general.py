"""Pins of the oracle's general parameterization (Eqs. msgpass-cp-alpha, msgpass-cp-beta,
Table 1, and the on-site contraction with parity-labelled inputs).

Each coupling category (Gaunt, Category alpha; surface curl, Category beta) and each output
parity sector (out_even, parity (-1)^l; out_odd, parity -(-1)^l) has its own input factors
and output weights: four blocks b = 2 * category + sector. On-site operands may each carry
a natural and a parity-flipped slot; the message-passing node feature too.

* Stacked factor forms reduce to one another exactly: [L,C,R] is four equal blocks, the
  per-category form [2,L,C,R] is blocks (g, g, c, c), per-sector output weights are equal
  Gaunt and curl weights.
* Routing: with one slot per operand only blocks 0 (Gaunt -> out_even) and 3 (curl ->
  out_odd) are read; the other two blocks may hold anything.
* Dense-grid brute force (scipy harmonics, finite-difference surface gradients, numpy
  quadrature) of the four blocks with distinct factors, on-site and message passing.
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


def _factors(rng, nb, lmax, C, R):
    return (rng.standard_normal((nb, lmax + 1, C, R)) / np.sqrt(C)).astype(np.float32)


def _onsite_d(lmax, n=3, C=3, R=4, seed=11):
    d = inputs.onsite_inputs(n, lmax, C, R, seed=seed, distinct_out=True)
    rng = np.random.default_rng(seed + 1000)
    K = (lmax + 1) ** 2
    d["A_flip"] = rng.standard_normal((n, C, K)).astype(np.float32)
    d["B_flip"] = rng.standard_normal((n, C, K)).astype(np.float32)
    d["UA4"] = _factors(rng, 4, lmax, C, R)
    d["UB4"] = _factors(rng, 4, lmax, C, R)
    d["Uoe2"] = _factors(rng, 2, lmax, C, R)
    d["Uoo2"] = _factors(rng, 2, lmax, C, R)
    return d


def _on(lmax, d, **over):
    a = dict(A=d["A"], B=d["B"], U_A=d["UA4"], U_B=d["UB4"], U_out_even=d["Uoe2"],
             U_out_odd=d["Uoo2"], A_flip=d["A_flip"], B_flip=d["B_flip"])
    a.update(over)
    return oracle.onsite(lmax, **a)


def _block(cat, rel):
    """Block of the coupling of category cat (0 Gaunt, 1 curl) for a slot pair of relative
    parity rel (0 equal, 1 mixed), by p = p1 p2 (Table 1)."""
    return 2 * cat + (rel if cat == 0 else 1 - rel)


def _sum_blocks(lmax, S, Uo, W, Y):
    """out_sec = sum over categories of the projection of the analysed block field."""
    outs = []
    for sec in range(2):
        o = 0.0
        for cat in range(2):
            b = 2 * cat + sec
            if S[b] is None:
                continue
            T = np.einsum("p,...rp,pk->...rk", W, S[b], Y)
            o = o + np.einsum("knr,...rk->...nk", Uo[b], T)
        outs.append(o)
    return outs


def _brute_onsite_general(lmax, d):
    Y, Dt, Dp, W = bf.sh_and_derivs(lmax)
    UA = [_per_k(d["UA4"][b].astype(np.float64), lmax) for b in range(4)]
    UB = [_per_k(d["UB4"][b].astype(np.float64), lmax) for b in range(4)]
    Uo = [_per_k(d["Uoe2" if b % 2 == 0 else "Uoo2"][b // 2].astype(np.float64), lmax)
          for b in range(4)]
    X1 = [d["A"].astype(np.float64), d["A_flip"].astype(np.float64)]
    X2 = [d["B"].astype(np.float64), d["B_flip"].astype(np.float64)]
    S = [None] * 4
    for s1 in range(2):
        for s2 in range(2):
            for cat in range(2):
                b = _block(cat, s1 != s2)
                h1 = np.einsum("knr,ink->irk", UA[b], X1[s1])
                h2 = np.einsum("knr,ink->irk", UB[b], X2[s2])
                a1, t1, p1 = _grid_fields(h1, Y, Dt, Dp)
                a2, t2, p2 = _grid_fields(h2, Y, Dt, Dp)
                v = a1 * a2 if cat == 0 else bf.bracket(t1, p1, t2, p2)
                S[b] = v if S[b] is None else S[b] + v
    return _sum_blocks(lmax, S, Uo, W, Y)


def test_onsite_factor_forms_reduce_exactly():
    lmax = 3
    d = _onsite_d(lmax)
    U, V = d["U_A"], d["U_B"]
    shared = _on(lmax, d, U_A=U, U_B=V, U_out_even=d["U_out_even"], U_out_odd=d["U_out_odd"])
    four = _on(lmax, d, U_A=np.stack([U] * 4), U_B=np.stack([V] * 4),
               U_out_even=np.stack([d["U_out_even"]] * 2), U_out_odd=np.stack([d["U_out_odd"]] * 2))
    g, c = d["UA4"][0], d["UA4"][3]
    two = _on(lmax, d, U_A=np.stack([g, c]))
    twof = _on(lmax, d, U_A=np.stack([g, g, c, c]))
    for x, y in ((shared, four), (two, twof)):
        assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])
    base = oracle.onsite(lmax, d["A"], d["B"], U, V, d["U_out_even"], d["U_out_odd"])
    one = _on(lmax, d, U_A=U, U_B=V, U_out_even=d["U_out_even"], U_out_odd=d["U_out_odd"],
              A_flip=None, B_flip=None)
    assert np.array_equal(base[0], one[0]) and np.array_equal(base[1], one[1])


def test_onsite_single_slot_reads_blocks_0_and_3_only():
    lmax = 4
    d = _onsite_d(lmax, seed=12)
    ref = _on(lmax, d, A_flip=None, B_flip=None)
    junk = {k: d[k].copy() for k in ("UA4", "UB4")}
    for k in junk:
        junk[k][1:3] = 7.0
    Uoe, Uoo = d["Uoe2"].copy(), d["Uoo2"].copy()
    Uoe[1] = -3.0     # curl weights of out_even: no curl coupling reaches it
    Uoo[0] = 5.0      # Gaunt weights of out_odd
    got = _on(lmax, d, A_flip=None, B_flip=None, U_A=junk["UA4"], U_B=junk["UB4"],
              U_out_even=Uoe, U_out_odd=Uoo)
    assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])
    # block 0 alone is the shared-factor Gaunt output, block 3 the curl output
    g = oracle.onsite(lmax, d["A"], d["B"], d["UA4"][0], d["UB4"][0], d["Uoe2"][0], d["Uoo2"][1])
    c = oracle.onsite(lmax, d["A"], d["B"], d["UA4"][3], d["UB4"][3], d["Uoe2"][0], d["Uoo2"][1])
    assert _rel(ref[0], g[0]) < 1e-14 and _rel(ref[1], c[1]) < 1e-14


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

def _mp_d(lmax, seed=5, C=3, R=2):
    d = inputs.mp_inputs(14, lmax, C, R, seed, density=0.1, r_cut=2.5, distinct_out=True,
                         two_slot=True)
    rng = np.random.default_rng(seed + 2000)
    d["UE4"] = _factors(rng, 4, lmax, C, R)
    d["UI4"] = _factors(rng, 4, lmax, C, R)
    d["Uoe2"] = _factors(rng, 2, lmax, C, R)
    d["Uoo2"] = _factors(rng, 2, lmax, C, R)
    return d


def _mp(lmax, d, rec, **over):
    a = dict(row_ptr=d["row_ptr"], col=d["col"], edge_unit=d["edge_unit"],
             edge_radial=d["edge_radial"], node_feat=d["node_feat"], U_E=d["UE4"], U_I=d["UI4"],
             U_out_even=d["Uoe2"], U_out_odd=d["Uoo2"], receivers=rec, node_flip=d["node_flip"])
    a.update(over)
    return oracle.message_pass(lmax, **a)


def test_mp_factor_forms_and_routing():
    lmax = 3
    d = _mp_d(lmax)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    shared = _mp(lmax, d, rec, U_E=d["U_E"], U_I=d["U_I"], U_out_even=d["U_out_even"],
                 U_out_odd=d["U_out_odd"])
    four = _mp(lmax, d, rec, U_E=np.stack([d["U_E"]] * 4), U_I=np.stack([d["U_I"]] * 4),
               U_out_even=np.stack([d["U_out_even"]] * 2),
               U_out_odd=np.stack([d["U_out_odd"]] * 2))
    assert np.array_equal(shared[0], four[0]) and np.array_equal(shared[1], four[1])
    ref = _mp(lmax, d, rec, node_flip=None)
    junk = {k: d[k].copy() for k in ("UE4", "UI4")}
    for k in junk:
        junk[k][1:3] = 7.0
    Uoe, Uoo = d["Uoe2"].copy(), d["Uoo2"].copy()
    Uoe[1], Uoo[0] = -3.0, 5.0
    got = _mp(lmax, d, rec, node_flip=None, U_E=junk["UE4"], U_I=junk["UI4"], U_out_even=Uoe,
              U_out_odd=Uoo)
    assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])


@pytest.mark.parametrize("lmax", [1, 2, 3])
def test_mp_general_matches_dense_bruteforce(lmax):
    d = _mp_d(lmax, seed=6)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    Y, Dt, Dp, W = bf.sh_and_derivs(lmax)
    UE = [_per_k(d["UE4"][b].astype(np.float64), lmax) for b in range(4)]
    UI = [_per_k(d["UI4"][b].astype(np.float64), lmax) for b in range(4)]
    Uo = [_per_k(d["Uoe2" if b % 2 == 0 else "Uoo2"][b // 2].astype(np.float64), lmax)
          for b in range(4)]
    Ye = bf.real_sh_xyz(lmax, d["edge_unit"].astype(np.float64))
    rad = d["edge_radial"].astype(np.float64)
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    X2 = [d["node_feat"].astype(np.float64), d["node_flip"].astype(np.float64)]
    rp, col = d["row_ptr"], d["col"]
    S = [np.zeros((len(rec), UE[0].shape[2], Y.shape[0])) for _ in range(4)]
    for q, i in enumerate(rec):
        for e in range(rp[i], rp[i + 1]):
            j = col[e]
            for s2 in range(2):
                for cat in range(2):
                    b = _block(cat, s2)
                    he = np.einsum("knr,nk->rk", UE[b], rad[e][:, lk]) * Ye[e][None, :]
                    hi = np.einsum("knr,nk->rk", UI[b], X2[s2][j])
                    ae, te, pe = _grid_fields(he, Y, Dt, Dp)
                    ai, ti, pi = _grid_fields(hi, Y, Dt, Dp)
                    S[b][q] += ae * ai if cat == 0 else bf.bracket(te, pe, ti, pi)
    bn, bo = _sum_blocks(lmax, S, Uo, W, Y)
    assert _rel(on, bn) < 1e-8
    assert _rel(oo, bo) < 1e-8
    assert np.abs(on).max() > 1e-2 and np.abs(oo).max() > 1e-2


def test_mp_general_inversion():
    lmax = 4
    d = _mp_d(lmax, seed=9)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    P = _parity_diag(lmax)
    inn, ino = _mp(lmax, d, rec, edge_unit=-d["edge_unit"].astype(np.float64),
                   node_feat=d["node_feat"] * P, node_flip=-d["node_flip"] * P)
    assert _rel(inn, on * P) < 1e-13
    assert _rel(ino, -oo * P) < 1e-13
