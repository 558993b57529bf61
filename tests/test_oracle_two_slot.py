"""Pins of the oracle's message passing with both node parity slots (Table 1, Cases A-D).

The node features carry a natural-parity slot, parity (-1)^l2, and a parity-flipped slot,
parity -(-1)^l2. The edge feature R Y has natural parity. By the parity rule p = p1 p2, the
natural-parity output of degree l collects the Gaunt coupling with the natural slot and the
surface-curl coupling with the flipped slot; the opposite-parity output the other two.

* Flipped slot zero: the single-slot result, exactly.
* Dense-grid brute force (scipy harmonics, finite-difference surface gradients, numpy
  quadrature) of all four couplings at tiny sizes.
* Inversion: with the edge directions reversed and each slot multiplied by its own parity,
  out_even picks up (-1)^l and out_odd -(-1)^l. Any other routing of the four couplings
  breaks this.
* The dispatch check of App. B: with the edge restricted to one degree l1 and only the
  slot of absolute parity +1 populated, only output sectors of parity (-1)^l1 are non-zero.
* Rotation equivariance with both slots populated.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.test_oracle_contractions import _grid_fields, _parity_diag, _per_k, _rel


def _tiny(lmax, seed=5, C=3, R=2):
    return inputs.mp_inputs(14, lmax, C, R, seed, density=0.1, r_cut=2.5, distinct_out=True,
                            two_slot=True)


def _mp(lmax, d, rec, **over):
    a = dict(row_ptr=d["row_ptr"], col=d["col"], edge_unit=d["edge_unit"],
             edge_radial=d["edge_radial"], node_feat=d["node_feat"], U_E=d["U_E"], U_I=d["U_I"],
             U_out_even=d["U_out_even"], U_out_odd=d["U_out_odd"], receivers=rec,
             node_flip=d["node_flip"])
    a.update(over)
    return oracle.message_pass(lmax, **a)


def _brute_two_slot(lmax, d, receivers):
    Y, Dt, Dp, W = bf.sh_and_derivs(lmax)
    UE, UI = _per_k(d["U_E"].astype(np.float64), lmax), _per_k(d["U_I"].astype(np.float64), lmax)
    Uoe, Uoo = (_per_k(d[k].astype(np.float64), lmax) for k in ("U_out_even", "U_out_odd"))
    rp, col = d["row_ptr"], d["col"]
    Hn = np.einsum("knr,ink->irk", UI, d["node_feat"].astype(np.float64))
    Hf = np.einsum("knr,ink->irk", UI, d["node_flip"].astype(np.float64))
    Ye = bf.real_sh_xyz(lmax, d["edge_unit"].astype(np.float64))
    rad = d["edge_radial"].astype(np.float64)
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    HE = np.einsum("knr,enk->erk", UE, rad[:, :, lk]) * Ye[:, None, :]
    out_n, out_o = [], []
    for i in receivers:
        Sn = np.zeros((Hn.shape[1], Y.shape[0]))
        So = np.zeros_like(Sn)
        for e in range(rp[i], rp[i + 1]):
            j = col[e]
            ae, te, pe = _grid_fields(HE[e], Y, Dt, Dp)
            an, tn, pn = _grid_fields(Hn[j], Y, Dt, Dp)
            af, tf, pf = _grid_fields(Hf[j], Y, Dt, Dp)
            Sn += ae * an + bf.bracket(te, pe, tf, pf)
            So += bf.bracket(te, pe, tn, pn) + ae * af
        Tn = np.einsum("p,rp,pk->rk", W, Sn, Y)
        To = np.einsum("p,rp,pk->rk", W, So, Y)
        out_n.append(np.einsum("knr,rk->nk", Uoe, Tn))
        out_o.append(np.einsum("knr,rk->nk", Uoo, To))
    return np.array(out_n), np.array(out_o)


def test_flipped_slot_zero_is_single_slot():
    lmax = 3
    d = _tiny(lmax)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    two = _mp(lmax, d, rec, node_flip=np.zeros_like(d["node_flip"]))
    one = _mp(lmax, d, rec, node_flip=None)
    assert np.array_equal(two[0], one[0]) and np.array_equal(two[1], one[1])


@pytest.mark.parametrize("lmax", [1, 2, 3])
def test_two_slot_matches_dense_bruteforce(lmax):
    d = _tiny(lmax, seed=6)
    assert d["n_edges"] > 10
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    bn, bo = _brute_two_slot(lmax, d, rec)
    # both outputs now hold a curl term: finite-difference gradients bound the agreement
    assert _rel(on, bn) < 1e-8
    assert _rel(oo, bo) < 1e-8
    assert np.abs(oo).max() > 1e-2 and np.abs(on).max() > 1e-2


@pytest.mark.parametrize("lmax", [2, 4])
def test_two_slot_inversion_parity(lmax):
    d = _tiny(lmax, seed=9)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    P = _parity_diag(lmax)
    # inversion: the edge direction reverses; the natural slot transforms with (-1)^l, the
    # flipped slot with -(-1)^l
    inn, ino = _mp(lmax, d, rec, edge_unit=-d["edge_unit"].astype(np.float64),
                   node_feat=d["node_feat"] * P, node_flip=-d["node_flip"] * P)
    assert _rel(inn, on * P) < 1e-13
    assert _rel(ino, -oo * P) < 1e-13
    # each output holds two couplings of the same parity: both are present
    for sub in ({"node_flip": np.zeros_like(d["node_flip"])},
                {"node_feat": np.zeros_like(d["node_feat"])}):
        pn, po = _mp(lmax, d, rec, **sub)
        assert np.abs(pn).max() > 1e-2 * np.abs(on).max()
        assert np.abs(po).max() > 1e-2 * np.abs(oo).max()


@pytest.mark.parametrize("l1", [0, 1])
def test_dispatch_rule_single_edge_degree(l1):
    """App. B: edge restricted to degree l1, node features only in the slot of absolute
    parity +1; the outputs of parity -(-1)^l1 vanish exactly, those of parity (-1)^l1 do
    not."""
    lmax = 2
    d = _tiny(lmax, seed=13)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    rad = d["edge_radial"].astype(np.float64).copy()
    keep = np.zeros(lmax + 1)
    keep[l1] = 1.0
    rad *= keep[None, None, :]
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    even_l = (lk % 2 == 0)
    X = d["node_feat"].astype(np.float64)
    nat = np.where(even_l[None, None, :], X, 0.0)     # absolute parity +1: natural at even l2
    flip = np.where(even_l[None, None, :], 0.0, X)    # ... and flipped at odd l2
    on, oo = _mp(lmax, d, rec, edge_radial=rad, node_feat=nat, node_flip=flip)
    # absolute output parity: out_even (natural) has (-1)^l, out_odd -(-1)^l
    p_even = np.where(even_l, 1, -1)
    p_odd = -p_even
    want = (-1) ** l1
    scale = max(np.abs(on).max(), np.abs(oo).max())
    for out, par in ((on, p_even), (oo, p_odd)):
        zero = out[:, :, par != want]
        live = out[:, :, par == want]
        assert np.abs(zero).max() <= 1e-14 * scale
        if live.size:
            assert np.abs(live).max() > 1e-3 * scale


def test_two_slot_rotation_equivariance():
    lmax = 3
    d = _tiny(lmax, seed=17)
    rec = np.arange(d["row_ptr"].shape[0] - 1)
    on, oo = _mp(lmax, d, rec)
    rng = np.random.default_rng(8)
    rot = bf.random_rotation(rng)
    D = bf.wigner_d_real(lmax, rot)
    rn, ro = _mp(lmax, d, rec, edge_unit=d["edge_unit"].astype(np.float64) @ rot.T,
                 node_feat=bf.rotate_coeffs(D, d["node_feat"].astype(np.float64)),
                 node_flip=bf.rotate_coeffs(D, d["node_flip"].astype(np.float64)))
    assert _rel(rn, bf.rotate_coeffs(D, on)) < 1e-12
    assert _rel(ro, bf.rotate_coeffs(D, oo)) < 1e-12
