"""GPU parity of message passing with both node parity slots (Table 1, Cases A-D):
libcgtp's cgtp_message_pass_two_slot against the fp64 oracle, element by element on the
same seeded inputs. fp32 bar: max|gpu - ref| / max|ref| <= 2e-5 per output slot; the fp64
build must agree to 1e-11. Covers the per-thread receiver (lmax <= 6, ranks not a multiple
of 16) and the MFMA receiver (lmax >= 7, ranks a multiple of 16)."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.gpu_util import (MP_KEYS, TOL_F32, TOL_F64, bench_order, rel_err, run_mp,
                            same_without_order, sample_rows, to_dev)

pytestmark = pytest.mark.gpu

KEYS2 = MP_KEYS + ("node_flip",)


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _mp2(lmax, n=48, C=5, R=6, seed=1, r_cut=3.5):
    return inputs.mp_inputs(n, lmax, C, R, seed, r_cut=r_cut, distinct_out=True, two_slot=True)


def _run2(cg, plan, t, **kw):
    return run_mp(cg, plan, t, node_flip=t["node_flip"], **kw)


def _oracle2(lmax, d, receivers=None):
    return oracle.message_pass(lmax, *(d[k] for k in MP_KEYS), receivers=receivers,
                               node_flip=d["node_flip"])


def _check(gpu, ref, tol, nodes=None):
    ge, go = gpu
    if nodes is not None:
        ge, go = ge[nodes], go[nodes]
    ee, eo = rel_err(ge, ref[0]), rel_err(go, ref[1])
    assert ee <= tol and eo <= tol, f"rel err even {ee:.3e} odd {eo:.3e} (tol {tol:g})"


@pytest.mark.parametrize("lmax,R", [(0, 3), (2, 6), (5, 8), (6, 9)])
def test_two_slot_per_thread_receiver(cg, lmax, R):
    d = _mp2(lmax, R=R, seed=80 + lmax)
    plan = cg.plan_create(lmax, 5, R)
    _check(_run2(cg, plan, to_dev(d, KEYS2)), _oracle2(lmax, d), TOL_F32)


@pytest.mark.parametrize("lmax,R", [(7, 16), (8, 32), (12, 16), (20, 16)])
def test_two_slot_mfma_receiver(cg, lmax, R):
    d = _mp2(lmax, n=40, C=4, R=R, seed=90 + lmax)
    plan = cg.plan_create(lmax, 4, R)
    _check(_run2(cg, plan, to_dev(d, KEYS2)), _oracle2(lmax, d), TOL_F32)


def test_two_slot_fp64_matches_oracle_tightly(cg):
    lmax = 4
    d = _mp2(lmax, n=40, C=3, R=4, seed=97)
    plan = cg.plan_create(lmax, 3, 4, dtype="f64")
    _check(_run2(cg, plan, to_dev(d, KEYS2, "f64")), _oracle2(lmax, d), TOL_F64)


@pytest.mark.parametrize("lmax,R", [(4, 6), (9, 16)])
def test_zero_flipped_slot_equals_single_slot(cg, lmax, R):
    import torch

    d = _mp2(lmax, n=40, C=4, R=R, seed=99)
    t = to_dev(d, KEYS2)
    plan = cg.plan_create(lmax, 4, R)
    one = run_mp(cg, plan, t)
    two = run_mp(cg, plan, t, node_flip=torch.zeros_like(t["node_flip"]))
    for a, b in zip(one, two):
        assert torch.equal(a, b)


def test_two_slot_inversion_on_gpu(cg):
    """Edge directions reversed and each slot multiplied by its own parity: out_even picks
    up (-1)^l and out_odd -(-1)^l (Table 1)."""
    lmax = 8
    d = _mp2(lmax, n=40, C=4, R=16, seed=101)
    plan = cg.plan_create(lmax, 4, 16)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in _run2(cg, plan, to_dev(d, KEYS2)))
    P = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(lmax + 1)])
    di = dict(d)
    di["edge_unit"] = -d["edge_unit"]
    di["node_feat"] = (d["node_feat"] * P).astype(np.float32)
    di["node_flip"] = (-d["node_flip"] * P).astype(np.float32)
    ie, io = _run2(cg, plan, to_dev(di, KEYS2))
    assert rel_err(ie, oe * P) <= TOL_F32
    assert rel_err(io, -oo * P) <= TOL_F32


def test_two_slot_rotation_equivariance_gpu(cg):
    lmax = 5
    d = _mp2(lmax, n=48, C=4, R=6, seed=103)
    plan = cg.plan_create(lmax, 4, 6)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in _run2(cg, plan, to_dev(d, KEYS2)))
    rot = bf.random_rotation(np.random.default_rng(11))
    D = bf.wigner_d_real(lmax, rot)
    dr = dict(d)
    dr["edge_unit"] = d["edge_unit"].astype(np.float64) @ rot.T
    dr["node_feat"] = bf.rotate_coeffs(D, d["node_feat"].astype(np.float64))
    dr["node_flip"] = bf.rotate_coeffs(D, d["node_flip"].astype(np.float64))
    re_, ro = _run2(cg, plan, to_dev(dr, KEYS2))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


def test_two_slot_workspace_and_errors(cg):
    import torch

    lmax = 3
    d = _mp2(lmax, n=30, C=3, R=4, seed=105, r_cut=3.0)
    t = to_dev(d, KEYS2)
    plan = cg.plan_create(lmax, 3, 4)
    N, E = d["node_feat"].shape[0], d["n_edges"]
    one = cg.workspace_bytes(plan, cg.CGTP_OP_MESSAGE_PASS, N, E)
    two = cg.workspace_bytes(plan, cg.CGTP_OP_MESSAGE_PASS_TWO_SLOT, N, E)
    assert two > one
    ws = torch.empty(two, dtype=torch.uint8, device="cuda")
    _check(_run2(cg, plan, t, workspace=ws), _oracle2(lmax, d), TOL_F32)
    with pytest.raises(cg.CgtpError) as ei:
        _run2(cg, plan, t, workspace=ws[: one])
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    sep = cg.plan_create(lmax, 3, 4, flags=cg.CGTP_EDGE_SEPARATED)
    with pytest.raises(cg.CgtpError) as ei:
        _run2(cg, sep, t)
    assert ei.value.status == cg.CGTP_ERR_UNSUPPORTED
    lib = cg.load_library()
    oe = torch.empty_like(t["node_feat"])
    st = lib.cgtp_message_pass_two_slot(
        plan.handle, N, E, t["row_ptr"].data_ptr(), t["col"].data_ptr(),
        t["edge_unit"].data_ptr(), t["edge_radial"].data_ptr(), t["node_feat"].data_ptr(), None,
        t["U_E"].data_ptr(), t["U_I"].data_ptr(), t["U_out_even"].data_ptr(),
        t["U_out_odd"].data_ptr(), oe.data_ptr(), None, None, ctypes.c_size_t(0), None)
    assert st == cg.CGTP_ERR_ARG


def test_two_slot_stage_times(cg):
    lmax = 2
    d = _mp2(lmax, n=30, C=3, R=4, seed=107, r_cut=3.0)
    t = to_dev(d, KEYS2)
    plan = cg.plan_create(lmax, 3, 4, flags=cg.CGTP_TIME_STAGES)
    for _ in range(2):
        _run2(cg, plan, t)
    stages, calls = cg.stage_times(plan, cg.CGTP_OP_MESSAGE_PASS_TWO_SLOT)
    assert calls == 2 and len(stages) == 7 and all(v >= 0 for v in stages.values())
    assert cg.stage_times(plan, cg.CGTP_OP_MESSAGE_PASS)[1] == 0


def test_mp2_10k_l6_sampled(cg):
    import torch

    w = inputs.WORKLOADS["mp2_10k_l6_c128"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    bench_order(cg, plan, d)
    t = to_dev(d, KEYS2)
    gpu = _run2(cg, plan, t)
    rec = sample_rows(w.n, 128, seed=3)
    assert len(rec) == 128
    _check(gpu, _oracle2(w.lmax, d, rec), TOL_F32, nodes=rec)
    again = _run2(cg, plan, t)
    assert torch.equal(gpu[0], again[0]) and torch.equal(gpu[1], again[1])
    same_without_order(cg, plan, lambda p: _run2(cg, p, t), gpu)


_L20 = {}


def _mp2_5k_l20(cg):
    """The lmax-20 two-slot workload run once on the GPU; its outputs are checked in eight
    parts so that each test's oracle work stays well inside the per-test time limit."""
    if "run" not in _L20:
        w = inputs.WORKLOADS["mp2_5k_l20_c64"]
        d = w.make()
        plan = cg.plan_create(w.lmax, w.C, w.R)
        bench_order(cg, plan, d)
        t = to_dev(d, KEYS2)
        ge, go = _run2(cg, plan, t)
        same_without_order(cg, plan, lambda p: _run2(cg, p, t), (ge, go))
        _L20["run"] = (w, d, ge.cpu().numpy(), go.cpu().numpy())
        plan.close()
    return _L20["run"]


@pytest.mark.parametrize("part", range(8))
def test_mp2_5k_l20_sampled(cg, part):
    w, d, ge, go = _mp2_5k_l20(cg)
    rec = sample_rows(w.n, 32, seed=5)
    assert len(rec) == 32
    rec = rec[part::8]
    _check((ge, go), _oracle2(w.lmax, d, rec), TOL_F32, nodes=rec)
    if part == 7:
        _L20.clear()
