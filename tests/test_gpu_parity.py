"""GPU parity: libcgtp (through its C ABI) against the fp64 oracle, element by
element on the same seeded inputs. fp32 bar: max|gpu - ref| / max|ref| <= 2e-5
per output slot; the fp64 build of the same kernels must agree to 1e-11.
Full-size workloads are run whole on the GPU and checked on sampled nodes or
receivers, which the oracle computes independently."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.gpu_util import (MP_KEYS, ONSITE_KEYS, TOL_F32, TOL_F64, bench_order, rel_err, run_mp,
                            run_onsite, same_without_order, sample_rows, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _oracle_onsite(lmax, d, nodes=None):
    A, B = d["A"], d["B"]
    if nodes is not None:
        A, B = A[nodes], B[nodes]
    return oracle.onsite(lmax, A, B, d["U_A"], d["U_B"], d["U_out_even"], d["U_out_odd"])


def _oracle_mp(lmax, d, receivers=None):
    return oracle.message_pass(lmax, *(d[k] for k in MP_KEYS), receivers=receivers)


def _check_pair(gpu, ref, tol, nodes=None):
    ge, go = gpu
    re_, ro = ref
    if nodes is not None:
        ge, go = ge[nodes], go[nodes]
    ee, eo = rel_err(ge, re_), rel_err(go, ro)
    assert ee <= tol and eo <= tol, f"rel err even {ee:.3e} odd {eo:.3e} (tol {tol:g})"
    return ee, eo


# ------------------------------------------------------------------ on-site ---

def test_onsite_tiny_n64_l2(cg):
    lmax = 2
    d = inputs.onsite_inputs(64, lmax, 8, 8, seed=0)
    plan = cg.plan_create(lmax, 8, 8)
    _check_pair(run_onsite(cg, plan, to_dev(d, ONSITE_KEYS)), _oracle_onsite(lmax, d), TOL_F32)


@pytest.mark.parametrize("lmax,n,C,R", [(0, 5, 3, 2), (1, 37, 5, 7), (3, 37, 6, 5), (5, 19, 9, 4),
                                        (8, 11, 4, 6), (13, 3, 3, 3), (24, 2, 2, 3)])
def test_onsite_lmax_sweep_ragged(cg, lmax, n, C, R):
    d = inputs.onsite_inputs(n, lmax, C, R, seed=100 + lmax, distinct_out=True)
    plan = cg.plan_create(lmax, C, R)
    _check_pair(run_onsite(cg, plan, to_dev(d, ONSITE_KEYS)), _oracle_onsite(lmax, d), TOL_F32)


@pytest.mark.parametrize("lmax,n,C,R", [(2, 9, 5, 17), (6, 7, 8, 33), (10, 6, 5, 31),
                                        (12, 5, 6, 19), (14, 3, 4, 23), (15, 3, 4, 7),
                                        (16, 4, 5, 18), (20, 3, 4, 18), (24, 2, 3, 5)])
def test_onsite_rank_blocks_and_high_lmax(cg, lmax, n, C, R):
    # rank counts that leave a partial rank block; up to lmax 14 the register-resident
    # folded grid stage runs, from lmax 15 the MFMA one
    d = inputs.onsite_inputs(n, lmax, C, R, seed=300 + lmax, distinct_out=True)
    plan = cg.plan_create(lmax, C, R)
    _check_pair(run_onsite(cg, plan, to_dev(d, ONSITE_KEYS)), _oracle_onsite(lmax, d), TOL_F32)


def test_onsite_ace_n2048_l4_self_coupled(cg):
    w = inputs.WORKLOADS["onsite_ace_n2048_l4_c64"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    t = to_dev(d, ONSITE_KEYS)
    assert t["A"].data_ptr() != t["B"].data_ptr()
    t["B"] = t["A"]                      # the B := A self-coupling of this workload
    gpu = run_onsite(cg, plan, t)
    ref = _oracle_onsite(w.lmax, d)
    _check_pair(gpu, ref, TOL_F32)
    assert np.abs(ref[1]).max() > 1e-2 * np.abs(ref[0]).max()   # U_A != U_B: odd is O(1)


def test_onsite_n4096_l12_sampled(cg):
    w = inputs.WORKLOADS["onsite_n4096_l12_c128"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    gpu = run_onsite(cg, plan, to_dev(d, ONSITE_KEYS))
    nodes = sample_rows(w.n, 64, seed=0)
    assert len(nodes) == 64
    _check_pair(gpu, _oracle_onsite(w.lmax, d, nodes), TOL_F32, nodes=nodes)


@pytest.mark.parametrize("lmax", [3, 7])
def test_onsite_fp64_matches_oracle_tightly(cg, lmax):
    d = inputs.onsite_inputs(9, lmax, 4, 5, seed=7, distinct_out=True)
    plan = cg.plan_create(lmax, 4, 5, dtype="f64")
    _check_pair(run_onsite(cg, plan, to_dev(d, ONSITE_KEYS, "f64")), _oracle_onsite(lmax, d),
                TOL_F64)


def test_onsite_self_coupled_symmetric_vanishes(cg):
    lmax = 4
    d = inputs.onsite_inputs(64, lmax, 16, 16, seed=1, per_degree=True, self_coupled=True)
    plan = cg.plan_create(lmax, 16, 16)
    t = to_dev(d, ONSITE_KEYS)
    oe, oo = cg.onsite(plan, t["A"], t["A"], t["U_A"], t["U_A"], t["U_out_even"], t["U_out_odd"])
    ge = oe.cpu().numpy()
    assert np.abs(oo.cpu().numpy()).max() <= TOL_F32 * np.abs(ge).max()


def test_onsite_operand_exchange_negates_odd(cg):
    lmax = 5
    d = inputs.onsite_inputs(32, lmax, 8, 8, seed=3)
    plan = cg.plan_create(lmax, 8, 8)
    t = to_dev(d, ONSITE_KEYS)
    oe, oo = run_onsite(cg, plan, t)
    se, so = cg.onsite(plan, t["B"], t["A"], t["U_B"], t["U_A"], t["U_out_even"], t["U_out_odd"])
    ref = np.abs(oo.cpu().numpy()).max()
    assert rel_err(so, -oo.cpu().numpy().astype(np.float64), ref) <= TOL_F32
    assert rel_err(se, oe.cpu().numpy().astype(np.float64)) <= TOL_F32


def test_onsite_skip_slots_and_grid_override(cg):
    lmax = 4
    d = inputs.onsite_inputs(20, lmax, 6, 6, seed=4, distinct_out=True)
    ref = _oracle_onsite(lmax, d)
    t = to_dev(d, ONSITE_KEYS)
    plan = cg.plan_create(lmax, 6, 6)
    oe, oo = run_onsite(cg, plan, t, out_odd=False)
    assert oo is None and rel_err(oe, ref[0]) <= TOL_F32
    oe, oo = run_onsite(cg, plan, t, out_even=False)
    assert oe is None and rel_err(oo, ref[1]) <= TOL_F32
    big = cg.plan_create(lmax, 6, 6, n_theta=11, n_phi=20)
    assert (big.n_theta, big.n_phi) == (11, 20)
    _check_pair(run_onsite(cg, big, t), ref, TOL_F32)
    odd_l = cg.plan_create(3, 6, 6)          # odd lmax: default grid is one node above minimum
    d3 = inputs.onsite_inputs(20, 3, 6, 6, seed=5)
    mn = cg.plan_create(3, 6, 6, n_theta=5, n_phi=10)
    t3 = to_dev(d3, ONSITE_KEYS)
    r3 = _oracle_onsite(3, d3)
    _check_pair(run_onsite(cg, odd_l, t3), r3, TOL_F32)
    _check_pair(run_onsite(cg, mn, t3), r3, TOL_F32)


def test_onsite_paired_launches_match_single_and_stage_times(cg):
    """The fp32 call contracts both operands in one launch and projects both output slots in
    one launch; a call that asks for one slot (or shares the operands) takes the single
    launches. The paired blocks run the same arithmetic, so the results agree bit for bit."""
    import torch

    lmax = 5
    d = inputs.onsite_inputs(70, lmax, 12, 20, seed=14, distinct_out=True)
    ref = _oracle_onsite(lmax, d)
    t = to_dev(d, ONSITE_KEYS)
    plan = cg.plan_create(lmax, 12, 20, flags=cg.CGTP_TIME_STAGES)
    both = run_onsite(cg, plan, t)
    _check_pair(both, ref, TOL_F32)
    even, _ = run_onsite(cg, plan, t, out_odd=False)
    _, odd = run_onsite(cg, plan, t, out_even=False)
    assert torch.equal(both[0], even) and torch.equal(both[1], odd)
    stages, calls = cg.stage_times(plan, cg.CGTP_OP_ONSITE)
    assert calls == 3 and tuple(stages) == cg.ONSITE_STAGES
    assert all(v > 0 for v in stages.values())


def test_onsite_caller_workspace_and_errors(cg):
    import torch

    lmax, n = 3, 10
    d = inputs.onsite_inputs(n, lmax, 4, 4, seed=6)
    t = to_dev(d, ONSITE_KEYS)
    plan = cg.plan_create(lmax, 4, 4)
    need = cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, n)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    a = run_onsite(cg, plan, t, workspace=ws)
    b = run_onsite(cg, plan, t)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    small = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(cg.CgtpError) as ei:
        run_onsite(cg, plan, t, workspace=small)
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    # a workspace off a 256-byte boundary is refused before anything is enqueued
    big = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(cg.CgtpError) as ei:
        run_onsite(cg, plan, t, workspace=big[4:])
    assert ei.value.status == cg.CGTP_ERR_ARG
    empty = {k: (v[:0] if k in ("A", "B") else v) for k, v in t.items()}
    oe, oo = run_onsite(cg, plan, empty)
    assert oe.shape[0] == 0 and oo.shape[0] == 0


def test_onsite_rotation_equivariance_gpu(cg):
    lmax = 6
    d = inputs.onsite_inputs(16, lmax, 8, 8, seed=8, distinct_out=True)
    plan = cg.plan_create(lmax, 8, 8)
    t = to_dev(d, ONSITE_KEYS)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in run_onsite(cg, plan, t))
    D = bf.wigner_d_real(lmax, bf.random_rotation(np.random.default_rng(5)))
    dr = dict(d)
    dr["A"] = bf.rotate_coeffs(D, d["A"].astype(np.float64))
    dr["B"] = bf.rotate_coeffs(D, d["B"].astype(np.float64))
    re_, ro = run_onsite(cg, plan, to_dev(dr, ONSITE_KEYS))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


def test_onsite_deterministic(cg):
    import torch

    lmax = 6
    d = inputs.onsite_inputs(64, lmax, 16, 16, seed=9)
    plan = cg.plan_create(lmax, 16, 16)
    t = to_dev(d, ONSITE_KEYS)
    a = run_onsite(cg, plan, t)
    b = run_onsite(cg, plan, t)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# ------------------------------------------------------------ message passing ---

def _tiny_mp(lmax, n=64, C=8, R=8, seed=1, r_cut=4.0):
    return inputs.mp_inputs(n, lmax, C, R, seed, r_cut=r_cut, distinct_out=True)


@pytest.mark.parametrize("lmax", [0, 1, 2, 4, 6, 9])
def test_mp_small_lmax_sweep(cg, lmax):
    d = _tiny_mp(lmax, C=5, R=6, seed=20 + lmax)
    plan = cg.plan_create(lmax, 5, 6)
    _check_pair(run_mp(cg, plan, to_dev(d, MP_KEYS)), _oracle_mp(lmax, d), TOL_F32)


@pytest.mark.parametrize("lmax", [2, 5])
def test_mp_separated_edge_synthesis(cg, lmax):
    d = _tiny_mp(lmax, C=4, R=5, seed=30 + lmax)
    t = to_dev(d, MP_KEYS)
    sep = cg.plan_create(lmax, 4, 5, flags=cg.CGTP_EDGE_SEPARATED)
    zon = cg.plan_create(lmax, 4, 5)
    ref = _oracle_mp(lmax, d)
    _check_pair(run_mp(cg, sep, t), ref, TOL_F32)
    _check_pair(run_mp(cg, zon, t), ref, TOL_F32)


@pytest.mark.parametrize("sep", [False, True])
def test_mp_fp64_matches_oracle_tightly(cg, sep):
    lmax = 4
    d = _tiny_mp(lmax, n=40, C=3, R=4, seed=41, r_cut=3.5)
    plan = cg.plan_create(lmax, 3, 4, dtype="f64", flags=cg.CGTP_EDGE_SEPARATED if sep else 0)
    _check_pair(run_mp(cg, plan, to_dev(d, MP_KEYS, "f64")), _oracle_mp(lmax, d), TOL_F64)


def test_mp_empty_rows_and_no_edges(cg):
    import torch

    lmax = 3
    d = _tiny_mp(lmax, n=30, C=4, R=4, seed=50, r_cut=1.5)
    deg = np.diff(d["row_ptr"])
    assert (deg == 0).any() and (deg > 0).any()
    plan = cg.plan_create(lmax, 4, 4, flags=cg.CGTP_VALIDATE_CSR)
    gpu = run_mp(cg, plan, to_dev(d, MP_KEYS))
    _check_pair(gpu, _oracle_mp(lmax, d), TOL_F32)
    for o in gpu:
        assert torch.count_nonzero(o[torch.from_numpy(deg == 0).cuda()]) == 0
    z = dict(d)
    z["row_ptr"] = np.zeros_like(d["row_ptr"])
    z["col"] = d["col"][:0]
    z["edge_unit"] = d["edge_unit"][:0]
    z["edge_radial"] = d["edge_radial"][:0]
    oe, oo = run_mp(cg, plan, to_dev(z, MP_KEYS))
    assert torch.count_nonzero(oe) == 0 and torch.count_nonzero(oo) == 0


def test_mp_validate_csr_rejects_bad_lists(cg):
    lmax = 2
    d = _tiny_mp(lmax, n=30, C=3, R=3, seed=51, r_cut=3.0)
    plan = cg.plan_create(lmax, 3, 3, flags=cg.CGTP_VALIDATE_CSR)
    bad_col = dict(d)
    bad_col["col"] = d["col"].copy()
    bad_col["col"][len(bad_col["col"]) // 2] = 30
    bad_rp = dict(d)
    bad_rp["row_ptr"] = d["row_ptr"].copy()
    bad_rp["row_ptr"][-1] += 1
    for bad in (bad_col, bad_rp):
        with pytest.raises(cg.CgtpError) as ei:
            run_mp(cg, plan, to_dev(bad, MP_KEYS))
        assert ei.value.status == cg.CGTP_ERR_CSR


def test_mp_rotation_equivariance_gpu(cg):
    lmax = 5
    d = _tiny_mp(lmax, C=6, R=6, seed=60)
    plan = cg.plan_create(lmax, 6, 6)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in run_mp(cg, plan, to_dev(d, MP_KEYS)))
    rot = bf.random_rotation(np.random.default_rng(9))
    D = bf.wigner_d_real(lmax, rot)
    dr = dict(d)
    dr["edge_unit"] = (d["edge_unit"].astype(np.float64) @ rot.T)
    dr["node_feat"] = bf.rotate_coeffs(D, d["node_feat"].astype(np.float64))
    re_, ro = run_mp(cg, plan, to_dev(dr, MP_KEYS))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


def test_mp_10k_l6_sampled(cg):
    import torch

    w = inputs.WORKLOADS["mp_10k_l6_c128"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    bench_order(cg, plan, d)  # the launch configuration bench.py times
    t = to_dev(d, MP_KEYS)
    gpu = run_mp(cg, plan, t)
    rec = sample_rows(w.n, 160, seed=1)
    assert len(rec) == 160
    _check_pair(gpu, _oracle_mp(w.lmax, d, rec), TOL_F32, nodes=rec)
    again = run_mp(cg, plan, t)
    assert torch.equal(gpu[0], again[0]) and torch.equal(gpu[1], again[1])
    same_without_order(cg, plan, lambda p: run_mp(cg, p, t), gpu)


_L20 = {}


def _mp_5k_l20(cg):
    """The lmax-20 workload run once on the GPU; its outputs are checked in four parts so
    that each test's oracle work stays well inside the per-test time limit."""
    if "run" not in _L20:
        w = inputs.WORKLOADS["mp_5k_l20_c64"]
        d = w.make()
        plan = cg.plan_create(w.lmax, w.C, w.R)
        bench_order(cg, plan, d)
        t = to_dev(d, MP_KEYS)
        ge, go = run_mp(cg, plan, t)
        same_without_order(cg, plan, lambda p: run_mp(cg, p, t), (ge, go))
        _L20["run"] = (w, d, ge.cpu().numpy(), go.cpu().numpy())
        plan.close()
    return _L20["run"]


@pytest.mark.parametrize("part", range(4))
def test_mp_5k_l20_sampled(cg, part):
    w, d, ge, go = _mp_5k_l20(cg)
    rec = sample_rows(w.n, 32, seed=4)
    assert len(rec) == 32
    rec = rec[part::4]
    _check_pair((ge, go), _oracle_mp(w.lmax, d, rec), TOL_F32, nodes=rec)
    if part == 3:
        _L20.clear()


@pytest.mark.parametrize("lmax,R", [(7, 16), (8, 48), (9, 16), (10, 32), (13, 16), (24, 16)])
def test_mp_mfma_receiver(cg, lmax, R):
    """Ranks in multiples of 16 at lmax >= 7 take the MFMA receiver pass."""
    d = _tiny_mp(lmax, n=48, C=4, R=R, seed=70 + lmax, r_cut=3.5)
    plan = cg.plan_create(lmax, 4, R)
    _check_pair(run_mp(cg, plan, to_dev(d, MP_KEYS)), _oracle_mp(lmax, d), TOL_F32)
