"""The on-site entry point that allocates nothing (cgtp_onsite_noalloc, fixed device scratch)
against cgtp_onsite on the same inputs, through the C ABI: two calls in a row, the second
smaller (the scratch keeps the first call's contents), an fp64 plan, and the rejection of a
call whose workspace exceeds the scratch."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests.gpu_util import ONSITE_KEYS, TOL_F32, TOL_F64, rel_err, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _both(cg, plan, t):
    import torch

    ref = cg.onsite(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"], t["U_out_odd"])
    oe = torch.full_like(t["A"], float("nan"))
    oo = torch.full_like(t["A"], float("nan"))
    got = cg.onsite_noalloc(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"],
                            t["U_out_odd"], oe, oo)
    torch.cuda.synchronize()
    return got, ref


def _check(cg, got, ref, d, lmax, tol, nodes):
    import torch

    for g, r in zip(got, ref):
        assert torch.equal(g, r), "fixed-scratch call differs from cgtp_onsite"
    re_, ro = oracle.onsite(lmax, d["A"][nodes], d["B"][nodes], d["U_A"], d["U_B"],
                            d["U_out_even"], d["U_out_odd"])
    ee, eo = rel_err(got[0][nodes], re_), rel_err(got[1][nodes], ro)
    assert ee <= tol and eo <= tol, (ee, eo)


def test_noalloc_two_calls_second_smaller(cg):
    lmax, C, R = 4, 64, 64
    plan = cg.plan_create(lmax, C, R)
    need = cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, 2048)
    assert need <= cg.CGTP_NOALLOC_SCRATCH_BYTES
    d1 = inputs.onsite_inputs(2048, lmax, C, R, seed=1, per_degree=True)
    got, ref = _both(cg, plan, to_dev(d1, ONSITE_KEYS))
    _check(cg, got, ref, d1, lmax, TOL_F32, np.array([0, 5, 777, 1500, 2047]))
    d2 = inputs.onsite_inputs(301, lmax, C, R, seed=11, per_degree=True)
    got, ref = _both(cg, plan, to_dev(d2, ONSITE_KEYS))
    _check(cg, got, ref, d2, lmax, TOL_F32, np.arange(301))
    plan.close()


def test_noalloc_fp64_and_self_coupled(cg):
    lmax, C, R = 3, 8, 16
    plan = cg.plan_create(lmax, C, R, dtype="f64")
    d = inputs.onsite_inputs(96, lmax, C, R, seed=5, self_coupled=True)
    t = to_dev(d, ONSITE_KEYS, dtype="f64")
    t["B"] = t["A"]
    got, ref = _both(cg, plan, t)
    _check(cg, got, ref, d, lmax, TOL_F64, np.arange(96))
    plan.close()


def test_noalloc_rejects_oversize_and_skips_slot(cg):
    import torch

    lmax, C, R = 12, 16, 128
    plan = cg.plan_create(lmax, C, R)
    per_node = (cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, 2)
                - cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, 1))
    n = cg.CGTP_NOALLOC_SCRATCH_BYTES // per_node + 8
    assert cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, n) > cg.CGTP_NOALLOC_SCRATCH_BYTES
    d = inputs.onsite_inputs(n, lmax, C, R, seed=7)
    t = to_dev(d, ONSITE_KEYS)
    oe = torch.full_like(t["A"], 3.0)
    oo = torch.full_like(t["A"], 3.0)
    with pytest.raises(cg.CgtpError) as ei:
        cg.onsite_noalloc(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"],
                          t["U_out_odd"], oe, oo)
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((oe == 3.0).all()) and bool((oo == 3.0).all()), "outputs touched"
    # a call that fits, with the odd slot skipped
    m = 40
    tm = {k: (v[:m].contiguous() if k in ("A", "B") else v) for k, v in t.items()}
    got = cg.onsite_noalloc(plan, tm["A"], tm["B"], tm["U_A"], tm["U_B"], tm["U_out_even"],
                            tm["U_out_odd"], torch.empty_like(tm["A"]), False)
    ref = cg.onsite(plan, tm["A"], tm["B"], tm["U_A"], tm["U_B"], tm["U_out_even"],
                    tm["U_out_odd"], out_odd=False)
    torch.cuda.synchronize()
    assert got[1] is None and torch.equal(got[0], ref[0])
    plan.close()
