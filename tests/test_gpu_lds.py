"""Kernels sized from the device's LDS (160 KiB per workgroup on MI355X) instead of a fixed
64 KiB: fp64 plans at lmax 19-24 need more than 64 KiB of LDS staging and are now built and
checked against the fp64 oracle; the fp32 default-grid kernels keep their rank blocks."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests.gpu_util import MP_KEYS, ONSITE_KEYS, TOL_F64, rel_err, run_mp, run_onsite, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _lds_bytes_fp64(lmax):
    U, V = (3 * lmax + 3) // 2, 3 * lmax + 1
    K, M = (lmax + 1) ** 2, 2 * lmax + 1
    return 8 * max(2 * K + 4 * M * U + 2 * U * V, V * M + 2 * U * V + K + 2 * M * U)


@pytest.mark.parametrize("lmax", [19, 24])
def test_fp64_high_lmax_onsite(cg, lmax):
    assert _lds_bytes_fp64(lmax) > 65536
    d = inputs.onsite_inputs(3, lmax, 2, 3, seed=40 + lmax, distinct_out=True)
    plan = cg.plan_create(lmax, 2, 3, dtype="f64")
    ge, go = run_onsite(cg, plan, to_dev(d, ONSITE_KEYS, "f64"))
    re_, ro = oracle.onsite(lmax, d["A"], d["B"], d["U_A"], d["U_B"], d["U_out_even"],
                            d["U_out_odd"])
    assert rel_err(ge, re_) <= TOL_F64 and rel_err(go, ro) <= TOL_F64


def test_fp64_high_lmax_message_pass(cg):
    lmax = 20
    d = inputs.mp_inputs(12, lmax, 2, 2, seed=61, r_cut=2.0, distinct_out=True)
    assert d["n_edges"] > 0
    plan = cg.plan_create(lmax, 2, 2, dtype="f64")
    ge, go = run_mp(cg, plan, to_dev(d, MP_KEYS, "f64"))
    re_, ro = oracle.message_pass(lmax, *(d[k] for k in MP_KEYS))
    assert rel_err(ge, re_) <= TOL_F64 and rel_err(go, ro) <= TOL_F64
