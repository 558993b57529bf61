"""GPU parity of the nu-body on-site product (cgtp_onsite_nbody) against the fp64 oracle,
element by element on the same seeded inputs (fp32 bar 2e-5 of max|ref|, fp64 1e-11), on
plans whose grid is the exact one for nu operands; plus nu = 2 against the bilinear call,
inversion and rotation on the GPU, the grid check and the workspace contract."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.gpu_util import TOL_F32, TOL_F64, rel_err, sample_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _dev(a, dtype="f32"):
    import torch

    return torch.from_numpy(np.ascontiguousarray(
        np.asarray(a).astype(np.float64 if dtype == "f64" else np.float32))).cuda()


def _run(cg, plan, d, dtype="f32", **kw):
    uniq = {}
    X = [uniq.setdefault(id(x), _dev(x, dtype)) for x in d["X"]]
    return cg.onsite_nbody(plan, X, [_dev(u, dtype) for u in d["U"]], _dev(d["U_out"], dtype),
                           **kw)


def _plan(cg, lmax, nu, C, R, **kw):
    nt, nph = cg.nbody_grid(lmax, nu)
    return cg.plan_create(lmax, C, R, n_theta=max(nt, (3 * lmax + 2) // 2 + lmax % 2),
                          n_phi=max(nph, 3 * lmax + 1), **kw)


@pytest.mark.parametrize("lmax,nu,R,selfc", [
    (0, 2, 3, False),
    (2, 3, 6, False),
    (3, 3, 5, True),
    (4, 4, 8, False),
    (6, 3, 16, True),
    (5, 5, 4, False),
    (3, 8, 4, True),
    (8, 2, 8, False),
    (10, 3, 8, True),
])
def test_nbody_vs_oracle(cg, lmax, nu, R, selfc):
    d = inputs.nbody_inputs(12, lmax, 4, R, 600 + lmax + nu, nu, self_coupled=selfc)
    plan = _plan(cg, lmax, nu, 4, R)
    ref = oracle.nbody(lmax, d["X"], d["U"], d["U_out"])
    err = rel_err(_run(cg, plan, d), ref)
    assert err <= TOL_F32, err


def test_nbody_fp64(cg):
    lmax, nu = 3, 4
    d = inputs.nbody_inputs(10, lmax, 3, 4, 611, nu, self_coupled=False)
    plan = _plan(cg, lmax, nu, 3, 4, dtype="f64")
    ref = oracle.nbody(lmax, d["X"], d["U"], d["U_out"])
    assert rel_err(_run(cg, plan, d, "f64"), ref) <= TOL_F64


def test_nu2_is_bilinear_onsite(cg):
    lmax = 5
    d = inputs.nbody_inputs(32, lmax, 4, 8, 613, 2, self_coupled=False)
    plan_n = _plan(cg, lmax, 2, 4, 8)
    plan = cg.plan_create(lmax, 4, 8)
    A, B = _dev(d["X"][0]), _dev(d["X"][1])
    Uo = _dev(d["U_out"])
    oe, _ = cg.onsite(plan, A, B, _dev(d["U"][0]), _dev(d["U"][1]), Uo, Uo)
    got = cg.onsite_nbody(plan_n, [A, B], [_dev(d["U"][0]), _dev(d["U"][1])], Uo)
    assert rel_err(got, oe.cpu().numpy().astype(np.float64)) <= 2 * TOL_F32


def test_nbody_inversion_and_rotation_gpu(cg):
    lmax, nu = 4, 3
    d = inputs.nbody_inputs(24, lmax, 4, 8, 615, nu, self_coupled=False)
    plan = _plan(cg, lmax, nu, 4, 8)
    out = _run(cg, plan, d).cpu().numpy().astype(np.float64)
    P = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(lmax + 1)])
    di = dict(d)
    di["X"] = [(x * P).astype(np.float32) for x in d["X"]]
    assert rel_err(_run(cg, plan, di), out * P) <= TOL_F32
    D = bf.wigner_d_real(lmax, bf.random_rotation(np.random.default_rng(17)))
    dr = dict(d)
    dr["X"] = [bf.rotate_coeffs(D, x.astype(np.float64)) for x in d["X"]]
    assert rel_err(_run(cg, plan, dr), bf.rotate_coeffs(D, out)) <= TOL_F32


def test_nbody_grid_check_workspace_and_stages(cg):
    import torch

    lmax, nu = 3, 3
    d = inputs.nbody_inputs(16, lmax, 3, 4, 617, nu, self_coupled=True)
    coarse = cg.plan_create(lmax, 3, 4)  # the bilinear grid is too coarse for nu = 3
    with pytest.raises(cg.CgtpError) as ei:
        _run(cg, coarse, d)
    assert ei.value.status == cg.CGTP_ERR_ARG
    plan = _plan(cg, lmax, nu, 3, 4, flags=cg.CGTP_TIME_STAGES)
    need = cg.workspace_bytes_nbody(plan, 16, nu)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    ref = oracle.nbody(lmax, d["X"], d["U"], d["U_out"])
    assert rel_err(_run(cg, plan, d, workspace=ws), ref) <= TOL_F32
    with pytest.raises(cg.CgtpError) as ei:
        _run(cg, plan, d, workspace=ws[: need - 256])
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    assert rel_err(_run(cg, plan, d), ref) <= TOL_F32
    stages, calls = cg.stage_times(plan, cg.CGTP_OP_ONSITE_NBODY)
    assert calls == 2 and len(stages) == 3 and all(v >= 0 for v in stages.values())


@pytest.mark.parametrize("name", ["nbody_n2048_l4_c64_nu3", "nbody_n2048_l8_c64_nu4"])
def test_nbody_workloads_sampled(cg, name):
    import torch

    w = inputs.WORKLOADS[name]
    d = w.make()
    plan = _plan(cg, w.lmax, w.nu, w.C, w.R)
    out = _run(cg, plan, d)
    rows = sample_rows(w.n, 32, seed=9)
    assert len(rows) == 32
    ref = oracle.nbody(w.lmax, [x[rows] for x in d["X"]], d["U"], d["U_out"])
    assert rel_err(out[rows], ref) <= TOL_F32
    assert torch.equal(out, _run(cg, plan, d))
