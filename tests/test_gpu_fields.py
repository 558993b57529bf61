"""GPU parity of message passing with two parity-bearing fields (Eq. twoparity-phi):
cgtp_message_pass_fields against the fp64 oracle, element by element on the same seeded
inputs (fp32 bar 2e-5 of max|ref| per output slot, fp64 1e-11), plus the identities that
tie it to the other entry points: an R Y edge field is cgtp_message_pass, one self-edge per
node is cgtp_onsite_general."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.gpu_util import TOL_F32, TOL_F64, bench_order, rel_err, same_without_order, sample_rows
from tests.test_gpu_general import _dev, _check

pytestmark = pytest.mark.gpu

FK = ("row_ptr", "col", "edge_feat", "edge_flip", "node_feat", "node_flip", "U_E", "U_I",
      "U_out_even", "U_out_odd")


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _d(lmax, n, C, R, seed, ef, nf, nin, nout, r_cut=3.5):
    return inputs.fields_mp_inputs(n, lmax, C, R, seed, edge_flip=ef, node_flip=nf,
                                   in_blocks=nin, out_blocks=nout, r_cut=r_cut)


def _gpu(cg, plan, t, **kw):
    return cg.message_pass_fields(plan, t["row_ptr"], t["col"], t["edge_feat"], t["node_feat"],
                                  t["U_E"], t["U_I"], t["U_out_even"], t["U_out_odd"],
                                  edge_flip=t["edge_flip"], node_flip=t["node_flip"], **kw)


def _ref(lmax, d, rec=None):
    return oracle.message_pass_fields(lmax, d["row_ptr"], d["col"], d["edge_feat"],
                                      d["node_feat"], d["U_E"], d["U_I"], d["U_out_even"],
                                      d["U_out_odd"], receivers=rec, edge_flip=d["edge_flip"],
                                      node_flip=d["node_flip"])


@pytest.mark.parametrize("lmax,R,ef,nf,nin,nout", [
    (0, 3, True, True, 4, 2),
    (2, 6, True, True, 4, 2),
    (3, 6, False, False, 1, 1),   # one slot each, shared factors
    (4, 5, True, False, 2, 1),
    (5, 6, True, True, 4, 2),     # split factors: the curl pass writes the curl values to plane 1
    (6, 9, False, True, 1, 2),
    (8, 8, True, True, 2, 2),
    (12, 8, False, False, 4, 2),
    (20, 4, True, True, 1, 1),
    (3, 32, True, True, 4, 2),    # ranks a multiple of 32: gathered projection
])
def test_fields_vs_oracle(cg, lmax, R, ef, nf, nin, nout):
    d = _d(lmax, 36, 4, R, 500 + lmax, ef, nf, nin, nout)
    plan = cg.plan_create(lmax, 4, R)
    gpu = _gpu(cg, plan, _dev(d, FK))
    rec = None if lmax < 12 else np.array([0, 17, 35])
    _check(gpu, _ref(lmax, d, rec), TOL_F32, rows=rec)


def test_fields_fp64(cg):
    lmax = 3
    d = _d(lmax, 30, 3, 4, 511, True, True, 4, 2, r_cut=3.0)
    plan = cg.plan_create(lmax, 3, 4, dtype="f64")
    _check(_gpu(cg, plan, _dev(d, FK, "f64")), _ref(lmax, d), TOL_F64)


def test_ry_edge_field_is_message_pass(cg):
    """The edge field R Y (real harmonics from scipy) reproduces cgtp_message_pass."""
    lmax = 7
    d = _d(lmax, 40, 4, 16, 513, False, False, 1, 1)
    lk = np.array([l for l in range(lmax + 1) for _ in range(2 * l + 1)])
    Y = bf.real_sh_xyz(lmax, d["edge_unit"].astype(np.float64))
    dd = dict(d)
    dd["edge_feat"] = (d["edge_radial"].astype(np.float64)[:, :, lk] * Y[:, None, :]).astype(np.float32)
    plan = cg.plan_create(lmax, 4, 16)
    t = _dev(dd, FK + ("edge_unit", "edge_radial"))
    fe, fo = _gpu(cg, plan, t)
    me, mo = cg.message_pass(plan, t["row_ptr"], t["col"], t["edge_unit"], t["edge_radial"],
                             t["node_feat"], t["U_E"], t["U_I"], t["U_out_even"], t["U_out_odd"])
    ref_e, ref_o = (x.cpu().numpy().astype(np.float64) for x in (me, mo))
    assert rel_err(fe, ref_e) <= 2 * TOL_F32 and rel_err(fo, ref_o) <= 2 * TOL_F32


def test_self_edges_are_onsite_general(cg):
    import torch

    lmax = 5
    g = inputs.general_onsite_inputs(40, lmax, 4, 6, 515, in_blocks=4, out_blocks=2)
    n = g["A"].shape[0]
    t = _dev(g, ("A", "B", "A_flip", "B_flip", "U_A", "U_B", "U_out_even", "U_out_odd"))
    rp = torch.arange(n + 1, dtype=torch.int32, device="cuda")
    col = torch.arange(n, dtype=torch.int32, device="cuda")
    plan = cg.plan_create(lmax, 4, 6)
    fe, fo = cg.message_pass_fields(plan, rp, col, t["A"], t["B"], t["U_A"], t["U_B"],
                                    t["U_out_even"], t["U_out_odd"], edge_flip=t["A_flip"],
                                    node_flip=t["B_flip"])
    oe, oo = cg.onsite_general(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"],
                               t["U_out_odd"], A_flip=t["A_flip"], B_flip=t["B_flip"])
    ref_e, ref_o = (x.cpu().numpy().astype(np.float64) for x in (oe, oo))
    assert rel_err(fe, ref_e) <= 2 * TOL_F32 and rel_err(fo, ref_o) <= 2 * TOL_F32


def test_fields_inversion_on_gpu(cg):
    lmax = 6
    d = _d(lmax, 36, 4, 8, 517, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, 8)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in _gpu(cg, plan, _dev(d, FK)))
    P = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(lmax + 1)])
    di = dict(d)
    for k in ("edge", "node"):
        di[k + "_feat"] = (d[k + "_feat"] * P).astype(np.float32)
        di[k + "_flip"] = (-d[k + "_flip"] * P).astype(np.float32)
    ie, io = _gpu(cg, plan, _dev(di, FK))
    assert rel_err(ie, oe * P) <= TOL_F32 and rel_err(io, -oo * P) <= TOL_F32


def test_fields_workspace_errors_and_stages(cg):
    import torch

    lmax = 2
    d = _d(lmax, 30, 3, 4, 519, True, True, 4, 2, r_cut=3.0)
    t = _dev(d, FK)
    plan = cg.plan_create(lmax, 3, 4, flags=cg.CGTP_TIME_STAGES)
    N, E = d["node_feat"].shape[0], d["n_edges"]
    op = cg.CGTP_OP_MESSAGE_PASS_FIELDS
    need = cg.workspace_bytes_general(plan, op, N, E, 3, 4, 2)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    ref = _ref(lmax, d)
    _check(_gpu(cg, plan, t, workspace=ws), ref, TOL_F32)
    with pytest.raises(cg.CgtpError) as ei:
        _gpu(cg, plan, t, workspace=ws[: need - 256])
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    _check(_gpu(cg, plan, t), ref, TOL_F32)
    stages, calls = cg.stage_times(plan, op)
    assert calls == 2 and len(stages) == 7 and all(v >= 0 for v in stages.values())


def test_mpf_5k_l6_sampled(cg):
    import torch

    w = inputs.WORKLOADS["mpf_5k_l6_c64"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    bench_order(cg, plan, d)
    t = _dev(d, FK)
    gpu = _gpu(cg, plan, t)
    rec = sample_rows(w.n, 24, seed=6)
    assert len(rec) == 24
    _check(gpu, _ref(w.lmax, d, rec), TOL_F32, rows=rec)
    again = _gpu(cg, plan, t)
    assert torch.equal(gpu[0], again[0]) and torch.equal(gpu[1], again[1])
    same_without_order(cg, plan, lambda p: _gpu(cg, p, t), gpu)
