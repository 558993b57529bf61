"""GPU parity of the general parameterization (Eqs. msgpass-cp-alpha, msgpass-cp-beta,
Table 1, on-site contraction with parity-labelled inputs): cgtp_onsite_general and
cgtp_message_pass_general against the fp64 oracle, element by element on the same seeded
inputs. fp32 bar: max|gpu - ref| / max|ref| <= 2e-5 per output slot; fp64 build 1e-11.

Cases cover every lowering: single slots with per-category factors, one or two flipped
slots, shared / per-category / per-block input factors, per-sector and per-category output
weights; the per-thread and MFMA grid stages (on-site lmax >= 13, receiver lmax >= 7 with
ranks a multiple of 16); the separated edge field; and the routes that reduce to the
plain entry points, which must agree with them bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests.gpu_util import TOL_F32, TOL_F64, bench_order, rel_err, same_without_order, sample_rows

pytestmark = pytest.mark.gpu

ONSITE_G = ("A", "B", "A_flip", "B_flip", "U_A", "U_B", "U_out_even", "U_out_odd")
MP_G = ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "node_flip", "U_E", "U_I",
        "U_out_even", "U_out_odd")


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _dev(d, keys, dtype="f32"):
    import torch

    out = {}
    for k in keys:
        a = d.get(k)
        if a is None:
            out[k] = None
        elif a.dtype == np.int32:
            out[k] = torch.from_numpy(np.ascontiguousarray(a)).cuda()
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(
                a.astype(np.float64 if dtype == "f64" else np.float32))).cuda()
    return out


def _check(gpu, ref, tol, rows=None):
    ge, go = gpu
    if rows is not None:
        ge, go = ge[rows], go[rows]
    ee, eo = rel_err(ge, ref[0]), rel_err(go, ref[1])
    assert ee <= tol and eo <= tol, f"rel err even {ee:.3e} odd {eo:.3e} (tol {tol:g})"


# ------------------------------------------------------------------------- on-site ---

def _on_d(lmax, n, C, R, seed, flip1, flip2, nin, nout):
    return inputs.general_onsite_inputs(n, lmax, C, R, seed, flip1=flip1, flip2=flip2,
                                        in_blocks=nin, out_blocks=nout)


def _on_gpu(cg, plan, t, **kw):
    return cg.onsite_general(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"],
                             t["U_out_odd"], A_flip=t["A_flip"], B_flip=t["B_flip"], **kw)


def _on_ref(lmax, d):
    return oracle.onsite(lmax, d["A"], d["B"], d["U_A"], d["U_B"], d["U_out_even"],
                         d["U_out_odd"], A_flip=d["A_flip"], B_flip=d["B_flip"])


@pytest.mark.parametrize("lmax,n,R,flip1,flip2,nin,nout", [
    (0, 20, 3, True, True, 4, 2),
    (2, 24, 6, True, True, 4, 2),
    (3, 24, 6, False, False, 2, 1),   # one slot each, independent Gaunt / curl factors
    (4, 20, 5, True, False, 1, 1),    # a flipped slot on the first operand only
    (5, 16, 6, True, True, 1, 2),
    (6, 12, 7, False, True, 4, 1),
    (8, 10, 16, True, True, 2, 1),
    (13, 6, 16, True, True, 4, 2),    # MFMA grid stage
    (4, 12, 32, True, True, 4, 2),    # ranks a multiple of 32: one gathered projection per sector
    (14, 5, 8, False, True, 2, 2),
])
def test_onsite_general_vs_oracle(cg, lmax, n, R, flip1, flip2, nin, nout):
    d = _on_d(lmax, n, 5, R, 300 + lmax, flip1, flip2, nin, nout)
    plan = cg.plan_create(lmax, 5, R)
    _check(_on_gpu(cg, plan, _dev(d, ONSITE_G)), _on_ref(lmax, d), TOL_F32)


def test_onsite_general_large_grid_override(cg):
    """A plan whose grid override is too large for the split kernel's LDS (lmax 12 on a 76 x 37
    grid) runs the general call on unsplit groups and the per-thread grid kernel."""
    lmax = 12
    d = _on_d(lmax, 6, 4, 4, 316, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, 4, n_theta=76, n_phi=37)
    _check(_on_gpu(cg, plan, _dev(d, ONSITE_G)), _on_ref(lmax, d), TOL_F32)


def test_onsite_general_fp64(cg):
    lmax = 3
    d = _on_d(lmax, 16, 4, 5, 311, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, 5, dtype="f64")
    _check(_on_gpu(cg, plan, _dev(d, ONSITE_G, "f64")), _on_ref(lmax, d), TOL_F64)


def test_onsite_general_fused_route_is_onsite(cg):
    """One slot each with shared input factors: the plain on-site call, bit for bit, with
    the Gaunt weights of out_even and the curl weights of out_odd."""
    import torch

    lmax = 5
    d = _on_d(lmax, 32, 6, 8, 313, False, False, 1, 2)
    t = _dev(d, ONSITE_G)
    plan = cg.plan_create(lmax, 6, 8)
    ge, go = _on_gpu(cg, plan, t)
    pe, po = cg.onsite(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"][0].contiguous(),
                       t["U_out_odd"][1].contiguous())
    assert torch.equal(ge, pe) and torch.equal(go, po)


def test_onsite_general_inversion_on_gpu(cg):
    """Each slot multiplied by its own parity: out_even picks up (-1)^l, out_odd -(-1)^l."""
    lmax = 6
    d = _on_d(lmax, 24, 4, 16, 315, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, 16)
    oe, oo = (x.cpu().numpy().astype(np.float64) for x in _on_gpu(cg, plan, _dev(d, ONSITE_G)))
    P = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(lmax + 1)])
    di = dict(d)
    for k in ("A", "B"):
        di[k] = (d[k] * P).astype(np.float32)
        di[k + "_flip"] = (-d[k + "_flip"] * P).astype(np.float32)
    ie, io = _on_gpu(cg, plan, _dev(di, ONSITE_G))
    assert rel_err(ie, oe * P) <= TOL_F32
    assert rel_err(io, -oo * P) <= TOL_F32


def test_onsite_general_workspace_errors_and_stages(cg):
    import torch

    lmax = 2
    d = _on_d(lmax, 16, 3, 4, 317, True, True, 4, 2)
    t = _dev(d, ONSITE_G)
    plan = cg.plan_create(lmax, 3, 4, flags=cg.CGTP_TIME_STAGES)
    N = d["A"].shape[0]
    need = cg.workspace_bytes_general(plan, cg.CGTP_OP_ONSITE_GENERAL, N, 0, 3, 4, 2)
    plain = cg.workspace_bytes(plan, cg.CGTP_OP_ONSITE, N)
    assert need > 2 * plain  # stacked rank groups (their number depends on the lowering)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    _check(_on_gpu(cg, plan, t, workspace=ws), _on_ref(lmax, d), TOL_F32)
    with pytest.raises(cg.CgtpError) as ei:
        _on_gpu(cg, plan, t, workspace=ws[: need - 256])
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    _on_gpu(cg, plan, t)  # a rejected call records no stages
    stages, calls = cg.stage_times(plan, cg.CGTP_OP_ONSITE_GENERAL)
    assert calls == 2 and len(stages) == 5 and all(v >= 0 for v in stages.values())
    lib = cg.load_library()
    oe = torch.empty_like(t["A"])
    st = lib.cgtp_onsite_general(plan.handle, N, t["A"].data_ptr(), None, t["B"].data_ptr(),
                                 None, 3, t["U_A"].data_ptr(), t["U_B"].data_ptr(), 2,
                                 t["U_out_even"].data_ptr(), t["U_out_odd"].data_ptr(),
                                 oe.data_ptr(), None, None, 0, None)
    assert st == cg.CGTP_ERR_ARG


def test_onsiteg_n4096_l12_sampled(cg):
    w = inputs.WORKLOADS["onsiteg_n4096_l12_c128"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    gpu = _on_gpu(cg, plan, _dev(d, ONSITE_G))
    rows = sample_rows(w.n, 24, seed=8)
    assert len(rows) == 24
    sub = {k: (v[rows] if k in ("A", "B", "A_flip", "B_flip") and v is not None else v)
           for k, v in d.items()}
    _check(gpu, _on_ref(w.lmax, sub), TOL_F32, rows=rows)


# ----------------------------------------------------------------- message passing ---

def _mp_d(lmax, n, C, R, seed, flip, nin, nout, r_cut=3.5):
    return inputs.general_mp_inputs(n, lmax, C, R, seed, flip=flip, in_blocks=nin,
                                    out_blocks=nout, r_cut=r_cut)


def _mp_gpu(cg, plan, t, **kw):
    return cg.message_pass_general(plan, *(t[k] for k in MP_G if k != "node_flip"),
                                   node_flip=t["node_flip"], **kw)


def _mp_ref(lmax, d, receivers=None):
    return oracle.message_pass(lmax, d["row_ptr"], d["col"], d["edge_unit"], d["edge_radial"],
                               d["node_feat"], d["U_E"], d["U_I"], d["U_out_even"],
                               d["U_out_odd"], receivers=receivers, node_flip=d["node_flip"])


@pytest.mark.parametrize("lmax,R,flip,nin,nout", [
    (0, 3, True, 4, 2),
    (3, 6, False, 2, 1),    # one slot, independent Gaunt / curl factors
    (5, 6, True, 1, 2),     # shared factors, per-category output weights
    (6, 9, True, 4, 2),
    (6, 8, True, 4, 2),     # split groups stacked to 16 ranks
    (7, 16, True, 4, 2),    # MFMA receiver at 4 x 16 ranks
    (4, 32, True, 4, 2),    # gathered projection
    (8, 32, False, 2, 2),   # gathered projection, one node slot
    (8, 16, False, 2, 2),
    (12, 16, True, 2, 1),
    (20, 16, True, 4, 2),
])
def test_mp_general_vs_oracle(cg, lmax, R, flip, nin, nout):
    d = _mp_d(lmax, 40, 4, R, 400 + lmax, flip, nin, nout)
    plan = cg.plan_create(lmax, 4, R)
    gpu = _mp_gpu(cg, plan, _dev(d, MP_G))
    # high degrees: the oracle at a sample of receivers (first, last and a middle one)
    rec = None if lmax < 12 else np.array([0, 17, 39])
    _check(gpu, _mp_ref(lmax, d, rec), TOL_F32, rows=rec)


def test_mp_general_fp64_and_separated(cg):
    lmax = 4
    d = _mp_d(lmax, 36, 3, 5, 411, True, 4, 2)
    ref = _mp_ref(lmax, d)
    plan64 = cg.plan_create(lmax, 3, 5, dtype="f64")
    _check(_mp_gpu(cg, plan64, _dev(d, MP_G, "f64")), ref, TOL_F64)
    sep = cg.plan_create(lmax, 3, 5, flags=cg.CGTP_EDGE_SEPARATED)
    _check(_mp_gpu(cg, sep, _dev(d, MP_G)), ref, TOL_F32)


def test_mp_general_fused_routes(cg):
    """Shared factors: one slot is cgtp_message_pass (Gaunt weights of out_even, curl weights
    of out_odd); two slots with per-sector weights are cgtp_message_pass_two_slot."""
    import torch

    lmax = 6
    one = _mp_d(lmax, 40, 4, 6, 413, False, 1, 2)
    t = _dev(one, MP_G)
    plan = cg.plan_create(lmax, 4, 6)
    ge, go = _mp_gpu(cg, plan, t)
    pe, po = cg.message_pass(plan, t["row_ptr"], t["col"], t["edge_unit"], t["edge_radial"],
                             t["node_feat"], t["U_E"], t["U_I"], t["U_out_even"][0].contiguous(),
                             t["U_out_odd"][1].contiguous())
    assert torch.equal(ge, pe) and torch.equal(go, po)
    two = _mp_d(lmax, 40, 4, 6, 415, True, 1, 1)
    t = _dev(two, MP_G)
    ge, go = _mp_gpu(cg, plan, t)
    pe, po = cg.message_pass(plan, t["row_ptr"], t["col"], t["edge_unit"], t["edge_radial"],
                             t["node_feat"], t["U_E"], t["U_I"], t["U_out_even"],
                             t["U_out_odd"], node_flip=t["node_flip"])
    assert torch.equal(ge, pe) and torch.equal(go, po)


def test_mp_general_workspace_and_errors(cg):
    import torch

    lmax = 3
    d = _mp_d(lmax, 30, 3, 4, 417, True, 4, 2, r_cut=3.0)
    t = _dev(d, MP_G)
    plan = cg.plan_create(lmax, 3, 4)
    N, E = d["node_feat"].shape[0], d["n_edges"]
    need = cg.workspace_bytes_general(plan, cg.CGTP_OP_MESSAGE_PASS_GENERAL, N, E, 2, 4, 2)
    # the rank groups (two slot pairs, split factors) need more than the one-slot call
    assert need > cg.workspace_bytes(plan, cg.CGTP_OP_MESSAGE_PASS, N, E)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    _check(_mp_gpu(cg, plan, t, workspace=ws), _mp_ref(lmax, d), TOL_F32)
    with pytest.raises(cg.CgtpError) as ei:
        _mp_gpu(cg, plan, t, workspace=ws[: need - 256])
    assert ei.value.status == cg.CGTP_ERR_WORKSPACE
    with pytest.raises(cg.CgtpError) as ei:
        cg.workspace_bytes_general(plan, cg.CGTP_OP_MESSAGE_PASS_GENERAL, N, E, 2, 3, 2)
    assert ei.value.status == cg.CGTP_ERR_ARG


def test_mpg_10k_l6_sampled(cg):
    import torch

    w = inputs.WORKLOADS["mpg_10k_l6_c128"]
    d = w.make()
    plan = cg.plan_create(w.lmax, w.C, w.R)
    bench_order(cg, plan, d)
    t = _dev(d, MP_G)
    gpu = _mp_gpu(cg, plan, t)
    rec = sample_rows(w.n, 48, seed=5)
    assert len(rec) == 48
    _check(gpu, _mp_ref(w.lmax, d, rec), TOL_F32, rows=rec)
    again = _mp_gpu(cg, plan, t)
    assert torch.equal(gpu[0], again[0]) and torch.equal(gpu[1], again[1])
    same_without_order(cg, plan, lambda p: _mp_gpu(cg, p, t), gpu)
