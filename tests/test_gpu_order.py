"""GPU tests of the receiver order (cgtp_receiver_order, cgtp_plan_set_receiver_order): the
neighbour sum of a receiver (Eq. msgpass-S) does not depend on the order the receivers run
in, and each receiver's sum runs in the same edge order either way, so every message-passing
path must give bitwise the same outputs with and without an order; plus the fp64 oracle on
one case, the node-count check and clearing the order."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2605_15073_amd import inputs
from tests.gpu_util import TOL_F32
from tests.test_gpu_general import MP_G, _check, _dev, _mp_d, _mp_gpu, _mp_ref

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


def _same_with_order(cg, plan, d, run):
    """run(plan) twice, without and with the order of d's graph; both results equal bitwise."""
    import torch

    base = run(plan)
    o = cg.receiver_order(d["row_ptr"], d["col"], d.get("edge_unit"))
    assert not np.array_equal(o, np.arange(o.shape[0]))  # a real permutation
    cg.set_receiver_order(plan, o)
    try:
        got = run(plan)
    finally:
        cg.set_receiver_order(plan, None)
    for a, b in zip(base, got):
        assert torch.equal(a, b)
    return got


@pytest.mark.parametrize("lmax,R,two,kw", [
    (3, 16, False, {}),                       # MFMA receiver, values-only, plain layout
    (8, 16, False, {}),                       # MFMA receiver, chunked sender layout
    (3, 6, False, {}),                        # per-thread receiver handing over to the analysis
    (8, 16, False, {"n_theta": 14}),          # MFMA receiver, three planes (grid override)
    (4, 6, False, {"n_theta": 8}),            # per-thread receiver, analysis inside
    (3, 4, False, {"dtype": "f64"}),
    (3, 4, False, {"flags": 2}),              # separated edge field
    (5, 16, True, {}),
    (5, 6, True, {}),
])
def test_message_pass_order_invariant(cg, lmax, R, two, kw):
    d = inputs.mp_inputs(60, lmax, 4, R, 900 + lmax, density=0.1, r_cut=3.5, two_slot=two)
    dt = kw.get("dtype", "f32")
    t = _dev(d, ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "node_flip", "U_E",
                 "U_I", "U_out_even", "U_out_odd"), dt)
    plan = cg.plan_create(lmax, 4, R, **kw)

    def run(p):
        return cg.message_pass(p, t["row_ptr"], t["col"], t["edge_unit"], t["edge_radial"],
                               t["node_feat"], t["U_E"], t["U_I"], t["U_out_even"],
                               t["U_out_odd"], node_flip=t["node_flip"])

    got = _same_with_order(cg, plan, d, run)
    if lmax == 3 and R == 16:
        ref = oracle.message_pass(lmax, d["row_ptr"], d["col"], d["edge_unit"], d["edge_radial"],
                                  d["node_feat"], d["U_E"], d["U_I"], d["U_out_even"],
                                  d["U_out_odd"])
        _check(got, ref, TOL_F32)


@pytest.mark.parametrize("lmax,R,nin", [(6, 8, 4), (4, 6, 2), (8, 16, 2)])
def test_message_pass_general_order_invariant(cg, lmax, R, nin):
    d = _mp_d(lmax, 50, 4, R, 930 + lmax, True, nin, 2)
    t = _dev(d, MP_G)
    plan = cg.plan_create(lmax, 4, R)
    got = _same_with_order(cg, plan, d, lambda p: _mp_gpu(cg, p, t))
    if lmax == 4:
        _check(got, _mp_ref(lmax, d), TOL_F32)


@pytest.mark.parametrize("lmax,R,kw", [(5, 6, {}), (3, 4, {"dtype": "f64"})])
def test_message_pass_fields_order_invariant(cg, lmax, R, kw):
    d = inputs.fields_mp_inputs(40, lmax, 4, R, 950 + lmax, edge_flip=True, node_flip=True,
                                in_blocks=4, out_blocks=2, r_cut=3.5)
    t = _dev(d, FK, kw.get("dtype", "f32"))
    plan = cg.plan_create(lmax, 4, R, **kw)

    def run(p):
        return cg.message_pass_fields(p, t["row_ptr"], t["col"], t["edge_feat"], t["node_feat"],
                                      t["U_E"], t["U_I"], t["U_out_even"], t["U_out_odd"],
                                      edge_flip=t["edge_flip"], node_flip=t["node_flip"])

    dd = dict(d)
    dd.pop("edge_unit", None)  # the fields call has no directions: breadth-first order
    _same_with_order(cg, plan, dd, run)


def test_order_node_count_and_probe(cg):
    import torch

    lmax, R = 6, 16
    d = inputs.mp_inputs(50, lmax, 4, R, 970, density=0.1, r_cut=3.5)
    t = _dev(d, ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "U_E", "U_I",
                 "U_out_even", "U_out_odd"))
    plan = cg.plan_create(lmax, 4, R)
    N = d["node_feat"].shape[0]
    o = cg.receiver_order(d["row_ptr"], d["col"], d["edge_unit"])
    with pytest.raises(cg.CgtpError) as ei:
        cg.set_receiver_order(plan, np.zeros(N, np.int32))  # not a permutation
    assert ei.value.status == cg.CGTP_ERR_ARG
    cg.set_receiver_order(plan, o)
    # the probe replays the receiver's loads in the same order
    fields = torch.zeros(N * R * 3 * ((plan.n_theta * plan.n_phi + 31) // 32 * 32),
                         dtype=torch.float32, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    cg.gather_probe(plan, t["row_ptr"], t["col"], fields, sink)
    torch.cuda.synchronize()
    assert sink.item() == 0.0
    # a call over another node count is refused while the order is set
    d2 = inputs.mp_inputs(30, lmax, 4, R, 971, density=0.1, r_cut=3.0)
    t2 = _dev(d2, ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "U_E", "U_I",
                   "U_out_even", "U_out_odd"))
    args = ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "U_E", "U_I",
            "U_out_even", "U_out_odd")
    with pytest.raises(cg.CgtpError) as ei:
        cg.message_pass(plan, *(t2[k] for k in args))
    assert ei.value.status == cg.CGTP_ERR_ARG
    cg.set_receiver_order(plan, None)
    cg.message_pass(plan, *(t2[k] for k in args))
    torch.cuda.synchronize()
