"""GPU edge cases of the general parameterization, the two-field message passing and the
nu-body product: calls with no nodes, graphs whose receivers have no neighbours or that have
no edges at all, rotation equivariance of every input slot on the GPU, and run-to-run
determinism (bit-identical outputs). Values are compared with the fp64 oracle at the fp32 bar
(2e-5 of max|ref| per output slot) or with the rotated GPU output itself."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2605_15073_amd import inputs
from tests import bruteforce as bf
from tests.gpu_util import TOL_F32, rel_err
from tests.test_gpu_fields import FK
from tests.test_gpu_fields import _d as _f_d
from tests.test_gpu_fields import _gpu as _f_gpu
from tests.test_gpu_fields import _ref as _f_ref
from tests.test_gpu_general import MP_G, ONSITE_G, _check, _dev, _mp_d, _mp_gpu, _mp_ref, _on_d, \
    _on_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2605_15073_amd as lib

    lib.load_library()
    return lib


def _np(x):
    return x.cpu().numpy().astype(np.float64)


def test_no_nodes(cg):
    """N = 0: every general entry point returns empty outputs without launching."""
    import torch

    lmax, C, R = 3, 4, 4
    K = (lmax + 1) ** 2
    plan = cg.plan_create(lmax, C, R)
    d = _on_d(lmax, 8, C, R, 700, True, True, 4, 2)
    t = _dev(d, ONSITE_G)
    for k in ("A", "B", "A_flip", "B_flip"):
        t[k] = t[k][:0]
    oe, oo = _on_gpu(cg, plan, t)
    assert oe.shape == (0, C, K) and oo.shape == (0, C, K)

    m = _dev(_mp_d(lmax, 40, C, R, 701, True, 4, 2), MP_G)
    m["row_ptr"] = torch.zeros(1, dtype=torch.int32, device="cuda")
    for k in ("col", "edge_unit", "edge_radial", "node_feat", "node_flip"):
        m[k] = m[k][:0]
    oe, oo = _mp_gpu(cg, plan, m)
    assert oe.shape == (0, C, K) and oo.shape == (0, C, K)

    f = _dev(_f_d(lmax, 36, C, R, 702, True, True, 4, 2), FK)
    f["row_ptr"] = torch.zeros(1, dtype=torch.int32, device="cuda")
    for k in ("col", "edge_feat", "edge_flip", "node_feat", "node_flip"):
        f[k] = f[k][:0]
    oe, oo = _f_gpu(cg, plan, f)
    assert oe.shape == (0, C, K) and oo.shape == (0, C, K)

    nt, nph = cg.nbody_grid(lmax, 3)
    pn = cg.plan_create(lmax, C, R, n_theta=nt, n_phi=nph)
    nb = inputs.nbody_inputs(4, lmax, C, R, 703, 3, self_coupled=False)
    X = [torch.from_numpy(x[:0].astype(np.float32)).cuda() for x in nb["X"]]
    Ut = [torch.from_numpy(u.astype(np.float32)).cuda() for u in nb["U"]]
    out = cg.onsite_nbody(pn, X, Ut, torch.from_numpy(nb["U_out"].astype(np.float32)).cuda())
    assert out.shape == (0, C, K)


def _isolate(d, keep):
    """The graph restricted to the edges whose receiver is in `keep` (others: empty rows)."""
    rp = d["row_ptr"]
    deg = np.diff(rp)
    recv = np.repeat(np.arange(len(deg)), deg)
    sel = np.isin(recv, keep)
    out = dict(d)
    new_deg = np.where(np.isin(np.arange(len(deg)), keep), deg, 0)
    out["row_ptr"] = np.concatenate([[0], np.cumsum(new_deg)]).astype(np.int32)
    out["col"] = d["col"][sel]
    for k in ("edge_unit", "edge_radial", "edge_feat", "edge_flip"):
        if d.get(k) is not None:
            out[k] = d[k][sel]
    out["n_edges"] = int(sel.sum())
    return out


def test_general_mp_empty_rows_and_no_edges(cg):
    import torch

    lmax, C, R = 4, 4, 6
    d = _mp_d(lmax, 40, C, R, 704, True, 4, 2)
    d = _isolate(d, np.arange(0, 40, 3))  # every third receiver keeps its neighbours
    deg = np.diff(d["row_ptr"])
    assert (deg == 0).any() and (deg > 0).any()
    plan = cg.plan_create(lmax, C, R, flags=cg.CGTP_VALIDATE_CSR)
    gpu = _mp_gpu(cg, plan, _dev(d, MP_G))
    _check(gpu, _mp_ref(lmax, d), TOL_F32)
    empty = torch.from_numpy(deg == 0).cuda()
    assert all(torch.count_nonzero(o[empty]) == 0 for o in gpu)
    z = _isolate(d, np.array([], dtype=np.int64))
    assert z["n_edges"] == 0
    oe, oo = _mp_gpu(cg, plan, _dev(z, MP_G))
    assert torch.count_nonzero(oe) == 0 and torch.count_nonzero(oo) == 0


def test_fields_empty_rows_and_no_edges(cg):
    import torch

    lmax, C, R = 3, 4, 5
    d = _isolate(_f_d(lmax, 36, C, R, 705, True, True, 4, 2), np.arange(1, 36, 4))
    deg = np.diff(d["row_ptr"])
    assert (deg == 0).any() and (deg > 0).any()
    plan = cg.plan_create(lmax, C, R)
    gpu = _f_gpu(cg, plan, _dev(d, FK))
    _check(gpu, _f_ref(lmax, d), TOL_F32)
    empty = torch.from_numpy(deg == 0).cuda()
    assert all(torch.count_nonzero(o[empty]) == 0 for o in gpu)
    z = _isolate(d, np.array([], dtype=np.int64))
    oe, oo = _f_gpu(cg, plan, _dev(z, FK))
    assert torch.count_nonzero(oe) == 0 and torch.count_nonzero(oo) == 0


def _rotation(lmax, seed):
    rot = bf.random_rotation(np.random.default_rng(seed))
    return rot, bf.wigner_d_real(lmax, rot)


# the phased split kernel (lmax <= 14), and above that unsplit groups on the matrix-core stage
@pytest.mark.parametrize("lmax,R", [(5, 6), (15, 4)])
def test_general_onsite_rotation(cg, lmax, R):
    """Rotating every input slot rotates both outputs (parity slots are ordinary SO(3)
    irreps; only inversion tells them apart)."""
    d = _on_d(lmax, 10, 4, R, 706 + lmax, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, R)
    oe, oo = (_np(x) for x in _on_gpu(cg, plan, _dev(d, ONSITE_G)))
    _, D = _rotation(lmax, 21)
    dr = dict(d)
    for k in ("A", "B", "A_flip", "B_flip"):
        dr[k] = bf.rotate_coeffs(D, d[k].astype(np.float64))
    re_, ro = _on_gpu(cg, plan, _dev(dr, ONSITE_G))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


@pytest.mark.parametrize("lmax,R", [(4, 6), (8, 16)])  # per-thread and matrix-core receivers
def test_general_mp_rotation(cg, lmax, R):
    d = _mp_d(lmax, 40, 4, R, 708 + lmax, True, 4, 2)
    plan = cg.plan_create(lmax, 4, R)
    oe, oo = (_np(x) for x in _mp_gpu(cg, plan, _dev(d, MP_G)))
    rot, D = _rotation(lmax, 22)
    dr = dict(d)
    dr["edge_unit"] = d["edge_unit"].astype(np.float64) @ rot.T
    for k in ("node_feat", "node_flip"):
        dr[k] = bf.rotate_coeffs(D, d[k].astype(np.float64))
    re_, ro = _mp_gpu(cg, plan, _dev(dr, MP_G))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


@pytest.mark.parametrize("lmax,R", [(3, 5), (6, 8)])
def test_fields_rotation(cg, lmax, R):
    """Both fields carry their own coefficients: rotating the edge field, the node field and
    their flipped slots rotates both outputs."""
    d = _f_d(lmax, 36, 4, R, 710 + lmax, True, True, 4, 2)
    plan = cg.plan_create(lmax, 4, R)
    oe, oo = (_np(x) for x in _f_gpu(cg, plan, _dev(d, FK)))
    _, D = _rotation(lmax, 23)
    dr = dict(d)
    for k in ("edge_feat", "edge_flip", "node_feat", "node_flip"):
        dr[k] = bf.rotate_coeffs(D, d[k].astype(np.float64))
    re_, ro = _f_gpu(cg, plan, _dev(dr, FK))
    assert rel_err(re_, bf.rotate_coeffs(D, oe)) <= TOL_F32
    assert rel_err(ro, bf.rotate_coeffs(D, oo)) <= TOL_F32


def test_general_calls_deterministic(cg):
    """The same inputs give bit-identical outputs on a second call (no atomics anywhere)."""
    import torch

    lmax = 6
    plan = cg.plan_create(lmax, 8, 8)
    t = _dev(_on_d(lmax, 50, 8, 8, 712, True, True, 4, 2), ONSITE_G)
    a, b = _on_gpu(cg, plan, t), _on_gpu(cg, plan, t)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    m = _dev(_mp_d(lmax, 60, 8, 8, 713, True, 4, 2), MP_G)
    a, b = _mp_gpu(cg, plan, m), _mp_gpu(cg, plan, m)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    f = _dev(_f_d(lmax, 40, 8, 8, 714, True, True, 4, 2), FK)
    a, b = _f_gpu(cg, plan, f), _f_gpu(cg, plan, f)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# grids larger than the defaults, up to the plan's cap of 2816 points: the kernels that assume
# the default grid hand over to their generic forms, which size their LDS from the plan
@pytest.mark.parametrize("lmax,R,nt,nph", [
    (4, 6, 20, 40),
    (6, 16, 40, 70),     # split groups stacked to 32 ranks, 2800 points
    (8, 16, 30, 60),     # matrix-core receiver range, off the default grid
])
def test_general_mp_grid_override(cg, lmax, R, nt, nph):
    d = _mp_d(lmax, 40, 4, R, 720 + lmax, True, 4, 2)
    plan = cg.plan_create(lmax, 4, R, n_theta=nt, n_phi=nph)
    _check(_mp_gpu(cg, plan, _dev(d, MP_G)), _mp_ref(lmax, d), TOL_F32)


# off the default grid the per-point receiver serves grids of up to 2048 points
@pytest.mark.parametrize("lmax,R,nt,nph", [(3, 5, 16, 30), (6, 8, 32, 64)])
def test_fields_grid_override(cg, lmax, R, nt, nph):
    d = _f_d(lmax, 30, 4, R, 724 + lmax, True, True, 4, 2, r_cut=3.0)
    plan = cg.plan_create(lmax, 4, R, n_theta=nt, n_phi=nph)
    _check(_f_gpu(cg, plan, _dev(d, FK)), _f_ref(lmax, d), TOL_F32)


def test_fields_grid_beyond_per_point_receiver(cg):
    """More than 2048 points off the default grid: a clear error, nothing launched."""
    lmax = 6
    d = _f_d(lmax, 30, 4, 8, 726, True, True, 4, 2, r_cut=3.0)
    plan = cg.plan_create(lmax, 4, 8, n_theta=40, n_phi=70)
    with pytest.raises(cg.CgtpError) as ei:
        _f_gpu(cg, plan, _dev(d, FK))
    assert ei.value.status == cg.CGTP_ERR_UNSUPPORTED and "2048" in str(ei.value)
