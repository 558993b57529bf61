"""CPU tests of cgtp_receiver_order (host only): a permutation of the nodes for any CSR,
deterministic, components contiguous, and, where positions are exact, a Hilbert-curve walk:
on a lattice whose edge vectors are the unit lattice steps, consecutive receivers are lattice
neighbours. No GPU call runs here."""
from __future__ import annotations

import numpy as np
import pytest

import paper_2605_15073_amd as cg
from paper_2605_15073_amd import inputs


@pytest.fixture(scope="module")
def lib():
    return cg.load_library()


def _lattice(nx, ny, nz, scale=1.0):
    idx = lambda x, y, z: (x * ny + y) * nz + z
    rows, cols, vec = [], [], []
    for x in range(nx):
        for y in range(ny):
            for z in range(nz):
                nb = []
                for d in ((1, 0, 0), (-1, 0, 0), (0, 1, 0), (0, -1, 0), (0, 0, 1), (0, 0, -1)):
                    X, Y, Z = x + d[0], y + d[1], z + d[2]
                    if 0 <= X < nx and 0 <= Y < ny and 0 <= Z < nz:
                        nb.append((idx(X, Y, Z), tuple(scale * c for c in d)))
                nb.sort()
                rows.append(len(nb))
                cols += [a for a, _ in nb]
                vec += [v for _, v in nb]
    rp = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    xyz = np.array([(i // (ny * nz), (i // nz) % ny, i % nz) for i in range(nx * ny * nz)])
    return rp, np.array(cols, np.int32), np.array(vec, np.float32), xyz


@pytest.mark.parametrize("side,scale", [(2, 1.0), (4, 1.0), (8, 1.0), (4, 2.5)])
def test_lattice_order_is_a_hilbert_walk(side, scale):
    rp, col, vec, xyz = _lattice(side, side, side, scale)
    o = cg.receiver_order(rp, col, vec)
    assert sorted(o.tolist()) == list(range(side ** 3))
    steps = np.abs(np.diff(xyz[o], axis=0)).sum(1)
    assert (steps == 1).all()


def test_lattice_with_edge_directions_only():
    # unit directions of a lattice with spacing 2.5 are the unit steps: same walk
    rp, col, vec, xyz = _lattice(4, 4, 4, 2.5)
    unit = vec / np.linalg.norm(vec, axis=1, keepdims=True)
    o = cg.receiver_order(rp, col, unit)
    assert (np.abs(np.diff(xyz[o], axis=0)).sum(1) == 1).all()


def test_permutation_components_and_determinism():
    d = inputs.mp_inputs(600, 1, 2, 2, 11, density=0.05, r_cut=2.5)
    rp, col, unit = d["row_ptr"], d["col"], d["edge_unit"]
    n = rp.shape[0] - 1
    o = cg.receiver_order(rp, col, unit)
    assert sorted(o.tolist()) == list(range(n))
    assert np.array_equal(o, cg.receiver_order(rp, col, unit))
    # components (undirected reachability) are contiguous runs of the order
    from scipy.sparse import csr_matrix
    from scipy.sparse.csgraph import connected_components
    A = csr_matrix((np.ones(col.shape[0]), col, rp), shape=(n, n))
    nc, lab = connected_components(A, directed=False)
    assert nc > 1  # isolated atoms at this density
    runs = lab[o]
    changes = np.flatnonzero(np.diff(runs)) + 1
    assert len(changes) == nc - 1
    # without edge vectors: breadth-first order, also a permutation with contiguous components
    b = cg.receiver_order(rp, col)
    assert sorted(b.tolist()) == list(range(n))
    assert len(np.flatnonzero(np.diff(lab[b]))) == nc - 1
    assert b[0] == 0


def test_breadth_first_order_on_a_path():
    # path 0 - 1 - ... - 9 stored as a CSR; breadth-first from 0 visits it in order
    n = 10
    rows = [[1]] + [[i - 1, i + 1] for i in range(1, n - 1)] + [[n - 2]]
    rp = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
    col = np.array([c for r in rows for c in r], np.int32)
    assert cg.receiver_order(rp, col).tolist() == list(range(n))


def test_empty_and_isolated():
    assert cg.receiver_order(np.zeros(1, np.int32), np.zeros(0, np.int32)).shape == (0,)
    o = cg.receiver_order(np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros((0, 3), np.float32))
    assert o.tolist() == list(range(5))


def test_csr_errors(lib):
    with pytest.raises(cg.CgtpError) as ei:
        cg.receiver_order(np.array([0, 2, 1], np.int32), np.array([1, 0], np.int32))
    assert ei.value.status == cg.CGTP_ERR_CSR
    with pytest.raises(cg.CgtpError) as ei:
        cg.receiver_order(np.array([0, 1, 2], np.int32), np.array([1, 5], np.int32))
    assert ei.value.status == cg.CGTP_ERR_CSR
    with pytest.raises(cg.CgtpError) as ei:
        cg.receiver_order(np.array([0, 1, 3], np.int32), np.array([1, 0], np.int32))
    assert ei.value.status == cg.CGTP_ERR_CSR
    assert lib.cgtp_receiver_order(-1, 0, None, None, None, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_receiver_order(3, 0, None, None, None, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_plan_set_receiver_order(None, 3, None) == cg.CGTP_ERR_ARG
