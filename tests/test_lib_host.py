"""CPU tests of the HIP library: it loads, exports every symbol the header
declares, its host-side grid tables are right, and descriptor errors are
reported without touching a GPU. No compute call runs here."""
from __future__ import annotations

import ctypes
import math
import os
import re

import numpy as np
import pytest
from scipy.special import lpmv

import paper_2605_15073_amd as cg

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "cgtp.h")


@pytest.fixture(scope="module")
def lib():
    return cg.load_library()


def test_header_symbols_exported(lib):
    src = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:int|const char \*)\s*(cgtp_\w+)\s*\(", src, re.M))
    assert declared == set(cg.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_header_constants_match_binding():
    src = open(HEADER).read()
    consts = dict(re.findall(r"#define (CGTP_\w+) \(?(-?\w+)u?\)?", src))
    for name, val in consts.items():
        if name == "CGTP_H" or not hasattr(cg, name):
            continue
        assert int(val.rstrip("u"), 0) == getattr(cg, name), name


@pytest.mark.parametrize("lmax", [0, 1, 2, 5, 12, 20, 24])
def test_gauss_legendre_matches_numpy(lmax):
    x, w, p, dp, q = cg.host_tables(lmax)
    U = (3 * lmax + 3) // 2
    assert x.shape == (U,)
    xr, wr = np.polynomial.legendre.leggauss(U)
    order = np.argsort(x)
    assert np.abs(x[order] - xr).max() < 1e-14
    assert np.abs(w[order] - wr).max() < 1e-14
    assert abs(w.sum() - 2) < 1e-14


def _pt_ref(l, m, x):
    """Pt_l^m without the Condon-Shortley phase, via scipy's lpmv (which has it)."""
    n = math.sqrt((2 * l + 1) / (4 * math.pi) * math.factorial(l - m) / math.factorial(l + m))
    return n * (-1) ** m * lpmv(m, l, x)


@pytest.mark.parametrize("lmax", [2, 6, 12, 20])
def test_legendre_tables_match_scipy(lmax):
    x, w, p, dp, q = cg.host_tables(lmax)
    h = 1e-6
    for l in range(lmax + 1):
        for m in range(l + 1):
            i = l * (l + 1) // 2 + m
            ref = _pt_ref(l, m, x)
            scale = max(1.0, np.abs(ref).max())
            assert np.abs(p[:, i] - ref).max() < 1e-12 * scale, (l, m)
            dref = (_pt_ref(l, m, x + h) - _pt_ref(l, m, x - h)) / (2 * h)
            dscale = max(1.0, np.abs(dref).max())
            assert np.abs(dp[:, i] - dref).max() < 1e-6 * dscale, (l, m)


def test_fourier_table():
    lmax, V = 4, 13
    *_, q = cg.host_tables(lmax)
    phi = 2 * np.pi * np.arange(V) / V
    for m in range(-lmax, lmax + 1):
        if m > 0:
            ref = np.sqrt(2) * np.cos(m * phi)
        elif m == 0:
            ref = np.ones(V)
        else:
            ref = np.sqrt(2) * np.sin(-m * phi)
        assert np.abs(q[:, m + lmax] - ref).max() < 1e-14


def test_grid_is_exact_for_degree_3lmax_products():
    """The default grid integrates Y_a Y_b Y_c exactly (orthonormality of the
    real basis assembled from the library's own p and q tables)."""
    for lmax in (1, 2, 3, 4):
        x, w, p, dp, q = cg.host_tables(lmax)
        V = q.shape[0]
        Y = []
        for l in range(lmax + 1):
            for m in range(-l, l + 1):
                Y.append(np.outer(p[:, l * (l + 1) // 2 + abs(m)], q[:, m + lmax]).ravel())
        Y = np.array(Y)
        W = np.repeat(w, V) * 2 * np.pi / V
        gram = (Y * W) @ Y.T
        assert np.abs(gram - np.eye(len(Y))).max() < 1e-13


def test_host_tables_reject_bad_grid(lib):
    assert lib.cgtp_host_tables(3, 4, 10, None, None, None, None, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_host_tables(3, 5, 9, None, None, None, None, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_host_tables(25, 0, 0, None, None, None, None, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_host_tables(3, 5, 10, None, None, None, None, None) == cg.CGTP_OK


def test_plan_create_rejects_bad_descriptors(lib):
    h = ctypes.c_void_p()
    bad = [
        cg._Desc(-1, 8, 8, 0, 0, 0, 0),
        cg._Desc(25, 8, 8, 0, 0, 0, 0),
        cg._Desc(4, 0, 8, 0, 0, 0, 0),
        cg._Desc(4, 8, 0, 0, 0, 0, 0),
        cg._Desc(4, 8, 8, 6, 0, 0, 0),     # below ceil((3*4+1)/2) = 7
        cg._Desc(4, 8, 8, 0, 12, 0, 0),    # below 13
        cg._Desc(4, 8, 8, 0, 0, 7, 0),     # unknown dtype
        cg._Desc(4, 8, 8, 0, 0, 0, 64),    # unknown flag
    ]
    for d in bad:
        assert lib.cgtp_plan_create(ctypes.byref(d), ctypes.byref(h)) == cg.CGTP_ERR_ARG
        assert h.value is None
        assert lib.cgtp_last_error()
    assert lib.cgtp_plan_create(None, ctypes.byref(h)) == cg.CGTP_ERR_ARG
    d = cg._Desc(4, 8, 8, 0, 0, 0, 0)
    assert lib.cgtp_plan_create(ctypes.byref(d), None) == cg.CGTP_ERR_ARG


def test_null_plan_calls_fail_cleanly(lib):
    assert lib.cgtp_onsite(None, 1, *([None] * 8), None, 0, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_message_pass(None, 1, 1, *([None] * 11), None, 0, None) == cg.CGTP_ERR_ARG
    assert lib.cgtp_destroy(None) == cg.CGTP_OK
    sz = ctypes.c_size_t()
    assert lib.cgtp_workspace_bytes(None, 0, 1, 0, ctypes.byref(sz)) == cg.CGTP_ERR_ARG
    for s in (0, -1, -2, -3, -4, -5, -99):
        assert lib.cgtp_status_string(s)
