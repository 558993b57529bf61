"""fp64 CPU oracle for the contracted Clebsch-Gordan products.

TEST INFRASTRUCTURE ONLY: tests/, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package; the product path
(``paper_2605_15073_amd``) never does, and the two share no code.

The arithmetic lives in ``cgtp_oracle.c`` (plain C, fp64, OpenMP over nodes);
this module only loads it with ctypes and marshals numpy arrays. See that file
for what is computed and which passages of the paper each part follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cgtp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile liboracle.so from cgtp_oracle.c with gcc (fp64, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
             "-o", tmp, _SRC, "-lm"],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    i32, i64, dbl = ctypes.c_int, ctypes.c_long, ctypes.c_double
    p = ctypes.c_void_p
    for name in ("cgo_wigner3j", "cgo_cg", "cgo_gaunt_conj", "cgo_curl_conj_im"):
        getattr(lib, name).restype = dbl
        getattr(lib, name).argtypes = [i32] * 6
    lib.cgo_kappa_inv_im.restype = dbl
    lib.cgo_kappa_inv_im.argtypes = [i32] * 3
    lib.cgo_real_entry.restype = dbl
    lib.cgo_real_entry.argtypes = [i32] * 7 + [ctypes.POINTER(dbl)]
    lib.cgo_real_table.restype = i64
    lib.cgo_real_table.argtypes = [i32, i32, i32, p, p, p, p, i64, ctypes.POINTER(dbl)]
    lib.cgo_real_sh.restype = None
    lib.cgo_real_sh.argtypes = [i32, dbl, dbl, dbl, p]
    lib.cgo_onsite.restype = i32
    lib.cgo_onsite.argtypes = [i32, i32, i32, i64] + [p] * 9 + [i32]
    lib.cgo_message_pass.restype = i32
    lib.cgo_message_pass.argtypes = [i32, i32, i32, i64, i64] + [p] * 9 + [p, i64, p, p, i32]
    lib.cgo_nbody.restype = i32
    lib.cgo_nbody.argtypes = [i32, i32, i32, i32, i64, p, p, p, p, i32]
    lib.cgo_message_pass_fields.restype = i32
    lib.cgo_message_pass_fields.argtypes = ([i32, i32, i32, i64, i64] + [p] * 9
                                            + [p, i64, p, p, i32])
    lib.cgo_max_threads.restype = i32
    lib.cgo_max_threads.argtypes = []
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


def max_threads() -> int:
    return int(_load().cgo_max_threads())


def wigner3j(j1, j2, j3, m1, m2, m3) -> float:
    return _load().cgo_wigner3j(j1, j2, j3, m1, m2, m3)


def cg(l1, m1, l2, m2, l, m) -> float:
    """<l1 m1 l2 m2 | l m> (Condon-Shortley)."""
    return _load().cgo_cg(l1, m1, l2, m2, l, m)


def gaunt_conj(l1, m1, l2, m2, l, m) -> float:
    """int Y_{l1m1} Y_{l2m2} Y*_{lm} (Eq. cg-integral), complex CS basis."""
    return _load().cgo_gaunt_conj(l1, m1, l2, m2, l, m)


def curl_conj_im(l1, m1, l2, m2, l, m) -> float:
    """Im int Y*_{lm} {Y_{l1m1}, Y_{l2m2}} (Eq. Q-CG); the value is purely imaginary."""
    return _load().cgo_curl_conj_im(l1, m1, l2, m2, l, m)


def kappa_inv_im(l1, l2, l) -> float:
    """Im kappa^-1(l1, l2, l) of Eq. kappa-inv-closed on the parity-odd support, else 0."""
    return _load().cgo_kappa_inv_im(l1, l2, l)


def real_entry(kind: int, l1, m1, l2, m2, l3, m3):
    """(value, imaginary residue) of int Y^R Y^R Y^R (kind 0) or int {Y^R, Y^R} Y^R (kind 1)."""
    im = ctypes.c_double(0.0)
    v = _load().cgo_real_entry(kind, l1, m1, l2, m2, l3, m3, ctypes.byref(im))
    return v, im.value


def real_table(kind: int, lmax_in: int, lmax_out: int | None = None):
    """Sparse real table: (k1, k2, k3, val, max_imag). kind 0 = Gaunt GR, 1 = curl QR."""
    lib = _load()
    if lmax_out is None:
        lmax_out = lmax_in
    mi = ctypes.c_double(0.0)
    n = lib.cgo_real_table(kind, lmax_in, lmax_out, None, None, None, None, 0, ctypes.byref(mi))
    k1 = np.zeros(max(n, 1), np.int32)
    k2 = np.zeros(max(n, 1), np.int32)
    k3 = np.zeros(max(n, 1), np.int32)
    v = np.zeros(max(n, 1), np.float64)
    lib.cgo_real_table(kind, lmax_in, lmax_out, _ptr(k1), _ptr(k2), _ptr(k3), _ptr(v), n,
                       ctypes.byref(mi))
    return k1[:n], k2[:n], k3[:n], v[:n], mi.value


def dense_table(kind: int, lmax_in: int, lmax_out: int | None = None) -> np.ndarray:
    """Dense [(lmax_in+1)^2, (lmax_in+1)^2, (lmax_out+1)^2] real table."""
    if lmax_out is None:
        lmax_out = lmax_in
    k1, k2, k3, v, _ = real_table(kind, lmax_in, lmax_out)
    n_in, n_out = (lmax_in + 1) ** 2, (lmax_out + 1) ** 2
    t = np.zeros((n_in, n_in, n_out))
    t[k1, k2, k3] = v
    return t


def real_sh(lmax: int, unit) -> np.ndarray:
    """Real SH of App. C Eq. realY at unit vectors [..., 3] -> [..., (lmax+1)^2]."""
    lib = _load()
    u = _f64(unit).reshape(-1, 3)
    out = np.zeros((u.shape[0], (lmax + 1) ** 2))
    row = np.zeros((lmax + 1) ** 2)
    for i in range(u.shape[0]):
        lib.cgo_real_sh(lmax, float(u[i, 0]), float(u[i, 1]), float(u[i, 2]), _ptr(row))
        out[i] = row
    return out.reshape(tuple(np.shape(unit)[:-1]) + ((lmax + 1) ** 2,))


def _in_blocks(U, lmax, C):
    """Input factors of the four blocks b = 2 * category + sector (category 0: Gaunt,
    1: curl; sector 0: out_even, 1: out_odd). U: [L, C, R] (all blocks share it),
    [2, L, C, R] (per category) or [4, L, C, R] (per block)."""
    U = _f64(U)
    if U.ndim == 3:
        blocks = [U] * 4
    elif U.shape[0] == 2:
        blocks = [U[0], U[0], U[1], U[1]]
    else:
        assert U.shape[0] == 4, "factor blocks: [L,C,R], [2,L,C,R] or [4,L,C,R]"
        blocks = [U[b] for b in range(4)]
    blocks = [np.ascontiguousarray(x) for x in blocks]
    for x in blocks:
        assert x.shape[:2] == (lmax + 1, C)
    return blocks


def _out_blocks(U_out_even, U_out_odd, lmax, C):
    """Output weights per block from the per-sector arrays: [L, C, R] (both categories share
    it) or [2, L, C, R] (Gaunt, curl)."""
    per = []
    for U in (U_out_even, U_out_odd):
        U = _f64(U)
        per.append([U, U] if U.ndim == 3 else [U[0], U[1]])
    blocks = [np.ascontiguousarray(per[b & 1][b >> 1]) for b in range(4)]
    for x in blocks:
        assert x.shape[:2] == (lmax + 1, C)
    return blocks


def _ptr_array(arrays):
    arr = (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])
    return arr, ctypes.cast(arr, ctypes.c_void_p)


def onsite(lmax, A, B, U_A, U_B, U_out_even, U_out_odd, nthreads: int = 0, A_flip=None,
           B_flip=None):
    """On-site contracted product, fp64. A, B: [N, C, L^2].

    A_flip, B_flip: parity-flipped slots of the two operands (None: absent). Slot pairs of
    equal relative parity send their Gaunt coupling to out_even (natural parity) and their
    curl coupling to out_odd; mixed pairs the other way round (p = p1 p2).
    U_A, U_B: input factors, [L, C, R] shared by all couplings, [2, L, C, R] per category
    (Gaunt, curl) or [4, L, C, R] per block 2 * category + sector (Eqs. msgpass-cp-alpha,
    msgpass-cp-beta). U_out_even, U_out_odd: [L, C, R], or [2, L, C, R] per category.
    Returns (out_even, out_odd), each [N, C, L^2] float64."""
    lib = _load()
    A, B = _f64(A), _f64(B)
    Af = None if A_flip is None else _f64(A_flip)
    Bf = None if B_flip is None else _f64(B_flip)
    N, C, L2 = A.shape
    assert L2 == (lmax + 1) ** 2 and B.shape == A.shape
    for X in (Af, Bf):
        assert X is None or X.shape == A.shape
    UA, UB = _in_blocks(U_A, lmax, C), _in_blocks(U_B, lmax, C)
    Uo = _out_blocks(U_out_even, U_out_odd, lmax, C)
    R = UA[0].shape[2]
    for x in UA + UB + Uo:
        assert x.shape == (lmax + 1, C, R)
    keep = [_ptr_array(x) for x in (UA, UB, Uo)]
    oe = np.zeros((N, C, L2))
    oo = np.zeros((N, C, L2))
    rc = lib.cgo_onsite(lmax, C, R, N, _ptr(A), _ptr(Af), _ptr(B), _ptr(Bf), keep[0][1],
                        keep[1][1], keep[2][1], _ptr(oe), _ptr(oo), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"cgo_onsite failed ({rc})")
    return oe, oo


def message_pass(lmax, row_ptr, col, edge_unit, edge_radial, node_feat, U_E, U_I,
                 U_out_even, U_out_odd, receivers=None, nthreads: int = 0, node_flip=None):
    """Message-passing contracted product, fp64, for a receiver subset.

    row_ptr [N+1], col [E] (int32 CSR by receiver), edge_unit [E,3],
    edge_radial [E,C,L], node_feat [N,C,L^2] (natural-parity slot), U_*: [L,C,R].
    node_flip: None, or the parity-flipped node slot [N,C,L^2] (Table 1, Cases C and D:
    out_even, the natural-parity output, gains the curl coupling with it and out_odd, the
    opposite-parity output, its Gaunt coupling).
    U_E, U_I: edge / node input factors, [L, C, R] shared by all couplings, [2, L, C, R]
    per category (Gaunt, curl) or [4, L, C, R] per block 2 * category + sector.
    U_out_even, U_out_odd: [L, C, R], or [2, L, C, R] per category.
    Returns (out_even, out_odd), each [len(receivers), C, L^2] (all receivers
    when receivers is None)."""
    if receivers is None:
        n = np.asarray(node_feat).shape[0]
        return _mp_rows(lmax, row_ptr, col, edge_unit, edge_radial, node_feat, node_flip, U_E,
                        U_I, U_out_even, U_out_odd, np.arange(n), nthreads)
    # Marshalling only: cut out the rows of the requested receivers and the
    # features of their senders, so large inputs are not converted to fp64 whole.
    row_ptr = np.asarray(row_ptr)
    rec = np.asarray(receivers, dtype=np.int64)
    starts, ends = row_ptr[rec].astype(np.int64), row_ptr[rec + 1].astype(np.int64)
    parts = [np.arange(a, b, dtype=np.int64) for a, b in zip(starts, ends)]
    eidx = np.concatenate(parts) if parts else np.zeros(0, np.int64)
    senders, local_col = np.unique(np.asarray(col)[eidx], return_inverse=True)
    # compact graph: node q < len(rec) is receiver rec[q]; node table rows are the senders
    n_compact = max(len(rec), len(senders), 1)
    def compact(a):
        full = np.asarray(a)
        out = np.zeros((n_compact,) + full.shape[1:], dtype=np.float64)
        out[:len(senders)] = full[senders]
        return out

    nf = compact(node_feat)
    nfl = None if node_flip is None else compact(node_flip)
    rp = np.zeros(n_compact + 1, np.int32)
    rp[1:len(rec) + 1] = np.cumsum(ends - starts)
    rp[len(rec) + 1:] = rp[len(rec)]
    return _mp_rows(lmax, rp, local_col.astype(np.int32), np.asarray(edge_unit)[eidx],
                    np.asarray(edge_radial)[eidx], nf, nfl, U_E, U_I,
                    U_out_even, U_out_odd, np.arange(len(rec)), nthreads)


def _mp_rows(lmax, row_ptr, col, edge_unit, edge_radial, node_feat, node_flip, U_E, U_I,
             U_out_even, U_out_odd, receivers, nthreads):
    lib = _load()
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col = np.ascontiguousarray(col, dtype=np.int32)
    eu, er, nf = _f64(edge_unit), _f64(edge_radial), _f64(node_feat)
    nfl = None if node_flip is None else _f64(node_flip)
    if nfl is not None:
        assert nfl.shape == nf.shape
    N, C, L2 = nf.shape
    UE, UI = _in_blocks(U_E, lmax, C), _in_blocks(U_I, lmax, C)
    Uo = _out_blocks(U_out_even, U_out_odd, lmax, C)
    R = UE[0].shape[2]
    for x in UE + UI + Uo:
        assert x.shape == (lmax + 1, C, R)
    E = col.shape[0]
    assert L2 == (lmax + 1) ** 2 and row_ptr.shape[0] == N + 1
    assert er.shape == (E, C, lmax + 1) and eu.shape == (E, 3)
    rec = np.ascontiguousarray(receivers, dtype=np.int64)
    keep = [_ptr_array(x) for x in (UE, UI, Uo)]
    oe = np.zeros((rec.shape[0], C, L2))
    oo = np.zeros((rec.shape[0], C, L2))
    rc = lib.cgo_message_pass(lmax, C, R, N, E, _ptr(row_ptr), _ptr(col), _ptr(eu), _ptr(er),
                              _ptr(nf), _ptr(nfl), keep[0][1], keep[1][1], keep[2][1], _ptr(rec),
                              rec.shape[0], _ptr(oe), _ptr(oo), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"cgo_message_pass failed ({rc})")
    return oe, oo


def message_pass_fields(lmax, row_ptr, col, edge_feat, node_feat, U_E, U_I, U_out_even,
                        U_out_odd, receivers=None, nthreads: int = 0, edge_flip=None,
                        node_flip=None):
    """Message passing with two parity-bearing fields (Eq. twoparity-phi), fp64.

    row_ptr [N+1], col [E] (int32 CSR by receiver); edge_feat [E, C, L^2] (natural-parity
    slot of the per-edge field) and edge_flip (its parity-flipped slot, or None);
    node_feat, node_flip [N, C, L^2]; factor arrays stacked as in onsite().
    Returns (out_even, out_odd), each [len(receivers), C, L^2] (all receivers when
    receivers is None)."""
    if receivers is None:
        n = np.asarray(node_feat).shape[0]
        return _mpf_rows(lmax, row_ptr, col, edge_feat, edge_flip, node_feat, node_flip, U_E,
                         U_I, U_out_even, U_out_odd, np.arange(n), nthreads)
    # Marshalling only: the rows of the requested receivers, their edges and the features
    # of their senders, so large inputs are not converted to fp64 whole.
    row_ptr = np.asarray(row_ptr)
    rec = np.asarray(receivers, dtype=np.int64)
    starts, ends = row_ptr[rec].astype(np.int64), row_ptr[rec + 1].astype(np.int64)
    parts = [np.arange(a, b, dtype=np.int64) for a, b in zip(starts, ends)]
    eidx = np.concatenate(parts) if parts else np.zeros(0, np.int64)
    senders, local_col = np.unique(np.asarray(col)[eidx], return_inverse=True)
    n_compact = max(len(rec), len(senders), 1)

    def compact(a):
        if a is None:
            return None
        full = np.asarray(a)
        out = np.zeros((n_compact,) + full.shape[1:], dtype=np.float64)
        out[:len(senders)] = full[senders]
        return out

    rp = np.zeros(n_compact + 1, np.int32)
    rp[1:len(rec) + 1] = np.cumsum(ends - starts)
    rp[len(rec) + 1:] = rp[len(rec)]
    cut = lambda a: None if a is None else np.asarray(a)[eidx]
    return _mpf_rows(lmax, rp, local_col.astype(np.int32), cut(edge_feat), cut(edge_flip),
                     compact(node_feat), compact(node_flip), U_E, U_I, U_out_even, U_out_odd,
                     np.arange(len(rec)), nthreads)


def _mpf_rows(lmax, row_ptr, col, edge_feat, edge_flip, node_feat, node_flip, U_E, U_I,
              U_out_even, U_out_odd, receivers, nthreads):
    lib = _load()
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col = np.ascontiguousarray(col, dtype=np.int32)
    ef, nf = _f64(edge_feat), _f64(node_feat)
    efl = None if edge_flip is None else _f64(edge_flip)
    nfl = None if node_flip is None else _f64(node_flip)
    N, C, L2 = nf.shape
    E = col.shape[0]
    assert L2 == (lmax + 1) ** 2 and row_ptr.shape[0] == N + 1 and ef.shape == (E, C, L2)
    assert efl is None or efl.shape == ef.shape
    assert nfl is None or nfl.shape == nf.shape
    UE, UI = _in_blocks(U_E, lmax, C), _in_blocks(U_I, lmax, C)
    Uo = _out_blocks(U_out_even, U_out_odd, lmax, C)
    R = UE[0].shape[2]
    for x in UE + UI + Uo:
        assert x.shape == (lmax + 1, C, R)
    rec = np.ascontiguousarray(receivers, dtype=np.int64)
    keep = [_ptr_array(x) for x in (UE, UI, Uo)]
    oe = np.zeros((rec.shape[0], C, L2))
    oo = np.zeros((rec.shape[0], C, L2))
    rc = lib.cgo_message_pass_fields(lmax, C, R, N, E, _ptr(row_ptr), _ptr(col), _ptr(ef),
                                     _ptr(efl), _ptr(nf), _ptr(nfl), keep[0][1], keep[1][1],
                                     keep[2][1], _ptr(rec), rec.shape[0], _ptr(oe), _ptr(oo),
                                     int(nthreads))
    if rc != 0:
        raise RuntimeError(f"cgo_message_pass_fields failed ({rc})")
    return oe, oo


def nbody(lmax, X, U, U_out, nthreads: int = 0):
    """nu-body on-site product, fp64: X, U lists of nu arrays [N, C, L^2] and [L, C, R];
    U_out [L, C, R]. Returns out [N, C, L^2] (natural parity)."""
    lib = _load()
    nu = len(X)
    assert nu == len(U) and nu >= 1
    Xs = [_f64(x) for x in X]
    Us = [_f64(u) for u in U]
    Uo = _f64(U_out)
    N, C, L2 = Xs[0].shape
    R = Us[0].shape[2]
    assert L2 == (lmax + 1) ** 2
    for x in Xs:
        assert x.shape == (N, C, L2)
    for u in Us + [Uo]:
        assert u.shape == (lmax + 1, C, R)
    kx, ku = _ptr_array(Xs), _ptr_array(Us)
    out = np.zeros((N, C, L2))
    rc = lib.cgo_nbody(lmax, C, R, nu, N, kx[1], ku[1], _ptr(Uo), _ptr(out), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"cgo_nbody failed ({rc})")
    return out
