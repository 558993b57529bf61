"""Independent brute-force references used to pin the oracle.

Nothing here imports the oracle or the GPU library. Spherical harmonics come
from ``scipy.special.sph_harm_y`` (complex, Condon-Shortley), turned into the
real basis of App. C (Eq. realY, no CS phase); integrals are dense
Gauss-Legendre x uniform-phi quadratures from ``numpy.polynomial.legendre``;
surface gradients are 4th-order central finite differences along the tangent
frame (e_theta, e_phi), so no analytic derivative of P_l^m is used.
"""
from __future__ import annotations

import numpy as np
from scipy.special import sph_harm_y


def lm_index(lmax: int):
    return [(l, m) for l in range(lmax + 1) for m in range(-l, l + 1)]


def real_sh_angles(lmax: int, theta, phi) -> np.ndarray:
    """Real SH of Eq. realY at polar angle theta, azimuth phi -> [..., (lmax+1)^2]."""
    theta = np.asarray(theta, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    out = np.zeros(theta.shape + ((lmax + 1) ** 2,))
    for l in range(lmax + 1):
        for m in range(-l, l + 1):
            k = l * l + l + m
            y = sph_harm_y(l, abs(m), theta, phi)   # CS phase (-1)^|m| included
            cs = (-1.0) ** abs(m)
            if m == 0:
                out[..., k] = y.real
            elif m > 0:
                out[..., k] = np.sqrt(2.0) * cs * y.real
            else:
                out[..., k] = np.sqrt(2.0) * cs * y.imag
    return out


def real_sh_xyz(lmax: int, xyz) -> np.ndarray:
    xyz = np.asarray(xyz, dtype=np.float64)
    r = np.linalg.norm(xyz, axis=-1)
    theta = np.arccos(np.clip(xyz[..., 2] / r, -1.0, 1.0))
    phi = np.arctan2(xyz[..., 1], xyz[..., 0])
    return real_sh_angles(lmax, theta, phi)


def dense_grid(n_theta: int = 24, n_phi: int = 48):
    """Points (unit vectors), their (theta, phi) and quadrature weights (sum 4 pi)."""
    x, w = np.polynomial.legendre.leggauss(n_theta)
    theta = np.arccos(x)
    phi = 2 * np.pi * np.arange(n_phi) / n_phi
    T, P = np.meshgrid(theta, phi, indexing="ij")
    W = np.repeat(w[:, None], n_phi, axis=1) * (2 * np.pi / n_phi)
    pts = np.stack([np.sin(T) * np.cos(P), np.sin(T) * np.sin(P), np.cos(T)], axis=-1)
    return pts.reshape(-1, 3), T.ravel(), P.ravel(), W.ravel()


def tangent_frame(theta, phi):
    e_t = np.stack([np.cos(theta) * np.cos(phi), np.cos(theta) * np.sin(phi), -np.sin(theta)], -1)
    e_p = np.stack([-np.sin(phi), np.cos(phi), np.zeros_like(phi)], -1)
    return e_t, e_p


def surface_derivs(f, pts, theta, phi, h=1e-3):
    """(D_{e_theta} f, D_{e_phi} f) at unit vectors pts, f: [P,3] -> [P, K]."""
    e_t, e_p = tangent_frame(theta, phi)

    def d(t):
        def at(s):
            q = pts + s * t
            return f(q / np.linalg.norm(q, axis=-1, keepdims=True))
        return (-at(2 * h) + 8 * at(h) - 8 * at(-h) + at(-2 * h)) / (12 * h)

    return d(e_t), d(e_p)


def sh_and_derivs(lmax: int, n_theta: int = 24, n_phi: int = 48):
    """Y [P,K], D_theta Y [P,K], D_phi Y [P,K], weights [P] on a dense grid."""
    pts, T, P, W = dense_grid(n_theta, n_phi)
    Y = real_sh_xyz(lmax, pts)
    Dt, Dp = surface_derivs(lambda q: real_sh_xyz(lmax, q), pts, T, P)
    return Y, Dt, Dp, W


def bracket(Dt_a, Dp_a, Dt_b, Dp_b):
    """r . (grad a x grad b) with grad = Dt e_theta + Dp e_phi and e_theta x e_phi = r."""
    return Dt_a * Dp_b - Dp_a * Dt_b


def random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    a, b, c, d = q
    return np.array([
        [a * a + b * b - c * c - d * d, 2 * (b * c - a * d), 2 * (b * d + a * c)],
        [2 * (b * c + a * d), a * a - b * b + c * c - d * d, 2 * (c * d - a * b)],
        [2 * (b * d - a * c), 2 * (c * d + a * b), a * a - b * b - c * c + d * d],
    ])


def wigner_d_real(lmax: int, rot: np.ndarray, rng: np.random.Generator | None = None):
    """Block-diagonal real Wigner matrix D for the active rotation ``rot``:
    a field f = sum_k c_k Y_k rotated as (rot f)(x) = f(rot^T x) has coefficients
    D @ c. Fitted by least squares from SH samples at random points."""
    rng = rng or np.random.default_rng(12345)
    n = (lmax + 1) ** 2
    pts = rng.standard_normal((4 * n + 32, 3))
    pts /= np.linalg.norm(pts, axis=1, keepdims=True)
    Y = real_sh_xyz(lmax, pts)                    # [P, K]
    Yr = real_sh_xyz(lmax, pts @ rot)             # rows: Y(rot^T x)
    # Y_k(rot^T x) = sum_j Y_j(x) M[j, k]  =>  new coefficients c' = M @ c
    M, *_ = np.linalg.lstsq(Y, Yr, rcond=None)
    keep = np.zeros((n, n), bool)
    for l in range(lmax + 1):                     # the exact block structure
        s = slice(l * l, (l + 1) * (l + 1))
        keep[s, s] = True
    M[~keep] = 0.0
    return M


def rotate_coeffs(D: np.ndarray, X: np.ndarray) -> np.ndarray:
    """Apply D on the last (L^2) axis."""
    return np.einsum("kj,...j->...k", D, X)
