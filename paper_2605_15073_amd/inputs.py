"""Seeded synthetic inputs for the contracted CG products.

This module only draws random numbers and builds neighbour lists; it holds none
of the method's arithmetic (no spherical harmonics, no coupling). Both the GPU
path and the fp64 oracle consume exactly the arrays produced here.

Recipe (the paper benchmarks on random atomic environments, Sec. "Numerical
performance"; no public dataset is involved):

* RNG: ``numpy.random.default_rng(seed)`` (PCG64), fp64 standard normals rounded
  to fp32 once, so every consumer sees identical values.
* CP factor matrices ``[L][C][R]`` per degree: N(0, 1/C).
* Coefficients ``[N][C][L^2]``: N(0, 1), optionally scaled by 1/(2l+1) per degree.
* Message passing: atoms uniform in a periodic cube of side (N/density)^(1/3);
  directed edges j -> i for 0 < |r_j - r_i| < r_cut (minimum image), CSR sorted
  by receiver i, senders ascending in a row, atoms in generator (random) order.
  ``edge_unit`` = (r_j - r_i)/|r_j - r_i|. Radial features
  R_{n l}(r) = sum_k W[l][n][k] g_k(r) with 8 Gaussians
  g_k(r) = exp(-(r - k r_cut/7)^2 / (2 (r_cut/7)^2)), W ~ N(0, 1/8).
* General parameterization: parity-flipped slots N(0, 1) like the natural ones; input
  factors stacked [n_blocks][L][C][R] and output weights [2][L][C][R] (Gaunt, curl), each
  block N(0, 1/C), drawn from a second generator seeded seed + 7919 so the graph and the
  natural slots are those of the plain workload of the same seed.
* Two parity-bearing fields: per-edge field coefficients [E][C][L^2] (and their flipped
  slot) N(0, 1) drawn directly in fp32 from 64 PCG64 streams spawned from
  SeedSequence(seed + 104729) (flipped slot: seed + 104730), each filling a fixed slice;
  factor blocks from a generator seeded seed + 104731.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def _normal(rng: np.random.Generator, shape, scale=1.0) -> np.ndarray:
    return (rng.standard_normal(shape) * scale).astype(np.float32)


def degree_scale(lmax: int) -> np.ndarray:
    """1/(2l+1) for every flattened index k = l*l + l + m."""
    return np.concatenate([np.full(2 * l + 1, 1.0 / (2 * l + 1)) for l in range(lmax + 1)])


def cp_factors(rng: np.random.Generator, lmax: int, C: int, R: int) -> np.ndarray:
    return _normal(rng, (lmax + 1, C, R), 1.0 / np.sqrt(C))


def coefficients(rng: np.random.Generator, n: int, C: int, lmax: int, per_degree: bool):
    x = rng.standard_normal((n, C, (lmax + 1) ** 2))
    if per_degree:
        x = x * degree_scale(lmax)[None, None, :]
    return x.astype(np.float32)


def onsite_inputs(n: int, lmax: int, C: int, R: int, seed: int, per_degree: bool = False,
                  self_coupled: bool = False, distinct_out: bool = False):
    """Draw order: A, B (skipped when B := A), U_A, U_B, U_out (, U_out_odd)."""
    rng = np.random.default_rng(seed)
    A = coefficients(rng, n, C, lmax, per_degree)
    B = A if self_coupled else coefficients(rng, n, C, lmax, per_degree)
    U_A = cp_factors(rng, lmax, C, R)
    U_B = cp_factors(rng, lmax, C, R)
    U_out = cp_factors(rng, lmax, C, R)
    U_out_odd = cp_factors(rng, lmax, C, R) if distinct_out else U_out
    return dict(A=A, B=B, U_A=U_A, U_B=U_B, U_out_even=U_out, U_out_odd=U_out_odd)


def periodic_neighbours(pos: np.ndarray, box: float, r_cut: float):
    """CSR (by receiver) of directed edges j -> i with 0 < |r_j - r_i|_min-image < r_cut."""
    from scipy.spatial import cKDTree

    if not r_cut < box / 2:
        raise ValueError("r_cut must be below half the box side for minimum-image edges")
    n = pos.shape[0]
    tree = cKDTree(pos, boxsize=box)
    pairs = tree.query_pairs(r_cut, output_type="ndarray")
    if pairs.size == 0:
        pairs = np.zeros((0, 2), dtype=np.int64)
    recv = np.concatenate([pairs[:, 0], pairs[:, 1]])
    send = np.concatenate([pairs[:, 1], pairs[:, 0]])
    order = np.lexsort((send, recv))
    recv, send = recv[order], send[order]
    d = pos[send] - pos[recv]
    d -= box * np.round(d / box)
    dist = np.linalg.norm(d, axis=1)
    keep = dist > 0
    recv, send, d, dist = recv[keep], send[keep], d[keep], dist[keep]
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    np.add.at(row_ptr, recv + 1, 1)
    row_ptr = np.cumsum(row_ptr)
    return row_ptr.astype(np.int32), send.astype(np.int32), d, dist


def gaussian_radial(dist: np.ndarray, r_cut: float, n_basis: int = 8) -> np.ndarray:
    mu = np.arange(n_basis) * r_cut / (n_basis - 1)
    sigma = r_cut / (n_basis - 1)
    return np.exp(-((dist[:, None] - mu[None, :]) ** 2) / (2 * sigma ** 2))


def mp_inputs(n_atoms: int, lmax: int, C: int, R: int, seed: int, density: float = 0.1,
              r_cut: float = 5.0, n_basis: int = 8, distinct_out: bool = False,
              two_slot: bool = False):
    """Draw order: positions, W_rad, I, U_E, U_I, U_out (, U_out_odd) (, I_flip).

    two_slot adds node_flip, the parity-flipped node slot [N, C, L^2], drawn last so the
    other arrays are the same as without it."""
    rng = np.random.default_rng(seed)
    box = (n_atoms / density) ** (1.0 / 3.0)
    pos = rng.uniform(0.0, box, size=(n_atoms, 3))
    W_rad = rng.standard_normal((lmax + 1, C, n_basis)) / np.sqrt(n_basis)
    node_feat = coefficients(rng, n_atoms, C, lmax, per_degree=False)
    U_E = cp_factors(rng, lmax, C, R)
    U_I = cp_factors(rng, lmax, C, R)
    U_out = cp_factors(rng, lmax, C, R)
    U_out_odd = cp_factors(rng, lmax, C, R) if distinct_out else U_out
    row_ptr, col, d, dist = periodic_neighbours(pos, box, r_cut)
    edge_unit = (d / dist[:, None]).astype(np.float32)
    g = gaussian_radial(dist, r_cut, n_basis)                    # [E, K]
    edge_radial = np.empty((g.shape[0], C, lmax + 1), dtype=np.float32)  # [E, C, L]
    for l in range(lmax + 1):
        edge_radial[:, :, l] = g @ W_rad[l].T
    out = dict(row_ptr=row_ptr, col=col, edge_unit=edge_unit, edge_radial=edge_radial,
               node_feat=node_feat, U_E=U_E, U_I=U_I, U_out_even=U_out, U_out_odd=U_out_odd,
               box=box, n_edges=int(col.shape[0]))
    if two_slot:
        out["node_flip"] = coefficients(rng, n_atoms, C, lmax, per_degree=False)
    return out


def _stacked(rng, n_blocks: int, lmax: int, C: int, R: int) -> np.ndarray:
    if n_blocks == 1:
        return cp_factors(rng, lmax, C, R)
    return np.stack([cp_factors(rng, lmax, C, R) for _ in range(n_blocks)])


def _general_factors(rng, names, lmax, C, R, in_blocks, out_blocks):
    out = {nm: _stacked(rng, in_blocks, lmax, C, R) for nm in names}
    for nm in ("U_out_even", "U_out_odd"):
        out[nm] = _stacked(rng, out_blocks, lmax, C, R)
    return out


def general_onsite_inputs(n: int, lmax: int, C: int, R: int, seed: int, flip1: bool = True,
                          flip2: bool = True, in_blocks: int = 4, out_blocks: int = 2,
                          per_degree: bool = False):
    """On-site operands with optional parity-flipped slots and stacked factor blocks.
    Draw order (second generator): A_flip, B_flip (each if present), U_A, U_B, U_out_even,
    U_out_odd."""
    d = onsite_inputs(n, lmax, C, R, seed, per_degree=per_degree)
    rng = np.random.default_rng(seed + 7919)
    d["A_flip"] = coefficients(rng, n, C, lmax, per_degree) if flip1 else None
    d["B_flip"] = coefficients(rng, n, C, lmax, per_degree) if flip2 else None
    d.update(_general_factors(rng, ("U_A", "U_B"), lmax, C, R, in_blocks, out_blocks))
    return d


def general_mp_inputs(n_atoms: int, lmax: int, C: int, R: int, seed: int, flip: bool = True,
                      in_blocks: int = 4, out_blocks: int = 2, density: float = 0.1,
                      r_cut: float = 5.0):
    """Message passing with an optional flipped node slot and stacked factor blocks (the
    graph, radial features and node slots of mp_inputs with the same seed). Draw order
    (second generator): U_E, U_I, U_out_even, U_out_odd."""
    d = mp_inputs(n_atoms, lmax, C, R, seed, density=density, r_cut=r_cut, two_slot=flip)
    if not flip:
        d["node_flip"] = None
    rng = np.random.default_rng(seed + 7919)
    d.update(_general_factors(rng, ("U_E", "U_I"), lmax, C, R, in_blocks, out_blocks))
    return d


def normal_f32_streams(seed: int, shape, streams: int = 64) -> np.ndarray:
    """N(0, 1) fp32 array filled from `streams` PCG64 generators spawned from
    SeedSequence(seed), stream c filling the c-th of `streams` equal slices of the flattened
    array. The values depend on seed, shape and streams only; the slices are filled by
    parallel threads (numpy releases the GIL while it draws)."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    out = np.empty(shape, dtype=np.float32)
    flat = out.reshape(-1)
    kids = np.random.SeedSequence(seed).spawn(streams)
    cuts = np.linspace(0, flat.size, streams + 1).astype(np.int64)

    def fill(c):
        np.random.default_rng(kids[c]).standard_normal(out=flat[cuts[c]:cuts[c + 1]],
                                                       dtype=np.float32)

    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(fill, range(streams)))
    return out


def fields_mp_inputs(n_atoms: int, lmax: int, C: int, R: int, seed: int, edge_flip: bool = True,
                     node_flip: bool = True, in_blocks: int = 4, out_blocks: int = 2,
                     density: float = 0.1, r_cut: float = 5.0):
    """Message passing with two parity-bearing fields: the graph and node slots of mp_inputs
    with the same seed, and a per-edge field [E][C][L^2] (and its flipped slot) of N(0, 1)
    coefficients in place of R Y, drawn in fp32 by normal_f32_streams (seeds seed + 104729
    and seed + 104730). The factor blocks come from a generator seeded seed + 104731, in the
    order U_E, U_I, U_out_even, U_out_odd."""
    d = mp_inputs(n_atoms, lmax, C, R, seed, density=density, r_cut=r_cut, two_slot=node_flip)
    if not node_flip:
        d["node_flip"] = None
    E = d["n_edges"]
    K = (lmax + 1) ** 2
    d["edge_feat"] = normal_f32_streams(seed + 104729, (E, C, K))
    d["edge_flip"] = normal_f32_streams(seed + 104730, (E, C, K)) if edge_flip else None
    rng = np.random.default_rng(seed + 104731)
    d.update(_general_factors(rng, ("U_E", "U_I"), lmax, C, R, in_blocks, out_blocks))
    return d


def nbody_inputs(n: int, lmax: int, C: int, R: int, seed: int, nu: int,
                 self_coupled: bool = True, per_degree: bool = True):
    """nu-body on-site operands: X (a list of nu [N][C][L^2] arrays; with self_coupled one
    array repeated, the ACE density raised to the nu-th power), U (nu factor matrices),
    U_out. Draw order: X (once, or nu times), U[0 .. nu-1], U_out."""
    rng = np.random.default_rng(seed)
    if self_coupled:
        A = coefficients(rng, n, C, lmax, per_degree)
        X = [A] * nu
    else:
        X = [coefficients(rng, n, C, lmax, per_degree) for _ in range(nu)]
    U = [cp_factors(rng, lmax, C, R) for _ in range(nu)]
    return dict(X=X, U=U, U_out=cp_factors(rng, lmax, C, R))


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str          # "onsite", "mp", "mp_fields" (two parity-bearing fields) or "nbody"
    n: int             # nodes (on-site) or atoms (message passing)
    lmax: int
    C: int
    R: int
    seed: int
    per_degree: bool = False
    self_coupled: bool = False
    r_cut: float = 5.0
    two_slot: bool = False   # message passing with both node parity slots (Cases A-D)
    # general parameterization (0: the plain calls): input factor blocks 1, 2 or 4 ...
    in_blocks: int = 0
    out_blocks: int = 1      # ... output weight blocks per sector (1 or 2)
    flip1: bool = False      # first operand (on-site A, or the edge field) has a flipped slot
    nu: int = 0              # body order of a "nbody" workload

    @property
    def general(self) -> bool:
        return self.in_blocks > 0

    def make(self, **kw):
        if self.kind == "nbody":
            return nbody_inputs(self.n, self.lmax, self.C, self.R, self.seed, self.nu,
                                self_coupled=self.self_coupled, per_degree=self.per_degree, **kw)
        if self.kind == "mp_fields":
            return fields_mp_inputs(self.n, self.lmax, self.C, self.R, self.seed,
                                    edge_flip=self.flip1, node_flip=self.two_slot,
                                    in_blocks=self.in_blocks, out_blocks=self.out_blocks,
                                    r_cut=self.r_cut, **kw)
        if self.general and self.kind == "onsite":
            return general_onsite_inputs(self.n, self.lmax, self.C, self.R, self.seed,
                                         flip1=self.flip1, flip2=self.two_slot,
                                         in_blocks=self.in_blocks, out_blocks=self.out_blocks,
                                         per_degree=self.per_degree, **kw)
        if self.general:
            return general_mp_inputs(self.n, self.lmax, self.C, self.R, self.seed,
                                     flip=self.two_slot, in_blocks=self.in_blocks,
                                     out_blocks=self.out_blocks, r_cut=self.r_cut, **kw)
        if self.kind == "onsite":
            return onsite_inputs(self.n, self.lmax, self.C, self.R, self.seed,
                                 per_degree=self.per_degree, self_coupled=self.self_coupled, **kw)
        return mp_inputs(self.n, self.lmax, self.C, self.R, self.seed, r_cut=self.r_cut,
                         two_slot=self.two_slot, **kw)


# The five workloads of the benchmark plan, named by what they are.
WORKLOADS = {
    "onsite_n64_l2_c8": Workload("onsite_n64_l2_c8", "onsite", 64, 2, 8, 8, seed=0),
    "onsite_ace_n2048_l4_c64": Workload("onsite_ace_n2048_l4_c64", "onsite", 2048, 4, 64, 64,
                                        seed=1, per_degree=True, self_coupled=True),
    "mp_10k_l6_c128": Workload("mp_10k_l6_c128", "mp", 10000, 6, 128, 128, seed=2),
    "onsite_n4096_l12_c128": Workload("onsite_n4096_l12_c128", "onsite", 4096, 12, 128, 128,
                                      seed=3, per_degree=True),
    "mp_5k_l20_c64": Workload("mp_5k_l20_c64", "mp", 5000, 20, 64, 64, seed=4),
    # the same two message-passing workloads at the cutoff that gives the edge counts quoted
    # for them (about 301k and 151k directed edges, r_cut = 4.153 A, Z about 30)
    "mp_10k_l6_c128_rc4153": Workload("mp_10k_l6_c128_rc4153", "mp", 10000, 6, 128, 128,
                                      seed=2, r_cut=4.153),
    "mp_5k_l20_c64_rc4153": Workload("mp_5k_l20_c64_rc4153", "mp", 5000, 20, 64, 64, seed=4,
                                     r_cut=4.153),
    # both node parity slots populated (natural and parity-flipped), Cases A-D of Table 1
    "mp2_10k_l6_c128": Workload("mp2_10k_l6_c128", "mp", 10000, 6, 128, 128, seed=2,
                                two_slot=True),
    "mp2_5k_l20_c64": Workload("mp2_5k_l20_c64", "mp", 5000, 20, 64, 64, seed=4, two_slot=True),
    # the general parameterization: both parity slots, input factors and output weights per
    # (category, sector) block (Eqs. msgpass-cp-alpha, msgpass-cp-beta)
    "mpg_10k_l6_c128": Workload("mpg_10k_l6_c128", "mp", 10000, 6, 128, 128, seed=2,
                                two_slot=True, in_blocks=4, out_blocks=2),
    "onsiteg_n4096_l12_c128": Workload("onsiteg_n4096_l12_c128", "onsite", 4096, 12, 128, 128,
                                       seed=3, per_degree=True, two_slot=True, flip1=True,
                                       in_blocks=4, out_blocks=2),
    # two parity-bearing fields (Eq. twoparity-phi): a per-edge field with both slots in place
    # of R Y, both node slots, per-block factors
    "mpf_5k_l6_c64": Workload("mpf_5k_l6_c64", "mp_fields", 5000, 6, 64, 64, seed=4,
                              two_slot=True, flip1=True, in_blocks=4, out_blocks=2),
    # nu-body grid products (ACE-style: the density A to the nu-th power, one factor matrix per
    # power, one inverse transform), on the grid exact for the (nu + 1) lmax integrand
    "nbody_n2048_l4_c64_nu3": Workload("nbody_n2048_l4_c64_nu3", "nbody", 2048, 4, 64, 64,
                                       seed=5, per_degree=True, self_coupled=True, nu=3),
    "nbody_n2048_l8_c64_nu4": Workload("nbody_n2048_l8_c64_nu4", "nbody", 2048, 8, 64, 64,
                                       seed=6, per_degree=True, self_coupled=True, nu=4),
}
