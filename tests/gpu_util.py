"""Helpers for the GPU parity tests: move seeded inputs to the device, call the
library through its binding, compare with the oracle per output slot."""
from __future__ import annotations

import numpy as np

ONSITE_KEYS = ("A", "B", "U_A", "U_B", "U_out_even", "U_out_odd")
MP_KEYS = ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "U_E", "U_I",
           "U_out_even", "U_out_odd")

TOL_F32 = 2e-5      # max|gpu - ref| / max|ref| per output slot (fp32 path)
TOL_F64 = 1e-11     # fp64 path of the same kernels


def to_dev(d, keys, dtype="f32"):
    import torch

    out = {}
    for k in keys:
        a = d[k]
        if a.dtype == np.int32:
            out[k] = torch.from_numpy(np.ascontiguousarray(a)).cuda()
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(
                a.astype(np.float64 if dtype == "f64" else np.float32))).cuda()
    return out


def rel_err(gpu, ref, scale=None):
    g = gpu.detach().cpu().numpy() if hasattr(gpu, "detach") else np.asarray(gpu)
    s = np.abs(ref).max() if scale is None else scale
    return float(np.abs(g.astype(np.float64) - ref).max() / max(s, 1e-300))


def run_onsite(cg, plan, t, **kw):
    return cg.onsite(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"], t["U_out_odd"],
                     **kw)


def run_mp(cg, plan, t, **kw):
    return cg.message_pass(plan, *(t[k] for k in MP_KEYS), **kw)


def sample_rows(n: int, k: int, seed: int):
    """k distinct rows of [0, n) drawn with a seeded generator over the whole range, always
    including the first and the last, sorted."""
    if k >= n:
        return np.arange(n)
    rng = np.random.default_rng(seed)
    inner = rng.choice(np.arange(1, n - 1), max(k - 2, 0), replace=False)
    return np.unique(np.concatenate([[0, n - 1], inner]))[:max(k, 1)]


def bench_order(cg, plan, d):
    """Set on plan the receiver order bench.py uses for the graph of d (cgtp_receiver_order
    from the edge directions when the inputs have them)."""
    cg.set_receiver_order(plan, cg.receiver_order(d["row_ptr"], d["col"], d.get("edge_unit")))


def same_without_order(cg, plan, run, got):
    """run(plan) in node order equals got (computed under a receiver order) bit for bit."""
    import torch

    cg.set_receiver_order(plan, None)
    base = run(plan)
    assert all(torch.equal(a, b) for a, b in zip(base, got))
