#!/usr/bin/env python
"""Benchmark of the contracted Clebsch-Gordan products on one MI355X.

A step is one call of the library on one batch of synthetic input. The default
workload is message passing on 10,000 atoms (periodic box at 0.1 atoms/A^3,
5 A cutoff, about 525k directed edges), lmax = 6, C = R = 128, fp32. One
cgtp_message_pass call runs every stage of the method: node-side channel
contraction and grid synthesis (A, dA/dx, dA/dphi), edge-radial contraction,
the receiver pass (edge-field synthesis, grid product and surface curl summed
over neighbours, quadrature analysis) and both output projections.

Prints ONE JSON line: throughput in nodes*channels/s (receivers x C per second),
the per-stage GPU times measured with HIP events on the library's stream over
the timed steps, the roofline of the dominant kernel, and the fp64 CPU oracle
timed on a bounded sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
  python bench.py --sweep-out FILE     # lmax sweeps, one JSON line per point in FILE
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 vector (and matrix) peak
CSRC = os.path.join(ROOT, "paper_2605_15073_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


def kernel_sha() -> str:
    """Hash of the library's device code (the .hip sources and their headers): traffic
    counters are only valid for this version of the kernels."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def grid_dims(lmax: int):
    U = (3 * lmax + 3) // 2
    V = 3 * lmax + 1
    return U, V


# ---------------------------------------------------------------- algorithmic work

def receiver_bytes(lmax: int, R: int, N: int, E: int, slots: int = 1, planes: int = 0,
                   rt_blocks: int = 1, t_fields: int = 2) -> int:
    """Bytes the receiver pass must move (fp32): per edge the sender grid fields the
    couplings read (planes R UV floats: the value A for a Gaunt coupling and, for a curl
    coupling, dA/dx and dA/dphi, or nothing more when the curl's derivatives are moved onto
    the analysis; default 3 per node slot), the edge radial
    coefficients (R L per distinct edge factor block), the unit vector and the sender
    index; per receiver the row pointer and the analysed fields (R K each)."""
    U, V = grid_dims(lmax)
    L, K = lmax + 1, (lmax + 1) ** 2
    planes = planes or 3 * slots
    per_edge = 4 * (planes * R * U * V + rt_blocks * R * L + 3 + 1)
    per_recv = 4 * (1 + t_fields * R * K)
    return E * per_edge + N * per_recv


def compulsory_receiver_bytes(lmax: int, R: int, N: int, E: int, planes: int = 3,
                              rt_blocks: int = 1, t_fields: int = 2) -> int:
    """Bytes the receiver stage must move to or from HBM at the least (fp32): every sender's
    grid fields once (the planes the couplings read, R U V floats each), the edge radial
    coefficients, unit vectors and sender indices once, the row pointers, and the analysed
    fields written once. Everything beyond this is served by the on-chip and memory-side
    caches or re-read."""
    U, V = grid_dims(lmax)
    L, K = lmax + 1, (lmax + 1) ** 2
    return (4 * N * planes * R * U * V + 4 * E * (rt_blocks * R * L + 3 + 1)
            + 4 * (N + 1) + 4 * N * t_fields * R * K)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def live_blocks(flip1: bool, flip2: bool):
    """Blocks b = 2 category + sector that receive a coupling: Gaunt sends equal slot pairs
    to the even sector and mixed ones to the odd sector, curl the other way round."""
    live = set()
    for s1 in (0, 1) if flip1 else (0,):
        for s2 in (0, 1) if flip2 else (0,):
            rel = int(s1 != s2)
            live.update({rel, 2 + (1 - rel)})
    return sorted(live)


def general_receiver_bytes(w, N: int, E: int) -> int:
    """Algorithmic receiver bytes of general message passing: one grid field per block (the
    sender values its factors give: the curl takes its derivatives on the analysis side); one
    edge factor per block (one when shared); one analysed field per block with per-category
    weights (two otherwise)."""
    live = live_blocks(False, w.two_slot)
    planes = len(live)
    rt = 1 if w.in_blocks == 1 else len(live)
    tf = len(live) if w.out_blocks == 2 else 2
    return receiver_bytes(w.lmax, w.R, N, E, planes=planes, rt_blocks=rt, t_fields=tf)


def onsite_grid_flops(lmax: int, R: int, N: int, kind: str = "both") -> int:
    """fp32 flops of the on-site grid stage with the paper's dense transforms, per
    (node, rank). Both products: Legendre synthesis of F and dF/dx for both operands
    (8 U L^2), Fourier synthesis of 3 fields per operand (12 U V M), product and curl
    (4 U V), Fourier analysis of 2 fields (4 U V M), Gauss-Legendre analysis (4 U L^2).
    Gaunt only: F of both operands, one field each, one product, one analysis. Curl
    only: F and dF/dx of both operands, two fields each, the bracket, one analysis."""
    U, V = grid_dims(lmax)
    L, M = lmax + 1, 2 * lmax + 1
    per = {"both": 12 * U * L * L + 16 * U * V * M + 4 * U * V,
           "gaunt": 6 * U * L * L + 6 * U * V * M + U * V,
           "curl": 10 * U * L * L + 10 * U * V * M + 3 * U * V}[kind]
    return N * R * per


def fields_receiver_flops(w, N: int, E: int) -> int:
    """Algorithmic flops of the edge-field receiver (two parity-bearing fields), dense
    transforms as in onsite_grid_flops. Per (edge, rank) of a slot pair: the edge field's
    Legendre and Fourier syntheses and the product; per (receiver, rank): the analysis. With
    shared factors a pair needs both products (F and dF/dx, three fields, product and
    bracket, two analysed fields); with per-block factors each (pair, category) needs its own
    (Gaunt: F, one field, one product, one analysed field; curl: F and dF/dx, two fields, the
    bracket, one analysed field)."""
    U, V = grid_dims(w.lmax)
    L, M = w.lmax + 1, 2 * w.lmax + 1
    pairs = (2 if w.flip1 else 1) * (2 if w.two_slot else 1)
    both_e, both_r = 4 * U * L * L + 6 * U * V * M + 4 * U * V, 4 * U * V * M + 4 * U * L * L
    g_e, g_r = 2 * U * L * L + 2 * U * V * M + U * V, 2 * U * V * M + 2 * U * L * L
    c_e, c_r = 4 * U * L * L + 4 * U * V * M + 3 * U * V, 2 * U * V * M + 2 * U * L * L
    if w.in_blocks == 1:
        return pairs * w.R * (E * both_e + N * both_r)
    return pairs * w.R * (E * (g_e + c_e) + N * (g_r + c_r))


def nbody_grid_flops(w) -> int:
    """Algorithmic flops of the nu-body grid stage on its grid (U, V) = the exact grid for
    nu operands, dense transforms, per (node, rank): value-only Legendre synthesis of nu
    operands (2 U L^2 each), one Fourier synthesis each (2 U V M), nu - 1 products per point,
    one Fourier analysis (2 U V M) and one Gauss-Legendre analysis (2 U L^2)."""
    deg = (w.nu + 1) * w.lmax
    U, V = max(1, (deg + 2) // 2), deg + 1
    L, M = w.lmax + 1, 2 * w.lmax + 1
    per = (w.nu + 1) * (2 * U * L * L + 2 * U * V * M) + (w.nu - 1) * U * V
    return w.n * w.R * per


def general_onsite_flops(w) -> int:
    """Algorithmic grid flops of the general on-site call: with shared factors every slot
    pair needs both products; with per-block factors every (slot pair, block) needs the
    product of its category only."""
    pairs = [(s1, s2) for s1 in ((0, 1) if w.flip1 else (0,))
             for s2 in ((0, 1) if w.two_slot else (0,))]
    if w.in_blocks == 1:
        return len(pairs) * onsite_grid_flops(w.lmax, w.R, w.n)
    return len(pairs) * (onsite_grid_flops(w.lmax, w.R, w.n, "gaunt")
                         + onsite_grid_flops(w.lmax, w.R, w.n, "curl"))


# ---------------------------------------------------------------- helpers

def to_dev(d, keys):
    import numpy as np
    import torch

    out = {}
    for k in keys:
        a = d.get(k)
        out[k] = None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return out


MP_KEYS = ("row_ptr", "col", "edge_unit", "edge_radial", "node_feat", "U_E", "U_I",
           "U_out_even", "U_out_odd")
MPF_KEYS = ("row_ptr", "col", "edge_feat", "node_feat", "U_E", "U_I", "U_out_even",
            "U_out_odd")
ONSITE_KEYS = ("A", "B", "U_A", "U_B", "U_out_even", "U_out_odd")


def load_traffic(workload: str):
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sha") != kernel_sha():
        return None                      # counters were taken on another kernel version
    return rec.get("bytes_per_launch")


def cpu_baseline(w, d, budget_s: float = 15.0, n_fixed: int = 0):
    """Time the fp64 oracle on a bounded sample of the same workload: the first n nodes or
    receivers, n chosen to take about budget_s (or n_fixed of them, the whole workload when
    n_fixed >= its size)."""
    import numpy as np

    import oracle

    cores = oracle.max_threads()
    if w.kind == "nbody":
        def run(n):
            return oracle.nbody(w.lmax, [x[:n] for x in d["X"]], d["U"], d["U_out"])
        unit_name = "nodes"
    elif w.kind == "mp_fields":
        def run(n):
            return oracle.message_pass_fields(w.lmax, *(d[k] for k in MPF_KEYS),
                                              receivers=np.arange(n), edge_flip=d["edge_flip"],
                                              node_flip=d["node_flip"])
        unit_name = "receivers"
    elif w.kind == "mp":
        def run(n):
            return oracle.message_pass(w.lmax, *(d[k] for k in MP_KEYS),
                                       receivers=np.arange(n), node_flip=d.get("node_flip"))
        unit_name = "receivers"
    else:
        def run(n):
            cut = lambda k: None if d.get(k) is None else d[k][:n]
            return oracle.onsite(w.lmax, d["A"][:n], d["B"][:n], d["U_A"], d["U_B"],
                                 d["U_out_even"], d["U_out_odd"], A_flip=cut("A_flip"),
                                 B_flip=cut("B_flip"))
        unit_name = "nodes"
    if n_fixed:
        n = min(w.n, n_fixed)
    else:
        probe = min(w.n, 16)
        t0 = time.perf_counter()
        run(probe)
        tp = time.perf_counter() - t0
        n = int(min(w.n, max(probe, probe * budget_s / max(tp, 1e-6))))
    t0 = time.perf_counter()
    run(n)
    t = time.perf_counter() - t0
    return {"value": n * w.C / t, "unit": "nodes*channels/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"first {n} {unit_name} (of {w.n}) of the same workload, fp64, "
                      f"{t:.1f} s on {cores} OpenMP threads"}


# ---------------------------------------------------------------- one workload

def set_order(plan, w, d, use_order: bool):
    """Message passing: compute the receiver order of the workload's graph on the host
    (cgtp_receiver_order, once per graph, before any timed step) and set it on the plan.
    Returns (kind, host ms) for the bench line."""
    import paper_2605_15073_amd as cg

    if w.kind not in ("mp", "mp_fields"):
        return None, None
    if not use_order:
        return "identity", None
    t0 = time.perf_counter()
    o = cg.receiver_order(d["row_ptr"], d["col"], d.get("edge_unit"))
    ms = 1e3 * (time.perf_counter() - t0)
    cg.set_receiver_order(plan, o)
    return ("hilbert" if d.get("edge_unit") is not None else "breadth_first"), ms


def bench_workload(w, steps: int, warmup: int, with_cpu: bool, d=None, quiet=False,
                   cpu_budget: float = 15.0, use_order: bool = True):
    import torch

    import paper_2605_15073_amd as cg

    if d is None:
        d = w.make()
    torch.empty(1, device="cuda")  # the GPU context exists before the plan is timed
    torch.cuda.synchronize()
    t_plan = time.perf_counter()
    if w.kind == "nbody":
        nt, nph = cg.nbody_grid(w.lmax, w.nu)
        plan = cg.plan_create(w.lmax, w.C, w.R, n_theta=nt, n_phi=nph,
                              flags=cg.CGTP_TIME_STAGES)
    else:
        plan = cg.plan_create(w.lmax, w.C, w.R, flags=cg.CGTP_TIME_STAGES)
    torch.cuda.synchronize()
    plan_ms = 1e3 * (time.perf_counter() - t_plan)  # tables built and uploaded, outside every step
    order_kind, order_ms = set_order(plan, w, d, use_order)
    if w.kind == "nbody":
        import numpy as np

        uniq = {}
        X = [uniq.setdefault(id(x), torch.from_numpy(np.ascontiguousarray(x)).cuda())
             for x in d["X"]]
        Ut = [torch.from_numpy(np.ascontiguousarray(u)).cuda() for u in d["U"]]
        Uo = torch.from_numpy(np.ascontiguousarray(d["U_out"])).cuda()
        E = 0
        op = cg.CGTP_OP_ONSITE_NBODY
        ws = torch.empty(cg.workspace_bytes_nbody(plan, w.n, w.nu), dtype=torch.uint8,
                         device="cuda")
        oe = torch.empty_like(X[0])
        oo = None

        def step():
            cg.onsite_nbody(plan, X, Ut, Uo, out=oe, workspace=ws)
    elif w.kind == "mp_fields":
        t = to_dev(d, MPF_KEYS + ("edge_flip", "node_flip"))
        E = int(d["n_edges"])
        op = cg.CGTP_OP_MESSAGE_PASS_FIELDS
        flips = (1 if w.flip1 else 0) | (2 if w.two_slot else 0)
        ws = torch.empty(cg.workspace_bytes_general(plan, op, w.n, E, flips, w.in_blocks,
                                                    w.out_blocks),
                         dtype=torch.uint8, device="cuda")
        oe = torch.empty_like(t["node_feat"])
        oo = torch.empty_like(t["node_feat"])

        def step():
            cg.message_pass_fields(plan, *(t[k] for k in MPF_KEYS), edge_flip=t["edge_flip"],
                                   node_flip=t["node_flip"], out_even=oe, out_odd=oo,
                                   workspace=ws)
    elif w.general and w.kind == "mp":
        t = to_dev(d, MP_KEYS + ("node_flip",))
        E = int(d["n_edges"])
        op = cg.CGTP_OP_MESSAGE_PASS_GENERAL
        ws = torch.empty(cg.workspace_bytes_general(plan, op, w.n, E, 2 if w.two_slot else 0,
                                                    w.in_blocks, w.out_blocks),
                         dtype=torch.uint8, device="cuda")
        oe = torch.empty_like(t["node_feat"])
        oo = torch.empty_like(t["node_feat"])

        def step():
            cg.message_pass_general(plan, *(t[k] for k in MP_KEYS), node_flip=t["node_flip"],
                                    out_even=oe, out_odd=oo, workspace=ws)
    elif w.general:
        t = to_dev(d, ONSITE_KEYS + ("A_flip", "B_flip"))
        E = 0
        op = cg.CGTP_OP_ONSITE_GENERAL
        flips = (1 if w.flip1 else 0) | (2 if w.two_slot else 0)
        ws = torch.empty(cg.workspace_bytes_general(plan, op, w.n, 0, flips, w.in_blocks,
                                                    w.out_blocks),
                         dtype=torch.uint8, device="cuda")
        oe = torch.empty_like(t["A"])
        oo = torch.empty_like(t["A"])

        def step():
            cg.onsite_general(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"],
                              t["U_out_odd"], A_flip=t["A_flip"], B_flip=t["B_flip"],
                              out_even=oe, out_odd=oo, workspace=ws)
    elif w.kind == "mp":
        two = w.two_slot
        t = to_dev(d, MP_KEYS + (("node_flip",) if two else ()))
        E = int(d["n_edges"])
        op = cg.CGTP_OP_MESSAGE_PASS_TWO_SLOT if two else cg.CGTP_OP_MESSAGE_PASS
        ws = torch.empty(cg.workspace_bytes(plan, op, w.n, E), dtype=torch.uint8, device="cuda")
        oe = torch.empty_like(t["node_feat"])
        oo = torch.empty_like(t["node_feat"])

        def step():
            cg.message_pass(plan, *(t[k] for k in MP_KEYS), out_even=oe, out_odd=oo, workspace=ws,
                            node_flip=t.get("node_flip"))
    else:
        t = to_dev(d, ONSITE_KEYS)
        if w.self_coupled:
            t["B"] = t["A"]
        E = 0
        op = cg.CGTP_OP_ONSITE
        ws = torch.empty(cg.workspace_bytes(plan, op, w.n), dtype=torch.uint8, device="cuda")
        oe = torch.empty_like(t["A"])
        oo = torch.empty_like(t["A"])

        def step():
            cg.onsite(plan, t["A"], t["B"], t["U_A"], t["U_B"], t["U_out_even"], t["U_out_odd"],
                      out_even=oe, out_odd=oo, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    cg.stage_times(plan, op)                     # drop the warm-up events
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    stages, calls = cg.stage_times(plan, op)
    assert calls == steps, (calls, steps)
    ms_step = 1e3 * wall / steps
    # per-step times for the median, from HIP events around single steps after the timed region
    cur = torch.cuda.current_stream()
    singles = []
    for _ in range(min(steps, 20)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        step()
        e1.record(cur)
        e1.synchronize()
        singles.append(e0.elapsed_time(e1))
    cg.stage_times(plan, op)                     # these steps do not enter the stage averages
    singles.sort()
    ms_median = (singles[len(singles) // 2] if len(singles) % 2
                 else 0.5 * (singles[len(singles) // 2 - 1] + singles[len(singles) // 2]))
    stage_avg = {k: v / steps for k, v in stages.items()}
    dom = max(stage_avg, key=stage_avg.get)
    U, V = grid_dims(w.lmax)
    rec = {
        "metric": "contracted CG products/sec (nodes*channels/s)",
        "value": w.n * w.C / (ms_step / 1e3),
        "unit": "nodes*channels/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": ms_median,
        "plan_create_ms": plan_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name,
                   "kind": "onsite_nbody" if w.kind == "nbody" else
                   "message_passing_two_fields" if w.kind == "mp_fields" else
                   ("message_passing" if w.kind == "mp" else "onsite")
                   + ("_general" if w.general else "_two_slot" if w.two_slot else ""),
                   "nodes": w.n, "edges": E, "lmax": w.lmax, "channels": w.C, "rank": w.R,
                   "grid": f"{U}x{V}", "seed": w.seed},
        "receiver_order": order_kind,
        "receiver_order_host_ms": order_ms,
        "stages_ms": {k: round(v, 4) for k, v in stage_avg.items()},
        "dominant_kernel": dom,
    }
    t_dom = stage_avg[dom] / 1e3
    if w.kind == "nbody":
        nt, nph = cg.nbody_grid(w.lmax, w.nu)
        rec["config"].update(nu=w.nu, grid=f"{nt}x{nph}", self_coupled=bool(w.self_coupled))
    if w.general:
        rec["config"].update(in_blocks=w.in_blocks, out_blocks=w.out_blocks,
                             flips=[bool(w.flip1), bool(w.two_slot)])
    if w.kind == "nbody" and dom == "contract_operands":
        # one per-degree channel contraction per power: 2 C R flops per (node, k)
        fl = w.nu * 2 * w.n * w.C * w.R * (w.lmax + 1) ** 2
        rec["roofline"] = {"bound": "mfma", "achieved": fl / t_dom / 1e12,
                           "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": fl / t_dom / 1e12 / FP32_PEAK_TFLOPS,
                           "traffic": load_traffic(w.name), "algorithmic_flops": fl}
    elif w.kind == "nbody" and dom == "grid_product_analysis":
        fl = nbody_grid_flops(w)
        rec["roofline"] = {"bound": "alu", "achieved": fl / t_dom / 1e12,
                           "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": fl / t_dom / 1e12 / FP32_PEAK_TFLOPS,
                           "traffic": load_traffic(w.name), "algorithmic_flops": fl}
    elif w.kind == "mp_fields" and dom == "receiver":
        fl = fields_receiver_flops(w, w.n, E)
        rec["roofline"] = {"bound": "alu", "achieved": fl / t_dom / 1e12,
                           "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": fl / t_dom / 1e12 / FP32_PEAK_TFLOPS,
                           "traffic": load_traffic(w.name), "algorithmic_flops": fl}
    elif w.kind == "mp" and dom == "receiver":
        if w.general:
            alg = general_receiver_bytes(w, w.n, E)
            live = live_blocks(False, w.two_slot)
            comp = compulsory_receiver_bytes(
                w.lmax, w.R, w.n, E, planes=len(live),
                rt_blocks=1 if w.in_blocks == 1 else len(live),
                t_fields=len(live) if w.out_blocks == 2 else 2)
        else:
            # with shared factors the receivers take the curl in the moved-derivative form and
            # read one plane (the sender values) per node slot
            per_slot = 1
            slots = 2 if w.two_slot else 1
            alg = receiver_bytes(w.lmax, w.R, w.n, E, slots, planes=per_slot * slots)
            comp = compulsory_receiver_bytes(w.lmax, w.R, w.n, E, per_slot * slots)
        traffic = load_traffic(w.name)
        # The receiver reads each sender's grid fields once per edge (about 52 times per
        # sender). Those gathers are served by the memory-side cache and the fabric into L2,
        # not by HBM: the fraction below is the effective gather (L2-fill) bandwidth against
        # the 8 TB/s HBM figure, and compulsory_hbm_* is what HBM itself must supply.
        rec["roofline"] = {"bound": "l2_fill", "achieved": alg / t_dom / 1e9,
                           "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": alg / t_dom / 1e9 / HBM_PEAK_GBS,
                           "traffic": traffic, "algorithmic_bytes": alg,
                           "compulsory_hbm_bytes": comp,
                           "compulsory_hbm_GBs": comp / t_dom / 1e9,
                           "compulsory_hbm_frac": comp / t_dom / 1e9 / HBM_PEAK_GBS}
        ceil = gather_ceiling(plan, w, t, E) if probe_ok(w) else None
        if ceil is not None:
            rec["roofline"]["gather_ceiling"] = ceil
            rec["roofline"]["frac_of_gather_ceiling"] = (alg / t_dom / 1e9) / ceil["GBs"]
    elif w.kind == "onsite" and dom == "grid_product_curl_analysis":
        fl = general_onsite_flops(w) if w.general else onsite_grid_flops(w.lmax, w.R, w.n)
        rec["roofline"] = {"bound": "alu", "achieved": fl / t_dom / 1e12,
                           "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": fl / t_dom / 1e12 / FP32_PEAK_TFLOPS,
                           "traffic": load_traffic(w.name), "algorithmic_flops": fl}
    else:
        rec["roofline"] = None
    rec["cpu_baseline"] = cpu_baseline(w, d, cpu_budget) if with_cpu else None
    plan.close()
    return rec


def probe_ok(w) -> bool:
    """The read-pattern probe replays the fp32 message-passing receiver in its values-only form
    on the plain sender layout (lmax <= 6, one node slot, shared factors)."""
    return w.kind == "mp" and not w.general and not w.two_slot and w.lmax <= 6


def gather_ceiling(plan, w, t, E, reps: int = 5):
    """Time cgtp_gather_probe (the receiver's sender-field loads alone, same blocks and order)
    on the workload's CSR over a zero-filled field buffer of the receiver's layout, with HIP
    events on the stream it runs on. Returns the bytes the receiver gathers per launch (the
    value plane: 4 R U V per edge), the mean launch time and their ratio."""
    import torch

    import paper_2605_15073_amd as cg

    U, V = grid_dims(w.lmax)
    uvs = (U * V + 31) // 32 * 32
    fields = torch.zeros(w.n * w.R * 3 * uvs, dtype=torch.float32, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    cur = torch.cuda.current_stream()
    for _ in range(2):
        cg.gather_probe(plan, t["row_ptr"], t["col"], fields, sink, stream=cur)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(cur)
    for _ in range(reps):
        cg.gather_probe(plan, t["row_ptr"], t["col"], fields, sink, stream=cur)
    e1.record(cur)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / reps
    gathered = 4 * E * w.R * U * V
    del fields
    return {"pattern": "per-edge sender value-plane loads of the receiver",
            "bytes": gathered, "ms": ms, "GBs": gathered / (ms / 1e3) / 1e9}


def sweep(path: str, steps: int, warmup: int):
    from paper_2605_15073_amd.inputs import Workload

    pts = []
    for lmax in range(2, 21, 2):
        pts.append(Workload(f"onsite_n4096_l{lmax}_c128", "onsite", 4096, lmax, 128, 128,
                            seed=3, per_degree=True))
        pts.append(Workload(f"onsite_n1000_l{lmax}_c64", "onsite", 1000, lmax, 64, 64, seed=3,
                            per_degree=True))
    for lmax in range(2, 21, 2):
        pts.append(Workload(f"mp_1000_l{lmax}_c64", "mp", 1000, lmax, 64, 64, seed=4))
        pts.append(Workload(f"mp_5k_l{lmax}_c64", "mp", 5000, lmax, 64, 64, seed=4))
    with open(path, "w") as f:
        for w in pts:
            # the oracle on a sample of about 2 s of host work next to every point
            rec = bench_workload(w, steps, warmup, with_cpu=True, cpu_budget=2.0)
            f.write(json.dumps(rec) + "\n")
            f.flush()
            print(f"sweep {w.name}: {rec['ms_per_step']:.3f} ms/step "
                  f"dominant {rec['dominant_kernel']}", flush=True)


def cpu_baselines(path: str):
    """The fp64 oracle on the host cores for the five benchmark workloads: the two smaller
    on-site ones and the lmax-12 on-site one whole, message passing at lmax 20 on its first
    64 receivers and at lmax 6 on a sample of about 15 s. One JSON line per workload."""
    from paper_2605_15073_amd.inputs import WORKLOADS

    plan = [("onsite_n64_l2_c8", 10 ** 9, 0), ("onsite_ace_n2048_l4_c64", 10 ** 9, 0),
            ("mp_10k_l6_c128", 0, 15.0), ("onsite_n4096_l12_c128", 10 ** 9, 0),
            ("mp_5k_l20_c64", 64, 0)]
    with open(path, "w") as f:
        for name, n_fixed, budget in plan:
            w = WORKLOADS[name]
            d = w.make()
            if w.self_coupled:
                d = dict(d, B=d["A"])
            rec = {"workload": name, **cpu_baseline(w, d, budget or 15.0, n_fixed)}
            f.write(json.dumps(rec) + "\n")
            f.flush()
            print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mp_10k_l6_c128")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep-out", default=None)
    ap.add_argument("--cpu-baselines", default=None,
                    help="time only the fp64 oracle on the five benchmark workloads (whole, "
                         "or on a stated sample) and write one JSON line each to this file")
    ap.add_argument("--gather-ceiling", action="store_true",
                    help="run only the receiver's read-pattern probe (cgtp_gather_probe) on the "
                         "workload's neighbour list, 5 launches after 2 warm-up launches")
    ap.add_argument("--no-receiver-order", action="store_true",
                    help="message passing: run the receivers in node order instead of the "
                         "locality order of cgtp_receiver_order")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="run only a plain device-to-device copy of this many bytes (3 times), "
                         "the calibration kernel for the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the method is "
                                   "measured on one MI355X (--gpus 1)"}), flush=True)
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(1)
    from paper_2605_15073_amd.inputs import WORKLOADS

    if args.cpu_baselines:
        cpu_baselines(args.cpu_baselines)
        return
    if args.copy_bytes:
        n = args.copy_bytes // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4, "copies": 3}), flush=True)
        return
    if args.gather_ceiling:
        import paper_2605_15073_amd as cg

        w = WORKLOADS[args.workload]
        if not probe_ok(w):
            print(json.dumps({"error": f"no read-pattern probe for {w.name}"}), flush=True)
            sys.exit(2)
        d = w.make()
        t = to_dev(d, ("row_ptr", "col"))
        plan = cg.plan_create(w.lmax, w.C, w.R)
        order_kind, _ = set_order(plan, w, d, not args.no_receiver_order)
        ceil = gather_ceiling(plan, w, t, int(d["n_edges"]))
        plan.close()
        print(json.dumps({"workload": w.name, "edges": int(d["n_edges"]),
                          "receiver_order": order_kind, "gather_ceiling": ceil}), flush=True)
        return
    if args.sweep_out:
        sweep(args.sweep_out, max(3, args.steps // 4), args.warmup)
        return
    w = WORKLOADS[args.workload]
    rec = bench_workload(w, args.steps, args.warmup, with_cpu=not args.no_cpu_baseline,
                         use_order=not args.no_receiver_order)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
