"""Python binding of libcgtp (contracted Clebsch-Gordan products on MI355X).

Thin ctypes marshalling over the C ABI declared in ``include/cgtp.h``: every
step of the computation runs in the HIP kernels of ``libcgtp.so``. Tensors are
torch device tensors (torch provides device memory and streams only). If the
shared library is missing this module raises on first use; there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcgtp.so")

CGTP_OK = 0
CGTP_ERR_ARG = -1
CGTP_ERR_WORKSPACE = -2
CGTP_ERR_CSR = -3
CGTP_ERR_HIP = -4
CGTP_ERR_UNSUPPORTED = -5
CGTP_F32 = 0
CGTP_F64 = 1
CGTP_VALIDATE_CSR = 1
CGTP_EDGE_SEPARATED = 2
CGTP_TIME_STAGES = 4
CGTP_OP_ONSITE = 0
CGTP_OP_MESSAGE_PASS = 1
CGTP_OP_MESSAGE_PASS_TWO_SLOT = 2
CGTP_OP_ONSITE_GENERAL = 3
CGTP_OP_MESSAGE_PASS_GENERAL = 4
CGTP_OP_MESSAGE_PASS_FIELDS = 5
CGTP_OP_ONSITE_NBODY = 6
CGTP_MAX_NU = 8
CGTP_MAX_LMAX = 24

EXPORTED = ("cgtp_plan_create", "cgtp_plan_grid", "cgtp_workspace_bytes", "cgtp_onsite",
            "cgtp_message_pass", "cgtp_message_pass_two_slot", "cgtp_workspace_bytes_general",
            "cgtp_onsite_general", "cgtp_message_pass_general", "cgtp_message_pass_fields",
            "cgtp_workspace_bytes_nbody", "cgtp_onsite_nbody", "cgtp_stage_times",
            "cgtp_destroy", "cgtp_status_string", "cgtp_last_error", "cgtp_host_tables",
            "cgtp_onsite_noalloc", "cgtp_gather_probe", "cgtp_receiver_order",
            "cgtp_plan_set_receiver_order")
CGTP_NOALLOC_SCRATCH_BYTES = 64 << 20
ONSITE_STAGES = ("contract_operands", "grid_product_curl_analysis", "project")
ONSITE_GENERAL_STAGES = ("contract_a", "contract_b", "grid_product_curl_analysis",
                         "project_even", "project_odd")
MP_STAGES = ("contract_node", "sender_fields", "contract_edge_radial", "receiver", "analysis",
             "project_even", "project_odd")
NBODY_STAGES = ("contract_operands", "grid_product_analysis", "project")


class CgtpError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class _Desc(ctypes.Structure):
    _fields_ = [("lmax", ctypes.c_int), ("channels", ctypes.c_int), ("rank", ctypes.c_int),
                ("n_theta", ctypes.c_int), ("n_phi", ctypes.c_int), ("dtype", ctypes.c_int),
                ("flags", ctypes.c_uint)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libcgtp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libcgtp.so not found at {path}: build it with "
                           "`python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    lib.cgtp_plan_create.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(vp)]
    lib.cgtp_plan_grid.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.cgtp_workspace_bytes.argtypes = [vp, i32, i64, i64, ctypes.POINTER(sz)]
    lib.cgtp_onsite.argtypes = [vp, i64] + [vp] * 8 + [vp, sz, vp]
    lib.cgtp_onsite_noalloc.argtypes = [vp, i64] + [vp] * 8 + [vp]
    lib.cgtp_gather_probe.argtypes = [vp, i64, i64, vp, vp, vp, sz, vp, vp]
    lib.cgtp_message_pass.argtypes = [vp, i64, i64] + [vp] * 11 + [vp, sz, vp]
    lib.cgtp_message_pass_two_slot.argtypes = [vp, i64, i64] + [vp] * 12 + [vp, sz, vp]
    lib.cgtp_workspace_bytes_general.argtypes = [vp, i32, i64, i64, i32, i32, i32,
                                                 ctypes.POINTER(sz)]
    lib.cgtp_onsite_general.argtypes = ([vp, i64] + [vp] * 4 + [i32, vp, vp, i32] + [vp] * 4
                                        + [vp, sz, vp])
    lib.cgtp_message_pass_general.argtypes = ([vp, i64, i64] + [vp] * 6 + [i32, vp, vp, i32]
                                              + [vp] * 4 + [vp, sz, vp])
    lib.cgtp_message_pass_fields.argtypes = lib.cgtp_message_pass_general.argtypes
    lib.cgtp_workspace_bytes_nbody.argtypes = [vp, i64, i32, ctypes.POINTER(sz)]
    lib.cgtp_onsite_nbody.argtypes = [vp, i64, i32, vp, vp, vp, vp, vp, sz, vp]
    lib.cgtp_stage_times.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double), i32,
                                     ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.cgtp_destroy.argtypes = [vp]
    lib.cgtp_status_string.argtypes = [i32]
    lib.cgtp_status_string.restype = ctypes.c_char_p
    lib.cgtp_last_error.argtypes = []
    lib.cgtp_last_error.restype = ctypes.c_char_p
    lib.cgtp_host_tables.argtypes = [i32, i32, i32] + [vp] * 5
    lib.cgtp_receiver_order.argtypes = [i64, i64, vp, vp, vp, vp]
    lib.cgtp_plan_set_receiver_order.argtypes = [vp, i64, vp]
    for name in ("cgtp_plan_create", "cgtp_plan_grid", "cgtp_workspace_bytes", "cgtp_onsite",
                 "cgtp_onsite_noalloc", "cgtp_gather_probe",
                 "cgtp_message_pass", "cgtp_message_pass_two_slot", "cgtp_stage_times",
                 "cgtp_destroy", "cgtp_host_tables", "cgtp_receiver_order",
                 "cgtp_plan_set_receiver_order"):
        getattr(lib, name).restype = i32
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != CGTP_OK:
        lib = load_library()
        detail = lib.cgtp_last_error().decode() or lib.cgtp_status_string(status).decode()
        raise CgtpError(status, where, detail)


class Plan:
    """Owns a cgtp_plan handle (grid tables on the current device)."""

    def __init__(self, lmax: int, channels: int, rank: int, n_theta: int = 0, n_phi: int = 0,
                 dtype: str = "f32", flags: int = 0):
        lib = load_library()
        self.lmax, self.channels, self.rank = lmax, channels, rank
        self.dtype = dtype
        desc = _Desc(lmax, channels, rank, n_theta, n_phi,
                     CGTP_F64 if dtype == "f64" else CGTP_F32, flags)
        h = ctypes.c_void_p()
        _check(lib.cgtp_plan_create(ctypes.byref(desc), ctypes.byref(h)), "cgtp_plan_create")
        self.handle = h
        u, v = ctypes.c_int(), ctypes.c_int()
        _check(lib.cgtp_plan_grid(h, ctypes.byref(u), ctypes.byref(v)), "cgtp_plan_grid")
        self.n_theta, self.n_phi = u.value, v.value

    def close(self):
        if getattr(self, "handle", None):
            _check(load_library().cgtp_destroy(self.handle), "cgtp_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def plan_create(lmax: int, channels: int, rank: int, n_theta: int = 0, n_phi: int = 0,
                dtype: str = "f32", flags: int = 0) -> Plan:
    return Plan(lmax, channels, rank, n_theta, n_phi, dtype, flags)


def destroy(plan: Plan) -> None:
    plan.close()


def workspace_bytes(plan: Plan, op: int, n_nodes: int, n_edges: int = 0) -> int:
    out = ctypes.c_size_t()
    _check(load_library().cgtp_workspace_bytes(plan.handle, op, n_nodes, n_edges,
                                               ctypes.byref(out)), "cgtp_workspace_bytes")
    return out.value


def stage_times(plan: Plan, op: int):
    """cgtp_stage_times: ({stage name: summed ms}, number of calls) since the last query."""
    ms = (ctypes.c_double * 8)()
    ns, nc = ctypes.c_int(), ctypes.c_int()
    _check(load_library().cgtp_stage_times(plan.handle, op, ms, 8, ctypes.byref(ns),
                                           ctypes.byref(nc)), "cgtp_stage_times")
    names = (NBODY_STAGES if op == CGTP_OP_ONSITE_NBODY else
             ONSITE_STAGES if op == CGTP_OP_ONSITE else
             ONSITE_GENERAL_STAGES if op == CGTP_OP_ONSITE_GENERAL else MP_STAGES)
    return {names[i]: ms[i] for i in range(ns.value)}, nc.value


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _want(plan: Plan, name: str, t, shape, dtype=None):
    torch = _torch()
    dt = dtype or (torch.float64 if plan.dtype == "f64" else torch.float32)
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda or t.dtype != dt or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected contiguous {dt} device tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def onsite(plan: Plan, A, B, U_A, U_B, U_out_even, U_out_odd, out_even=None, out_odd=None,
           workspace=None, stream=None):
    """cgtp_onsite. A, B [N, C, K]; U_* [L, C, R]; outputs [N, C, K] (allocated if not given
    and not explicitly skipped with out_even=False / out_odd=False)."""
    torch = _torch()
    N, C, K = A.shape
    L = plan.lmax + 1
    _want(plan, "A", A, (N, plan.channels, L * L))
    _want(plan, "B", B, A.shape)
    for nm, U in (("U_A", U_A), ("U_B", U_B)):
        _want(plan, nm, U, (L, plan.channels, plan.rank))
    outs = []
    for nm, o, U in (("out_even", out_even, U_out_even), ("out_odd", out_odd, U_out_odd)):
        if o is False:
            outs.append(None)
            continue
        _want(plan, nm.replace("out", "U_out"), U, (L, plan.channels, plan.rank))
        if o is None:
            o = torch.empty_like(A)
        _want(plan, nm, o, A.shape)
        outs.append(o)
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(load_library().cgtp_onsite(plan.handle, N, _ptr(A), _ptr(B), _ptr(U_A), _ptr(U_B),
                                      _ptr(U_out_even), _ptr(U_out_odd), _ptr(outs[0]),
                                      _ptr(outs[1]), ws_ptr, ws_len, _stream_handle(stream)),
           "cgtp_onsite")
    return outs[0], outs[1]


def onsite_noalloc(plan: Plan, A, B, U_A, U_B, U_out_even, U_out_odd, out_even, out_odd,
                   stream=None):
    """cgtp_onsite_noalloc: cgtp_onsite on the library's fixed device scratch
    (CGTP_NOALLOC_SCRATCH_BYTES per GPU). The caller passes the outputs (either may be
    False to skip that slot); nothing is allocated, here or in the library."""
    N, C, K = A.shape
    L = plan.lmax + 1
    _want(plan, "A", A, (N, plan.channels, L * L))
    _want(plan, "B", B, A.shape)
    for nm, U in (("U_A", U_A), ("U_B", U_B)):
        _want(plan, nm, U, (L, plan.channels, plan.rank))
    outs = []
    for nm, o, U in (("out_even", out_even, U_out_even), ("out_odd", out_odd, U_out_odd)):
        if o is False:
            outs.append(None)
            continue
        _want(plan, nm.replace("out", "U_out"), U, (L, plan.channels, plan.rank))
        _want(plan, nm, o, A.shape)
        outs.append(o)
    _check(load_library().cgtp_onsite_noalloc(plan.handle, N, _ptr(A), _ptr(B), _ptr(U_A),
                                              _ptr(U_B), _ptr(U_out_even), _ptr(U_out_odd),
                                              _ptr(outs[0]), _ptr(outs[1]),
                                              _stream_handle(stream)),
           "cgtp_onsite_noalloc")
    return outs[0], outs[1]


def _host(a, dtype):
    """A contiguous numpy array of dtype on the host (from numpy or a torch tensor)."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=dtype)


def receiver_order(row_ptr, col, edge_vec=None):
    """cgtp_receiver_order on the host: a locality-preserving permutation of the receivers
    of the CSR (row_ptr [N+1], col [E]), from the edge vectors [E, 3] if given, else the
    breadth-first order. Returns an int32 numpy array [N]."""
    rp = _host(row_ptr, np.int32)
    cl = _host(col, np.int32)
    N, E = rp.shape[0] - 1, cl.shape[0]
    ev = None if edge_vec is None else _host(edge_vec, np.float32)
    if ev is not None and ev.shape != (E, 3):
        raise ValueError(f"edge_vec: expected shape ({E}, 3), got {ev.shape}")
    out = np.empty(N, dtype=np.int32)
    vp = ctypes.c_void_p
    _check(load_library().cgtp_receiver_order(
        N, E, vp(rp.ctypes.data), vp(cl.ctypes.data),
        None if ev is None else vp(ev.ctypes.data), vp(out.ctypes.data)), "cgtp_receiver_order")
    return out


def set_receiver_order(plan: Plan, order=None) -> None:
    """cgtp_plan_set_receiver_order: run the plan's message-passing receivers in this order
    (a permutation of the N nodes; None restores the identity)."""
    lib = load_library()
    if order is None:
        _check(lib.cgtp_plan_set_receiver_order(plan.handle, 0, None),
               "cgtp_plan_set_receiver_order")
        return
    o = _host(order, np.int32)
    _check(lib.cgtp_plan_set_receiver_order(plan.handle, o.shape[0], ctypes.c_void_p(o.ctypes.data)),
           "cgtp_plan_set_receiver_order")


def gather_probe(plan: Plan, row_ptr, col, fields, sink, stream=None):
    """cgtp_gather_probe: replay the receiver's sender-field loads over fields (a device
    buffer of at least N R 3 UVs floats) for the CSR (row_ptr, col); sink: a device float."""
    torch = _torch()
    N = row_ptr.shape[0] - 1
    E = col.shape[0]
    _want(plan, "row_ptr", row_ptr, (N + 1,), torch.int32)
    _want(plan, "col", col, (E,), torch.int32)
    if not fields.is_cuda or not sink.is_cuda:
        raise ValueError("fields and sink must be device tensors")
    _check(load_library().cgtp_gather_probe(plan.handle, N, E, _ptr(row_ptr), _ptr(col),
                                            _ptr(fields), fields.numel() * fields.element_size(),
                                            _ptr(sink), _stream_handle(stream)),
           "cgtp_gather_probe")


def message_pass(plan: Plan, row_ptr, col, edge_unit, edge_radial, node_feat, U_E, U_I,
                 U_out_even, U_out_odd, out_even=None, out_odd=None, workspace=None,
                 stream=None, node_flip=None):
    """cgtp_message_pass (or cgtp_message_pass_two_slot when node_flip is given).
    row_ptr [N+1], col [E] int32; edge_unit [E, 3]; edge_radial [E, C, L];
    node_feat [N, C, K] (natural-parity slot); node_flip [N, C, K] (parity-flipped slot);
    U_* [L, C, R]; outputs [N, C, K]."""
    torch = _torch()
    N = node_feat.shape[0]
    E = col.shape[0]
    L = plan.lmax + 1
    _want(plan, "row_ptr", row_ptr, (N + 1,), torch.int32)
    _want(plan, "col", col, (E,), torch.int32)
    _want(plan, "edge_unit", edge_unit, (E, 3))
    _want(plan, "edge_radial", edge_radial, (E, plan.channels, L))
    _want(plan, "node_feat", node_feat, (N, plan.channels, L * L))
    if node_flip is not None:
        _want(plan, "node_flip", node_flip, (N, plan.channels, L * L))
    for nm, U in (("U_E", U_E), ("U_I", U_I)):
        _want(plan, nm, U, (L, plan.channels, plan.rank))
    outs = []
    for nm, o, U in (("out_even", out_even, U_out_even), ("out_odd", out_odd, U_out_odd)):
        if o is False:
            outs.append(None)
            continue
        _want(plan, nm.replace("out", "U_out"), U, (L, plan.channels, plan.rank))
        if o is None:
            o = torch.empty_like(node_feat)
        _want(plan, nm, o, node_feat.shape)
        outs.append(o)
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    lib = load_library()
    head = (plan.handle, N, E, _ptr(row_ptr), _ptr(col), _ptr(edge_unit), _ptr(edge_radial),
            _ptr(node_feat))
    tail = (_ptr(U_E), _ptr(U_I), _ptr(U_out_even), _ptr(U_out_odd), _ptr(outs[0]),
            _ptr(outs[1]), ws_ptr, ws_len, _stream_handle(stream))
    if node_flip is None:
        _check(lib.cgtp_message_pass(*head, *tail), "cgtp_message_pass")
    else:
        _check(lib.cgtp_message_pass_two_slot(*head, _ptr(node_flip), *tail),
               "cgtp_message_pass_two_slot")
    return outs[0], outs[1]


def workspace_bytes_general(plan: Plan, op: int, n_nodes: int, n_edges: int = 0, flips: int = 0,
                            in_blocks: int = 1, out_blocks: int = 1) -> int:
    """cgtp_workspace_bytes_general (flips: bit 0 first on-site operand, bit 1 second operand
    or node feature)."""
    out = ctypes.c_size_t()
    _check(load_library().cgtp_workspace_bytes_general(plan.handle, op, n_nodes, n_edges, flips,
                                                       in_blocks, out_blocks, ctypes.byref(out)),
           "cgtp_workspace_bytes_general")
    return out.value


def _blocks(plan: Plan, name: str, U, allowed):
    """Number of factor blocks of a stacked factor tensor: [L, C, R] is 1, [n, L, C, R] is n."""
    L = plan.lmax + 1
    base = (L, plan.channels, plan.rank)
    n = 1 if U is not None and U.dim() == 3 else (U.shape[0] if U is not None else 0)
    if n not in allowed:
        raise ValueError(f"{name}: expected {allowed} stacked blocks of {base}")
    _want(plan, name, U, base if n == 1 else (n,) + base)
    return n


def _outputs(plan: Plan, like, out_even, out_odd, U_out_even, U_out_odd):
    torch = _torch()
    outs, nout = [], set()
    for nm, o, U in (("out_even", out_even, U_out_even), ("out_odd", out_odd, U_out_odd)):
        if o is False:
            outs.append(None)
            continue
        nout.add(_blocks(plan, nm.replace("out", "U_out"), U, (1, 2)))
        if o is None:
            o = torch.empty_like(like)
        _want(plan, nm, o, like.shape)
        outs.append(o)
    if len(nout) != 1:
        raise ValueError("U_out_even and U_out_odd must have the same number of blocks")
    return outs, nout.pop()


def onsite_general(plan: Plan, A, B, U_A, U_B, U_out_even, U_out_odd, A_flip=None, B_flip=None,
                   out_even=None, out_odd=None, workspace=None, stream=None):
    """cgtp_onsite_general. A, B (and the flipped slots A_flip, B_flip) [N, C, K].
    U_A, U_B: [L, C, R], or stacked [2, L, C, R] (Gaunt, curl) or [4, L, C, R] (block
    2 * category + sector). U_out_even, U_out_odd: [L, C, R] or [2, L, C, R] (Gaunt, curl)."""
    N = A.shape[0]
    L = plan.lmax + 1
    _want(plan, "A", A, (N, plan.channels, L * L))
    for nm, X in (("B", B), ("A_flip", A_flip), ("B_flip", B_flip)):
        if X is not None or nm == "B":
            _want(plan, nm, X, A.shape)
    nin = _blocks(plan, "U_A", U_A, (1, 2, 4))
    if _blocks(plan, "U_B", U_B, (1, 2, 4)) != nin:
        raise ValueError("U_A and U_B must have the same number of blocks")
    outs, nout = _outputs(plan, A, out_even, out_odd, U_out_even, U_out_odd)
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(load_library().cgtp_onsite_general(
        plan.handle, N, _ptr(A), _ptr(A_flip), _ptr(B), _ptr(B_flip), nin, _ptr(U_A), _ptr(U_B),
        nout, _ptr(U_out_even), _ptr(U_out_odd), _ptr(outs[0]), _ptr(outs[1]), ws_ptr, ws_len,
        _stream_handle(stream)), "cgtp_onsite_general")
    return outs[0], outs[1]


def message_pass_general(plan: Plan, row_ptr, col, edge_unit, edge_radial, node_feat, U_E, U_I,
                         U_out_even, U_out_odd, node_flip=None, out_even=None, out_odd=None,
                         workspace=None, stream=None):
    """cgtp_message_pass_general. Arguments as in message_pass; U_E, U_I and U_out_* stacked
    as in onsite_general."""
    torch = _torch()
    N = node_feat.shape[0]
    E = col.shape[0]
    L = plan.lmax + 1
    _want(plan, "row_ptr", row_ptr, (N + 1,), torch.int32)
    _want(plan, "col", col, (E,), torch.int32)
    _want(plan, "edge_unit", edge_unit, (E, 3))
    _want(plan, "edge_radial", edge_radial, (E, plan.channels, L))
    _want(plan, "node_feat", node_feat, (N, plan.channels, L * L))
    if node_flip is not None:
        _want(plan, "node_flip", node_flip, node_feat.shape)
    nin = _blocks(plan, "U_E", U_E, (1, 2, 4))
    if _blocks(plan, "U_I", U_I, (1, 2, 4)) != nin:
        raise ValueError("U_E and U_I must have the same number of blocks")
    outs, nout = _outputs(plan, node_feat, out_even, out_odd, U_out_even, U_out_odd)
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(load_library().cgtp_message_pass_general(
        plan.handle, N, E, _ptr(row_ptr), _ptr(col), _ptr(edge_unit), _ptr(edge_radial),
        _ptr(node_feat), _ptr(node_flip), nin, _ptr(U_E), _ptr(U_I), nout, _ptr(U_out_even),
        _ptr(U_out_odd), _ptr(outs[0]), _ptr(outs[1]), ws_ptr, ws_len, _stream_handle(stream)),
        "cgtp_message_pass_general")
    return outs[0], outs[1]


def message_pass_fields(plan: Plan, row_ptr, col, edge_feat, node_feat, U_E, U_I, U_out_even,
                        U_out_odd, edge_flip=None, node_flip=None, out_even=None, out_odd=None,
                        workspace=None, stream=None):
    """cgtp_message_pass_fields (two parity-bearing fields). row_ptr [N+1], col [E] int32;
    edge_feat, edge_flip [E, C, K]; node_feat, node_flip [N, C, K]; factors stacked as in
    onsite_general."""
    torch = _torch()
    N = node_feat.shape[0]
    E = col.shape[0]
    L = plan.lmax + 1
    _want(plan, "row_ptr", row_ptr, (N + 1,), torch.int32)
    _want(plan, "col", col, (E,), torch.int32)
    _want(plan, "edge_feat", edge_feat, (E, plan.channels, L * L))
    if edge_flip is not None:
        _want(plan, "edge_flip", edge_flip, edge_feat.shape)
    _want(plan, "node_feat", node_feat, (N, plan.channels, L * L))
    if node_flip is not None:
        _want(plan, "node_flip", node_flip, node_feat.shape)
    nin = _blocks(plan, "U_E", U_E, (1, 2, 4))
    if _blocks(plan, "U_I", U_I, (1, 2, 4)) != nin:
        raise ValueError("U_E and U_I must have the same number of blocks")
    outs, nout = _outputs(plan, node_feat, out_even, out_odd, U_out_even, U_out_odd)
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(load_library().cgtp_message_pass_fields(
        plan.handle, N, E, _ptr(row_ptr), _ptr(col), _ptr(edge_feat), _ptr(edge_flip),
        _ptr(node_feat), _ptr(node_flip), nin, _ptr(U_E), _ptr(U_I), nout, _ptr(U_out_even),
        _ptr(U_out_odd), _ptr(outs[0]), _ptr(outs[1]), ws_ptr, ws_len, _stream_handle(stream)),
        "cgtp_message_pass_fields")
    return outs[0], outs[1]


def nbody_grid(lmax: int, nu: int):
    """Smallest (n_theta, n_phi) on which cgtp_onsite_nbody is exact for nu operands."""
    deg = (nu + 1) * lmax
    return max(1, (deg + 2) // 2), deg + 1


def workspace_bytes_nbody(plan: Plan, n_nodes: int, nu: int) -> int:
    out = ctypes.c_size_t()
    _check(load_library().cgtp_workspace_bytes_nbody(plan.handle, n_nodes, nu,
                                                     ctypes.byref(out)),
           "cgtp_workspace_bytes_nbody")
    return out.value


def onsite_nbody(plan: Plan, X, U, U_out, out=None, workspace=None, stream=None):
    """cgtp_onsite_nbody. X: sequence of nu device tensors [N, C, K]; U: nu factor tensors
    [L, C, R]; U_out [L, C, R]. The plan's grid must be at least nbody_grid(lmax, nu)."""
    torch = _torch()
    nu = len(X)
    if nu != len(U) or nu < 1:
        raise ValueError("X and U must hold the same number (>= 1) of operands")
    L = plan.lmax + 1
    N = X[0].shape[0]
    for t in range(nu):
        _want(plan, f"X[{t}]", X[t], (N, plan.channels, L * L))
        _want(plan, f"U[{t}]", U[t], (L, plan.channels, plan.rank))
    _want(plan, "U_out", U_out, (L, plan.channels, plan.rank))
    if out is None:
        out = torch.empty_like(X[0])
    _want(plan, "out", out, X[0].shape)
    xs = (ctypes.c_void_p * nu)(*[x.data_ptr() for x in X])
    us = (ctypes.c_void_p * nu)(*[u.data_ptr() for u in U])
    ws_ptr, ws_len = None, 0
    if workspace is not None:
        ws_ptr, ws_len = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(load_library().cgtp_onsite_nbody(plan.handle, N, nu, ctypes.cast(xs, ctypes.c_void_p),
                                            ctypes.cast(us, ctypes.c_void_p), _ptr(U_out),
                                            _ptr(out), ws_ptr, ws_len, _stream_handle(stream)),
           "cgtp_onsite_nbody")
    return out


def host_tables(lmax: int, n_theta: int = 0, n_phi: int = 0):
    """fp64 grid tables (x, w, p, dp, q) as the plan builds them; host only."""
    import numpy as np

    lib = load_library()
    u, v = n_theta, n_phi
    if u == 0:
        u = (3 * lmax + 3) // 2
    if v == 0:
        v = 3 * lmax + 1
    P = (lmax + 1) * (lmax + 2) // 2
    x, w = np.zeros(u), np.zeros(u)
    p, dp = np.zeros((u, P)), np.zeros((u, P))
    q = np.zeros((v, 2 * lmax + 1))
    args = [ctypes.c_void_p(a.ctypes.data) for a in (x, w, p, dp, q)]
    _check(lib.cgtp_host_tables(lmax, n_theta, n_phi, *args), "cgtp_host_tables")
    return x, w, p, dp, q
