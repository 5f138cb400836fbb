"""Python binding of libsla (ctypes).  Argument marshalling only: every step of
the SLA path runs in the HIP library; torch supplies device memory and the
current stream.  There is no fallback: if the library is missing or no GPU is
present the calls raise.

Functions mirror the C ABI in include/sla.h:
    plan_bytes(n, num_windows)
    plan_layout(n, num_windows)
    build_segments(ids | offsets, num_windows, chunk_rows=0) -> Plan
    forward(plan, q, k, v, out=None, feature_map=None, eps=None) -> o
    backward(plan, q, k, v, dout, dq=None, dk=None, dv=None, feature_map=None, eps=None)
        -> (dq, dk, dv)
        (feature_map "elu1" | "relu" and eps >= 0 select sla_forward_ex /
        sla_backward_ex; leaving both None calls sla_forward / sla_backward)
    forward_projected(plan, x, w_qkv, w_o, heads, b_qkv=None, b_o=None, o=None, y=None,
                      feature_map="elu1", eps=0.0) -> (o, y)
    cwi_map_bytes(gx, gy, gz)
    cwi_build_map(coords, grid, map=None) -> (map, conflicts)
    cwi_forward(map, grid, coords, x, w_x, w_y, w_3, order=None, y=None) -> y
    cwi_backward(map, grid, coords, x, w_x, w_y, w_3, dy, order=None) -> (dx, dw_x, dw_y, dw_3)
    scatter_workspace_bytes(n, heads, head_dim)
    forward_scatter(plan, q, k, v, out=None, workspace=None) -> o   (naive comparator)
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsla.so")

SLA_OK, SLA_E_ARG, SLA_E_UNSUPPORTED, SLA_E_WORKSPACE, SLA_E_HIP = range(5)

FEATURE_MAPS = {"elu1": 0, "relu": 1}   # sla_feature_map_t

EXPORTED = (
    "sla_abi_version",
    "sla_status_string",
    "sla_max_windows",
    "sla_default_chunk_rows",
    "sla_plan_bytes",
    "sla_plan_layout",
    "sla_build_segments",
    "sla_forward",
    "sla_backward",
    "sla_forward_ex",
    "sla_backward_ex",
    "sla_forward_projected",
    "sla_backward_projected_workspace_bytes",
    "sla_backward_projected",
    "sla_cwi_map_bytes",
    "sla_cwi_build_map",
    "sla_cwi_forward",
    "sla_cwi_backward_workspace_bytes",
    "sla_cwi_backward",
    "sla_scatter_workspace_bytes",
    "sla_forward_scatter",
    "sla_forward_xca",
    "sla_xca_backward_workspace_bytes",
    "sla_backward_xca",
    "sla_backward_xca_noalloc",
)


class SlaError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)}")


class PlanLayout(ctypes.Structure):
    _fields_ = [
        ("header", ctypes.c_size_t),
        ("perm", ctypes.c_size_t),
        ("offsets", ctypes.c_size_t),
        ("chunks", ctypes.c_size_t),
        ("longs", ctypes.c_size_t),
        ("total", ctypes.c_size_t),
        ("max_chunks", ctypes.c_int32),
        ("max_long", ctypes.c_int32),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsla.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libsla.so not built at {LIB_PATH}; run python -m paper_2401_00912_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    i32, i64, sz, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    L.sla_abi_version.restype = i32
    L.sla_abi_version.argtypes = []
    L.sla_status_string.restype = ctypes.c_char_p
    L.sla_status_string.argtypes = [ctypes.c_int]
    L.sla_max_windows.restype = i32
    L.sla_max_windows.argtypes = []
    L.sla_default_chunk_rows.restype = i32
    L.sla_default_chunk_rows.argtypes = []
    L.sla_plan_bytes.restype = sz
    L.sla_plan_bytes.argtypes = [i64, i32]
    L.sla_plan_layout.restype = ctypes.c_int
    L.sla_plan_layout.argtypes = [i64, i32, ctypes.POINTER(PlanLayout)]
    L.sla_build_segments.restype = ctypes.c_int
    L.sla_build_segments.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, sz, vp]
    L.sla_forward.restype = ctypes.c_int
    L.sla_forward.argtypes = [vp, sz, i64, i32, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp]
    L.sla_backward.restype = ctypes.c_int
    L.sla_backward.argtypes = [vp, sz, i64, i32, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    f32, en = ctypes.c_float, ctypes.c_int
    L.sla_forward_ex.restype = ctypes.c_int
    L.sla_forward_ex.argtypes = [vp, sz, i64, i32, en, i32, i32, en, f32, vp, vp, vp, vp, vp]
    L.sla_backward_ex.restype = ctypes.c_int
    L.sla_backward_ex.argtypes = [vp, sz, i64, i32, en, i32, i32, en, f32, vp, vp, vp, vp, vp, vp, vp, vp]
    L.sla_forward_projected.restype = ctypes.c_int
    L.sla_forward_projected.argtypes = [vp, sz, i64, i32, en, i32, i32, en, f32] + [vp] * 9
    L.sla_backward_projected_workspace_bytes.restype = sz
    L.sla_backward_projected_workspace_bytes.argtypes = [i64, i32, i32]
    L.sla_backward_projected.restype = ctypes.c_int
    L.sla_backward_projected.argtypes = [vp, sz, i64, i32, en, i32, i32, en, f32] + [vp] * 12 + [vp, sz, vp]
    L.sla_cwi_map_bytes.restype = sz
    L.sla_cwi_map_bytes.argtypes = [i32, i32, i32]
    L.sla_cwi_build_map.restype = ctypes.c_int
    L.sla_cwi_build_map.argtypes = [vp, i64, i32, i32, i32, vp, sz, vp, vp]
    L.sla_cwi_forward.restype = ctypes.c_int
    L.sla_cwi_forward.argtypes = [vp, i32, i32, i32, vp, i64, vp, en, i32, i32, i32, vp, vp, vp, vp, vp, vp]
    L.sla_cwi_backward_workspace_bytes.restype = sz
    L.sla_cwi_backward_workspace_bytes.argtypes = [i64, en, i32, i32, i32]
    L.sla_cwi_backward.restype = ctypes.c_int
    L.sla_cwi_backward.argtypes = [vp, i32, i32, i32, vp, i64, vp, en, i32, i32, i32, vp, vp, vp, vp, vp, vp,
                                   vp, vp, vp, vp, sz, vp]
    L.sla_scatter_workspace_bytes.restype = sz
    L.sla_scatter_workspace_bytes.argtypes = [i64, i32, i32]
    L.sla_forward_scatter.restype = ctypes.c_int
    L.sla_forward_scatter.argtypes = [vp, sz, i64, i32, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp, sz, vp]
    L.sla_forward_xca.restype = ctypes.c_int
    L.sla_forward_xca.argtypes = [vp, sz, i64, i32, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp, vp]
    L.sla_backward_xca_noalloc.restype = ctypes.c_int
    L.sla_backward_xca_noalloc.argtypes = [vp, sz, i64, i32, en, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.sla_xca_backward_workspace_bytes.restype = sz
    L.sla_xca_backward_workspace_bytes.argtypes = [i32, i32]
    L.sla_backward_xca.restype = ctypes.c_int
    L.sla_backward_xca.argtypes = [vp, sz, i64, i32, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp, sz, vp]
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().sla_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != SLA_OK:
        raise SlaError(status, what)


def plan_bytes(n: int, num_windows: int) -> int:
    return int(lib().sla_plan_bytes(int(n), int(num_windows)))


def plan_layout(n: int, num_windows: int) -> PlanLayout:
    out = PlanLayout()
    _check(lib().sla_plan_layout(int(n), int(num_windows), ctypes.byref(out)), "sla_plan_layout")
    return out


# ----------------------------------------------------------------- torch glue
def _torch():
    import torch

    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(dt) -> int:
    torch = _torch()
    codes = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}
    if dt not in codes:
        raise TypeError(f"SLA supports float32, float16 and bfloat16, not {dt}")
    return codes[dt]


@dataclass
class Plan:
    """Device plan of one scene: window-sorted row order, offsets, chunks and
    long windows."""

    buf: object          # torch uint8 tensor on the device (the plan bytes)
    n: int
    num_windows: int
    chunk_rows: int
    perm: object         # int32 [n] copy of the permutation, or None (CSR mode)
    offsets: object      # int32 [num_windows + 1]
    invalid: object      # int32 [1]

    @property
    def nbytes(self) -> int:
        return int(self.buf.numel())


def new_plan_buffer(n: int, num_windows: int, device):
    torch = _torch()
    nb = plan_bytes(n, num_windows)
    if nb == 0:
        raise SlaError(SLA_E_ARG, "sla_plan_bytes")
    # zero-filled once: the builder keeps its window totals at zero between builds
    return torch.zeros(nb, dtype=torch.uint8, device=device)


def build_segments(ids=None, num_windows: int = 0, chunk_rows: int = 0, offsets=None,
                   plan_buf=None, want_perm: bool = True, n: int | None = None) -> Plan:
    """Mode A: ids (int32 [n] device tensor).  Mode B: offsets (int32 [W+1]) of
    already window-sorted rows, with n given."""
    torch = _torch()
    if ids is not None:
        if ids.dtype != torch.int32 or not ids.is_contiguous():
            raise TypeError("window ids must be a contiguous int32 tensor")
        n = ids.numel()
        device = ids.device
    else:
        if offsets is None or n is None:
            raise ValueError("give ids, or offsets and n")
        device = offsets.device
    if plan_buf is None:
        plan_buf = new_plan_buffer(n, num_windows, device)
    invalid = torch.empty(1, dtype=torch.int32, device=device)  # always written by the builder
    perm = None
    ids_arg = ids
    if ids is not None:
        perm = torch.empty(n, dtype=torch.int32, device=device) if want_perm else None
        if offsets is None:
            offsets = torch.empty(num_windows + 1, dtype=torch.int32, device=device)
        if n == 0:
            # an empty tensor has a NULL data pointer, which the C ABI reads as CSR mode
            ids_arg = torch.zeros(1, dtype=torch.int32, device=device)
    st = lib().sla_build_segments(_ptr(ids_arg), int(n), int(num_windows), int(chunk_rows), _ptr(perm),
                                  _ptr(offsets), _ptr(invalid), _ptr(plan_buf),
                                  int(plan_buf.numel()), _stream(device))
    _check(st, "sla_build_segments")
    cr = chunk_rows if chunk_rows else int(lib().sla_default_chunk_rows())
    return Plan(plan_buf, int(n), int(num_windows), cr, perm, offsets, invalid)


def _check_rows(name, t, n, like=None):
    if t.dim() != 3 or t.shape[0] != n or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous [n, heads, head_dim] tensor with n={n}")
    if like is not None and (t.shape != like.shape or t.dtype != like.dtype or t.device != like.device):
        raise ValueError(f"{name} must match q in shape, dtype and device")


def _check_workspace(ws, device):
    """A caller's workspace: a contiguous tensor on the call's device (its size in
    bytes, numel x element size, is checked by the library)."""
    if ws.device != device or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor on the inputs' device")


def _variant(feature_map, eps):
    """None for the plain Eq. (3) calls, else (sla_feature_map_t, eps)."""
    if feature_map is None and eps is None:
        return None
    fm = "elu1" if feature_map is None else feature_map
    if fm not in FEATURE_MAPS:
        raise ValueError(f"feature_map must be one of {sorted(FEATURE_MAPS)}, not {fm!r}")
    return FEATURE_MAPS[fm], float(0.0 if eps is None else eps)


def forward(plan: Plan, q, k, v, out=None, feature_map=None, eps=None):
    torch = _torch()
    _check_rows("q", q, plan.n)
    _check_rows("k", k, plan.n, q)
    _check_rows("v", v, plan.n, q)
    if out is None:
        out = torch.empty_like(q)
    _check_rows("out", out, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    var = _variant(feature_map, eps)
    if var is None:
        st = lib().sla_forward(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows, _dtype_code(q.dtype),
                               H, d, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _stream(q.device))
        _check(st, "sla_forward")
    else:
        st = lib().sla_forward_ex(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                  _dtype_code(q.dtype), H, d, var[0], var[1], _ptr(q), _ptr(k), _ptr(v),
                                  _ptr(out), _stream(q.device))
        _check(st, "sla_forward_ex")
    return out


def backward(plan: Plan, q, k, v, dout, dq=None, dk=None, dv=None, feature_map=None, eps=None):
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v), ("dout", dout)):
        _check_rows(name, t, plan.n, q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check_rows(name, t, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    var = _variant(feature_map, eps)
    if var is None:
        st = lib().sla_backward(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows, _dtype_code(q.dtype),
                                H, d, _ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
                                _stream(q.device))
        _check(st, "sla_backward")
    else:
        st = lib().sla_backward_ex(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                   _dtype_code(q.dtype), H, d, var[0], var[1], _ptr(q), _ptr(k), _ptr(v),
                                   _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _stream(q.device))
        _check(st, "sla_backward_ex")
    return dq, dk, dv


def forward_xca(plan: Plan, q, k, v, tau, out=None):
    """XCA inside every window (sla_forward_xca); tau: float32 [heads] on q's device."""
    torch = _torch()
    _check_rows("q", q, plan.n)
    _check_rows("k", k, plan.n, q)
    _check_rows("v", v, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    if (tau.dtype != torch.float32 or tau.dim() != 1 or tau.shape[0] != H or not tau.is_contiguous()
            or tau.device != q.device):
        raise ValueError("tau must be a contiguous float32 [heads] tensor on q's device")
    if out is None:
        out = torch.empty_like(q)
    _check_rows("out", out, plan.n, q)
    st = lib().sla_forward_xca(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows, _dtype_code(q.dtype),
                               H, d, _ptr(tau), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _stream(q.device))
    _check(st, "sla_forward_xca")
    return out


def backward_xca(plan: Plan, q, k, v, tau, dout, dq=None, dk=None, dv=None, dtau=None, workspace=None):
    """Gradients of forward_xca (sla_backward_xca): (dq, dk, dv, dtau)."""
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v), ("dout", dout)):
        _check_rows(name, t, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    if (tau.dtype != torch.float32 or tau.dim() != 1 or tau.shape[0] != H or not tau.is_contiguous()
            or tau.device != q.device):
        raise ValueError("tau must be a contiguous float32 [heads] tensor on q's device")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check_rows(name, t, plan.n, q)
    dtau = torch.empty_like(tau) if dtau is None else dtau
    if (dtau.dtype != torch.float32 or dtau.dim() != 1 or dtau.shape[0] != H or not dtau.is_contiguous()
            or dtau.device != q.device):
        raise ValueError("dtau must be a contiguous float32 [heads] tensor on q's device")
    need = int(lib().sla_xca_backward_workspace_bytes(plan.num_windows, H))
    if workspace is None:
        workspace = torch.empty(max(need, 4), dtype=torch.uint8, device=q.device)
    _check_workspace(workspace, q.device)
    st = lib().sla_backward_xca(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows, _dtype_code(q.dtype),
                                H, d, _ptr(tau), _ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(dq), _ptr(dk),
                                _ptr(dv), _ptr(dtau), _ptr(workspace),
                                int(workspace.numel() * workspace.element_size()), _stream(q.device))
    _check(st, "sla_backward_xca")
    return dq, dk, dv, dtau


def backward_xca_noalloc(plan: Plan, q, k, v, tau, dout, dq=None, dk=None, dv=None, dtau=None):
    """backward_xca through sla_backward_xca_noalloc: the dtau partials live in the
    library's static device buffer (no workspace; calls on one GPU must not overlap)."""
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v), ("dout", dout)):
        _check_rows(name, t, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    if (tau.dtype != torch.float32 or tau.dim() != 1 or tau.shape[0] != H or not tau.is_contiguous()
            or tau.device != q.device):
        raise ValueError("tau must be a contiguous float32 [heads] tensor on q's device")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check_rows(name, t, plan.n, q)
    dtau = torch.empty_like(tau) if dtau is None else dtau
    if (dtau.dtype != torch.float32 or dtau.dim() != 1 or dtau.shape[0] != H or not dtau.is_contiguous()
            or dtau.device != q.device):
        raise ValueError("dtau must be a contiguous float32 [heads] tensor on q's device")
    st = lib().sla_backward_xca_noalloc(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                        _dtype_code(q.dtype), H, d, _ptr(tau), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dtau), _stream(q.device))
    _check(st, "sla_backward_xca_noalloc")
    return dq, dk, dv, dtau


def forward_projected(plan: Plan, x, w_qkv, w_o, heads: int, b_qkv=None, b_o=None, o=None, y=None,
                      feature_map="elu1", eps=0.0, qkv_out=None):
    """Projection layer, SLA and output projection (sla_forward_projected):
    x [n, C], w_qkv [3C, C], w_o [C, C], optional biases [3C], [C]; returns (o, y)
    with o [n, heads, C // heads] and y [n, C].  qkv_out, a contiguous [3, n, C]
    tensor like x, also receives q, k, v for backward_projected(qkv=...)."""
    torch = _torch()
    if x.dim() != 2 or x.shape[0] != plan.n or not x.is_contiguous():
        raise ValueError(f"x must be a contiguous [n, C] tensor with n={plan.n}")
    n, C = x.shape
    if C % heads:
        raise ValueError("C must be a multiple of heads")
    d = C // heads
    for name, t, shape in (("w_qkv", w_qkv, (3 * C, C)), ("w_o", w_o, (C, C)),
                           ("b_qkv", b_qkv, (3 * C,)), ("b_o", b_o, (C,))):
        if t is None:
            continue
        if tuple(t.shape) != shape or t.dtype != x.dtype or t.device != x.device or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor like x")
    o = torch.empty((n, heads, d), dtype=x.dtype, device=x.device) if o is None else o
    y = torch.empty_like(x) if y is None else y
    _check_rows("o", o, n)
    if y.shape != x.shape or y.dtype != x.dtype or not y.is_contiguous():
        raise ValueError("y must be a contiguous tensor like x")
    if feature_map not in FEATURE_MAPS:
        raise ValueError(f"feature_map must be one of {sorted(FEATURE_MAPS)}, not {feature_map!r}")
    _check_qkv("qkv_out", qkv_out, x)
    st = lib().sla_forward_projected(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                     _dtype_code(x.dtype), heads, d, FEATURE_MAPS[feature_map], float(eps),
                                     _ptr(x), _ptr(w_qkv), _ptr(b_qkv), _ptr(w_o), _ptr(b_o), _ptr(o), _ptr(y),
                                     _ptr(qkv_out), _stream(x.device))
    _check(st, "sla_forward_projected")
    return o, y


def _check_qkv(name, t, x):
    if t is None:
        return
    n, C = x.shape
    if tuple(t.shape) != (3, n, C) or t.dtype != x.dtype or t.device != x.device or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous (3, {n}, {C}) tensor like x")


def backward_projected_workspace_bytes(n: int, heads: int, head_dim: int) -> int:
    return int(lib().sla_backward_projected_workspace_bytes(int(n), int(heads), int(head_dim)))


def backward_projected(plan: Plan, x, w_qkv, w_o, o, dy, heads: int, b_qkv=None, feature_map="elu1", eps=0.0,
                       dx=None, workspace=None, bias_grads=True, qkv=None):
    """Gradients of sla_forward_projected (sla_backward_projected): x, dy [n, C],
    w_qkv [3C, C], w_o [C, C], o the forward's SLA output ([n, heads, d] or [n, C]),
    optional b_qkv [3C], optional qkv (the forward's qkv_out, [3, n, C]; q, k, v
    are recomputed without it).  Returns (dx, dw_qkv, db_qkv, dw_o, db_o): dx like
    x, the weight and bias gradients float32 (the bias ones None with
    bias_grads=False)."""
    torch = _torch()
    if x.dim() != 2 or x.shape[0] != plan.n or not x.is_contiguous():
        raise ValueError(f"x must be a contiguous [n, C] tensor with n={plan.n}")
    n, C = x.shape
    if C % heads:
        raise ValueError("C must be a multiple of heads")
    d = C // heads
    for name, t, shape in (("w_qkv", w_qkv, (3 * C, C)), ("w_o", w_o, (C, C)), ("b_qkv", b_qkv, (3 * C,)),
                           ("dy", dy, (n, C))):
        if t is None:
            continue
        if tuple(t.shape) != shape or t.dtype != x.dtype or t.device != x.device or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor like x")
    if o.dtype != x.dtype or o.device != x.device or not o.is_contiguous() or o.numel() != n * C:
        raise ValueError("o must be the forward's contiguous [n, C] output, like x")
    dx = torch.empty_like(x) if dx is None else dx
    if dx.shape != x.shape or dx.dtype != x.dtype or not dx.is_contiguous() or dx.device != x.device:
        raise ValueError("dx must be a contiguous tensor like x")
    f32 = dict(dtype=torch.float32, device=x.device)
    dw_qkv, dw_o = torch.empty((3 * C, C), **f32), torch.empty((C, C), **f32)
    db_qkv = torch.empty(3 * C, **f32) if bias_grads else None
    db_o = torch.empty(C, **f32) if bias_grads else None
    need = backward_projected_workspace_bytes(n, heads, d)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check_workspace(workspace, x.device)
    if feature_map not in FEATURE_MAPS:
        raise ValueError(f"feature_map must be one of {sorted(FEATURE_MAPS)}, not {feature_map!r}")
    _check_qkv("qkv", qkv, x)
    st = lib().sla_backward_projected(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                      _dtype_code(x.dtype), heads, d, FEATURE_MAPS[feature_map], float(eps),
                                      _ptr(x), _ptr(w_qkv), _ptr(b_qkv), _ptr(w_o), _ptr(o), _ptr(dy), _ptr(dx),
                                      _ptr(dw_qkv), _ptr(db_qkv), _ptr(dw_o), _ptr(db_o), _ptr(qkv),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(x.device))
    _check(st, "sla_backward_projected")
    return dx, dw_qkv, db_qkv, dw_o, db_o


def cwi_map_bytes(gx: int, gy: int, gz: int) -> int:
    return int(lib().sla_cwi_map_bytes(int(gx), int(gy), int(gz)))


def cwi_build_map(coords, grid, map=None):
    """Cell -> row table of a scene for the cross-window interaction: coords int32
    [n, 3] (x, y, z) on the device, grid (gx, gy, gz).  Returns (map, conflicts),
    conflicts an int32 [1] device tensor (rows outside the grid or on a taken cell)."""
    torch = _torch()
    gx, gy, gz = (int(g) for g in grid)
    if coords.dtype != torch.int32 or coords.dim() != 2 or coords.shape[1] != 3 or not coords.is_contiguous():
        raise ValueError("coords must be a contiguous int32 [n, 3] tensor")
    nb = cwi_map_bytes(gx, gy, gz)
    if nb == 0:
        raise SlaError(SLA_E_ARG, "sla_cwi_map_bytes")
    if map is None:
        map = torch.empty(nb // 4, dtype=torch.int32, device=coords.device)
    conflicts = torch.empty(1, dtype=torch.int32, device=coords.device)
    n = coords.shape[0]
    cptr = _ptr(coords) if n else ctypes.c_void_p(0)
    st = lib().sla_cwi_build_map(cptr, n, gx, gy, gz, _ptr(map), int(map.numel() * 4), _ptr(conflicts),
                                 _stream(coords.device))
    _check(st, "sla_cwi_build_map")
    return map, conflicts


def _cwi_check(map, grid, coords, x, w_x, w_y, w_3, order, **like_x):
    """Shapes, dtypes, devices and layouts of a cross-window interaction call (the
    C entry points take the cell table without its size, so it is checked here)."""
    torch = _torch()
    gx, gy, gz = (int(g) for g in grid)
    if x.dim() != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous [n, channels] tensor")
    n, C = x.shape
    c = C // 4
    for name, t, rows in (("w_x", w_x, None), ("w_y", w_y, None), ("w_3", w_3, 27)):
        if t.dim() != 2 or t.shape[1] != c or (rows and t.shape[0] != rows) or t.dtype != x.dtype \
                or not t.is_contiguous() or t.device != x.device:
            raise ValueError(f"{name} must be a contiguous [taps, {c}] tensor like x")
    if coords.shape != (n, 3) or coords.dtype != torch.int32 or not coords.is_contiguous() \
            or coords.device != x.device:
        raise ValueError("coords must be a contiguous int32 [n, 3] tensor on x's device")
    need = cwi_map_bytes(gx, gy, gz)
    if need == 0 or map.dtype != torch.int32 or map.numel() * 4 < need or not map.is_contiguous() \
            or map.device != x.device:
        raise ValueError("map must be the int32 cell table of this grid (cwi_build_map)")
    if order is not None and (order.shape != (n,) or order.dtype != torch.int32 or not order.is_contiguous()
                              or order.device != x.device):
        raise ValueError("order must be a contiguous int32 [n] tensor on x's device")
    for name, t in like_x.items():
        if t is not None and (t.shape != x.shape or t.dtype != x.dtype or not t.is_contiguous()
                              or t.device != x.device):
            raise ValueError(f"{name} must be a contiguous tensor like x")
    return gx, gy, gz, n, C


def cwi_forward(map, grid, coords, x, w_x, w_y, w_3, order=None, y=None):
    """Cross-window interaction (sla_cwi_forward): x [n, 4c], w_x [K_x, c], w_y
    [K_y, c], w_3 [27, c]; order an int32 [n] visiting order or None."""
    torch = _torch()
    gx, gy, gz, n, C = _cwi_check(map, grid, coords, x, w_x, w_y, w_3, order, y=y)
    y = torch.empty_like(x) if y is None else y
    st = lib().sla_cwi_forward(_ptr(map), gx, gy, gz, _ptr(coords), n, _ptr(order), _dtype_code(x.dtype), C,
                               int(w_x.shape[0]), int(w_y.shape[0]), _ptr(x), _ptr(w_x), _ptr(w_y), _ptr(w_3),
                               _ptr(y), _stream(x.device))
    _check(st, "sla_cwi_forward")
    return y


def cwi_backward_workspace_bytes(n: int, dtype, channels: int, taps_x: int, taps_y: int) -> int:
    """Workspace of cwi_backward (0: unsupported shape); dtype a torch dtype."""
    return int(lib().sla_cwi_backward_workspace_bytes(int(n), _dtype_code(dtype), int(channels), int(taps_x),
                                                      int(taps_y)))


def cwi_backward(map, grid, coords, x, w_x, w_y, w_3, dy, order=None, workspace=None, out=None):
    """Backward of cwi_forward (sla_cwi_backward): returns (dx, dw_x, dw_y, dw_3),
    written into `out` when given (tensors shaped like x, w_x, w_y, w_3)."""
    torch = _torch()
    gx, gy, gz, n, C = _cwi_check(map, grid, coords, x, w_x, w_y, w_3, order, dy=dy)
    code = _dtype_code(x.dtype)
    need = cwi_backward_workspace_bytes(n, x.dtype, C, w_x.shape[0], w_y.shape[0])
    if need == 0:
        raise SlaError(SLA_E_UNSUPPORTED, "sla_cwi_backward_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    _check_workspace(workspace, x.device)
    if out is None:
        dx = torch.empty_like(x)
        dws = [torch.empty_like(w) for w in (w_x, w_y, w_3)]
    else:
        dx, dws = out[0], list(out[1:])
        for t, ref in zip(out, (x, w_x, w_y, w_3)):
            if t.shape != ref.shape or t.dtype != ref.dtype or not t.is_contiguous():
                raise ValueError("out tensors must be contiguous and shaped like x, w_x, w_y, w_3")
    st = lib().sla_cwi_backward(_ptr(map), gx, gy, gz, _ptr(coords), n, _ptr(order), code, C,
                                int(w_x.shape[0]), int(w_y.shape[0]), _ptr(x), _ptr(w_x), _ptr(w_y), _ptr(w_3),
                                _ptr(dy), _ptr(dx), *(_ptr(t) for t in dws), _ptr(workspace),
                                int(workspace.numel() * workspace.element_size()), _stream(x.device))
    _check(st, "sla_cwi_backward")
    return (dx, *dws)


def scatter_workspace_bytes(n: int, heads: int, head_dim: int) -> int:
    return int(lib().sla_scatter_workspace_bytes(int(n), int(heads), int(head_dim)))


def forward_scatter(plan: Plan, q, k, v, out=None, workspace=None):
    """The naive scatter-based forward (per-voxel kv cache + per-window sums),
    the comparator of the chunk-wise sla_forward."""
    torch = _torch()
    _check_rows("q", q, plan.n)
    _check_rows("k", k, plan.n, q)
    _check_rows("v", v, plan.n, q)
    if out is None:
        out = torch.empty_like(q)
    _check_rows("out", out, plan.n, q)
    H, d = q.shape[1], q.shape[2]
    need = scatter_workspace_bytes(plan.n, H, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _check_workspace(workspace, q.device)
    st = lib().sla_forward_scatter(_ptr(plan.buf), plan.nbytes, plan.n, plan.num_windows,
                                   _dtype_code(q.dtype), H, d, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                   _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                   _stream(q.device))
    _check(st, "sla_forward_scatter")
    return out


def read_plan(plan: Plan):
    """Host copy of the plan's header, perm, offsets, chunk table and long-window
    table (tests)."""
    import numpy as np

    lay = plan_layout(plan.n, plan.num_windows)
    raw = plan.buf.cpu().numpy()
    hdr = raw[lay.header: lay.header + 64].view(np.int32)
    header = dict(zip(("magic", "n", "num_windows", "chunk_rows", "n_chunks", "csr", "invalid",
                       "n_long", "n_long4"), hdr[:9].tolist()))
    perm = raw[lay.perm: lay.perm + 4 * plan.n].view(np.int32)
    offs = raw[lay.offsets: lay.offsets + 4 * (plan.num_windows + 1)].view(np.int32)
    nc = max(0, min(header["n_chunks"], lay.max_chunks))
    chunks = raw[lay.chunks: lay.chunks + 16 * nc].view(np.int32).reshape(nc, 4)
    nl = max(0, min(header["n_long"], lay.max_long))
    longs = raw[lay.longs: lay.longs + 16 * nl].view(np.int32).reshape(nl, 4)
    return header, perm, offs, chunks, longs
