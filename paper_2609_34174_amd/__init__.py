"""GradLev fast-weight scans on MI355X (gfx950): thin Python binding.

Every function here only marshals arguments (shapes, dtypes, device
pointers, the current HIP stream) into the C ABI of ``libgradlev.so``
(declared in ``include/gradlev.h``).  All arithmetic runs in the library's
HIP kernels; there is no fallback: if the library is not built, or a tensor
is not on a ROCm device, a call raises.

    import paper_2609_34174_amd as gl
    Y = gl.scan_fwd(W0, X, G, eta=0.1)
    out = gl.scan_bwd(W0, X, G, dY, eta=0.1)     # dict of gradients
    y = gl.decode_step(W, x, g, eta=0.1)          # updates W in place

Shapes: W0 [H,m,d] fp32; X [B,H,T,d], G/dY [B,H,T,m] (fp32 or bf16, all
three the same); eta a float or an fp32 [B,H,T] tensor.
"""

from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "libgradlev.so")

F32, BF16 = 0, 1
EXCLUSIVE, INCLUSIVE = 0, 1
OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_ALIGN, ERR_WORKSPACE, ERR_HIP, ERR_SCRATCH = 0, -1, -2, -3, -4, -5, -6
STATIC_SCRATCH_BYTES = 64 << 20  # GRADLEV_STATIC_SCRATCH_BYTES

_PREFIX = {"exclusive": EXCLUSIVE, "inclusive": INCLUSIVE}


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("H", ctypes.c_int64), ("T", ctypes.c_int64),
                ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64),
                ("chunk", ctypes.c_int64), ("segment", ctypes.c_int64),
                ("in_dtype", ctypes.c_int32), ("prefix", ctypes.c_int32)]


class Plan(ctypes.Structure):
    _fields_ = [("fwd_chunk", ctypes.c_int64), ("fwd_segment", ctypes.c_int64),
                ("fwd_nseg", ctypes.c_int64), ("bwd_chunk", ctypes.c_int64),
                ("bwd_segment", ctypes.c_int64), ("bwd_nseg", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_size_t)]


class Gates(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_void_p), ("alpha_scalar", ctypes.c_float),
                ("reset", ctypes.c_void_p)]


class MlpShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("H", ctypes.c_int64), ("T", ctypes.c_int64),
                ("d_in", ctypes.c_int64), ("hidden", ctypes.c_int64), ("d_out", ctypes.c_int64),
                ("segment", ctypes.c_int64), ("in_dtype", ctypes.c_int32), ("act", ctypes.c_int32)]


ACT = {"tanh": 0, "gelu": 1, "gelu_tanh": 2}


class GradLevError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"{what}: {error_string(code)} (status {code})")
        self.code = code


_lib = None


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"GradLev HIP library not built ({LIB_PATH}); run "
                               "`python -m paper_2609_34174_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, f32p = ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p
        L.gradlev_version.restype = ctypes.c_int
        L.gradlev_error_string.restype = ctypes.c_char_p
        L.gradlev_error_string.argtypes = [ctypes.c_int]
        L.gradlev_scan_plan.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(Plan)]
        L.gradlev_scan_workspace_bytes.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(ctypes.c_size_t)]
        L.gradlev_scan_fwd.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                       f32p, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_fwd_static.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                              f32p, vp]
        L.gradlev_scan_bwd.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                       vp, f32p, f32p, f32p, f32p, f32p, vp, ctypes.c_size_t, vp]
        L.gradlev_decode_step.argtypes = [i64, i64, i64, i64, f32p, f32p, f32p, f32p,
                                          ctypes.c_float, f32p, vp]
        szp = ctypes.POINTER(ctypes.c_size_t)
        L.gradlev_scan_saved_bytes.argtypes = [ctypes.POINTER(Shape), szp, szp]
        L.gradlev_scan_fwd_save.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                            f32p, f32p, ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_bwd_saved.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                             vp, f32p, ctypes.c_size_t, f32p, f32p, f32p, f32p, f32p,
                                             vp, ctypes.c_size_t, vp]
        L.gradlev_scan_reset_saved_bytes.argtypes = [ctypes.POINTER(Shape), szp, szp]
        L.gradlev_scan_fwd_reset_save.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float, vp,
                                                  f32p, f32p, ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_bwd_reset_saved.argtypes = [ctypes.POINTER(Shape), f32p, vp, vp, f32p, ctypes.c_float,
                                                   vp, vp, f32p, ctypes.c_size_t, f32p, f32p, f32p, f32p, f32p,
                                                   vp, ctypes.c_size_t, vp]
        gp = ctypes.POINTER(Gates)
        L.gradlev_scan_gated_workspace_bytes.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(ctypes.c_size_t)]
        L.gradlev_scan_fwd_gated.argtypes = [ctypes.POINTER(Shape), gp, f32p, vp, vp, f32p, ctypes.c_float,
                                             f32p, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_bwd_gated.argtypes = [ctypes.POINTER(Shape), gp, f32p, vp, vp, f32p, ctypes.c_float,
                                             vp, f32p, f32p, f32p, f32p, f32p, f32p, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_gated_saved_bytes.argtypes = [ctypes.POINTER(Shape), szp, szp]
        L.gradlev_scan_fwd_gated_save.argtypes = [ctypes.POINTER(Shape), gp, f32p, vp, vp, f32p, ctypes.c_float,
                                                  f32p, f32p, ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.gradlev_scan_bwd_gated_saved.argtypes = [ctypes.POINTER(Shape), gp, f32p, vp, vp, f32p, ctypes.c_float,
                                                   vp, f32p, ctypes.c_size_t, f32p, f32p, f32p, f32p, f32p, f32p,
                                                   vp, ctypes.c_size_t, vp]
        L.gradlev_decode_step_gated.argtypes = [i64, i64, i64, i64, f32p, f32p, f32p, f32p, f32p,
                                                ctypes.c_float, f32p, ctypes.c_float, vp, f32p, vp]
        mp = ctypes.POINTER(MlpShape)
        L.gradlev_mlp_workspace_bytes.argtypes = [mp, ctypes.POINTER(ctypes.c_size_t)]
        L.gradlev_mlp_fwd.argtypes = [mp, gp, f32p, f32p, vp, vp, vp, f32p, ctypes.c_float,
                                      f32p, vp, f32p, vp, ctypes.c_size_t, vp]
        L.gradlev_mlp_reverse.argtypes = [mp, gp, f32p, f32p, vp, vp, vp, f32p, ctypes.c_float,
                                          f32p, vp, vp, f32p, f32p, f32p, f32p, f32p, f32p, vp,
                                          ctypes.c_size_t, vp]
        L.gradlev_timing_enable.argtypes = [ctypes.c_int]
        L.gradlev_timing_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_int64)]
        for name in ("gradlev_scan_plan", "gradlev_scan_workspace_bytes", "gradlev_scan_fwd", "gradlev_scan_fwd_static",
                     "gradlev_scan_bwd", "gradlev_scan_saved_bytes", "gradlev_scan_fwd_save",
                     "gradlev_scan_bwd_saved", "gradlev_decode_step", "gradlev_scan_gated_workspace_bytes",
                     "gradlev_scan_reset_saved_bytes", "gradlev_scan_fwd_reset_save", "gradlev_scan_bwd_reset_saved",
                     "gradlev_scan_fwd_gated", "gradlev_scan_bwd_gated", "gradlev_decode_step_gated",
                     "gradlev_scan_gated_saved_bytes", "gradlev_scan_fwd_gated_save", "gradlev_scan_bwd_gated_saved",
                     "gradlev_mlp_workspace_bytes", "gradlev_mlp_fwd", "gradlev_mlp_reverse",
                     "gradlev_timing_enable",
                     "gradlev_timing_reset", "gradlev_timing_read"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def error_string(code: int) -> str:
    return lib().gradlev_error_string(int(code)).decode()


def make_shape(B, H, T, d_in, d_out, dtype=BF16, prefix="exclusive", chunk=0, segment=0) -> Shape:
    return Shape(int(B), int(H), int(T), int(d_in), int(d_out), int(chunk), int(segment),
                 int(dtype), _PREFIX[prefix] if isinstance(prefix, str) else int(prefix))


def plan(shape: Shape) -> Plan:
    p = Plan()
    rc = lib().gradlev_scan_plan(ctypes.byref(shape), ctypes.byref(p))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_plan")
    return p


def workspace_bytes(shape: Shape) -> int:
    n = ctypes.c_size_t(0)
    rc = lib().gradlev_scan_workspace_bytes(ctypes.byref(shape), ctypes.byref(n))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_workspace_bytes")
    return int(n.value)


def saved_bytes(shape: Shape):
    """(saved-state bytes, workspace bytes) of the save-for-backward pair."""
    sv, ws = ctypes.c_size_t(0), ctypes.c_size_t(0)
    rc = lib().gradlev_scan_saved_bytes(ctypes.byref(shape), ctypes.byref(sv), ctypes.byref(ws))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_saved_bytes")
    return int(sv.value), int(ws.value)


# ---------------------------------------------------------------------------
# torch marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_dev(name, t, dtype=None, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a ROCm GPU (got {t.device}); there is no CPU path")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _scan_shape(W0, X, G, prefix, chunk, segment):
    torch = _torch()
    _check_dev("X", X)
    if X.dim() != 4:
        raise ValueError("X must be [B, H, T, d]")
    B, H, T, d = X.shape
    if X.dtype == torch.bfloat16:
        dt = BF16
    elif X.dtype == torch.float32:
        dt = F32
    else:
        raise TypeError("X must be float32 or bfloat16")
    _check_dev("G", G, X.dtype)
    if G.dim() != 4 or tuple(G.shape[:3]) != (B, H, T):
        raise ValueError("G must be [B, H, T, m]")
    m = G.shape[3]
    _check_dev("W0", W0, torch.float32, (H, m, d))
    return make_shape(B, H, T, d, m, dt, prefix, chunk, segment)


def _eta_args(eta, B, H, T, X):
    torch = _torch()
    if isinstance(eta, torch.Tensor):
        _check_dev("eta", eta, torch.float32, (B, H, T))
        if eta.device != X.device:
            raise ValueError("eta must be on the same device as X")
        return eta, 0.0
    return None, float(eta)


def _workspace(shape, device, workspace):
    torch = _torch()
    need = workspace_bytes(shape)
    if need == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    return workspace, workspace.numel() * workspace.element_size()


def scan_fwd(W0, X, G, eta=0.1, *, prefix="exclusive", chunk=0, segment=0, out=None, workspace=None):
    """Forward scan; returns Y [B,H,T,m] fp32 (see gradlev_scan_fwd)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, prefix, chunk, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    ws, wsn = _workspace(s, X.device, workspace)
    rc = lib().gradlev_scan_fwd(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(out),
                                _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd")
    return out


def scan_fwd_static(W0, X, G, eta=0.1, *, prefix="exclusive", chunk=0, segment=0, out=None):
    """Forward scan with no workspace: the library's static per-device scratch
    holds what scan_fwd keeps in its workspace (see gradlev_scan_fwd_static;
    calls that may overlap on one GPU race on that scratch)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, prefix, chunk, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    with torch.cuda.device(X.device):
        rc = lib().gradlev_scan_fwd_static(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(out),
                                           _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd_static")
    return out


BWD_OUTPUTS = ("gtilde", "dx", "dg", "deta", "dw0")


def scan_bwd(W0, X, G, dY, eta=0.1, *, prefix="exclusive", chunk=0, segment=0,
             outputs=BWD_OUTPUTS, out=None, workspace=None):
    """Backward of the forward scan; returns a dict with the requested outputs.

    outputs: any of "gtilde" [B,H,T,d], "dx" [B,H,T,d], "dg" [B,H,T,m],
    "deta" [B,H,T], "dw0" [H,m,d] (all fp32).  ``out`` may pre-supply tensors.
    """
    torch = _torch()
    s = _scan_shape(W0, X, G, prefix, chunk, segment)
    _check_dev("dY", dY, X.dtype, (s.B, s.H, s.T, s.d_out))
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    shapes = {"gtilde": (s.B, s.H, s.T, s.d_in), "dx": (s.B, s.H, s.T, s.d_in),
              "dg": (s.B, s.H, s.T, s.d_out), "deta": (s.B, s.H, s.T), "dw0": (s.H, s.d_out, s.d_in)}
    res = dict(out or {})
    for k in outputs:
        if k not in shapes:
            raise ValueError(f"unknown output {k!r}")
        if k not in res:
            res[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
        _check_dev(k, res[k], torch.float32, shapes[k])
    ws, wsn = _workspace(s, X.device, workspace)
    rc = lib().gradlev_scan_bwd(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(dY),
                                _ptr(res.get("gtilde")), _ptr(res.get("dx")), _ptr(res.get("dg")),
                                _ptr(res.get("deta")), _ptr(res.get("dw0")), _ptr(ws), wsn,
                                _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_bwd")
    return res


def _bytes_of(name, t, need):
    torch = _torch()
    if t is None:
        return None, 0
    _check_dev(name, t)
    n = t.numel() * t.element_size()
    if n < need:
        raise ValueError(f"{name} too small: need {need} bytes")
    return t, n


def scan_fwd_save(W0, X, G, eta=0.1, *, prefix="exclusive", chunk=0, segment=0, out=None, saved=None,
                  workspace=None):
    """Forward scan that also keeps each segment's end state for scan_bwd_saved.

    Returns (Y, saved): Y [B,H,T,m] fp32 and the saved state, a flat fp32
    device tensor (see gradlev_scan_fwd_save)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, prefix, chunk, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    sv_need, ws_need = saved_bytes(s)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    if saved is None:
        saved = torch.empty(sv_need // 4, dtype=torch.float32, device=X.device)
    saved, svn = _bytes_of("saved", saved, sv_need)
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_fwd_save(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(out),
                                     _ptr(saved), svn, _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd_save")
    return out, saved


def scan_bwd_saved(W0, X, G, dY, saved, eta=0.1, *, prefix="exclusive", chunk=0, segment=0,
                   outputs=BWD_OUTPUTS, out=None, workspace=None):
    """scan_bwd starting from the state scan_fwd_save kept (same inputs, same
    prefix/chunk/segment); returns the same dict as scan_bwd."""
    torch = _torch()
    s = _scan_shape(W0, X, G, prefix, chunk, segment)
    _check_dev("dY", dY, X.dtype, (s.B, s.H, s.T, s.d_out))
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    sv_need, ws_need = saved_bytes(s)
    shapes = {"gtilde": (s.B, s.H, s.T, s.d_in), "dx": (s.B, s.H, s.T, s.d_in),
              "dg": (s.B, s.H, s.T, s.d_out), "deta": (s.B, s.H, s.T), "dw0": (s.H, s.d_out, s.d_in)}
    res = dict(out or {})
    for k in outputs:
        if k not in shapes:
            raise ValueError(f"unknown output {k!r}")
        if k not in res:
            res[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
        _check_dev(k, res[k], torch.float32, shapes[k])
    saved, svn = _bytes_of("saved", saved, sv_need)
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_bwd_saved(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(dY),
                                      _ptr(saved), svn, _ptr(res.get("gtilde")), _ptr(res.get("dx")),
                                      _ptr(res.get("dg")), _ptr(res.get("deta")), _ptr(res.get("dw0")),
                                      _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_bwd_saved")
    return res



def reset_saved_bytes(shape: Shape):
    """(saved-state bytes, workspace bytes) of the reset pair."""
    sv, ws = ctypes.c_size_t(0), ctypes.c_size_t(0)
    rc = lib().gradlev_scan_reset_saved_bytes(ctypes.byref(shape), ctypes.byref(sv), ctypes.byref(ws))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_reset_saved_bytes")
    return int(sv.value), int(ws.value)


def _reset_arg(reset, B, T, X):
    torch = _torch()
    if reset is None:
        return None
    _check_dev("reset", reset, torch.uint8, (B, T))
    if reset.device != X.device:
        raise ValueError("reset must be on the same device as X")
    return reset


def scan_fwd_reset_save(W0, X, G, eta=0.1, reset=None, *, segment=0, out=None, saved=None, workspace=None):
    """Forward of the reset pair (unit retention, document starts reset [B,T]
    uint8); returns (Y, saved) for scan_bwd_reset_saved."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", 0, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    r = _reset_arg(reset, s.B, s.T, X)
    sv_need, ws_need = reset_saved_bytes(s)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    if saved is None:
        saved = torch.empty(sv_need // 4, dtype=torch.float32, device=X.device)
    saved, svn = _bytes_of("saved", saved, sv_need)
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_fwd_reset_save(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(r),
                                           _ptr(out), _ptr(saved), svn, _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd_reset_save")
    return out, saved


def scan_bwd_reset_saved(W0, X, G, dY, saved, eta=0.1, reset=None, *, segment=0, outputs=BWD_OUTPUTS, out=None,
                         workspace=None):
    """Backward of the reset pair from the state scan_fwd_reset_save kept
    (same inputs, flags and segment hint); returns the dict of scan_bwd."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", 0, segment)
    _check_dev("dY", dY, X.dtype, (s.B, s.H, s.T, s.d_out))
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    r = _reset_arg(reset, s.B, s.T, X)
    sv_need, ws_need = reset_saved_bytes(s)
    saved, svn = _bytes_of("saved", saved, sv_need)
    shapes = {"gtilde": (s.B, s.H, s.T, s.d_in), "dx": (s.B, s.H, s.T, s.d_in),
              "dg": (s.B, s.H, s.T, s.d_out), "deta": (s.B, s.H, s.T), "dw0": (s.H, s.d_out, s.d_in)}
    res = dict(out or {})
    for k in outputs:
        if k not in shapes:
            raise ValueError(f"unknown output {k!r}")
        if k not in res:
            res[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
        _check_dev(k, res[k], torch.float32, shapes[k])
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_bwd_reset_saved(ctypes.byref(s), _ptr(W0), _ptr(X), _ptr(G), _ptr(e), es, _ptr(dY),
                                            _ptr(r), _ptr(saved), svn, _ptr(res.get("gtilde")), _ptr(res.get("dx")),
                                            _ptr(res.get("dg")), _ptr(res.get("deta")), _ptr(res.get("dw0")),
                                            _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_bwd_reset_saved")
    return res

def decode_step(W, x, g, eta=0.1, *, out=None):
    """One deployment step: returns y = W x and updates W <- W - eta g x^T in place."""
    torch = _torch()
    _check_dev("W", W, torch.float32)
    if W.dim() != 4:
        raise ValueError("W must be [S, H, m, d]")
    S, H, m, d = W.shape
    _check_dev("x", x, torch.float32, (S, H, d))
    _check_dev("g", g, torch.float32, (S, H, m))
    if isinstance(eta, torch.Tensor):
        _check_dev("eta", eta, torch.float32, (S, H))
        e, es = eta, 0.0
    else:
        e, es = None, float(eta)
    if out is None:
        out = torch.empty(S, H, m, dtype=torch.float32, device=W.device)
    _check_dev("out", out, torch.float32, (S, H, m))
    rc = lib().gradlev_decode_step(S, H, d, m, _ptr(W), _ptr(x), _ptr(g), _ptr(e), es, _ptr(out),
                                   _stream(W.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_decode_step")
    return out


# ---------------------------------------------------------------------------
# Gated scans: retention alpha and document resets
# ---------------------------------------------------------------------------

def gated_workspace_bytes(shape: Shape) -> int:
    n = ctypes.c_size_t(0)
    rc = lib().gradlev_scan_gated_workspace_bytes(ctypes.byref(shape), ctypes.byref(n))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_gated_workspace_bytes")
    return int(n.value)


def _gates(alpha, reset, B, H, T, X, name="alpha", alpha_shape=None):
    torch = _torch()
    g = Gates()
    if isinstance(alpha, torch.Tensor):
        _check_dev(name, alpha, torch.float32, alpha_shape or (B, H, T))
        g.alpha, g.alpha_scalar = alpha.data_ptr(), 0.0
    else:
        g.alpha, g.alpha_scalar = None, float(alpha)
    if reset is not None:
        _check_dev("reset", reset, torch.uint8, (B, T) if alpha_shape is None else (B,))
        g.reset = reset.data_ptr()
    else:
        g.reset = None
    return g


def _gated_ws(shape, device, workspace):
    torch = _torch()
    need = gated_workspace_bytes(shape)
    if need == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    return workspace, workspace.numel() * workspace.element_size()


def scan_fwd_gated(W0, X, G, eta=0.1, alpha=1.0, reset=None, *, chunk=0, segment=0, out=None,
                   workspace=None):
    """Gated forward scan (retention alpha: float or fp32 [B,H,T]; reset: uint8 [B,T] or None)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", chunk, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    ws, wsn = _gated_ws(s, X.device, workspace)
    rc = lib().gradlev_scan_fwd_gated(ctypes.byref(s), ctypes.byref(gt), _ptr(W0), _ptr(X), _ptr(G), _ptr(e),
                                      es, _ptr(out), _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd_gated")
    return out


GATED_OUTPUTS = ("gtilde", "dx", "dg", "deta", "dalpha", "dw0")


def scan_bwd_gated(W0, X, G, dY, eta=0.1, alpha=1.0, reset=None, *, chunk=0, segment=0,
                   outputs=GATED_OUTPUTS, out=None, workspace=None):
    """Backward of the gated forward scan; dict with the requested outputs (``dalpha`` [B,H,T] too)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", chunk, segment)
    _check_dev("dY", dY, X.dtype, (s.B, s.H, s.T, s.d_out))
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    shapes = {"gtilde": (s.B, s.H, s.T, s.d_in), "dx": (s.B, s.H, s.T, s.d_in),
              "dg": (s.B, s.H, s.T, s.d_out), "deta": (s.B, s.H, s.T), "dalpha": (s.B, s.H, s.T),
              "dw0": (s.H, s.d_out, s.d_in)}
    res = dict(out or {})
    for k in outputs:
        if k not in shapes:
            raise ValueError(f"unknown output {k!r}")
        if k not in res:
            res[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
        _check_dev(k, res[k], torch.float32, shapes[k])
    ws, wsn = _gated_ws(s, X.device, workspace)
    rc = lib().gradlev_scan_bwd_gated(ctypes.byref(s), ctypes.byref(gt), _ptr(W0), _ptr(X), _ptr(G), _ptr(e),
                                      es, _ptr(dY), _ptr(res.get("gtilde")), _ptr(res.get("dx")),
                                      _ptr(res.get("dg")), _ptr(res.get("deta")), _ptr(res.get("dalpha")),
                                      _ptr(res.get("dw0")), _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_bwd_gated")
    return res


def gated_saved_bytes(shape: Shape):
    """(saved-state bytes, workspace bytes) of the gated save-for-backward pair."""
    sv, ws = ctypes.c_size_t(0), ctypes.c_size_t(0)
    rc = lib().gradlev_scan_gated_saved_bytes(ctypes.byref(shape), ctypes.byref(sv), ctypes.byref(ws))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_gated_saved_bytes")
    return int(sv.value), int(ws.value)


def scan_fwd_gated_save(W0, X, G, eta=0.1, alpha=1.0, reset=None, *, chunk=0, segment=0, out=None, saved=None,
                        workspace=None):
    """Gated forward that also keeps the backward's chunk-start states.

    Returns (Y, saved) (see gradlev_scan_fwd_gated_save)."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", chunk, segment)
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    sv_need, ws_need = gated_saved_bytes(s)
    if out is None:
        out = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    _check_dev("out", out, torch.float32, (s.B, s.H, s.T, s.d_out))
    if saved is None:
        saved = torch.empty(sv_need // 4, dtype=torch.float32, device=X.device)
    saved, svn = _bytes_of("saved", saved, sv_need)
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_fwd_gated_save(ctypes.byref(s), ctypes.byref(gt), _ptr(W0), _ptr(X), _ptr(G), _ptr(e),
                                           es, _ptr(out), _ptr(saved), svn, _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_fwd_gated_save")
    return out, saved


def scan_bwd_gated_saved(W0, X, G, dY, saved, eta=0.1, alpha=1.0, reset=None, *, chunk=0, segment=0,
                         outputs=GATED_OUTPUTS, out=None, workspace=None):
    """scan_bwd_gated starting from the states scan_fwd_gated_save kept."""
    torch = _torch()
    s = _scan_shape(W0, X, G, "exclusive", chunk, segment)
    _check_dev("dY", dY, X.dtype, (s.B, s.H, s.T, s.d_out))
    e, es = _eta_args(eta, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    sv_need, ws_need = gated_saved_bytes(s)
    shapes = {"gtilde": (s.B, s.H, s.T, s.d_in), "dx": (s.B, s.H, s.T, s.d_in),
              "dg": (s.B, s.H, s.T, s.d_out), "deta": (s.B, s.H, s.T), "dalpha": (s.B, s.H, s.T),
              "dw0": (s.H, s.d_out, s.d_in)}
    res = dict(out or {})
    for k in outputs:
        if k not in shapes:
            raise ValueError(f"unknown output {k!r}")
        if k not in res:
            res[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
        _check_dev(k, res[k], torch.float32, shapes[k])
    saved, svn = _bytes_of("saved", saved, sv_need)
    if workspace is None and ws_need:
        workspace = torch.empty(ws_need, dtype=torch.uint8, device=X.device)
    ws, wsn = _bytes_of("workspace", workspace, ws_need)
    rc = lib().gradlev_scan_bwd_gated_saved(ctypes.byref(s), ctypes.byref(gt), _ptr(W0), _ptr(X), _ptr(G),
                                            _ptr(e), es, _ptr(dY), _ptr(saved), svn, _ptr(res.get("gtilde")),
                                            _ptr(res.get("dx")), _ptr(res.get("dg")), _ptr(res.get("deta")),
                                            _ptr(res.get("dalpha")), _ptr(res.get("dw0")), _ptr(ws), wsn,
                                            _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_scan_bwd_gated_saved")
    return res


def decode_step_gated(W, W0, x, g, eta=0.1, alpha=1.0, reset=None, *, out=None):
    """Gated deployment step: y = W x (W0 after a reset), then W <- W0 + alpha (W - W0) - eta g x^T."""
    torch = _torch()
    _check_dev("W", W, torch.float32)
    if W.dim() != 4:
        raise ValueError("W must be [S, H, m, d]")
    S, H, m, d = W.shape
    _check_dev("W0", W0, torch.float32, (H, m, d))
    _check_dev("x", x, torch.float32, (S, H, d))
    _check_dev("g", g, torch.float32, (S, H, m))
    if isinstance(eta, torch.Tensor):
        _check_dev("eta", eta, torch.float32, (S, H))
        e, es = eta, 0.0
    else:
        e, es = None, float(eta)
    if isinstance(alpha, torch.Tensor):
        _check_dev("alpha", alpha, torch.float32, (S, H))
        a, as_ = alpha, 0.0
    else:
        a, as_ = None, float(alpha)
    if reset is not None:
        _check_dev("reset", reset, torch.uint8, (S,))
    if out is None:
        out = torch.empty(S, H, m, dtype=torch.float32, device=W.device)
    _check_dev("out", out, torch.float32, (S, H, m))
    rc = lib().gradlev_decode_step_gated(S, H, d, m, _ptr(W), _ptr(W0), _ptr(x), _ptr(g), _ptr(e), es,
                                         _ptr(a), as_, _ptr(reset), _ptr(out), _stream(W.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_decode_step_gated")
    return out


# ---------------------------------------------------------------------------
# Two-map online MLP
# ---------------------------------------------------------------------------

def _mlp_shape(W10, W20, X, Gz, Gy, act, segment):
    torch = _torch()
    _check_dev("X", X)
    if X.dim() != 4:
        raise ValueError("X must be [B, H, T, d_in]")
    B, H, T, d = X.shape
    if X.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("X must be float32 or bfloat16")
    _check_dev("W1_0", W10, torch.float32)
    if W10.dim() != 3 or W10.shape[0] != H or W10.shape[2] != d:
        raise ValueError("W1_0 must be [H, hidden, d_in]")
    hid = W10.shape[1]
    _check_dev("W2_0", W20, torch.float32)
    if W20.dim() != 3 or W20.shape[0] != H or W20.shape[2] != hid:
        raise ValueError("W2_0 must be [H, d_out, hidden]")
    o = W20.shape[1]
    _check_dev("Gz", Gz, X.dtype, (B, H, T, hid))
    _check_dev("Gy", Gy, X.dtype, (B, H, T, o))
    return MlpShape(B, H, T, d, hid, o, int(segment), BF16 if X.dtype == torch.bfloat16 else F32, ACT[act])


def _mlp_ws(s, device, workspace):
    torch = _torch()
    n = ctypes.c_size_t(0)
    rc = lib().gradlev_mlp_workspace_bytes(ctypes.byref(s), ctypes.byref(n))
    if rc != OK:
        raise GradLevError(rc, "gradlev_mlp_workspace_bytes")
    need = max(int(n.value), 256)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    return workspace, workspace.numel() * workspace.element_size()


def mlp_fwd(W10, W20, X, Gz, Gy, mu=0.9, alpha=1.0, reset=None, *, act="tanh", segment=0, workspace=None):
    """Two-map MLP forward from costate proposals; returns (Z fp32, Hid in X's dtype, Y fp32)."""
    torch = _torch()
    s = _mlp_shape(W10, W20, X, Gz, Gy, act, segment)
    m, ms = _eta_args(mu, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    Z = torch.empty(s.B, s.H, s.T, s.hidden, dtype=torch.float32, device=X.device)
    Hid = torch.empty(s.B, s.H, s.T, s.hidden, dtype=X.dtype, device=X.device)
    Y = torch.empty(s.B, s.H, s.T, s.d_out, dtype=torch.float32, device=X.device)
    ws, wsn = _mlp_ws(s, X.device, workspace)
    rc = lib().gradlev_mlp_fwd(ctypes.byref(s), ctypes.byref(gt), _ptr(W10), _ptr(W20), _ptr(X), _ptr(Gz),
                               _ptr(Gy), _ptr(m), ms, _ptr(Z), _ptr(Hid), _ptr(Y), _ptr(ws), wsn,
                               _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_mlp_fwd")
    return Z, Hid, Y


MLP_GRADS = ("dmu", "dalpha", "dw10", "dw20")


def mlp_reverse(W10, W20, X, Gz, Gy, Z, Hid, gY, mu=0.9, alpha=1.0, reset=None, *, act="tanh",
                with_gx=True, grads=(), segment=0, workspace=None):
    """Reverse targets of the MLP: returns (gZ, gX or None), fp32; with
    ``grads`` (any of "dmu" [B,H,T], "dalpha" [B,H,T], "dw10" [H,hidden,d_in],
    "dw20" [H,d_out,hidden]) returns (gZ, gX, dict of those training
    gradients) - see gradlev_mlp_reverse."""
    torch = _torch()
    s = _mlp_shape(W10, W20, X, Gz, Gy, act, segment)
    _check_dev("Z", Z, torch.float32, (s.B, s.H, s.T, s.hidden))
    _check_dev("Hid", Hid, X.dtype, (s.B, s.H, s.T, s.hidden))
    _check_dev("gY", gY, X.dtype, (s.B, s.H, s.T, s.d_out))
    m, ms = _eta_args(mu, s.B, s.H, s.T, X)
    gt = _gates(alpha, reset, s.B, s.H, s.T, X)
    gZ = torch.empty(s.B, s.H, s.T, s.hidden, dtype=torch.float32, device=X.device)
    gX = torch.empty(s.B, s.H, s.T, s.d_in, dtype=torch.float32, device=X.device) if with_gx else None
    shapes = {"dmu": (s.B, s.H, s.T), "dalpha": (s.B, s.H, s.T), "dw10": (s.H, s.hidden, s.d_in),
              "dw20": (s.H, s.d_out, s.hidden)}
    g = {}
    for k in grads:
        if k not in shapes:
            raise ValueError(f"unknown gradient {k!r}")
        g[k] = torch.empty(shapes[k], dtype=torch.float32, device=X.device)
    ws, wsn = _mlp_ws(s, X.device, workspace)
    rc = lib().gradlev_mlp_reverse(ctypes.byref(s), ctypes.byref(gt), _ptr(W10), _ptr(W20), _ptr(X), _ptr(Gz),
                                   _ptr(Gy), _ptr(m), ms, _ptr(Z), _ptr(Hid), _ptr(gY), _ptr(gZ), _ptr(gX),
                                   _ptr(g.get("dmu")), _ptr(g.get("dalpha")), _ptr(g.get("dw10")),
                                   _ptr(g.get("dw20")), _ptr(ws), wsn, _stream(X.device))
    if rc != OK:
        raise GradLevError(rc, "gradlev_mlp_reverse")
    return (gZ, gX, g) if grads else (gZ, gX)


# ---------------------------------------------------------------------------
# Kernel timing (HIP events recorded by the library around each launch)
# ---------------------------------------------------------------------------

KERNELS = ("fwd_agg", "fwd_main", "bwd_agg", "bwd_main", "bwd_dw0", "decode",
           "gated_agg", "gated_fwd", "gated_states", "gated_bwd", "wide_score", "wide_out")


def timing_enable(on: bool = True, kernels=None) -> int:
    """Turn per-launch event timing on (for ``kernels``, default all families) or off.

    Returns the previous family mask."""
    if not on:
        mask = 0
    elif kernels is None:
        mask = (1 << len(KERNELS)) - 1
    else:
        mask = 0
        for k in kernels:
            mask |= 1 << KERNELS.index(k)
    return int(lib().gradlev_timing_enable(mask))


def timing_reset() -> None:
    lib().gradlev_timing_reset()


def timing_read() -> dict:
    """{kernel: (total_ms, launches)} since the last reset (waits for the events)."""
    out = {}
    for i, name in enumerate(KERNELS):
        ms, n = ctypes.c_double(0.0), ctypes.c_int64(0)
        rc = lib().gradlev_timing_read(i, ctypes.byref(ms), ctypes.byref(n))
        if rc != OK:
            raise GradLevError(rc, "gradlev_timing_read")
        out[name] = (ms.value, int(n.value))
    return out


__all__ = ["timing_enable", "timing_reset", "timing_read", "KERNELS", "scan_fwd", "scan_bwd", "decode_step",
           "scan_fwd_gated", "scan_bwd_gated", "decode_step_gated", "gated_workspace_bytes", "Gates",
           "GATED_OUTPUTS", "mlp_fwd", "mlp_reverse", "MlpShape", "ACT", "plan", "workspace_bytes", "make_shape",
           "error_string", "lib", "GradLevError", "Shape", "Plan", "F32", "BF16",
           "EXCLUSIVE", "INCLUSIVE", "BWD_OUTPUTS"]
