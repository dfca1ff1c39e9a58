"""Python binding of the CCQ C ABI (libccq.so): argument marshalling only.

Every entry point has the same name as its C function.  Tensors are torch
tensors on the GPU; the binding checks dtypes/shapes, allocates outputs and
the workspace with torch when the caller does not pass them, and hands raw
device pointers plus the current HIP stream to the library.  All arithmetic
runs in the library's HIP kernels.  There is no fallback: if libccq.so is
missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libccq.so")

CCQ_F32, CCQ_BF16 = 0, 1
CCQ_GLA, CCQ_GDN = 0, 1
_STATUS = {0: "CCQ_OK", 1: "CCQ_ERR_INVALID_ARG", 2: "CCQ_ERR_UNSUPPORTED",
           3: "CCQ_ERR_WORKSPACE", 4: "CCQ_ERR_HIP"}
EXPORTS = ("ccq_workspace_size", "ccq_gla_fwd", "ccq_gdn_fwd", "ccq_gdn_fwd_noalloc", "ccq_fwd_bwd",
           "ccq_varlen_workspace_size", "ccq_gla_fwd_varlen", "ccq_gdn_fwd_varlen",
           "ccq_fwd_bwd_varlen", "ccq_decode_workspace_size", "ccq_decode", "ccq_prep",
           "ccq_fwd_raw_workspace_size", "ccq_fwd_raw",
           "ccq_trace_events", "ccq_status_string", "ccq_version")


class CcqError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__("%s returned %s (%d): %s" % (fn, _STATUS.get(code, "?"), code,
                                                      ccq_status_string(code)))
        self.code = code


class Shape(ctypes.Structure):
    """Mirror of ccq_shape (include/ccq.h)."""
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("gate_dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("centered", ctypes.c_int32),
                ("decay_aligned", ctypes.c_int32), ("t0", ctypes.c_int64)]


_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """Load libccq.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libccq.so is not built (%s); run "
                                   "`python -m paper_2606_01294_amd.build`" % LIB_PATH)
            L = ctypes.CDLL(LIB_PATH)
            P, S = ctypes.c_void_p, ctypes.c_size_t
            SP = ctypes.POINTER(Shape)
            L.ccq_workspace_size.argtypes = [SP, ctypes.c_int, ctypes.c_int]
            L.ccq_workspace_size.restype = S
            L.ccq_gla_fwd.argtypes = [SP] + [P] * 14 + [S, P]
            L.ccq_gla_fwd.restype = ctypes.c_int
            L.ccq_gdn_fwd.argtypes = [SP] + [P] * 15 + [S, P]
            L.ccq_gdn_fwd.restype = ctypes.c_int
            L.ccq_gdn_fwd_noalloc.argtypes = [SP] + [P] * 15
            L.ccq_gdn_fwd_noalloc.restype = ctypes.c_int
            L.ccq_fwd_bwd.argtypes = [SP, ctypes.c_int] + [P] * 15 + [S, P]
            L.ccq_fwd_bwd.restype = ctypes.c_int
            L.ccq_varlen_workspace_size.argtypes = [SP, ctypes.c_int, ctypes.c_int]
            L.ccq_varlen_workspace_size.restype = S
            L.ccq_gla_fwd_varlen.argtypes = [SP] + [P] * 14 + [S, P]
            L.ccq_gla_fwd_varlen.restype = ctypes.c_int
            L.ccq_gdn_fwd_varlen.argtypes = [SP] + [P] * 15 + [S, P]
            L.ccq_gdn_fwd_varlen.restype = ctypes.c_int
            L.ccq_fwd_bwd_varlen.argtypes = [SP, ctypes.c_int] + [P] * 16 + [S, P]
            L.ccq_fwd_bwd_varlen.restype = ctypes.c_int
            L.ccq_decode_workspace_size.argtypes = [SP]
            L.ccq_decode_workspace_size.restype = S
            L.ccq_decode.argtypes = [SP, ctypes.c_int] + [P] * 11 + [S, P]
            L.ccq_decode.restype = ctypes.c_int
            L.ccq_prep.argtypes = [SP] + [P] * 8
            L.ccq_prep.restype = ctypes.c_int
            L.ccq_fwd_raw_workspace_size.argtypes = [SP, ctypes.c_int]
            L.ccq_fwd_raw_workspace_size.restype = S
            L.ccq_fwd_raw.argtypes = [SP, ctypes.c_int] + [P] * 15 + [P, S, P]
            L.ccq_fwd_raw.restype = ctypes.c_int
            L.ccq_trace_events.argtypes = [P, ctypes.c_int]
            L.ccq_trace_events.restype = ctypes.c_int
            L.ccq_status_string.argtypes = [ctypes.c_int]
            L.ccq_status_string.restype = ctypes.c_char_p
            L.ccq_version.argtypes = []
            L.ccq_version.restype = ctypes.c_char_p
            _lib = L
    return _lib


def ccq_status_string(code: int) -> str:
    return lib().ccq_status_string(int(code)).decode()


def ccq_version() -> str:
    return lib().ccq_version().decode()


def ccq_trace_events(events) -> None:
    """Per-kernel timing hook: `events` is a list of torch.cuda.Event(enable_timing=True)
    (2 per kernel: before, after) or None to switch tracing off.  The caller keeps the
    list alive while tracing is on."""
    if not events:
        rc = lib().ccq_trace_events(None, 0)
    else:
        for e in events:
            e.record() if e.cuda_event == 0 else None  # make sure the event exists
        arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        ccq_trace_events._keep = arr
        rc = lib().ccq_trace_events(ctypes.cast(arr, ctypes.c_void_p), len(events))
    if rc != 0:
        raise CcqError("ccq_trace_events", rc)


def _dt(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return CCQ_BF16
    if t == torch.float32:
        return CCQ_F32
    raise TypeError("unsupported dtype %s (float32 or bfloat16)" % t)


def make_shape(B, T, H, dk, dv, io_dtype, gate_dtype=None, scale=1.0, centered=True, t0=0,
               chunk=64, decay_aligned=False) -> Shape:
    gd = io_dtype if gate_dtype is None else gate_dtype
    return Shape(int(B), int(T), int(H), int(dk), int(dv), int(chunk), _dt(io_dtype), _dt(gd),
                 float(scale), int(bool(centered)), int(bool(decay_aligned)), int(t0))


def ccq_workspace_size(shape: Shape, backbone: int, with_bwd: bool = False) -> int:
    return int(lib().ccq_workspace_size(ctypes.byref(shape), int(backbone), int(bool(with_bwd))))


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _record(stream, *objs):
    """Tensors the binding allocated on torch's current stream but handed to the
    library on another stream `stream`: mark them as used there, so that the caching
    allocator does not give their memory to a later allocation on the current stream
    while the library's kernels on `stream` may still use it (the workspace is freed
    when the call returns)."""
    if stream is None:
        return
    for o in objs:
        for t in (o.values() if isinstance(o, dict) else (o,)):
            if isinstance(t, torch.Tensor) and t.is_cuda and \
                    stream != torch.cuda.current_stream(t.device):
                t.record_stream(stream)


def _check(t, name, shape, dtype, device):
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s: shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if t.dtype != dtype:
        raise TypeError("%s: dtype %s, expected %s" % (name, t.dtype, dtype))
    if t.device != device:
        raise ValueError("%s: on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _workspace(shape, backbone, with_bwd, workspace, device):
    need = ccq_workspace_size(shape, backbone, with_bwd)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    return workspace, need


def _fwd(backbone, q, k, v, gate, lam, beta, S0, C0, mu0, scale, centered, t0, chunk,
         want_states, want_qclean, out, workspace, stream, decay_aligned=False):
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    gate_dtype = gate.dtype if backbone == CCQ_GLA else q.dtype
    shape = make_shape(B, T, H, dk, dv, q.dtype, gate_dtype, scale, centered, t0, chunk,
                       decay_aligned)
    _check(k, "k", (B, T, H, dk), q.dtype, dev)
    _check(v, "v", (B, T, H, dv), q.dtype, dev)
    if backbone == CCQ_GLA:
        _check(gate, "g", (B, T, H, dk), gate.dtype, dev)
    else:
        _check(gate, "logalpha", (B, T, H), torch.float32, dev)
        _check(beta, "beta", (B, T, H), torch.float32, dev)
    _check(lam, "lam", (B, T, H), torch.float32, dev)
    _check(S0, "S0", (B, H, dv, dk), torch.float32, dev)
    _check(C0, "C0", (B, H, dk, dk), torch.float32, dev)
    _check(mu0, "mu0", (B, H, dk), torch.float32, dev)
    out = dict(out or {})
    if "o" not in out:
        out["o"] = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    if want_states:
        out.setdefault("ST", torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev))
        out.setdefault("CT", torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev))
        out.setdefault("muT", torch.empty((B, H, dk), dtype=torch.float32, device=dev))
    if want_qclean:
        out.setdefault("qclean", torch.empty((B, T, H, dk), dtype=torch.float32, device=dev))
    workspace, need = _workspace(shape, backbone, False, workspace, dev)
    st = _stream(stream)
    if backbone == CCQ_GLA:
        rc = lib().ccq_gla_fwd(ctypes.byref(shape), _p(q), _p(k), _p(v), _p(gate), _p(lam),
                               _p(S0), _p(C0), _p(mu0), _p(out["o"]), _p(out.get("ST")),
                               _p(out.get("CT")), _p(out.get("muT")), _p(out.get("qclean")),
                               _p(workspace), workspace.numel(), st)
        fn = "ccq_gla_fwd"
    else:
        rc = lib().ccq_gdn_fwd(ctypes.byref(shape), _p(q), _p(k), _p(v), _p(gate), _p(beta),
                               _p(lam), _p(S0), _p(C0), _p(mu0), _p(out["o"]),
                               _p(out.get("ST")), _p(out.get("CT")), _p(out.get("muT")),
                               _p(out.get("qclean")), _p(workspace), workspace.numel(), st)
        fn = "ccq_gdn_fwd"
    _record(stream, workspace, out)
    if rc != 0:
        raise CcqError(fn, rc)
    return out


def ccq_gla_fwd(q, k, v, g, lam, S0=None, C0=None, mu0=None, scale=1.0, centered=True, t0=0,
                chunk=64, want_states=True, want_qclean=False, out=None, workspace=None,
                stream=None):
    """CCQ-GLA chunkwise forward.  Returns dict o[, ST, CT, muT][, qclean]."""
    return _fwd(CCQ_GLA, q, k, v, g, lam, None, S0, C0, mu0, scale, centered, t0, chunk,
                want_states, want_qclean, out, workspace, stream)


def ccq_gdn_fwd(q, k, v, logalpha, beta, lam, S0=None, C0=None, mu0=None, scale=1.0,
                centered=True, t0=0, chunk=64, want_states=True, want_qclean=False, out=None,
                workspace=None, stream=None, decay_aligned=False):
    """CCQ-Gated-DeltaNet chunkwise forward.  Returns dict o[, ST, CT, muT][, qclean].
    decay_aligned=True: the decay-aligned statistics (ccq_shape.decay_aligned)."""
    return _fwd(CCQ_GDN, q, k, v, logalpha, lam, beta, S0, C0, mu0, scale, centered, t0, chunk,
                want_states, want_qclean, out, workspace, stream, decay_aligned)


# CCQ_NOALLOC_SCRATCH_BYTES of include/ccq.h
NOALLOC_SCRATCH_BYTES = 64 << 20


def ccq_gdn_fwd_noalloc(q, k, v, logalpha, beta, lam, S0=None, C0=None, mu0=None, scale=1.0,
                        centered=True, t0=0, chunk=64, want_states=True, want_qclean=False,
                        out=None, stream=None):
    """CCQ-Gated-DeltaNet forward without a workspace: the library's own per-device
    scratch (CCQ_NOALLOC_SCRATCH_BYTES) serves the kernels.  The binding allocates
    only the outputs it is not given; pass every output in `out` to allocate nothing.
    Returns dict o[, ST, CT, muT][, qclean]."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    shape = make_shape(B, T, H, dk, dv, q.dtype, q.dtype, scale, centered, t0, chunk)
    _check(k, "k", (B, T, H, dk), q.dtype, dev)
    _check(v, "v", (B, T, H, dv), q.dtype, dev)
    _check(logalpha, "logalpha", (B, T, H), torch.float32, dev)
    _check(beta, "beta", (B, T, H), torch.float32, dev)
    _check(lam, "lam", (B, T, H), torch.float32, dev)
    _check(S0, "S0", (B, H, dv, dk), torch.float32, dev)
    _check(C0, "C0", (B, H, dk, dk), torch.float32, dev)
    _check(mu0, "mu0", (B, H, dk), torch.float32, dev)
    out = dict(out or {})
    if "o" not in out:
        out["o"] = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    if want_states:
        out.setdefault("ST", torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev))
        out.setdefault("CT", torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev))
        out.setdefault("muT", torch.empty((B, H, dk), dtype=torch.float32, device=dev))
    if want_qclean:
        out.setdefault("qclean", torch.empty((B, T, H, dk), dtype=torch.float32, device=dev))
    rc = lib().ccq_gdn_fwd_noalloc(ctypes.byref(shape), _p(q), _p(k), _p(v), _p(logalpha),
                                   _p(beta), _p(lam), _p(S0), _p(C0), _p(mu0), _p(out["o"]),
                                   _p(out.get("ST")), _p(out.get("CT")), _p(out.get("muT")),
                                   _p(out.get("qclean")), _stream(stream))
    _record(stream, out)
    if rc != 0:
        raise CcqError("ccq_gdn_fwd_noalloc", rc)
    return out


def ccq_fwd_bwd(q, k, v, g, lam, dO, scale=1.0, centered=True, chunk=64, out=None,
                workspace=None, stream=None, backbone=CCQ_GLA, beta=None):
    """CCQ training step: o and the gradients of sum <dO, o>.

    GLA: g is the log-forget gate [B,T,H,dk]; returns dict o, dq, dk, dv, dg, dlam.
    Gated DeltaNet (backbone=CCQ_GDN): g is log alpha [B,T,H] fp32 and beta
    [B,T,H] fp32 is required; returns o, dq, dk, dv, dg (= d log alpha), dbeta,
    dlam."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    gate_dtype = g.dtype if backbone == CCQ_GLA else q.dtype
    shape = make_shape(B, T, H, dk, dv, q.dtype, gate_dtype, scale, centered, 0, chunk)
    if backbone == CCQ_GLA:
        _check(g, "g", (B, T, H, dk), g.dtype, dev)
    else:
        if beta is None:
            raise ValueError("beta is required for the Gated DeltaNet training step")
        _check(g, "logalpha", (B, T, H), torch.float32, dev)
        _check(beta, "beta", (B, T, H), torch.float32, dev)
    _check(k, "k", (B, T, H, dk), q.dtype, dev)
    _check(v, "v", (B, T, H, dv), q.dtype, dev)
    _check(dO, "dO", (B, T, H, dv), q.dtype, dev)
    _check(lam, "lam", (B, T, H), torch.float32, dev)
    out = dict(out or {})
    out.setdefault("o", torch.empty((B, T, H, dv), dtype=q.dtype, device=dev))
    out.setdefault("dq", torch.empty((B, T, H, dk), dtype=q.dtype, device=dev))
    out.setdefault("dk", torch.empty((B, T, H, dk), dtype=q.dtype, device=dev))
    out.setdefault("dv", torch.empty((B, T, H, dv), dtype=q.dtype, device=dev))
    out.setdefault("dg", torch.empty(tuple(g.shape), dtype=g.dtype, device=dev))
    out.setdefault("dlam", torch.empty((B, T, H), dtype=torch.float32, device=dev))
    if backbone == CCQ_GDN:
        out.setdefault("dbeta", torch.empty((B, T, H), dtype=torch.float32, device=dev))
    workspace, need = _workspace(shape, backbone, True, workspace, dev)
    rc = lib().ccq_fwd_bwd(ctypes.byref(shape), int(backbone), _p(q), _p(k), _p(v), _p(g),
                           _p(beta), _p(lam), _p(dO), _p(out["o"]), _p(out["dq"]),
                           _p(out["dk"]), _p(out["dv"]), _p(out["dg"]), _p(out.get("dbeta")),
                           _p(out["dlam"]), _p(workspace), workspace.numel(), _stream(stream))
    _record(stream, workspace, out)
    if rc != 0:
        raise CcqError("ccq_fwd_bwd", rc)
    return out


def ccq_varlen_workspace_size(shape: Shape, backbone: int, with_bwd: bool = False) -> int:
    return int(lib().ccq_varlen_workspace_size(ctypes.byref(shape), int(backbone),
                                               int(bool(with_bwd))))


def _varlen_shape(backbone, q, v, gate, cu_seqlens, max_len, scale, centered, t0,
                  decay_aligned=False):
    if cu_seqlens.dtype != torch.int32 or cu_seqlens.dim() != 1 or cu_seqlens.numel() < 1:
        raise TypeError("cu_seqlens must be a 1-D int32 tensor of B + 1 offsets")
    if cu_seqlens.device != q.device or not cu_seqlens.is_contiguous():
        raise ValueError("cu_seqlens must be contiguous on the device of q")
    rows, H, dk = q.shape
    B = cu_seqlens.numel() - 1
    gate_dtype = gate.dtype if backbone == CCQ_GLA else q.dtype
    return make_shape(B, max_len, H, dk, v.shape[-1], q.dtype, gate_dtype, scale, centered, t0,
                      decay_aligned=decay_aligned)


def _varlen_ws(shape, backbone, with_bwd, workspace, device):
    need = ccq_varlen_workspace_size(shape, backbone, with_bwd)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    return workspace


def _varlen_fwd(backbone, q, k, v, gate, beta, lam, cu_seqlens, max_len, S0, C0, mu0, scale,
                centered, t0, want_states, out, workspace, stream, decay_aligned=False):
    rows, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    shape = _varlen_shape(backbone, q, v, gate, cu_seqlens, max_len, scale, centered, t0,
                          decay_aligned)
    B = shape.B
    _check(k, "k", (rows, H, dk), q.dtype, dev)
    _check(v, "v", (rows, H, dv), q.dtype, dev)
    if backbone == CCQ_GLA:
        _check(gate, "g", (rows, H, dk), gate.dtype, dev)
    else:
        if beta is None:
            raise ValueError("beta is required for Gated DeltaNet")
        _check(gate, "logalpha", (rows, H), torch.float32, dev)
        _check(beta, "beta", (rows, H), torch.float32, dev)
    _check(lam, "lam", (rows, H), torch.float32, dev)
    _check(S0, "S0", (B, H, dv, dk), torch.float32, dev)
    _check(C0, "C0", (B, H, dk, dk), torch.float32, dev)
    _check(mu0, "mu0", (B, H, dk), torch.float32, dev)
    out = dict(out or {})
    out.setdefault("o", torch.empty((rows, H, dv), dtype=q.dtype, device=dev))
    if want_states:
        out.setdefault("ST", torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev))
        out.setdefault("CT", torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev))
        out.setdefault("muT", torch.empty((B, H, dk), dtype=torch.float32, device=dev))
    workspace = _varlen_ws(shape, backbone, False, workspace, dev)
    st = _stream(stream)
    if backbone == CCQ_GLA:
        rc = lib().ccq_gla_fwd_varlen(ctypes.byref(shape), _p(cu_seqlens), _p(q), _p(k), _p(v),
                                      _p(gate), _p(lam), _p(S0), _p(C0), _p(mu0), _p(out["o"]),
                                      _p(out.get("ST")), _p(out.get("CT")), _p(out.get("muT")),
                                      _p(workspace), workspace.numel(), st)
        fn = "ccq_gla_fwd_varlen"
    else:
        rc = lib().ccq_gdn_fwd_varlen(ctypes.byref(shape), _p(cu_seqlens), _p(q), _p(k), _p(v),
                                      _p(gate), _p(beta), _p(lam), _p(S0), _p(C0), _p(mu0),
                                      _p(out["o"]), _p(out.get("ST")), _p(out.get("CT")),
                                      _p(out.get("muT")), _p(workspace), workspace.numel(), st)
        fn = "ccq_gdn_fwd_varlen"
    _record(stream, workspace, out)
    if rc != 0:
        raise CcqError(fn, rc)
    return out


def ccq_gla_fwd_varlen(q, k, v, g, lam, cu_seqlens, max_len, S0=None, C0=None, mu0=None,
                       scale=1.0, centered=True, t0=0, want_states=True, out=None,
                       workspace=None, stream=None):
    """CCQ-GLA forward on a packed batch: q, k, g [rows,H,dk], v [rows,H,dv], lam
    [rows,H]; sequence b is rows cu_seqlens[b]..cu_seqlens[b+1]-1 (int32 device
    tensor of B + 1 offsets), at most max_len rows long.  Returns dict o
    [rows,H,dv][, ST, CT, muT per sequence]."""
    return _varlen_fwd(CCQ_GLA, q, k, v, g, None, lam, cu_seqlens, max_len, S0, C0, mu0, scale,
                       centered, t0, want_states, out, workspace, stream)


def ccq_gdn_fwd_varlen(q, k, v, logalpha, beta, lam, cu_seqlens, max_len, S0=None, C0=None,
                       mu0=None, scale=1.0, centered=True, t0=0, want_states=True, out=None,
                       workspace=None, stream=None, decay_aligned=False):
    """CCQ-Gated-DeltaNet forward on a packed batch (layout as ccq_gla_fwd_varlen;
    logalpha, beta [rows,H] fp32).  decay_aligned as ccq_gdn_fwd."""
    return _varlen_fwd(CCQ_GDN, q, k, v, logalpha, beta, lam, cu_seqlens, max_len, S0, C0, mu0,
                       scale, centered, t0, want_states, out, workspace, stream, decay_aligned)


def ccq_fwd_bwd_varlen(q, k, v, g, lam, dO, cu_seqlens, max_len, scale=1.0, centered=True,
                       out=None, workspace=None, stream=None, backbone=CCQ_GLA, beta=None):
    """Training step on a packed batch (layout as ccq_gla_fwd_varlen; dO [rows,H,dv]).
    Returns the same dict as ccq_fwd_bwd, packed."""
    rows, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    shape = _varlen_shape(backbone, q, v, g, cu_seqlens, max_len, scale, centered, 0)
    if backbone == CCQ_GLA:
        _check(g, "g", (rows, H, dk), g.dtype, dev)
    else:
        if beta is None:
            raise ValueError("beta is required for the Gated DeltaNet training step")
        _check(g, "logalpha", (rows, H), torch.float32, dev)
        _check(beta, "beta", (rows, H), torch.float32, dev)
    _check(k, "k", (rows, H, dk), q.dtype, dev)
    _check(v, "v", (rows, H, dv), q.dtype, dev)
    _check(dO, "dO", (rows, H, dv), q.dtype, dev)
    _check(lam, "lam", (rows, H), torch.float32, dev)
    out = dict(out or {})
    out.setdefault("o", torch.empty((rows, H, dv), dtype=q.dtype, device=dev))
    out.setdefault("dq", torch.empty((rows, H, dk), dtype=q.dtype, device=dev))
    out.setdefault("dk", torch.empty((rows, H, dk), dtype=q.dtype, device=dev))
    out.setdefault("dv", torch.empty((rows, H, dv), dtype=q.dtype, device=dev))
    out.setdefault("dg", torch.empty(tuple(g.shape), dtype=g.dtype, device=dev))
    out.setdefault("dlam", torch.empty((rows, H), dtype=torch.float32, device=dev))
    if backbone == CCQ_GDN:
        out.setdefault("dbeta", torch.empty((rows, H), dtype=torch.float32, device=dev))
    workspace = _varlen_ws(shape, backbone, True, workspace, dev)
    rc = lib().ccq_fwd_bwd_varlen(ctypes.byref(shape), int(backbone), _p(cu_seqlens), _p(q),
                                  _p(k), _p(v), _p(g), _p(beta), _p(lam), _p(dO), _p(out["o"]),
                                  _p(out["dq"]), _p(out["dk"]), _p(out["dv"]), _p(out["dg"]),
                                  _p(out.get("dbeta")), _p(out["dlam"]), _p(workspace),
                                  workspace.numel(), _stream(stream))
    _record(stream, workspace, out)
    if rc != 0:
        raise CcqError("ccq_fwd_bwd_varlen", rc)
    return out


def ccq_decode_workspace_size(shape: Shape) -> int:
    return int(lib().ccq_decode_workspace_size(ctypes.byref(shape)))


def ccq_decode(q, k, v, gate, lam, S, C, mu, t0, backbone=CCQ_GLA, beta=None, scale=1.0,
               centered=True, out=None, workspace=None, stream=None):
    """One recurrent CCQ step per sequence (Alg. 2) on the cache (S, C, mu), which is
    updated in place.  q, k [B,H,dk] and v [B,H,dv] (one token); GLA gate [B,H,dk],
    Gated DeltaNet log alpha [B,H] fp32 plus beta [B,H] fp32; lam [B,H] fp32;
    S [B,H,dv,dk], C [B,H,dk,dk], mu [B,H,dk] fp32; t0 = tokens already absorbed.
    Returns o [B,H,dv]."""
    B, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    gate_dtype = gate.dtype if backbone == CCQ_GLA else q.dtype
    shape = make_shape(B, 1, H, dk, dv, q.dtype, gate_dtype, scale, centered, t0)
    _check(k, "k", (B, H, dk), q.dtype, dev)
    _check(v, "v", (B, H, dv), q.dtype, dev)
    _check(lam, "lam", (B, H), torch.float32, dev)
    if backbone == CCQ_GLA:
        _check(gate, "g", (B, H, dk), gate.dtype, dev)
    else:
        if beta is None:
            raise ValueError("beta is required for Gated DeltaNet")
        _check(gate, "logalpha", (B, H), torch.float32, dev)
        _check(beta, "beta", (B, H), torch.float32, dev)
    for t, name, shp in ((S, "S", (B, H, dv, dk)), (C, "C", (B, H, dk, dk)), (mu, "mu", (B, H, dk))):
        if t is None:
            raise ValueError("%s (the cache) is required" % name)
        _check(t, name, shp, torch.float32, dev)
    o = out if out is not None else torch.empty((B, H, dv), dtype=q.dtype, device=dev)
    _check(o, "o", (B, H, dv), q.dtype, dev)
    need = ccq_decode_workspace_size(shape)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    rc = lib().ccq_decode(ctypes.byref(shape), int(backbone), _p(q), _p(k), _p(v), _p(gate),
                          _p(beta), _p(lam), _p(S), _p(C), _p(mu), _p(o), _p(workspace),
                          0 if workspace is None else workspace.numel(), _stream(stream))
    _record(stream, workspace, o)
    if rc != 0:
        raise CcqError("ccq_decode", rc)
    return o


def ccq_prep(q_raw, k_raw, w_lam, b_lam, out=None, stream=None):
    """Per-head l2 normalisation of raw q, k [B,T,H,dk] and the gate
    lam = sigmoid(w_lam qraw + b_lam) [B,T,H] from the token's query before the head
    split (w_lam [H, H*dk] fp32, b_lam [H] fp32).  Returns dict q, k, lam; pass
    out=dict(q=q_raw, k=k_raw) to normalise in place."""
    B, T, H, dk = q_raw.shape
    dev = q_raw.device
    _check(k_raw, "k_raw", (B, T, H, dk), q_raw.dtype, dev)
    _check(w_lam, "w_lam", (H, H * dk), torch.float32, dev)
    _check(b_lam, "b_lam", (H,), torch.float32, dev)
    out = dict(out or {})
    out.setdefault("q", torch.empty_like(q_raw))
    out.setdefault("k", torch.empty_like(k_raw))
    out.setdefault("lam", torch.empty((B, T, H), dtype=torch.float32, device=dev))
    shape = make_shape(B, T, H, dk, dk, q_raw.dtype)
    rc = lib().ccq_prep(ctypes.byref(shape), _p(q_raw), _p(k_raw), _p(w_lam), _p(b_lam),
                        _p(out["q"]), _p(out["k"]), _p(out["lam"]), _stream(stream))
    _record(stream, out)
    if rc != 0:
        raise CcqError("ccq_prep", rc)
    return out


def ccq_fwd_raw_workspace_size(shape: Shape, backbone: int) -> int:
    return int(lib().ccq_fwd_raw_workspace_size(ctypes.byref(shape), int(backbone)))


def ccq_fwd_raw(q_raw, k_raw, w_lam, b_lam, v, gate, beta=None, backbone=CCQ_GLA, S0=None, C0=None,
                mu0=None, scale=1.0, centered=True, t0=0, chunk=64, want_states=True,
                want_lam=False, out=None, workspace=None, stream=None):
    """Forward from raw q, k [B,T,H,dk]: the l2 normalisation and the gate
    lam = sigmoid(w_lam qraw + b_lam) (w_lam [H, H*dk], b_lam [H] fp32) folded into the
    forward.  gate: the GLA log-forget gate [B,T,H,dk], or Gated DeltaNet log alpha
    [B,T,H] fp32 with beta [B,T,H] fp32.  Returns dict o[, ST, CT, muT][, lam]."""
    B, T, H, dk = q_raw.shape
    dv = v.shape[-1]
    dev = q_raw.device
    gate_dtype = gate.dtype if backbone == CCQ_GLA else q_raw.dtype
    shape = make_shape(B, T, H, dk, dv, q_raw.dtype, gate_dtype, scale, centered, t0, chunk)
    _check(k_raw, "k_raw", (B, T, H, dk), q_raw.dtype, dev)
    _check(v, "v", (B, T, H, dv), q_raw.dtype, dev)
    _check(w_lam, "w_lam", (H, H * dk), torch.float32, dev)
    _check(b_lam, "b_lam", (H,), torch.float32, dev)
    if backbone == CCQ_GLA:
        _check(gate, "g", (B, T, H, dk), gate.dtype, dev)
    else:
        if beta is None:
            raise ValueError("beta is required for Gated DeltaNet")
        _check(gate, "logalpha", (B, T, H), torch.float32, dev)
        _check(beta, "beta", (B, T, H), torch.float32, dev)
    _check(S0, "S0", (B, H, dv, dk), torch.float32, dev)
    _check(C0, "C0", (B, H, dk, dk), torch.float32, dev)
    _check(mu0, "mu0", (B, H, dk), torch.float32, dev)
    out = dict(out or {})
    out.setdefault("o", torch.empty((B, T, H, dv), dtype=q_raw.dtype, device=dev))
    if want_states:
        out.setdefault("ST", torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev))
        out.setdefault("CT", torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev))
        out.setdefault("muT", torch.empty((B, H, dk), dtype=torch.float32, device=dev))
    if want_lam:
        out.setdefault("lam", torch.empty((B, T, H), dtype=torch.float32, device=dev))
    need = ccq_fwd_raw_workspace_size(shape, backbone)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lib().ccq_fwd_raw(ctypes.byref(shape), int(backbone), _p(q_raw), _p(k_raw), _p(w_lam),
                           _p(b_lam), _p(v), _p(gate), _p(beta), _p(S0), _p(C0), _p(mu0),
                           _p(out["o"]), _p(out.get("ST")), _p(out.get("CT")), _p(out.get("muT")),
                           _p(out.get("lam")), _p(workspace), workspace.numel(), _stream(stream))
    _record(stream, workspace, out)
    if rc != 0:
        raise CcqError("ccq_fwd_raw", rc)
    return out
