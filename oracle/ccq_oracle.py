"""fp64 CPU oracle for Curvature-Conditioned Query (CCQ) -- test infrastructure.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It wraps ``ccq_oracle.c`` (plain C, fp64, OpenMP over
(batch, head) pairs) through ctypes and builds it with gcc on first use.  It
imports nothing from the HIP library and the HIP library imports nothing from
here.

Functions (all arrays are numpy float64, row-major):
  fwd(...)          token-by-token forward (form 0: raw sums; form 1: the
                    running-mean recurrence of Alg. 2)
  chunk_fwd(...)    Alg. 1 chunkwise forward with the GLA / Gated DeltaNet
                    chunk forms of the backbone update
  gla_fwd_bwd(...)  reverse pass of CCQ-GLA for L = sum <dO, o>
  gdn_fwd_bwd(...)  reverse pass of CCQ-Gated DeltaNet for L = sum <dO, o>
  prep(...)         per-head l2 normalisation of raw q, k and the gate
                    lambda = sigmoid(W qraw + b) from the query before the head split
  varlen_fwd(...), varlen_fwd_bwd(...)
                    packed batches: the per-sequence forward / reverse pass applied
                    to each sequence of the batch on its own
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ccq_oracle.c")
_LIB = os.path.join(_HERE, "libccq_oracle.so")
_lock = threading.Lock()
_lib = None

GLA, GDN = 0, 1


class Shape(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
        ("dk", ctypes.c_int32), ("dv", ctypes.c_int32),
        ("backbone", ctypes.c_int32), ("centered", ctypes.c_int32), ("decay", ctypes.c_int32),
        ("scale", ctypes.c_double), ("t0", ctypes.c_int64),
    ]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no fast-math) into libccq_oracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB)
            P = ctypes.c_void_p
            lib.ccq_oracle_fwd.argtypes = [ctypes.POINTER(Shape), ctypes.c_int] + [P] * 14
            lib.ccq_oracle_chunk_fwd.argtypes = [ctypes.POINTER(Shape), ctypes.c_int] + [P] * 14
            lib.ccq_oracle_gla_fwd_bwd.argtypes = [ctypes.POINTER(Shape), ctypes.c_int] + [P] * 12
            lib.ccq_oracle_gdn_fwd_bwd.argtypes = [ctypes.POINTER(Shape), ctypes.c_int] + [P] * 14
            lib.ccq_oracle_prep.argtypes = [ctypes.c_int32] * 4 + [P] * 7
            lib.ccq_oracle_prep.restype = ctypes.c_int
            for f in (lib.ccq_oracle_fwd, lib.ccq_oracle_chunk_fwd, lib.ccq_oracle_gla_fwd_bwd,
                      lib.ccq_oracle_gdn_fwd_bwd):
                f.restype = ctypes.c_int
            lib.ccq_oracle_threads.restype = ctypes.c_int
            _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle runs on."""
    return _load().ccq_oracle_threads()


def _f64(x):
    if x is None:
        return None
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _shape(q, v, backbone, centered, scale, t0, decay=False):
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    return Shape(B, T, H, dk, dv, backbone, int(centered), int(decay), float(scale), int(t0))


def _inputs(q, k, v, gate, beta, lam, backbone):
    q, k, v, gate, lam = _f64(q), _f64(k), _f64(v), _f64(gate), _f64(lam)
    beta = _f64(beta) if backbone == GDN else None
    B, T, H, dk = q.shape
    assert k.shape == q.shape and v.shape[:3] == (B, T, H) and lam.shape == (B, T, H)
    if backbone == GLA:
        assert gate.shape == q.shape
    else:
        assert gate.shape == (B, T, H) and beta.shape == (B, T, H)
    return q, k, v, gate, beta, lam


def _outputs(q, v):
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    return (np.zeros((B, T, H, dv)), np.zeros((B, H, dv, dk)), np.zeros((B, H, dk, dk)),
            np.zeros((B, H, dk)), np.zeros((B, T, H, dk)))


def fwd(q, k, v, gate, lam, beta=None, backbone=GLA, S0=None, C0=None, mu0=None,
        scale=1.0, centered=True, t0=0, form=0, decay=False):
    """Token-by-token CCQ forward.  Returns dict o, ST, CT, muT, qclean.
    decay=True (Gated DeltaNet, t0 = 0, no C0/mu0): the decay-aligned statistics,
    each key weighted by the product of the later alphas and t replaced by the
    decayed count W_t = alpha_t W_{t-1} + 1."""
    q, k, v, gate, beta, lam = _inputs(q, k, v, gate, beta, lam, backbone)
    S0, C0, mu0 = _f64(S0), _f64(C0), _f64(mu0)
    o, ST, CT, muT, qc = _outputs(q, v)
    sh = _shape(q, v, backbone, centered, scale, t0, decay)
    rc = _load().ccq_oracle_fwd(ctypes.byref(sh), int(form), _ptr(q), _ptr(k), _ptr(v), _ptr(gate),
                                _ptr(beta), _ptr(lam), _ptr(S0), _ptr(C0), _ptr(mu0), _ptr(o),
                                _ptr(ST), _ptr(CT), _ptr(muT), _ptr(qc))
    if rc != 0:
        raise RuntimeError("ccq_oracle_fwd failed with code %d" % rc)
    return dict(o=o, ST=ST, CT=CT, muT=muT, qclean=qc)


def chunk_fwd(q, k, v, gate, lam, beta=None, backbone=GLA, chunk=64, S0=None, C0=None,
              mu0=None, scale=1.0, centered=True, t0=0):
    """Alg. 1 chunkwise CCQ forward.  Returns dict o, ST, CT, muT, qclean."""
    q, k, v, gate, beta, lam = _inputs(q, k, v, gate, beta, lam, backbone)
    S0, C0, mu0 = _f64(S0), _f64(C0), _f64(mu0)
    o, ST, CT, muT, qc = _outputs(q, v)
    sh = _shape(q, v, backbone, centered, scale, t0)
    rc = _load().ccq_oracle_chunk_fwd(ctypes.byref(sh), int(chunk), _ptr(q), _ptr(k), _ptr(v),
                                      _ptr(gate), _ptr(beta), _ptr(lam), _ptr(S0), _ptr(C0),
                                      _ptr(mu0), _ptr(o), _ptr(ST), _ptr(CT), _ptr(muT), _ptr(qc))
    if rc != 0:
        raise RuntimeError("ccq_oracle_chunk_fwd failed with code %d" % rc)
    return dict(o=o, ST=ST, CT=CT, muT=muT, qclean=qc)


def gla_fwd_bwd(q, k, v, g, lam, dO, scale=1.0, centered=True, seg=64):
    """Reverse pass of CCQ-GLA (zero initial state).  Returns o, dq, dk, dv, dg, dlam."""
    q, k, v, g, _, lam = _inputs(q, k, v, g, None, lam, GLA)
    dO = _f64(dO)
    assert dO.shape == q.shape[:3] + (v.shape[-1],)
    o = np.zeros(dO.shape)
    dq, dk, dg = np.zeros(q.shape), np.zeros(q.shape), np.zeros(q.shape)
    dv = np.zeros(v.shape)
    dlam = np.zeros(lam.shape)
    sh = _shape(q, v, GLA, centered, scale, 0)
    rc = _load().ccq_oracle_gla_fwd_bwd(ctypes.byref(sh), int(seg), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(g), _ptr(lam), _ptr(dO), _ptr(o), _ptr(dq), _ptr(dk),
                                        _ptr(dv), _ptr(dg), _ptr(dlam))
    if rc != 0:
        raise RuntimeError("ccq_oracle_gla_fwd_bwd failed with code %d" % rc)
    return dict(o=o, dq=dq, dk=dk, dv=dv, dg=dg, dlam=dlam)


def gdn_fwd_bwd(q, k, v, logalpha, beta, lam, dO, scale=1.0, centered=True, seg=64):
    """Reverse pass of CCQ-Gated DeltaNet (zero initial state).  Returns o, dq, dk, dv,
    dlogalpha, dbeta, dlam."""
    q, k, v, logalpha, beta, lam = _inputs(q, k, v, logalpha, beta, lam, GDN)
    dO = _f64(dO)
    assert dO.shape == q.shape[:3] + (v.shape[-1],)
    o = np.zeros(dO.shape)
    dq, dk = np.zeros(q.shape), np.zeros(q.shape)
    dv = np.zeros(v.shape)
    dla, dbeta, dlam = np.zeros(lam.shape), np.zeros(lam.shape), np.zeros(lam.shape)
    sh = _shape(q, v, GDN, centered, scale, 0)
    rc = _load().ccq_oracle_gdn_fwd_bwd(ctypes.byref(sh), int(seg), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(logalpha), _ptr(beta), _ptr(lam), _ptr(dO), _ptr(o),
                                        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dla), _ptr(dbeta),
                                        _ptr(dlam))
    if rc != 0:
        raise RuntimeError("ccq_oracle_gdn_fwd_bwd failed with code %d" % rc)
    return dict(o=o, dq=dq, dk=dk, dv=dv, dlogalpha=dla, dbeta=dbeta, dlam=dlam)


def prep(q, k, W, b):
    """Raw q, k [B,T,H,dk], W [H, H*dk], b [H] -> dict q, k (per-head unit rows) and
    lam [B,T,H] = sigmoid(W qraw + b), qraw the token's query over all heads."""
    q, k, W, b = _f64(q), _f64(k), _f64(W), _f64(b)
    B, T, H, dk = q.shape
    assert k.shape == q.shape and W.shape == (H, H * dk) and b.shape == (H,)
    qb, kb, lam = np.zeros(q.shape), np.zeros(q.shape), np.zeros((B, T, H))
    rc = _load().ccq_oracle_prep(B, T, H, dk, _ptr(q), _ptr(k), _ptr(W), _ptr(b), _ptr(qb),
                                 _ptr(kb), _ptr(lam))
    if rc != 0:
        raise RuntimeError("ccq_oracle_prep failed with code %d" % rc)
    return dict(q=qb, k=kb, lam=lam)


def _seq_slices(cu):
    cu = [int(x) for x in np.asarray(cu).reshape(-1)]
    return [(cu[b], cu[b + 1]) for b in range(len(cu) - 1)]


def varlen_fwd(q, k, v, gate, lam, cu, beta=None, backbone=GLA, S0=None, C0=None, mu0=None,
               scale=1.0, centered=True, t0=0):
    """Forward of a packed batch: sequence b is rows cu[b]..cu[b+1]-1 of q, k
    [rows,H,dk], v [rows,H,dv], gate, lam (and beta); each runs through fwd on its
    own, from its own initial states.  Returns o [rows,H,dv] and the per-sequence
    ST, CT, muT."""
    q, k, v, gate, lam = _f64(q), _f64(k), _f64(v), _f64(gate), _f64(lam)
    beta = _f64(beta) if backbone == GDN else None
    rows, H, dk = q.shape
    dv = v.shape[-1]
    sl = _seq_slices(cu)
    B = len(sl)
    o = np.zeros((rows, H, dv))
    ST, CT, muT = np.zeros((B, H, dv, dk)), np.zeros((B, H, dk, dk)), np.zeros((B, H, dk))
    for b, (r0, r1) in enumerate(sl):
        init = [None if x is None else _f64(x)[b:b + 1] for x in (S0, C0, mu0)]
        if r1 == r0:
            ST[b] = 0.0 if init[0] is None else init[0][0]
            CT[b] = 0.0 if init[1] is None else init[1][0]
            muT[b] = 0.0 if init[2] is None else init[2][0]
            continue
        r = fwd(q[None, r0:r1], k[None, r0:r1], v[None, r0:r1], gate[None, r0:r1], lam[None, r0:r1],
                beta=None if beta is None else beta[None, r0:r1], backbone=backbone, S0=init[0],
                C0=init[1], mu0=init[2], scale=scale, centered=centered, t0=t0)
        o[r0:r1] = r["o"][0]
        ST[b], CT[b], muT[b] = r["ST"][0], r["CT"][0], r["muT"][0]
    return dict(o=o, ST=ST, CT=CT, muT=muT)


def varlen_fwd_bwd(q, k, v, gate, lam, dO, cu, beta=None, backbone=GLA, scale=1.0, centered=True):
    """Reverse pass of a packed batch (L = sum <dO, o>), each sequence on its own from
    zero states.  Returns packed o, dq, dk, dv, dg, dlam (and dbeta for Gated DeltaNet)."""
    arrs = {"q": _f64(q), "k": _f64(k), "v": _f64(v), "g": _f64(gate), "lam": _f64(lam),
            "dO": _f64(dO)}
    if backbone == GDN:
        arrs["beta"] = _f64(beta)
    keys = ("o", "dq", "dk", "dv", "dg", "dlam") + (("dbeta",) if backbone == GDN else ())
    like = {"o": "dO", "dq": "q", "dk": "k", "dv": "v", "dg": "g", "dlam": "lam", "dbeta": "lam"}
    out = {key: np.zeros_like(arrs[like[key]]) for key in keys}
    for r0, r1 in _seq_slices(cu):
        if r1 == r0:
            continue
        a = {n: x[None, r0:r1] for n, x in arrs.items()}
        if backbone == GLA:
            r = gla_fwd_bwd(a["q"], a["k"], a["v"], a["g"], a["lam"], a["dO"], scale=scale,
                            centered=centered)
        else:
            r = gdn_fwd_bwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["lam"], a["dO"],
                            scale=scale, centered=centered)
        for key in keys:
            out[key][r0:r1] = r["dlogalpha" if (key == "dg" and backbone == GDN) else key][0]
    return out
