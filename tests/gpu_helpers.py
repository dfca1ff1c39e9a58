"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and measure errors.

Two error measures are computed per output tensor:
  nerr       max |gpu - ref| / max |ref|                 (the asserted bar)
  elem_err   max |gpu - ref| / (|ref| + 0.01 max |ref|)  (element-wise, floored;
             reported so that errors in small-magnitude entries stay visible)
"""
import numpy as np
import torch

from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, GLA, make_inputs, to_device, to_f64

# max |gpu - ref| / max |ref| per output tensor
TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}
ELEM_FLOOR = 0.01


def nerr(gpu, ref):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(gpu))) if gpu.size else 0.0
    return float(np.max(np.abs(gpu - ref)) / den)


def elem_err(gpu, ref, floor=ELEM_FLOOR):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if not ref.size:
        return 0.0
    den = np.abs(ref) + floor * np.max(np.abs(ref))
    if not np.all(den > 0):
        return float(np.max(np.abs(gpu - ref)))
    return float(np.max(np.abs(gpu - ref) / den))


def np64(t):
    return t.detach().double().cpu().numpy()


def gpu_fwd(backbone, d, **kw):
    """Run the HIP path on device copies of the input dict d (CPU tensors)."""
    g = to_device(d)
    if backbone == GLA:
        out = ccq.ccq_gla_fwd(g["q"], g["k"], g["v"], g["g"], g["lam"], want_qclean=True, **kw)
    else:
        out = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                              want_qclean=True, **kw)
    torch.cuda.synchronize()
    return {k: np64(v) for k, v in out.items()}


def oracle_fwd(backbone, d, **kw):
    f = to_f64(d)
    if backbone == GLA:
        return O.fwd(f["q"], f["k"], f["v"], f["g"], f["lam"], backbone=O.GLA, **kw)
    return O.fwd(f["q"], f["k"], f["v"], f["logalpha"], f["lam"], beta=f["beta"],
                 backbone=O.GDN, **kw)


def fwd_errors(gout, ref, q, states=True, sl=(slice(None),) * 4):
    """Errors of o, the final states and the correction lambda_t Sigma_t q_t (from the
    fp32 q_clean export) for the token/state slices sl = (b, h) index pair of slices."""
    b, h = sl[0], sl[1]
    errs = {"o": nerr(gout["o"][b, :, h], ref["o"])}
    elem = {"o": elem_err(gout["o"][b, :, h], ref["o"])}
    if states:
        for key in ("ST", "CT", "muT"):
            errs[key] = nerr(gout[key][b, h], ref[key])
    errs["corr"] = nerr(q - gout["qclean"][b, :, h], q - ref["qclean"])
    elem["corr"] = elem_err(q - gout["qclean"][b, :, h], q - ref["qclean"])
    return errs, elem


def compare(backbone, d, dtype, tol=None, states=True, **kw):
    """Element-wise comparison of o, the final states and the correction term."""
    tol = TOL[dtype] if tol is None else tol
    kw_t = {k: (torch.from_numpy(np.ascontiguousarray(v)).float().cuda()
                if isinstance(v, np.ndarray) else v) for k, v in kw.items()}
    gout = gpu_fwd(backbone, d, **kw_t)
    ref = oracle_fwd(backbone, d, **kw)
    q = to_f64(d)["q"]
    errs, elem = fwd_errors(gout, ref, q, states)
    print("  errors", errs, "element-wise", elem, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, "errors above %g: %s (all: %s)" % (tol, bad, errs)
    return errs, gout, ref
