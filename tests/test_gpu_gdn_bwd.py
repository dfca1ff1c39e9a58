"""Parity of the CCQ-Gated DeltaNet training step (ccq_fwd_bwd through the C ABI)
with the fp64 oracle's reverse pass (itself pinned by finite differences on the
CPU).

Same bar as the forward: max |gpu - ref| / max |ref| <= 1e-4 (fp32 io) or
<= 2e-2 (bf16 io) for o, dq, dk, dv, dlogalpha, dbeta and dlam.
"""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, elem_err, nerr, np64
from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, WORKLOADS, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu
F32, BF16 = torch.float32, torch.bfloat16
KEYS = ("o", "dq", "dk", "dv", "dlogalpha", "dbeta", "dlam")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_gpu(d, **kw):
    g = to_device(d)
    out = ccq.ccq_fwd_bwd(g["q"], g["k"], g["v"], g["logalpha"], g["lam"], g["dO"],
                          backbone=ccq.CCQ_GDN, beta=g["beta"], **kw)
    torch.cuda.synchronize()
    res = {k: np64(v) for k, v in out.items()}
    res["dlogalpha"] = res.pop("dg")
    return res


def run_oracle(d, **kw):
    f = to_f64(d)
    return O.gdn_fwd_bwd(f["q"], f["k"], f["v"], f["logalpha"], f["beta"], f["lam"], f["dO"],
                         **kw)


def check(d, dtype, tol=None, **kw):
    tol = TOL[dtype] if tol is None else tol
    gout = run_gpu(d, **kw)
    ref = run_oracle(d, **kw)
    errs = {key: nerr(gout[key], ref[key]) for key in KEYS}
    say("  errors", errs)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, "errors above %g: %s" % (tol, errs)
    return gout, ref


CASES = [
    # dtype, B, T, H, dk, dv, keys, lam
    (F32, 1, 256, 2, 64, 64, "iso", "const"),
    (F32, 1, 150, 2, 64, 128, "aniso", "random"),
    (BF16, 1, 200, 2, 128, 256, "iso", "random"),
    (BF16, 2, 130, 2, 64, 64, "aniso", "random"),
    (BF16, 1, 97, 1, 128, 512, "meanshift", "random"),
    (BF16, 1, 64, 2, 128, 128, "iso", "const"),
    (BF16, 1, 3, 2, 64, 64, "iso", "random"),
    (BF16, 3, 330, 3, 128, 64, "iso", "random"),
    # dk = 256, the 1.3B layer's head size
    (BF16, 1, 200, 2, 256, 256, "iso", "random"),
    (BF16, 2, 130, 2, 256, 128, "aniso", "random"),
    (BF16, 1, 97, 1, 256, 512, "meanshift", "random"),
    (BF16, 1, 3, 2, 256, 64, "iso", "const"),
    (BF16, 1, 600, 1, 256, 256, "aniso", "random"),
]


# The reverse state scan at dk = 256 splits value slices by how many there are
# (B * H * dv / 16): >= 2048 (four tiles per workgroup), >= 1024 (two), fewer
# (two, each over two waves); these shapes reach the first two, the cases above
# the third.
@pytest.mark.parametrize("B,H", [(8, 16), (4, 16)])
def test_gdn_fwd_bwd_dk256_state_splits(B, H):
    say("gdn fwd_bwd dk256 split", B, H)
    d = make_inputs(GDN, B, 70, H, 256, 256, BF16, seed=500 + B * H, keys="aniso", lam="random",
                    with_dO=True)
    check(d, BF16)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-B%d-T%d-dk%d-dv%d-%s" % (
    str(c[0]).split(".")[-1], c[1], c[2], c[4], c[5], c[6]))
def test_gdn_fwd_bwd_small(case):
    dtype, B, T, H, dk, dv, keys, lam = case
    say("gdn fwd_bwd", case)
    d = make_inputs(GDN, B, T, H, dk, dv, dtype, seed=400 + T, keys=keys, lam=lam, with_dO=True)
    check(d, dtype)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_gdn_fwd_bwd_uncentred_scaled(dtype):
    say("gdn fwd_bwd uncentred/scaled", dtype)
    d = make_inputs(GDN, 1, 170, 2, 64, 128, dtype, seed=27, lam="random", with_dO=True)
    check(d, dtype, centered=False, scale=0.25)


def test_gdn_fwd_bwd_matches_forward_entry_point():
    """The training step's o equals ccq_gdn_fwd's o bit for bit (same kernels)."""
    d = make_inputs(GDN, 2, 190, 2, 128, 256, BF16, seed=29, lam="random", with_dO=True)
    g = to_device(d)
    a = ccq.ccq_fwd_bwd(g["q"], g["k"], g["v"], g["logalpha"], g["lam"], g["dO"],
                        backbone=ccq.CCQ_GDN, beta=g["beta"])
    b = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"])
    torch.cuda.synchronize()
    assert torch.equal(a["o"], b["o"])


def test_gdn_fwd_bwd_deterministic():
    d = make_inputs(GDN, 1, 300, 2, 128, 256, BF16, seed=31, lam="random", with_dO=True)
    a, b = run_gpu(d), run_gpu(d)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])



def full_size_all_heads(w, d):
    """Every (batch, head) sequence of the training workload, each normalised by its own
    reference; the worst errors are printed with their element-wise counterparts."""
    gout = run_gpu(d)
    ref = run_oracle(d)
    worst, worst_elem = {}, {}
    for b in range(w.B):
        for h in range(w.H):
            errs = {}
            for key in KEYS:
                gv, rv = gout[key][b:b + 1, :, h:h + 1], ref[key][b:b + 1, :, h:h + 1]
                errs[key] = nerr(gv, rv)
                worst_elem[key] = max(worst_elem.get(key, 0.0), elem_err(gv, rv))
            for key, v in errs.items():
                worst[key] = max(worst.get(key, 0.0), v)
            assert all(v <= TOL[w.dtype] for v in errs.values()), (b, h, errs)
    say("  %d sequences, worst" % (w.B * w.H), worst, "element-wise", worst_elem)


def test_gdn_fwd_bwd_full_size():
    """The Gated DeltaNet training workload as the benchmark runs it; the oracle
    recomputes every (batch, head) sequence."""
    w = WORKLOADS["gdn_train_t4k"]
    say("full size", w)
    d = make_inputs(GDN, w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=w.seed, with_dO=True)
    full_size_all_heads(w, d)
