"""Parity of the pre-processing kernel (ccq_prep through the C ABI) with the oracle's
(pinned on the CPU by unit norms, scale invariance and closed-form gates), and the
composed path: raw q, k -> ccq_prep -> chunkwise forward, against the oracle's
pre-processing followed by its forward.

Bar: max |gpu - ref| / max |ref| <= 1e-4 (fp32 io) or <= 2e-2 (bf16 io)."""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, nerr, np64
from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq

pytestmark = pytest.mark.gpu
F32, BF16 = torch.float32, torch.bfloat16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def raw_inputs(B, T, H, dk, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    q = (torch.randn(B, T, H, dk, generator=g) * 3.0).to(dtype)
    k = torch.randn(B, T, H, dk, generator=g).to(dtype)
    w = torch.randn(H, H * dk, generator=g) / (H * dk) ** 0.5
    b = torch.randn(H, generator=g)
    return q, k, w, b


@pytest.mark.parametrize("dtype,B,T,H,dk", [(F32, 2, 100, 4, 64), (BF16, 1, 70, 8, 256),
                                            (BF16, 2, 33, 16, 64), (F32, 1, 17, 2, 128)])
def test_prep_matches_oracle(dtype, B, T, H, dk):
    q, k, w, b = raw_inputs(B, T, H, dk, dtype, 600 + dk)
    out = ccq.ccq_prep(q.cuda(), k.cuda(), w.cuda(), b.cuda())
    torch.cuda.synchronize()
    ref = O.prep(q.double().numpy(), k.double().numpy(), w.double().numpy(), b.double().numpy())
    errs = {key: nerr(np64(out[key]), ref[key]) for key in ("q", "k", "lam")}
    say("prep", dtype, B, T, H, dk, errs)
    assert all(v <= TOL[dtype] for v in errs.values()), errs


def test_prep_in_place():
    q, k, w, b = raw_inputs(2, 50, 4, 128, BF16, 7)
    qd, kd = q.cuda(), k.cuda()
    a = ccq.ccq_prep(qd, kd, w.cuda(), b.cuda())
    qi, ki = qd.clone(), kd.clone()
    c = ccq.ccq_prep(qi, ki, w.cuda(), b.cuda(), out=dict(q=qi, k=ki))
    torch.cuda.synchronize()
    assert torch.equal(a["q"], qi) and torch.equal(a["k"], ki) and torch.equal(a["lam"], c["lam"])


def test_prep_then_forward_matches_oracle():
    """Raw q, k -> ccq_prep -> ccq_gdn_fwd against oracle prep -> oracle forward (the
    oracle is fed the same bf16-rounded normalised q, k the HIP forward receives, so
    the comparison measures the forward, as everywhere else)."""
    B, T, H, dk, dv = 1, 150, 4, 128, 128
    q, k, w, b = raw_inputs(B, T, H, dk, BF16, 11)
    g = torch.Generator().manual_seed(12)
    v = torch.randn(B, T, H, dv, generator=g).to(BF16)
    beta = torch.sigmoid(torch.randn(B, T, H, generator=g))
    la = -torch.nn.functional.softplus(torch.randn(B, T, H, generator=g) - 3.0)
    p = ccq.ccq_prep(q.cuda(), k.cuda(), w.cuda(), b.cuda())
    o = ccq.ccq_gdn_fwd(p["q"], p["k"], v.cuda(), la.cuda(), beta.cuda(), p["lam"])
    torch.cuda.synchronize()
    ref_p = O.prep(q.double().numpy(), k.double().numpy(), w.double().numpy(), b.double().numpy())
    assert nerr(np64(p["lam"]), ref_p["lam"]) <= 2e-2
    ref = O.fwd(np64(p["q"]), np64(p["k"]), v.double().numpy(), la.double().numpy(),
                ref_p["lam"], beta=beta.double().numpy(), backbone=O.GDN)
    err = nerr(np64(o["o"]), ref["o"])
    say("prep+fwd", err)
    assert err <= 2e-2
