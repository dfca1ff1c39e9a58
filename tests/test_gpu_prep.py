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


# ---------------------------------------------------------------- forward from raw q, k


def raw_case(backbone, B, T, H, dk, dv, dtype, seed):
    q, k, w, b = raw_inputs(B, T, H, dk, dtype, seed)
    g = torch.Generator().manual_seed(seed + 1)
    v = torch.randn(B, T, H, dv, generator=g).to(dtype)
    if backbone == ccq.CCQ_GLA:
        gate = (torch.nn.functional.logsigmoid(torch.randn(B, T, H, dk, generator=g) + 4.0) / 16).to(dtype)
        beta = None
    else:
        beta = torch.sigmoid(torch.randn(B, T, H, generator=g))
        gate = -torch.nn.functional.softplus(torch.randn(B, T, H, generator=g) - 3.0)
    return q, k, w, b, v, gate, beta


def oracle_raw(backbone, q, k, w, b, v, gate, beta, dtype, **kw):
    """Oracle pre-processing, its normalised q, k rounded once to the io dtype (as the
    kernels round the scaled rows they stage), then the oracle forward."""
    ref_p = O.prep(q.double().numpy(), k.double().numpy(), w.double().numpy(), b.double().numpy())
    qn = torch.from_numpy(ref_p["q"]).to(dtype).double().numpy()
    kn = torch.from_numpy(ref_p["k"]).to(dtype).double().numpy()
    ref = O.fwd(qn, kn, v.double().numpy(), gate.double().numpy(), ref_p["lam"],
                beta=None if beta is None else beta.double().numpy(),
                backbone=O.GLA if backbone == ccq.CCQ_GLA else O.GDN, **kw)
    return ref, ref_p


RAW_CASES = [
    # backbone, dtype, B, T, H, dk, dv
    (ccq.CCQ_GLA, BF16, 2, 200, 4, 128, 256),
    (ccq.CCQ_GLA, F32, 1, 130, 2, 64, 64),
    (ccq.CCQ_GDN, BF16, 1, 150, 4, 128, 128),
    (ccq.CCQ_GDN, BF16, 1, 97, 8, 256, 256),
    (ccq.CCQ_GDN, F32, 2, 70, 2, 64, 128),
]


@pytest.mark.parametrize("case", RAW_CASES, ids=lambda c: "%s-%s-T%d-dk%d" % (
    "gla" if c[0] == ccq.CCQ_GLA else "gdn", str(c[1]).split(".")[-1], c[3], c[5]))
def test_forward_from_raw_matches_oracle(case):
    backbone, dtype, B, T, H, dk, dv = case
    say("raw fwd", case)
    q, k, w, b, v, gate, beta = raw_case(backbone, B, T, H, dk, dv, dtype, 700 + T)
    out = ccq.ccq_fwd_raw(q.cuda(), k.cuda(), w.cuda(), b.cuda(), v.cuda(), gate.cuda(),
                          None if beta is None else beta.cuda(), backbone=backbone, want_lam=True)
    torch.cuda.synchronize()
    ref, ref_p = oracle_raw(backbone, q, k, w, b, v, gate, beta, dtype)
    errs = {n: nerr(np64(out[n]), ref[n]) for n in ("o", "ST", "CT", "muT")}
    errs["lam"] = nerr(np64(out["lam"]), ref_p["lam"])
    say("  errors", errs)
    assert all(x <= TOL[dtype] for x in errs.values()), errs


@pytest.mark.parametrize("backbone", [ccq.CCQ_GLA, ccq.CCQ_GDN])
def test_forward_from_raw_matches_two_pass(backbone):
    """The folded path against ccq_prep followed by the forward on the normalised
    q, k (both through the HIP path), with initial states and t0 > 0: the gate bit for
    bit (the same kernel arithmetic), the outputs to the bf16 bar (the folded path
    scales the raw rows itself, one rounding of the same values)."""
    B, T, H, dk, dv = 2, 170, 4, 128, 128
    q, k, w, b, v, gate, beta = raw_case(backbone, B, T, H, dk, dv, BF16, 31)
    rng = np.random.default_rng(4)
    S0 = torch.from_numpy(rng.standard_normal((B, H, dv, dk)) * 0.2).float().cuda()
    Kp = rng.standard_normal((B, H, 20, dk))
    Kp /= np.linalg.norm(Kp, axis=-1, keepdims=True)
    C0 = torch.from_numpy(np.einsum("bhnc,bhnd->bhcd", Kp, Kp) / 20).float().cuda()
    mu0 = torch.from_numpy(Kp.mean(axis=2)).float().cuda()
    g = {n: x.cuda() for n, x in dict(q=q, k=k, w=w, b=b, v=v, gate=gate).items()}
    bt = None if beta is None else beta.cuda()
    a = ccq.ccq_fwd_raw(g["q"], g["k"], g["w"], g["b"], g["v"], g["gate"], bt, backbone=backbone,
                        S0=S0, C0=C0, mu0=mu0, t0=20, want_lam=True)
    p = ccq.ccq_prep(g["q"], g["k"], g["w"], g["b"])
    if backbone == ccq.CCQ_GLA:
        c = ccq.ccq_gla_fwd(p["q"], p["k"], g["v"], g["gate"], p["lam"], S0=S0, C0=C0, mu0=mu0, t0=20)
    else:
        c = ccq.ccq_gdn_fwd(p["q"], p["k"], g["v"], g["gate"], bt, p["lam"], S0=S0, C0=C0, mu0=mu0,
                            t0=20)
    torch.cuda.synchronize()
    assert torch.equal(a["lam"], p["lam"])
    errs = {n: nerr(np64(a[n]), np64(c[n])) for n in ("o", "ST", "CT", "muT")}
    say("  folded vs two-pass", backbone, errs)
    assert all(x <= TOL[BF16] for x in errs.values()), errs


def test_forward_from_raw_full_size_gdn():
    """The Gated DeltaNet 1.3B-layer shape (B=4, T=4096, H=8, dk=dv=256, bf16) from raw
    q, k; every (batch, head) sequence against the oracle."""
    B, T, H, dk, dv = 4, 4096, 8, 256, 256
    say("raw fwd full size")
    q, k, w, b, v, gate, beta = raw_case(ccq.CCQ_GDN, B, T, H, dk, dv, BF16, 2)
    out = ccq.ccq_fwd_raw(q.cuda(), k.cuda(), w.cuda(), b.cuda(), v.cuda(), gate.cuda(), beta.cuda(),
                          backbone=ccq.CCQ_GDN)
    torch.cuda.synchronize()
    ref, _ = oracle_raw(ccq.CCQ_GDN, q, k, w, b, v, gate, beta, BF16)
    o = np64(out["o"])
    worst = 0.0
    for bb in range(B):
        for h in range(H):
            e = nerr(o[bb, :, h], ref["o"][bb, :, h])
            worst = max(worst, e)
            assert e <= TOL[BF16], (bb, h, e)
    es = {n: nerr(np64(out[n]), ref[n]) for n in ("ST", "CT", "muT")}
    say("  worst o", worst, "states", es)
    assert all(x <= TOL[BF16] for x in es.values()), es
