"""Parity of the recurrent decode step (ccq_decode through the C ABI, Alg. 2) with
the fp64 oracle's running-mean recurrence (form 1 of its forward, pinned on the CPU
against the sum form, brute-force covariances and the chunkwise form).

The bar is the forward's: max |gpu - ref| / max |ref| <= 1e-4 (fp32 io) or
<= 2e-2 (bf16 io) for o and the updated cache (S, Cbar, mu), which is fp32 in both.
"""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, nerr, np64
from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, GLA, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu
F32, BF16 = torch.float32, torch.bfloat16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gate_key(backbone):
    return "g" if backbone == GLA else "logalpha"


def token(d, t):
    """The inputs of token t as decode-step tensors ([B,H,...]) on the GPU."""
    res = {}
    for key, x in d.items():
        res[key] = x[:, t].contiguous().cuda()
    return res


def oracle_run(backbone, f, S0=None, C0=None, mu0=None, t0=0, **kw):
    return O.fwd(f["q"], f["k"], f["v"], f[gate_key(backbone)], f["lam"],
                 beta=f.get("beta"), backbone=O.GLA if backbone == GLA else O.GDN,
                 S0=S0, C0=C0, mu0=mu0, t0=t0, form=1, **kw)


def decode_steps(backbone, d, S, C, mu, t0, steps, **kw):
    outs = []
    for i in range(steps):
        x = token(d, i)
        o = ccq.ccq_decode(x["q"], x["k"], x["v"], x[gate_key(backbone)], x["lam"], S, C, mu,
                           t0 + i, backbone=backbone, beta=x.get("beta"), **kw)
        outs.append(np64(o))
    torch.cuda.synchronize()
    return np.stack(outs, axis=1)


CASES = [
    # backbone, dtype, B, H, dk, dv, keys
    (GLA, F32, 2, 2, 64, 64, "iso"),
    (GLA, BF16, 2, 3, 128, 256, "aniso"),
    (GLA, BF16, 1, 2, 256, 512, "meanshift"),
    (GDN, F32, 2, 2, 64, 128, "iso"),
    (GDN, BF16, 2, 2, 256, 256, "aniso"),
    (GDN, BF16, 1, 3, 128, 64, "meanshift"),
    # S in several register batches (dk = 256, dv = 512), one short batch (dv = 64),
    # and a narrow head with a tall S (dk = 64, dv = 512)
    (GDN, BF16, 1, 2, 256, 512, "iso"),
    (GDN, F32, 1, 2, 256, 64, "aniso"),
    (GLA, F32, 1, 2, 64, 512, "aniso"),
    (GLA, BF16, 2, 2, 256, 128, "iso"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-%s-dk%d-dv%d-%s" % (
    "gla" if c[0] == GLA else "gdn", str(c[1]).split(".")[-1], c[4], c[5], c[6]))
def test_decode_continues_a_prefix(case):
    """Cache from the oracle over a 70-token prefix, then 6 decode steps on the GPU,
    against the oracle over the whole 76 tokens."""
    backbone, dtype, B, H, dk, dv, keys = case
    say("decode", case)
    P, n = 70, 6
    d = make_inputs(backbone, B, P + n, H, dk, dv, dtype, seed=500 + dk + dv, keys=keys,
                    lam="random")
    f = to_f64(d)
    pre = oracle_run(backbone, {k: v[:, :P] for k, v in f.items()})
    full = oracle_run(backbone, f)
    S = torch.from_numpy(pre["ST"]).float().cuda()
    C = torch.from_numpy(pre["CT"]).float().cuda()
    mu = torch.from_numpy(pre["muT"]).float().cuda()
    # one workspace for all the steps, as a serving loop would keep
    need = ccq.ccq_decode_workspace_size(ccq.make_shape(B, 1, H, dk, dv, dtype))
    ws = torch.zeros(max(need, 1), dtype=torch.uint8, device="cuda")
    o = decode_steps(backbone, {k: v[:, P:] for k, v in d.items()}, S, C, mu, P, n, workspace=ws)
    errs = {"o": nerr(o, full["o"][:, P:]), "S": nerr(np64(S), full["ST"]),
            "C": nerr(np64(C), full["CT"]), "mu": nerr(np64(mu), full["muT"])}
    say("  errors", errs)
    assert all(v <= TOL[dtype] for v in errs.values()), errs


@pytest.mark.parametrize("backbone", [GLA, GDN])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_decode_from_empty_cache(backbone, dtype):
    """A fresh sequence decoded token by token (zero cache, t0 = 0, 1, ...) equals the
    oracle's forward over the same tokens, uncentred and with a read scale."""
    say("decode from empty", backbone, dtype)
    B, T, H, dk, dv = 2, 40, 2, 128, 128
    d = make_inputs(backbone, B, T, H, dk, dv, dtype, seed=77, lam="random")
    f = to_f64(d)
    for centered, scale in ((True, 1.0), (False, 0.5)):
        ref = oracle_run(backbone, f, centered=centered, scale=scale)
        S = torch.zeros(B, H, dv, dk, device="cuda")
        C = torch.zeros(B, H, dk, dk, device="cuda")
        mu = torch.zeros(B, H, dk, device="cuda")
        o = decode_steps(backbone, d, S, C, mu, 0, T, centered=centered, scale=scale)
        errs = {"o": nerr(o, ref["o"]), "S": nerr(np64(S), ref["ST"]),
                "C": nerr(np64(C), ref["CT"]), "mu": nerr(np64(mu), ref["muT"])}
        say("  centered=%d" % centered, errs)
        assert all(v <= TOL[dtype] for v in errs.values()), errs


@pytest.mark.parametrize("backbone", [GLA, GDN])
def test_decode_after_chunked_prefill(backbone):
    """The chunkwise forward's final (S_T, Cbar_T, mu_T) is the decode cache: prefill 200
    tokens with the HIP forward, decode 4 more, compare with the oracle over 204."""
    dtype = BF16
    B, H, dk, dv, P, n = 2, 2, 128, 256, 200, 4
    d = make_inputs(backbone, B, P + n, H, dk, dv, dtype, seed=91, lam="random")
    g = {k: v[:, :P].contiguous().cuda() for k, v in d.items()}
    if backbone == GLA:
        pre = ccq.ccq_gla_fwd(g["q"], g["k"], g["v"], g["g"], g["lam"])
    else:
        pre = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"])
    S, C, mu = pre["ST"], pre["CT"], pre["muT"]
    o = decode_steps(backbone, {k: v[:, P:] for k, v in d.items()}, S, C, mu, P, n)
    full = oracle_run(backbone, to_f64(d))
    errs = {"o": nerr(o, full["o"][:, P:]), "S": nerr(np64(S), full["ST"]),
            "C": nerr(np64(C), full["CT"]), "mu": nerr(np64(mu), full["muT"])}
    say("  prefill+decode", backbone, errs)
    assert all(v <= TOL[dtype] for v in errs.values()), errs


def test_decode_lambda_zero_is_plain_backbone_read():
    """With lam = 0 the read uses the raw query: o equals S_t q from a decode step whose
    cache statistics are arbitrary (here deliberately not a valid second moment)."""
    B, H, dk, dv = 1, 2, 64, 64
    d = make_inputs(GLA, B, 1, H, dk, dv, F32, seed=5, lam="const", lam_value=0.0)
    x = token(d, 0)
    S = torch.randn(B, H, dv, dk, device="cuda")
    C = torch.randn(B, H, dk, dk, device="cuda") * 100
    mu = torch.randn(B, H, dk, device="cuda") * 100
    S_ref = S.clone()
    o = ccq.ccq_decode(x["q"], x["k"], x["v"], x["g"], x["lam"], S, C, mu, 9)
    S_new = S_ref * torch.exp(x["g"].float())[:, :, None, :] + x["v"][:, :, :, None] * x["k"][:, :, None, :]
    ref = torch.einsum("bhvk,bhk->bhv", S_new.double().cpu(), x["q"].double().cpu())
    torch.cuda.synchronize()
    assert nerr(np64(o), ref.numpy()) <= 1e-5
