"""Parity of the packed-batch entry points (ccq_gla_fwd_varlen, ccq_gdn_fwd_varlen,
ccq_fwd_bwd_varlen through the C ABI) with the oracle run on every sequence on its own.

Lengths mix empty, sub-chunk, exact-chunk and ragged multi-chunk sequences; max_len
is either the longest length or a looser bound.  Same bar as the padded calls:
max |gpu - ref| / max |ref| <= 1e-4 (fp32 io) or <= 2e-2 (bf16 io), per tensor.
"""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, nerr, np64
from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, GLA, make_inputs, to_f64

pytestmark = pytest.mark.gpu
F32, BF16 = torch.float32, torch.bfloat16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def packed(backbone, lens, H, dk, dv, dtype, seed, with_dO=False):
    """Seeded batch of max(lens) tokens per sequence, packed to the given lengths."""
    T = max(max(lens), 1)
    d = make_inputs(backbone, len(lens), T, H, dk, dv, dtype, seed=seed, keys="aniso",
                    lam="random", with_dO=with_dO)
    p = {n: torch.cat([x[b, :L] for b, L in enumerate(lens)], dim=0).contiguous()
         for n, x in d.items()}
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return p, cu


def initial_states(rng, B, H, dk, dv):
    S0 = rng.standard_normal((B, H, dv, dk)) * 0.2
    Kp = rng.standard_normal((B, H, 30, dk))
    Kp /= np.linalg.norm(Kp, axis=-1, keepdims=True)
    C0 = np.einsum("bhnc,bhnd->bhcd", Kp, Kp) / 30
    mu0 = Kp.mean(axis=2)
    return [x.astype(np.float32) for x in (S0, C0, mu0)]


def run_fwd(backbone, p, cu, max_len, init, t0):
    g = {n: x.cuda() for n, x in p.items()}
    cu_d = torch.from_numpy(cu).cuda()
    kw = {}
    if init is not None:
        kw = dict(S0=torch.from_numpy(init[0]).cuda(), C0=torch.from_numpy(init[1]).cuda(),
                  mu0=torch.from_numpy(init[2]).cuda(), t0=t0)
    if backbone == GLA:
        out = ccq.ccq_gla_fwd_varlen(g["q"], g["k"], g["v"], g["g"], g["lam"], cu_d, max_len, **kw)
    else:
        out = ccq.ccq_gdn_fwd_varlen(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                                     cu_d, max_len, **kw)
    torch.cuda.synchronize()
    return {n: np64(x) for n, x in out.items()}


FWD_CASES = [
    # backbone, dtype, lengths, H, dk, dv, max_len slack, initial states
    (GLA, BF16, [37, 200, 0, 64, 129], 2, 128, 256, 0, False),
    (GLA, F32, [5, 70, 128], 2, 64, 128, 40, True),
    (GDN, BF16, [150, 1, 64, 0, 90], 2, 256, 256, 0, True),
    (GDN, F32, [66, 130], 2, 64, 64, 8, False),
    # few heads and many chunks: the GLA state pass runs in segments, the
    # shorter sequences' last segments are empty
    (GLA, BF16, [1100, 300, 0, 700], 1, 128, 256, 0, True),
    (GDN, BF16, [700, 64, 333], 1, 128, 128, 0, False),
]


@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "%s-%s-%s" % (
    "gla" if c[0] == GLA else "gdn", str(c[1]).split(".")[-1], "-".join(map(str, c[2]))))
def test_varlen_forward(case):
    backbone, dtype, lens, H, dk, dv, slack, with_init = case
    say("varlen fwd", case)
    p, cu = packed(backbone, lens, H, dk, dv, dtype, seed=500 + sum(lens))
    rng = np.random.default_rng(9)
    init = initial_states(rng, len(lens), H, dk, dv) if with_init else None
    t0 = 30 if with_init else 0
    gout = run_fwd(backbone, p, cu, max(lens) + slack, init, t0)
    f = to_f64(p)
    gate = f["g"] if backbone == GLA else f["logalpha"]
    kw = {} if init is None else dict(S0=init[0].astype(np.float64), C0=init[1].astype(np.float64),
                                      mu0=init[2].astype(np.float64), t0=t0)
    ref = O.varlen_fwd(f["q"], f["k"], f["v"], gate, f["lam"], cu, beta=f.get("beta"),
                       backbone=backbone, **kw)
    errs = {n: nerr(gout[n], ref[n]) for n in ("o", "ST", "CT", "muT")}
    # every sequence's own output too, so that a short one is not hidden by the others
    for b in range(len(lens)):
        if lens[b]:
            errs["o%d" % b] = nerr(gout["o"][cu[b]:cu[b + 1]], ref["o"][cu[b]:cu[b + 1]])
    say("  errors", errs)
    tol = TOL[dtype]
    assert all(v <= tol for v in errs.values()), errs


def test_varlen_equals_separate_calls():
    """Each sequence of a packed bf16 batch gives the output of a padded call of its own
    length (both through the HIP path) to within two bf16 roundings: the two calls may
    group chunks differently (segments, output groups), which changes summation order
    only.  The states, kept in fp32, agree far more closely."""
    lens = [100, 64, 3]
    H, dk, dv = 2, 128, 128
    p, cu = packed(GLA, lens, H, dk, dv, BF16, seed=77)
    gout = run_fwd(GLA, p, cu, max(lens), None, 0)
    for b, L in enumerate(lens):
        s = {n: x[cu[b]:cu[b + 1]].unsqueeze(0).cuda().contiguous() for n, x in p.items()}
        one = ccq.ccq_gla_fwd(s["q"], s["k"], s["v"], s["g"], s["lam"])
        torch.cuda.synchronize()
        e = nerr(gout["o"][cu[b]:cu[b + 1]], np64(one["o"][0]))
        es = nerr(gout["ST"][b], np64(one["ST"][0]))
        ec = nerr(gout["CT"][b], np64(one["CT"][0]))
        say("  seq", b, e, es, ec)
        assert e <= 8e-3 and es <= 1e-4 and ec <= 1e-5


BWD_CASES = [
    (GLA, BF16, [100, 37, 64], 2, 64, 128),
    (GLA, F32, [70, 0, 20], 1, 64, 64),
    (GDN, BF16, [90, 64, 5], 2, 128, 128),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: "%s-%s-%s" % (
    "gla" if c[0] == GLA else "gdn", str(c[1]).split(".")[-1], "-".join(map(str, c[2]))))
def test_varlen_training_step(case):
    backbone, dtype, lens, H, dk, dv = case
    say("varlen fwd_bwd", case)
    p, cu = packed(backbone, lens, H, dk, dv, dtype, seed=600 + sum(lens), with_dO=True)
    g = {n: x.cuda() for n, x in p.items()}
    cu_d = torch.from_numpy(cu).cuda()
    gate = g["g"] if backbone == GLA else g["logalpha"]
    out = ccq.ccq_fwd_bwd_varlen(g["q"], g["k"], g["v"], gate, g["lam"], g["dO"], cu_d, max(lens),
                                 backbone=backbone, beta=g.get("beta"))
    torch.cuda.synchronize()
    gout = {n: np64(x) for n, x in out.items()}
    f = to_f64(p)
    ref = O.varlen_fwd_bwd(f["q"], f["k"], f["v"], f["g"] if backbone == GLA else f["logalpha"],
                           f["lam"], f["dO"], cu, beta=f.get("beta"), backbone=backbone)
    keys = ("o", "dq", "dk", "dv", "dg", "dlam") + (("dbeta",) if backbone == GDN else ())
    errs = {n: nerr(gout[n], ref[n]) for n in keys}
    say("  errors", errs)
    tol = TOL[dtype]
    assert all(v <= tol for v in errs.values()), errs


def test_varlen_sequence_cut_at_max_len():
    """A sequence longer than max_len is cut there: only its first max_len rows are read
    and written, and the next sequence's packed rows (which start past B * max_len) are
    still found through the offsets."""
    lens, max_len, H, dk, dv = [200, 50, 90], 100, 2, 64, 128
    for backbone in (GLA, GDN):
        p, cu = packed(backbone, lens, H, dk, dv, BF16, seed=88)
        gout = run_fwd(backbone, p, cu, max_len, None, 0)
        cut = [min(L, max_len) for L in lens]
        keep = np.concatenate([np.arange(cu[b], cu[b] + cut[b]) for b in range(len(lens))])
        f = to_f64(p)
        fc = {n: x[keep] for n, x in f.items()}
        cuc = np.concatenate([[0], np.cumsum(cut)]).astype(np.int32)
        gate = fc["g"] if backbone == GLA else fc["logalpha"]
        ref = O.varlen_fwd(fc["q"], fc["k"], fc["v"], gate, fc["lam"], cuc, beta=fc.get("beta"),
                           backbone=backbone)
        errs = {"o": nerr(gout["o"][keep], ref["o"])}
        errs.update({n: nerr(gout[n], ref[n]) for n in ("ST", "CT", "muT")})
        say("  cut", backbone, errs)
        assert all(v <= TOL[BF16] for v in errs.values()), errs


def test_varlen_full_size_gdn():
    """The packed Gated DeltaNet workload of the benchmark: 8 sequences of 1024 to 3072
    tokens, H=8, dk=dv=256, bf16, every sequence compared with the oracle."""
    from paper_2606_01294_amd.inputs import WORKLOADS, varlen_lengths
    w = WORKLOADS["gdn_1p3b_t4k"]
    lens = varlen_lengths(w)
    say("varlen full size", lens)
    T = max(lens)
    d = make_inputs(GDN, len(lens), T, w.H, w.dk, w.dv, w.dtype, seed=w.seed)
    p = {n: torch.cat([x[b, :L] for b, L in enumerate(lens)], dim=0).contiguous()
         for n, x in d.items()}
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    gout = run_fwd(GDN, p, cu, T, None, 0)
    f = to_f64(p)
    ref = O.varlen_fwd(f["q"], f["k"], f["v"], f["logalpha"], f["lam"], cu, beta=f["beta"],
                       backbone=GDN)
    worst = {}
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        e = {"o": nerr(gout["o"][sl], ref["o"][sl]), "ST": nerr(gout["ST"][b], ref["ST"][b]),
             "CT": nerr(gout["CT"][b], ref["CT"][b]), "muT": nerr(gout["muT"][b], ref["muT"][b])}
        for n, v in e.items():
            worst[n] = max(worst.get(n, 0.0), v)
        assert all(v <= TOL[w.dtype] for v in e.values()), (b, e)
    say("  worst", worst)
