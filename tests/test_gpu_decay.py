"""Parity of the decay-aligned contraction (ccq_shape.decay_aligned, Gated DeltaNet)
with the fp64 oracle's decay=True forward, which is pinned on the CPU to numpy's
weighted covariance, to Sigma_t at alpha = 1 and to its own running-mean form.

Same bar as the other forward tests: max |gpu - ref| / max |ref| <= 1e-4 (fp32 io) or
<= 2e-2 (bf16 io) on o, the final (S, Cbar^gamma, mu^gamma) and the correction term.
"""
import sys

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from gpu_helpers import TOL, elem_err, nerr, np64
from oracle import ccq_oracle as O
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, WORKLOADS, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu
F32, BF16 = torch.float32, torch.bfloat16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def decay_inputs(dtype, B, T, H, dk, dv, seed, keys="iso", forget="mild"):
    """make_inputs' Gated DeltaNet recipe; forget="strong" draws log decays of
    -softplus(N(0,1) + 1) (about 1.3 per token) and "reset" adds a few tokens with
    log decay -30 (almost everything forgotten there)."""
    d = make_inputs(GDN, B, T, H, dk, dv, dtype, seed=seed, keys=keys, lam="random")
    gen = torch.Generator().manual_seed(seed + 7)
    if forget in ("strong", "reset"):
        d["logalpha"] = -F.softplus(torch.randn(B, T, H, generator=gen) + 1.0)
    if forget == "reset":
        idx = torch.randint(0, T, (max(1, T // 50),), generator=gen)
        d["logalpha"][:, idx] = -30.0
    return d


def run_gpu(d, **kw):
    g = to_device(d)
    out = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                          want_qclean=True, decay_aligned=True, **kw)
    torch.cuda.synchronize()
    return {k: np64(v) for k, v in out.items()}


def run_oracle(d):
    f = to_f64(d)
    return O.fwd(f["q"], f["k"], f["v"], f["logalpha"], f["lam"], beta=f["beta"],
                 backbone=O.GDN, decay=True)


def errors(gout, ref, q64):
    e = {k: nerr(gout[k], ref[k]) for k in ("o", "ST", "CT", "muT")}
    # the correction lambda Sigma^gamma q itself, normalised by its own size
    e["corr"] = nerr(q64 - gout["qclean"], q64 - ref["qclean"])
    return e


def check(d, dtype):
    gout, ref = run_gpu(d), run_oracle(d)
    q64 = to_f64(d)["q"]
    e = errors(gout, ref, q64)
    say("  errors", e, "element-wise o %.3g" % elem_err(gout["o"], ref["o"]))
    assert all(v <= TOL[dtype] for v in e.values()), e
    return gout, ref


CASES = [
    # dtype, B, T, H, dk, dv, keys, forget
    (F32, 1, 200, 2, 64, 64, "iso", "mild"),
    (F32, 1, 130, 2, 128, 128, "meanshift", "strong"),
    (F32, 2, 333, 1, 64, 128, "aniso", "reset"),
    (BF16, 1, 150, 2, 256, 256, "iso", "mild"),
    (BF16, 1, 200, 2, 256, 256, "meanshift", "strong"),
    (BF16, 2, 100, 2, 128, 512, "aniso", "reset"),
    (BF16, 1, 97, 3, 64, 64, "meanshift", "mild"),
    (BF16, 1, 1, 2, 256, 256, "iso", "strong"),
    (BF16, 1, 63, 1, 128, 128, "iso", "reset"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-T%d-dk%d-dv%d-%s-%s" % (
    str(c[0]).split(".")[-1], c[2], c[4], c[5], c[6], c[7]))
def test_decay_aligned_small(case):
    dtype, B, T, H, dk, dv, keys, forget = case
    say("decay small", case)
    check(decay_inputs(dtype, B, T, H, dk, dv, seed=700 + T, keys=keys, forget=forget), dtype)


# Few heads and many chunks: the contraction runs in segments whose decayed sums are
# joined by the segment prefix (segments of 2 chunks here).
@pytest.mark.parametrize("dtype, dk", [(F32, 64), (BF16, 256)])
def test_decay_aligned_segments(dtype, dk):
    say("decay segments", dtype, dk)
    check(decay_inputs(dtype, 1, 1100, 2, dk, dk, seed=711, keys="meanshift", forget="strong"),
          dtype)


def test_decay_aligned_changes_the_correction():
    """With forgetting the decay-aligned correction differs from the undecayed one (and
    the oracle agrees on by how much): the flag is not silently ignored."""
    d = decay_inputs(F32, 1, 300, 2, 64, 64, seed=720, keys="meanshift", forget="strong")
    g = to_device(d)
    plain = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                            want_qclean=True)
    torch.cuda.synchronize()
    gout = run_gpu(d)
    ref = run_oracle(d)
    f = to_f64(d)
    ref_plain = O.fwd(f["q"], f["k"], f["v"], f["logalpha"], f["lam"], beta=f["beta"],
                      backbone=O.GDN)
    gap_gpu = np64(plain["qclean"]) - gout["qclean"]
    gap_ref = ref_plain["qclean"] - ref["qclean"]
    say("  correction gap", np.abs(gap_ref).max())
    assert np.abs(gap_ref).max() > 1e-2
    assert nerr(gap_gpu, gap_ref) <= 1e-3


def test_decay_aligned_packed_batch():
    """Packed rows: each sequence's statistics start empty and see only its own keys."""
    lens = [150, 1, 97, 300]
    dk = dv = 128
    d = decay_inputs(BF16, 1, sum(lens), 2, dk, dv, seed=730, keys="aniso", forget="strong")
    flat = {k: t[0] for k, t in d.items()}  # [rows, H, ...]
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda")
    g = to_device(flat)
    out = ccq.ccq_gdn_fwd_varlen(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"], cu,
                                 max(lens), decay_aligned=True)
    torch.cuda.synchronize()
    o = np64(out["o"])
    r0 = 0
    for b, L in enumerate(lens):
        part = {k: t[:, r0:r0 + L] for k, t in d.items()}
        ref = run_oracle(part)
        e = {"o": nerr(o[r0:r0 + L], ref["o"][0]), "ST": nerr(np64(out["ST"][b]), ref["ST"][0]),
             "CT": nerr(np64(out["CT"][b]), ref["CT"][0])}
        say("  sequence", b, L, e)
        assert all(v <= TOL[BF16] for v in e.values()), (b, e)
        r0 += L


def test_decay_aligned_full_size():
    """The 1.3B Gated DeltaNet layer (B=4, T=4096, H=8, dk=dv=256) with the decay-aligned
    statistics, every (batch, head) sequence against the oracle."""
    w = WORKLOADS["gdn_1p3b_t4k"]
    say("decay full size", w)
    d = make_inputs(GDN, w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=w.seed)
    gout, ref = run_gpu(d), run_oracle(d)
    q64 = to_f64(d)["q"]
    worst = {}
    for b in range(w.B):
        for h in range(w.H):
            sl = lambda x: x[b:b + 1, :, h:h + 1]
            sh = lambda x: x[b:b + 1, h:h + 1]
            e = {"o": nerr(sl(gout["o"]), sl(ref["o"])), "ST": nerr(sh(gout["ST"]), sh(ref["ST"])),
                 "CT": nerr(sh(gout["CT"]), sh(ref["CT"])),
                 "corr": nerr(sl(q64) - sl(gout["qclean"]), sl(q64) - sl(ref["qclean"]))}
            for k_, v in e.items():
                worst[k_] = max(worst.get(k_, 0.0), v)
            assert all(v <= TOL[w.dtype] for v in e.values()), (b, h, e)
    say("  %d sequences, worst" % (w.B * w.H), worst)
