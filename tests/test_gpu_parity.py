"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Small cases compare every element, at sizes that span several 64-token chunks
and end in a ragged chunk.  The full-size workloads run exactly as the
benchmark launches them and compare every (batch, head) sequence with the
oracle, each normalised by its own reference.  Tolerance: max |gpu - ref| / max |ref| per
tensor <= 1e-4 (fp32 io) or <= 2e-2 (bf16 io, fp32 accumulation), applied to
o, the final (S, Cbar, mu) and the correction lambda_t Sigma_t q_t itself.
"""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, compare, fwd_errors, gpu_fwd, nerr, np64, oracle_fwd
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, GLA, WORKLOADS, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu

F32, BF16 = torch.float32, torch.bfloat16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# ------------------------------------------------------------- small, element-wise

GLA_CASES = [
    # dtype, B, T, H, dk, dv, keys, lam, gates, gate_dtype
    (F32, 1, 256, 2, 64, 64, "iso", "const", "config", F32),
    (F32, 2, 130, 2, 128, 128, "aniso", "random", "config", F32),
    (F32, 1, 65, 3, 64, 512, "meanshift", "random", "strong", F32),
    (BF16, 2, 200, 2, 128, 256, "iso", "const", "config", BF16),
    (BF16, 1, 150, 2, 128, 256, "aniso", "random", "config", F32),
    (BF16, 1, 97, 2, 64, 128, "meanshift", "const", "strong", BF16),
    (BF16, 1, 70, 2, 64, 512, "aniso", "random", "config", BF16),
    (BF16, 1, 1, 2, 128, 256, "iso", "random", "config", BF16),
    (BF16, 1, 63, 1, 128, 256, "iso", "random", "config", BF16),
]


@pytest.mark.parametrize("case", GLA_CASES, ids=lambda c: "%s-T%d-dk%d-dv%d-%s" % (
    str(c[0]).split(".")[-1], c[2], c[4], c[5], c[6]))
def test_gla_parity_small(case):
    dtype, B, T, H, dk, dv, keys, lam, gates, gdt = case
    say("gla small", case)
    d = make_inputs(GLA, B, T, H, dk, dv, dtype, gate_dtype=gdt, seed=100 + T, keys=keys,
                    lam=lam, gates=gates)
    compare(GLA, d, dtype)


# More than 8 chunks with few heads: the GLA state pass runs in segments of 8
# chunks (the last one short and ending in a ragged chunk), joined by the
# segment scan; with an initial state, which enters segment 0 only.
GLA_SEG_CASES = [
    # dtype, B, T, H, dk, dv, gate dtype
    (F32, 1, 600, 2, 64, 64, F32),
    (BF16, 2, 1100, 1, 128, 256, BF16),
    (BF16, 1, 530, 2, 64, 512, F32),
]


@pytest.mark.parametrize("case", GLA_SEG_CASES, ids=lambda c: "%s-T%d-dk%d-dv%d" % (
    str(c[0]).split(".")[-1], c[2], c[4], c[5]))
def test_gla_parity_segments(case):
    dtype, B, T, H, dk, dv, gdt = case
    say("gla segments", case)
    d = make_inputs(GLA, B, T, H, dk, dv, dtype, gate_dtype=gdt, seed=400 + T, keys="aniso",
                    lam="random")
    S0 = np.random.default_rng(T).standard_normal((B, H, dv, dk)) * 0.2
    compare(GLA, d, dtype, S0=S0.astype(np.float32).astype(np.float64))


# The bf16 GLA forward (dv <= 256) carries S through groups of chunks per
# output workgroup, reading one stored state per group (the group size follows
# from B * H and the chunk count): the small and segment cases above take
# groups of 2 (across segment entries in the segment cases), these shapes
# groups of 8 (all 6 chunks of a head, one partial group), 4 (16 chunks, the
# last ragged) and 4 (one group of 3 chunks); the full-size workloads below add
# groups of 4 (T = 2048) and 8 (T = 20480, across the state pass's segments).
GLA_GROUP_CASES = [
    # dtype, B, T, H, dk, dv
    (BF16, 16, 337, 16, 64, 64),
    (BF16, 8, 1000, 8, 128, 128),
    (BF16, 16, 150, 16, 64, 128),
]


@pytest.mark.parametrize("case", GLA_GROUP_CASES, ids=lambda c: "%s-B%dT%dH%d-dk%d-dv%d" % (
    str(c[0]).split(".")[-1], c[1], c[2], c[3], c[4], c[5]))
def test_gla_parity_output_groups(case):
    dtype, B, T, H, dk, dv = case
    say("gla groups", case)
    d = make_inputs(GLA, B, T, H, dk, dv, dtype, seed=500 + T, keys="aniso", lam="random")
    compare(GLA, d, dtype)


GDN_CASES = [
    (F32, 1, 200, 2, 64, 64, "iso", "const"),
    (F32, 1, 130, 2, 128, 256, "aniso", "random"),
    (BF16, 1, 150, 2, 256, 256, "iso", "const"),
    (BF16, 2, 100, 2, 128, 512, "aniso", "random"),
    (BF16, 1, 90, 3, 64, 64, "meanshift", "random"),
    (BF16, 1, 5, 1, 256, 256, "iso", "random"),
]


@pytest.mark.parametrize("case", GDN_CASES, ids=lambda c: "%s-T%d-dk%d-dv%d-%s" % (
    str(c[0]).split(".")[-1], c[2], c[4], c[5], c[6]))
def test_gdn_parity_small(case):
    dtype, B, T, H, dk, dv, keys, lam = case
    say("gdn small", case)
    d = make_inputs(GDN, B, T, H, dk, dv, dtype, seed=200 + T, keys=keys, lam=lam)
    compare(GDN, d, dtype)


# The Gated DeltaNet state pass splits each 16-wide value slice over 1, 2, 4 or
# 8 waves depending on how many slices (B * H * dv / 16) the call has; these
# batch shapes reach every split the small cases above do not.
GDN_SPLIT_CASES = [
    # dtype, B, H, dk, dv  -> slices
    (BF16, 4, 16, 256, 256),   # 1024: one wave per slice
    (BF16, 2, 16, 256, 256),   # 512: two
    (BF16, 1, 16, 256, 256),   # 256: four
    (BF16, 4, 16, 128, 256),   # 1024: one
    (BF16, 2, 16, 128, 256),   # 512: two
    (BF16, 8, 16, 64, 128),    # 1024: one
    (F32, 8, 16, 128, 128),    # 1024: one
    (F32, 4, 16, 64, 128),     # 512: two
]


@pytest.mark.parametrize("case", GDN_SPLIT_CASES, ids=lambda c: "%s-B%dH%d-dk%d-dv%d" % (
    str(c[0]).split(".")[-1], c[1], c[2], c[3], c[4]))
def test_gdn_parity_state_splits(case):
    dtype, B, H, dk, dv = case
    say("gdn split", case)
    d = make_inputs(GDN, B, 70, H, dk, dv, dtype, seed=300 + B * H + dk, keys="aniso", lam="random")
    compare(GDN, d, dtype)


# With enough (batch, head) pairs the Gated DeltaNet output kernel takes
# groups of chunks per workgroup, carrying S from one stored state through the
# group (the group size follows from B * H and the chunk count); these shapes
# reach groups of 8 (here all 6 chunks of a head, one partial group), 4 (3
# chunks) and 2 (groups {0, 1} and {2}) with ragged last chunks, four value
# tiles per wave with and without the carry, and fp32.  The full-size
# workloads below add groups of 8 and 4 over many groups per head.
GDN_GROUP_CASES = [
    # dtype, B, T, H, dk, dv
    (BF16, 16, 337, 16, 64, 64),    # 6 chunks, one group
    (BF16, 8, 150, 16, 64, 128),    # 3 chunks, groups of 2
    (F32, 16, 337, 16, 64, 64),
    (BF16, 16, 150, 16, 128, 512),  # four value tiles per wave, one group of 3
    (F32, 16, 150, 16, 128, 256),
    (BF16, 16, 150, 16, 256, 512),  # S too large to carry: one chunk per workgroup
]


@pytest.mark.parametrize("case", GDN_GROUP_CASES, ids=lambda c: "%s-B%dT%dH%d-dk%d-dv%d" % (
    str(c[0]).split(".")[-1], c[1], c[2], c[3], c[4], c[5]))
def test_gdn_parity_output_groups(case):
    dtype, B, T, H, dk, dv = case
    say("gdn groups", case)
    d = make_inputs(GDN, B, T, H, dk, dv, dtype, seed=400 + T + dv, keys="aniso", lam="random")
    compare(GDN, d, dtype)


@pytest.mark.parametrize("backbone", [GLA, GDN])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_uncentred_scaled_with_initial_states(backbone, dtype):
    """Uncentred ablation Sigma := Cbar, read scale != 1, t0 > 0 and initial states."""
    say("uncentred/scale/t0", backbone, dtype)
    B, T, H, dk, dv = 1, 140, 2, 64, 128
    d = make_inputs(backbone, B, T, H, dk, dv, dtype, seed=7, lam="random")
    rng = np.random.default_rng(3)
    S0 = rng.standard_normal((B, H, dv, dk)) * 0.2
    Kp = rng.standard_normal((B, H, 30, dk))
    Kp /= np.linalg.norm(Kp, axis=-1, keepdims=True)
    C0 = np.einsum("bhnc,bhnd->bhcd", Kp, Kp) / 30
    mu0 = Kp.mean(axis=2)
    for centered in (True, False):
        compare(backbone, d, dtype, S0=S0.astype(np.float32).astype(np.float64),
                C0=C0.astype(np.float32).astype(np.float64),
                mu0=mu0.astype(np.float32).astype(np.float64), t0=30, centered=centered,
                scale=0.125)


def test_correction_changes_output_fp32():
    """fp32: Delta o = o(lam) - o(lam = 0) against the oracle's Delta o, so that a kernel that
    skipped the contraction would fail even where the correction is small."""
    w = WORKLOADS["gla_small_fp32"]
    say("delta-o", w)
    d = make_inputs(GLA, w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=w.seed)
    d0 = dict(d)
    d0["lam"] = torch.zeros_like(d["lam"])
    g1, g0 = gpu_fwd(GLA, d), gpu_fwd(GLA, d0)
    r1, r0 = oracle_fwd(GLA, d), oracle_fwd(GLA, d0)
    e = nerr(g1["o"] - g0["o"], r1["o"] - r0["o"])
    assert e <= 1e-3, e
    assert np.max(np.abs(r1["o"] - r0["o"])) > 1e-3  # the correction is visible


@pytest.mark.parametrize("backbone", [GLA, GDN])
def test_lambda_zero_is_plain_backbone(backbone):
    d = make_inputs(backbone, 1, 129, 2, 128, 128, BF16, seed=9, lam="const", lam_value=0.0)
    errs, gout, ref = compare(backbone, d, BF16)
    np.testing.assert_array_equal(gout["qclean"], to_f64(d)["q"])


@pytest.mark.parametrize("backbone", [GLA, GDN])
@pytest.mark.parametrize("split", [64, 100])
def test_split_sequence_continuation(backbone, split):
    """fwd(T) equals fwd(T1) followed by fwd(T - T1) from the returned (S, Cbar, mu) and
    t0 = T1, chunk-aligned or not."""
    say("split", backbone, split)
    dtype = F32
    d = make_inputs(backbone, 1, 230, 2, 64, 64, dtype, seed=11, lam="random")
    full = gpu_fwd(backbone, d)
    a = {k: v[:, :split].contiguous() for k, v in d.items()}
    b = {k: v[:, split:].contiguous() for k, v in d.items()}
    ra = gpu_fwd(backbone, a)
    st = {k: torch.from_numpy(ra[k]).float().cuda() for k in ("ST", "CT", "muT")}
    rb = gpu_fwd(backbone, b, S0=st["ST"], C0=st["CT"], mu0=st["muT"], t0=split)
    assert nerr(rb["o"], full["o"][:, split:]) <= 1e-4
    assert nerr(rb["ST"], full["ST"]) <= 1e-4
    assert nerr(rb["CT"], full["CT"]) <= 1e-5


@pytest.mark.parametrize("backbone", [GLA, GDN])
def test_deterministic(backbone):
    d = make_inputs(backbone, 2, 300, 2, 128, 256, BF16, seed=13, lam="random")
    a, b = gpu_fwd(backbone, d), gpu_fwd(backbone, d)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])


@pytest.mark.parametrize("backbone", [GLA, GDN])
def test_empty_sequence_returns_initial_states(backbone):
    d = make_inputs(backbone, 1, 0, 2, 64, 64, F32, seed=1)
    S0 = torch.randn(1, 2, 64, 64, device="cuda")
    C0 = torch.randn(1, 2, 64, 64, device="cuda")
    mu0 = torch.randn(1, 2, 64, device="cuda")
    out = gpu_fwd(backbone, d, S0=S0, C0=C0, mu0=mu0, t0=3)
    np.testing.assert_array_equal(out["ST"], np64(S0))
    np.testing.assert_array_equal(out["CT"], np64(C0))
    np.testing.assert_array_equal(out["muT"], np64(mu0))


def test_head_permutation_equivariance():
    d = make_inputs(GLA, 2, 100, 3, 64, 64, BF16, seed=17, lam="random")
    perm = [2, 0, 1]
    dp = {k: v[:, :, perm].contiguous() for k, v in d.items()}
    a, b = gpu_fwd(GLA, d), gpu_fwd(GLA, dp)
    np.testing.assert_array_equal(a["o"][:, :, perm], b["o"])
    np.testing.assert_array_equal(a["ST"][:, perm], b["ST"])


# ------------------------------------------------ full workloads, every sequence


def per_head_check(w_backbone, dtype, d, gout, ref, label):
    """Assert the bar on every (batch, head) sequence on its own: o, the final states and
    the correction term, each normalised by that sequence's own reference."""
    q = to_f64(d)["q"]
    B, H = q.shape[0], q.shape[2]
    worst, worst_elem = {}, {}
    tol = TOL[dtype]
    for b in range(B):
        for h in range(H):
            sl = (slice(b, b + 1), slice(h, h + 1))
            r = {k: (v[sl[0], :, sl[1]] if v.ndim == 4 and k in ("o", "qclean") else v[sl[0], sl[1]])
                 for k, v in ref.items() if k in ("o", "qclean", "ST", "CT", "muT")}
            errs, elem = fwd_errors(gout, r, q[sl[0], :, sl[1]], True, sl)
            for k, v in errs.items():
                worst[k] = max(worst.get(k, 0.0), v)
            for k, v in elem.items():
                worst_elem[k] = max(worst_elem.get(k, 0.0), v)
            assert all(v <= tol for v in errs.values()), (label, b, h, errs)
    say("  %s: %d sequences, worst" % (label, B * H), worst, "element-wise", worst_elem)


def full_size_check(name, **input_kw):
    """The workload exactly as the benchmark launches it; the oracle recomputes every
    (batch, head) sequence."""
    w = WORKLOADS[name]
    say("full size", name, input_kw)
    d = make_inputs(w.backbone, w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=w.seed, **input_kw)
    gout = gpu_fwd(w.backbone, d)
    ref = oracle_fwd(w.backbone, d)
    per_head_check(w.backbone, w.dtype, d, gout, ref, name)


def test_full_gla_500m_t2k():
    full_size_check("gla_500m_t2k")


def test_full_gdn_1p3b_t4k():
    full_size_check("gdn_1p3b_t4k")


def test_full_gla_500m_t20k():
    full_size_check("gla_500m_t20k")


def test_full_gdn_1p3b_t20k():
    full_size_check("gdn_1p3b_t20k")


# Long-context stress of the running statistics (App. B's 1/t normalisation at large
# t; App. G): at T = 20480 with a strong common key direction (mean-shifted keys,
# where Cbar - mu mu^T cancels heavily) or a strongly anisotropic key spread, and a
# random contraction gate, every head compared with the oracle.
@pytest.mark.parametrize("keys", ["meanshift", "aniso"])
@pytest.mark.parametrize("name", ["gla_500m_t20k", "gdn_1p3b_t20k"])
def test_full_t20k_key_stress(name, keys):
    full_size_check(name, keys=keys, lam="random")
