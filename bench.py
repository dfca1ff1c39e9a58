#!/usr/bin/env python3
"""Benchmark of the CCQ chunkwise forward on one MI355X.

One step = one CCQ-GLA forward on the ~500M-layer shape (B=8, T=2048, H=4,
dk=128, dv=256) plus one CCQ-Gated-DeltaNet forward on the ~1.3B-layer shape
(B=4, T=4096, H=8, dk=dv=256), bf16 io, fp32 states, chunk 64, inputs resident
in HBM.  `value` is the tokens of both calls divided by the mean step time of
`--steps` steps timed without per-kernel events; the same number of steps is
then timed again with the library's per-kernel HIP events recorded around every
launch (`ms_per_step_traced`), and those events give the per-kernel durations.
The line also carries the per-kernel HIP-event timings, the roofline of the
dominant kernel, per-workload figures (including T=20480, the GLA and Gated
DeltaNet training steps and the one-token recurrent decode step on the cache)
and the fp64 CPU oracle timed on a bounded sample of the same inputs.

    python bench.py [--gpus 1] [--steps 40] [--warmup 20]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "CCQ chunkwise fwd tokens/s per GPU (GLA & GDN, T=4K); % of MFMA peak"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
CHUNK = 64


def gla_seg(bh: int, nc: int, dk: int, dv: int) -> int:
    """Chunks per segment of the GLA state pass (the library's policy; 0 = one
    segment): the segment count minimising rounds of 512 workgroups x chunks per
    segment (+2 for the scan when segmented), the fewest segments on a tie."""
    tiles = bh * (dk // 64) * (dv // 64)
    best_ns, best_cost = 1, None
    for ns in range(1, min(64, nc) + 1):
        sl = -(-nc // ns)
        if -(-nc // sl) != ns or (ns > 1 and sl < 4):
            continue
        cost = -(-(tiles * ns) // 512) * sl + (2 if ns > 1 else 0)
        if best_cost is None or cost < best_cost:
            best_ns, best_cost = ns, cost
    return -(-nc // best_ns) if best_ns > 1 else 0


def clean_seg(bh: int, nc: int) -> int:
    """Chunks per segment of the query contraction (the library's policy: the length
    from 2 to 64 minimising rounds of 256 workgroups x chunks per segment, the longest
    on a tie)."""
    best, best_cost = 2, None
    for seg in range(2, 65):
        cost = -(-(bh * -(-nc // seg)) // 256) * min(seg, nc)
        if best_cost is None or cost <= best_cost:
            best, best_cost = seg, cost
    return best


def gdn_group(w) -> int:
    """Chunks per Gated DeltaNet output workgroup (one stored state per group), as
    the library picks it; 1 for training."""
    if getattr(w, "train", False):
        return 1
    vpw = max(1, w.dv // 128)   # the output kernel carries S only where it fits the registers
    if w.dk * vpw * (2 if w.dtype == __import__("torch").bfloat16 else 4) > 1024:
        return 1
    nc = -(-w.T // CHUNK)
    best, best_cost = 1, None
    for g in (1, 2, 4, 8):   # rounds of 256 workgroups x (group + 1), the largest on a tie
        cost = -(-(w.B * w.H * -(-nc // g)) // 256) * (g + 1)
        if best_cost is None or cost <= best_cost:
            best, best_cost = g, cost
    return best


def gla_group(w) -> int:
    """Chunks per GLA output workgroup (one stored state per group), as the library
    picks it; 1 for training, fp32 and dv > 256."""
    import torch
    if getattr(w, "train", False) or w.dtype != torch.bfloat16 or w.dv > 256 or w.dk not in (64, 128):
        return 1
    nc, bh = -(-w.T // CHUNK), w.B * w.H
    best, best_cost = 1, -(-(bh * nc) // 512) * 3   # one chunk per workgroup, two per compute unit
    for g in (2, 4, 8):   # rounds of 256 workgroups x (group + 1), the largest on a tie
        cost = -(-(bh * -(-nc // g)) // 256) * (g + 1)
        if cost <= best_cost:
            best, best_cost = g, cost
    return best


def kernel_cost(kernel: str, w, io_bytes: int = 2, gate_bytes: int = 2):
    """Algorithmic (bytes, flops) of one launch of `kernel` on workload w: every
    input read once, every output written once; products counted at 2 flops per
    multiply-add, the C x C chunk blocks counted dense."""
    BH, ntok = w.B * w.H, w.B * w.T * w.H
    dk, dv, C = w.dk, w.dv, CHUNK
    NC = -(-w.T // C)
    NS = -(-NC // clean_seg(BH, NC))
    gs = gla_seg(BH, NC, dk, dv)
    GS = -(-NC // gs) if gs else 1   # segments of the GLA state pass
    if kernel in ("gla_state", "gla_out") and getattr(w, "train", False):
        GS = 1
    stats = BH * NS * dk * dk               # elements of the segment statistics
    if kernel == "clean_gram":      # k in; segment Gram (fp32), chunk and segment key sums out
        by = ntok * dk * io_bytes + stats * 4 + BH * (NC + NS) * dk * 4
        fl = ntok * 2 * dk * dk
    elif kernel == "clean_prefix":  # Gram (fp32) and segment key sums in; entry moments out (io)
        by = stats * (4 + io_bytes) + BH * NS * dk * 4 + BH * dk * 4
        fl = stats * 6
    elif kernel in ("clean_out", "clean_out_train", "clean_dq"):
        # x, k, lam, entry moments, chunk key sums in; x_clean out (+ Sigma x, m.x)
        by = ntok * (3 * dk * io_bytes + 4) + stats * io_bytes + BH * NC * dk * 4
        if kernel == "clean_out_train":
            by += ntok * (4 * dk + 4)
        elif kernel == "clean_dq":
            by += ntok * (4 * dk + 4)
        fl = ntok * (2 * dk * dk + 4 * C * dk)
    elif kernel == "gla_state":     # k, g, v in; group-entry (segment-local) states, segment totals out
        NG = -(-NC // gla_group(w))
        by = ntok * (dk * io_bytes + dk * gate_bytes + dv * io_bytes) + BH * NG * dv * dk * io_bytes \
            + BH * GS * dv * dk * 4 + (BH * (GS + NC) * dk * 4 if GS > 1 else 0)
        fl = ntok * (2 * dk * dv)
    elif kernel == "gla_scan":      # segment totals in; segment entry states and final state out
        by = BH * GS * (dv * dk * 4 + dk * 4) + BH * (GS - 1) * dv * dk * io_bytes + BH * dv * dk * 4
        fl = BH * GS * dv * dk * 2
    elif kernel == "gla_out":       # q_clean, k, g, v, group-entry states, segment entry states in; o out
        NG = -(-NC // gla_group(w))
        by = ntok * (2 * dk * io_bytes + dk * gate_bytes + 2 * dv * io_bytes) + BH * NG * dv * dk * io_bytes \
            + (BH * (GS - 1) * dv * dk * io_bytes + BH * NG * dk * 4 if GS > 1 else 0)
        # plus the state carried through each group: S <- S diag(e^{b_C}) + V Kd^T
        fl = ntok * (2 * C * dk + 2 * dk * dv + 2 * C * dv) + BH * (NC - NG) * 2 * C * dk * dv
    elif kernel == "gdn_tri":       # k, log alpha, beta in; chunk transforms Tm and decays out
        by = ntok * (dk * io_bytes + 8 + C * io_bytes + 4)
        fl = ntok * (2 * C * dk)
    elif kernel == "gdn_state":     # k, v, Tm, decays, beta in; group-entry states, U, final state out
        G = gdn_group(w)
        by = ntok * (dk * io_bytes + dv * io_bytes + C * io_bytes + 8 + dv * io_bytes) \
            + BH * -(-NC // G) * dv * dk * io_bytes + (0 if getattr(w, "train", False) else BH * dv * dk * 4)
        fl = ntok * (4 * dk * dv + 2 * C * dv)
    elif kernel == "gdn_out":       # q_clean, k, group-entry states, U, decays in; o out
        G = gdn_group(w)
        by = ntok * (2 * dk * io_bytes + 2 * dv * io_bytes + 4) + BH * -(-NC // G) * dv * dk * io_bytes
        # plus the state carried through each group: S <- e^{gamma_C} S + U^T diag(.) K
        fl = ntok * (2 * C * dk + 2 * dk * dv + 2 * C * dv) + BH * (NC - -(-NC // G)) * 2 * C * dk * dv
    elif kernel == "gla_dstate":
        by = ntok * (dk * io_bytes + dk * gate_bytes + dv * io_bytes + dv * dk * io_bytes // C)
        fl = ntok * (2 * dk * dv)
    elif kernel == "gla_bwd_chunk":
        by = ntok * (2 * dk * io_bytes + dk * gate_bytes + 3 * dv * io_bytes + 2 * dv * dk * io_bytes // C
                     + 4 * dk + 12 * dk + dk * io_bytes + 4)
        fl = ntok * (6 * dk * dv + 4 * C * dv + 6 * C * dk)
    elif kernel == "gla_dg":
        by = ntok * (4 * dk + dk * gate_bytes)
        fl = ntok * dk
    elif kernel == "gdn_bwd_prep":  # q_clean, k, gamma, Tm in; decayed scores P^T and Tm^T out
        by = ntok * (2 * dk * io_bytes + 4 + 3 * C * io_bytes)
        fl = ntok * (2 * C * dk)
    elif kernel == "gdn_dstate":    # q_clean, k, dO, P^T, Tm^T, decays in; dS_{r+1}, dR out
        by = ntok * (2 * dk * io_bytes + 2 * dv * io_bytes + 2 * C * io_bytes + 16
                     + dv * dk * io_bytes // C)
        fl = ntok * (6 * dk * dv + 4 * C * dv)
    elif kernel == "gdn_bwd_chunk":  # q_clean, k, v, dO, dR, U, S_r, dS_{r+1}, Sigma q, decays in;
        # dq_clean (fp32 and io), backbone dk (fp32), dv, dlogalpha, dbeta, dlam out
        by = ntok * (3 * dk * io_bytes + 5 * dv * io_bytes + 2 * dv * dk * io_bytes // C
                     + 12 * dk + 28)
        fl = ntok * (6 * dk * dv + 4 * C * dv + 12 * C * dk)
    elif kernel in ("decode", "decode_split"):  # cache (S, Cbar fp32) read and written once,
        # mu, q, k, v, gates, o
        gb = dk * gate_bytes if w.backbone == 0 else 8
        by = BH * (8 * dv * dk + 8 * dk * dk + dk * (2 * io_bytes + 20) + 2 * dv * io_bytes + gb + 4)
        fl = BH * (5 * dk * dk + 6 * dv * dk)
    elif kernel == "prep":          # raw q, k in; normalised q, k and the gate out (W_lambda once)
        by = ntok * (4 * dk * io_bytes + 4) + w.H * w.H * dk * 4 + w.H * 4
        fl = ntok * (2 * w.H * dk + 6 * dk)
    elif kernel == "prep_scales":   # raw q, k in; the two row scales and the gate out
        by = ntok * (2 * dk * io_bytes + 12) + w.H * w.H * dk * 4 + w.H * 4
        fl = ntok * (2 * w.H * dk + 4 * dk)
    elif kernel == "ccq_dk":
        by = ntok * (3 * dk * io_bytes + 12 + 4 * dk + dk * io_bytes)
        fl = ntok * (6 * dk * dk + 8 * C * dk)
    elif kernel.startswith("varlen_"):
        # packed rows read and padded rows written (gathers), padded rows read and
        # packed rows written (scatter); rows of H heads
        real = getattr(w, "packed_rows", w.B * w.T)
        pad = w.B * w.T
        rb = {"varlen_gather_qk": dk * io_bytes, "varlen_gather_v": dv * io_bytes,
              "varlen_gather_scalar": 4, "varlen_scatter_o": dv * io_bytes}.get(kernel, 0) * w.H
        if kernel == "varlen_fix":
            by, fl = BH * (dk * dk + dk) * 8, 0
        elif kernel == "varlen_scatter_o":
            by, fl = 2 * real * rb, 0
        else:
            by, fl = (real + pad) * rb, 0
    else:
        raise KeyError(kernel)
    return by, fl


def method_cost(w, io_bytes=None, gate_bytes=None):
    """Algorithmic (bytes, flops) of the method itself on workload w, per forward call
    (the work the call must do, whatever the kernels): per token and head
      F_CCQ = 4 dk^2 + 4 C dk                               (statistics and contraction)
      F_GLA = 2 C (dk + dv) + 4 dk dv                       (chunk read and write)
      F_GDN = 6 C dk + 4 C dv + 6 dk dv + C^2 / 3           (WY/UT transform, read, write)
    with the C x C blocks counted dense; bytes = q, k, v, o, the gates and lambda read or
    written once, plus the final (S, Cbar, mu) in fp32.  A training step counts three
    times the forward flops (the backward taken as twice the forward) and also reads dO
    and writes dq, dk, dv, the gate gradients and dlambda once."""
    import torch
    io_bytes = io_bytes or (2 if w.dtype == torch.bfloat16 else 4)
    gate_bytes = gate_bytes or io_bytes
    BH = w.B * w.H
    n = getattr(w, "packed_rows", w.B * w.T) * w.H   # a packed batch: its real tokens only
    dk, dv, C = w.dk, w.dv, CHUNK
    f = 4 * dk * dk + 4 * C * dk
    if w.backbone == 0:
        f += 2 * C * (dk + dv) + 4 * dk * dv
        gates = dk * gate_bytes
    else:
        f += 6 * C * dk + 4 * C * dv + 6 * dk * dv + C * C / 3
        gates = 8
    tok = (2 * dk + 2 * dv) * io_bytes + gates + 4
    states = BH * (dv * dk + dk * dk + dk) * 4
    if getattr(w, "train", False):
        return n * (2 * tok + 4) + states, 3 * f * n
    return n * tok + states, f * n


def method_roofline(w, ms, traffic=None):
    """Roofline of one whole call (all of its kernels) on the method's own work: the
    bound is whichever of flops / MFMA peak and bytes / HBM peak is longer; `achieved`
    is that work over the measured call time; `traffic` the rocprofv3 HBM bytes summed
    over the call's kernels (None when any is missing or stale)."""
    by, fl = method_cost(w)
    sec = ms * 1e-3
    t_mfma = fl / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = by / (PEAK_HBM_GBS * 1e9)
    if t_mfma >= t_hbm:
        ach = fl / sec / 1e12
        r = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
             "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4)}
    else:
        ach = by / sec / 1e9
        r = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(ach / PEAK_HBM_GBS, 4)}
    r["traffic"] = traffic
    r["traffic_ratio"] = round(traffic / by, 3) if traffic else None
    r["method_bytes"] = by
    r["method_flops"] = int(fl)
    r["roofline_us"] = round(max(t_mfma, t_hbm) * 1e6, 2)
    r["ms_per_call"] = round(ms, 5)
    r["mfma_frac"] = round(fl / sec / 1e12 / PEAK_BF16_TFLOPS, 4)
    r["hbm_frac"] = round(by / sec / 1e9 / PEAK_HBM_GBS, 4)
    return r


def call_traffic(kernels, workload):
    """rocprofv3 HBM bytes of one call: the committed per-kernel counter figures summed,
    or None when any kernel's figure is missing or stale."""
    tot = 0
    for k in kernels:
        t = measured_traffic(k, workload)
        if t is None:
            return None
        tot += t
    return tot


CLEAN = ["clean_gram", "clean_prefix"]
KERNELS = {0: ["gla_state"] + CLEAN + ["clean_out", "gla_out"],
           "gla_seg": ["gla_state", "gla_scan"] + CLEAN + ["clean_out", "gla_out"],
           1: ["gdn_tri", "gdn_state"] + CLEAN + ["clean_out", "gdn_out"],
           "train": CLEAN + ["clean_out_train", "gla_state", "gla_out", "gla_dstate",
                             "gla_bwd_chunk", "gla_dg", "clean_dq", "ccq_dk"],
           "gdn_train": CLEAN + ["clean_out_train", "gdn_tri", "gdn_state", "gdn_out",
                                 "gdn_bwd_prep", "gdn_dstate", "gdn_bwd_chunk", "clean_dq",
                                 "ccq_dk"]}
VARLEN_GDN = KERNELS[1]  # the forward kernels read the packed rows themselves
KERNEL_SYMBOL = {"prep_scales": "prep_kernel (row scales)", "varlen_gather_qk": "varlen_copy_kernel", "varlen_gather_v": "varlen_copy_kernel",
                 "varlen_gather_scalar": "varlen_copy_kernel", "varlen_scatter_o": "varlen_copy_kernel",
                 "varlen_fix": "varlen_cache_fix_kernel", "prep": "prep_kernel", "decode": "decode_kernel", "decode_split": "decode_cbar_kernel+decode_s_kernel", "clean_gram": "clean_gram_kernel",
                 "clean_prefix": "clean_prefix_kernel", "clean_out": "clean_out_kernel",
                 "clean_out_train": "clean_out_kernel", "clean_dq": "clean_out_kernel",
                 "gla_state": "gla_state_kernel", "gla_scan": "gla_scan_kernel", "gla_out": "gla_out_kernel",
                 "gdn_tri": "gdn_tri_kernel", "gdn_state": "gdn_state_dma_kernel",
                 "gdn_out": "gdn_out_kernel", "gla_dstate": "gla_state_kernel (reverse)",
                 "gla_bwd_chunk": "gla_bwd_chunk_kernel", "gla_dg": "gla_dg_kernel",
                 "gdn_bwd_prep": "gdn_bwd_prep_kernel", "gdn_dstate": "gdn_dstate_kernel",
                 "gdn_bwd_chunk": "gdn_bwd_chunk_kernel", "ccq_dk": "ccq_dk_kernel"}


def _source(kernel: str) -> str:
    if kernel.startswith("clean"):
        return "ccq_clean.hip"
    if kernel in ("gla_state", "gla_scan", "gla_out", "gla_dstate"):
        return "ccq_gla.hip"
    if kernel in ("gdn_bwd_prep", "gdn_dstate", "gdn_bwd_chunk"):
        return "ccq_gdn_bwd.hip"
    if kernel.startswith("decode"):
        return "ccq_decode.hip"
    if kernel in ("prep", "prep_scales"):
        return "ccq_prep.hip"
    if kernel.startswith("varlen"):
        return "ccq_varlen.hip"
    if kernel.startswith("gdn"):
        return "ccq_gdn.hip"
    return "ccq_bwd.hip"


KERNEL_SOURCE = {k: _source(k) for k in KERNEL_SYMBOL}


def source_sha(kernel: str) -> str:
    p = os.path.join(ROOT, "paper_2606_01294_amd", "csrc", KERNEL_SOURCE[kernel])
    h = hashlib.sha256()
    for f in (p, os.path.join(ROOT, "paper_2606_01294_amd", "csrc", "ccq_device.h")):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or None when the
    kernel's source changed since they were taken."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        rec = json.load(open(p)).get("%s@%s" % (kernel, workload))
    except (ValueError, OSError):
        return None
    if not rec or rec.get("source_sha") != source_sha(kernel):
        return None
    return rec.get("bytes_per_launch")


class Call:
    """One pre-allocated CCQ forward call on a workload (inputs resident on the GPU)."""

    def __init__(self, w, torch, ccq, inputs):
        self.w = w
        d = inputs.workload_inputs(w)
        self.cpu = d
        self.d = inputs.to_device(d)
        dev = self.d["q"].device
        B, T, H, dk, dv = w.B, w.T, w.H, w.dk, w.dv
        self.out = {"o": torch.empty((B, T, H, dv), dtype=w.dtype, device=dev),
                    "ST": torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev),
                    "CT": torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev),
                    "muT": torch.empty((B, H, dk), dtype=torch.float32, device=dev)}
        shape = ccq.make_shape(B, T, H, dk, dv, w.dtype, w.dtype)
        self.ws = torch.empty(max(1, ccq.ccq_workspace_size(shape, w.backbone, w.train)),
                              dtype=torch.uint8, device=dev)
        if w.train:
            self.out = {"o": self.out["o"]}
            gate = "g" if w.backbone == 0 else "logalpha"
            for name, ref in (("dq", "q"), ("dk", "k"), ("dv", "v"), ("dg", gate)):
                self.out[name] = torch.empty_like(self.d[ref])
            self.out["dlam"] = torch.empty_like(self.d["lam"])
            if w.backbone == 1:
                self.out["dbeta"] = torch.empty_like(self.d["beta"])
        self.ccq = ccq
        if w.train:
            self.kernels = KERNELS["train" if w.backbone == 0 else "gdn_train"]
        elif w.backbone == 0 and gla_seg(B * H, -(-T // CHUNK), dk, dv):
            self.kernels = KERNELS["gla_seg"]   # the state pass in segments adds a scan
        else:
            self.kernels = KERNELS[w.backbone]

    def __call__(self):
        d = self.d
        if self.w.train and self.w.backbone == 0:
            self.ccq.ccq_fwd_bwd(d["q"], d["k"], d["v"], d["g"], d["lam"], d["dO"], out=self.out,
                                 workspace=self.ws)
        elif self.w.train:
            self.ccq.ccq_fwd_bwd(d["q"], d["k"], d["v"], d["logalpha"], d["lam"], d["dO"],
                                 out=self.out, workspace=self.ws, backbone=1, beta=d["beta"])
        elif self.w.backbone == 0:
            self.ccq.ccq_gla_fwd(d["q"], d["k"], d["v"], d["g"], d["lam"], out=self.out,
                                 workspace=self.ws)
        else:
            self.ccq.ccq_gdn_fwd(d["q"], d["k"], d["v"], d["logalpha"], d["beta"], d["lam"],
                                 out=self.out, workspace=self.ws)


class DecayCall(Call):
    """The Gated DeltaNet forward with the decay-aligned statistics (ccq_shape.decay_aligned)."""

    def __call__(self):
        d = self.d
        self.ccq.ccq_gdn_fwd(d["q"], d["k"], d["v"], d["logalpha"], d["beta"], d["lam"],
                             out=self.out, workspace=self.ws, decay_aligned=True)


class DecodeCall:
    """One recurrent decode step (one token per sequence) at position T + 1 of a
    workload's shape, with the cache resident on the GPU (updated in place)."""

    def __init__(self, w, torch, ccq, inputs):
        import dataclasses
        self.w = dataclasses.replace(w, name=w.name.replace("_t", "_decode_t"), T=1)
        self.t0 = w.T
        d = inputs.make_inputs(w.backbone, w.B, 1, w.H, w.dk, w.dv, w.dtype, seed=w.seed)
        self.d = {k: v[:, 0].contiguous().cuda() for k, v in d.items()}
        dev = self.d["q"].device
        gen = torch.Generator(device="cpu").manual_seed(w.seed)
        B, H, dk, dv = w.B, w.H, w.dk, w.dv
        self.S = (0.1 * torch.randn(B, H, dv, dk, generator=gen)).to(dev)
        self.C = (torch.randn(B, H, dk, dk, generator=gen) / dk).to(dev)
        self.mu = (torch.randn(B, H, dk, generator=gen) / dk).to(dev)
        self.o = torch.empty((B, H, dv), dtype=w.dtype, device=dev)
        # the decode workspace is allocated once and kept, as a serving loop would
        need = ccq.ccq_decode_workspace_size(ccq.make_shape(B, 1, H, dk, dv, w.dtype))
        self.ws = torch.empty(max(1, need), dtype=torch.uint8, device=dev)
        self.ccq = ccq
        # a workspace is needed exactly when the step is split into two launches
        self.kernels = ["decode_split" if need else "decode"]

    def __call__(self):
        d = self.d
        gate = d["g"] if self.w.backbone == 0 else d["logalpha"]
        self.ccq.ccq_decode(d["q"], d["k"], d["v"], gate, d["lam"], self.S, self.C, self.mu,
                            self.t0, backbone=self.w.backbone, beta=d.get("beta"), out=self.o,
                            workspace=self.ws)


class PrepCall:
    """Pre-processing of a workload's raw q, k (l2 normalisation per head and the gate
    from the pre-split query), inputs resident on the GPU."""

    def __init__(self, w, torch, ccq, inputs):
        import dataclasses
        self.w = dataclasses.replace(w, name=w.name.replace("_t", "_prep_t"))
        gen = torch.Generator().manual_seed(w.seed)
        B, T, H, dk = w.B, w.T, w.H, w.dk
        self.q = torch.randn(B, T, H, dk, generator=gen).to(w.dtype).cuda()
        self.k = torch.randn(B, T, H, dk, generator=gen).to(w.dtype).cuda()
        self.wl = (torch.randn(H, H * dk, generator=gen) / (H * dk) ** 0.5).cuda()
        self.bl = torch.randn(H, generator=gen).cuda()
        self.out = {"q": torch.empty_like(self.q), "k": torch.empty_like(self.k),
                    "lam": torch.empty((B, T, H), dtype=torch.float32, device=self.q.device)}
        self.ccq = ccq
        self.kernels = ["prep"]

    def __call__(self):
        self.ccq.ccq_prep(self.q, self.k, self.wl, self.bl, out=self.out)


class RawCall:
    """The Gated DeltaNet forward from raw q, k (ccq_fwd_raw: the l2 normalisation and
    the gate folded into the forward), inputs resident on the GPU; the same raw tensors
    as the pre-processing workload."""

    def __init__(self, w, torch, ccq, inputs):
        import dataclasses
        self.w = dataclasses.replace(w, name=w.name.replace("_t", "_raw_t"))
        gen = torch.Generator().manual_seed(w.seed)
        B, T, H, dk, dv = w.B, w.T, w.H, w.dk, w.dv
        self.q = torch.randn(B, T, H, dk, generator=gen).to(w.dtype).cuda()
        self.k = torch.randn(B, T, H, dk, generator=gen).to(w.dtype).cuda()
        self.wl = (torch.randn(H, H * dk, generator=gen) / (H * dk) ** 0.5).cuda()
        self.bl = torch.randn(H, generator=gen).cuda()
        d = inputs.workload_inputs(w)
        self.v, self.la, self.beta = d["v"].cuda(), d["logalpha"].cuda(), d["beta"].cuda()
        self.out = {"o": torch.empty((B, T, H, dv), dtype=w.dtype, device="cuda"),
                    "ST": torch.empty((B, H, dv, dk), dtype=torch.float32, device="cuda"),
                    "CT": torch.empty((B, H, dk, dk), dtype=torch.float32, device="cuda"),
                    "muT": torch.empty((B, H, dk), dtype=torch.float32, device="cuda")}
        shape = ccq.make_shape(B, T, H, dk, dv, w.dtype, w.dtype)
        self.ws = torch.empty(max(1, ccq.ccq_fwd_raw_workspace_size(shape, 1)), dtype=torch.uint8,
                              device="cuda")
        self.ccq = ccq
        self.kernels = ["prep_scales"] + KERNELS[1]

    def __call__(self):
        self.ccq.ccq_fwd_raw(self.q, self.k, self.wl, self.bl, self.v, self.la, self.beta,
                             backbone=1, out=self.out, workspace=self.ws)


class VarlenCall:
    """The Gated DeltaNet forward on a packed batch: 2B sequences of lengths uniform in
    [T/4, 3T/4] (about the tokens of the B x T workload), read by the kernels straight
    from the packed rows (inputs resident on the GPU)."""

    def __init__(self, w, torch, ccq, inputs):
        import dataclasses
        lens = inputs.varlen_lengths(w)
        self.lens = lens
        T = max(lens)
        self.w = dataclasses.replace(w, name=w.name.replace("_t", "_varlen_t"), B=len(lens), T=T)
        object.__setattr__(self.w, "packed_rows", sum(lens))  # rows of H heads actually present
        d = inputs.make_inputs(w.backbone, len(lens), T, w.H, w.dk, w.dv, w.dtype, seed=w.seed)
        self.d = inputs.to_device(inputs.pack(d, lens))
        dev = self.d["q"].device
        offs = [0]
        for L in lens:
            offs.append(offs[-1] + L)
        self.cu = torch.tensor(offs, dtype=torch.int32, device=dev)
        B, H, dk, dv = len(lens), w.H, w.dk, w.dv
        self.out = {"o": torch.empty((sum(lens), H, dv), dtype=w.dtype, device=dev),
                    "ST": torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev),
                    "CT": torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev),
                    "muT": torch.empty((B, H, dk), dtype=torch.float32, device=dev)}
        shape = ccq.make_shape(B, T, H, dk, dv, w.dtype, w.dtype)
        self.ws = torch.empty(max(1, ccq.ccq_varlen_workspace_size(shape, w.backbone)),
                              dtype=torch.uint8, device=dev)
        self.ccq = ccq
        self.kernels = VARLEN_GDN

    def __call__(self):
        d = self.d
        self.ccq.ccq_gdn_fwd_varlen(d["q"], d["k"], d["v"], d["logalpha"], d["beta"], d["lam"],
                                    self.cu, self.w.T, out=self.out, workspace=self.ws)


def time_calls(torch, ccq, calls, steps, warmup, with_plain=False):
    """Warm up, then time exactly `steps` steps (each step = every call once) between two
    synchronisations; per-kernel durations come from HIP events the library records on
    its stream around each of its launches.  With with_plain, exactly `steps` more steps
    are timed first without any events (the event records add dispatch gaps of their
    own), and that time is returned as well, then `steps` more with one pair of events
    around each whole call (every launch of a call is on torch's current stream), whose
    mean durations are stored as `ms_call` on each call."""
    for _ in range(warmup):
        for c in calls:
            c()
    torch.cuda.synchronize()
    ms_plain = None
    if with_plain:
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for i in range(steps):
            for c in calls:
                c()
        end.record()
        torch.cuda.synchronize()
        ms_plain = start.elapsed_time(end) / steps
        cev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in calls] for _ in range(steps)]
        for i in range(steps):
            for j, c in enumerate(calls):
                cev[i][j][0].record()
                c()
                cev[i][j][1].record()
        torch.cuda.synchronize()
        for j, c in enumerate(calls):
            c.ms_call = sum(cev[i][j][0].elapsed_time(cev[i][j][1]) for i in range(steps)) / steps
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2 * len(c.kernels))]
           for c in calls] for _ in range(steps)]
    for step_ev in ev:
        for evs in step_ev:
            for e in evs:
                e.record()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        for j, c in enumerate(calls):
            ccq.ccq_trace_events(ev[i][j])
            c()
    ccq.ccq_trace_events(None)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / steps
    if with_plain:
        return ms_plain, ms_step, per_kernel_times(calls, ev, steps)
    return ms_step, per_kernel_times(calls, ev, steps)


def per_kernel_times(calls, ev, steps):
    per_kernel = []
    for j, c in enumerate(calls):
        for kidx, name in enumerate(c.kernels):
            ts = [ev[i][j][2 * kidx].elapsed_time(ev[i][j][2 * kidx + 1]) for i in range(steps)]
            per_kernel.append({"workload": c.w.name, "kernel": name,
                               "symbol": KERNEL_SYMBOL[name],
                               "ms_mean": sum(ts) / len(ts),
                               "ms_std": (sum((t - sum(ts) / len(ts)) ** 2 for t in ts) /
                                          max(1, len(ts) - 1)) ** 0.5})
    return per_kernel


def roofline(entry, w, name=None):
    """The kernel's own roofline on workload w (`name`: the workload's label when it
    differs from w's, e.g. a variant of the statistics on w's shape)."""
    wn = name or w.name
    by, fl = kernel_cost(entry["kernel"], w)
    sec = entry["ms_mean"] * 1e-3
    intensity = fl / by
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    if intensity < ridge:
        ach = by / sec / 1e9
        r = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(ach / PEAK_HBM_GBS, 4)}
    else:
        ach = fl / sec / 1e12
        r = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
             "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4)}
    r["traffic"] = measured_traffic(entry["kernel"], wn)
    r["kernel"] = entry["symbol"]
    r["workload"] = wn
    r["algorithmic_bytes"] = by
    r["algorithmic_flops"] = fl
    r["ms_per_launch"] = round(entry["ms_mean"], 5)
    return r


EXTRA = ("gla_500m_t2k", "gdn_1p3b_t4k", "gla_500m_t20k", "gdn_1p3b_t20k", "gla_train_t4k",
         "gdn_train_t4k", "gla_500m_decode_t2k", "gdn_1p3b_decode_t4k", "gdn_1p3b_prep_t4k",
         "gdn_1p3b_raw_t4k", "gdn_1p3b_varlen_t4k", "gdn_1p3b_decay_t4k")


def measure_extra(name, torch, ccq, inputs, steps, existing):
    """Figures of one workload on its own: tokens/s from untimed-event steps, per-kernel
    durations and the dominant kernel's roofline from the traced steps."""
    W = inputs.WORKLOADS
    if "_prep_" in name:
        c = PrepCall(W[name.replace("_prep_t", "_t")], torch, ccq, inputs)
        ms, ms_tr, pk = time_calls(torch, ccq, [c], max(20, steps), 5, with_plain=True)
        res = {"tokens_per_s": round(c.w.tokens / (ms * 1e-3), 1), "ms": round(ms, 5),
               "ms_traced": round(ms_tr, 5),
               "kernels_ms": [[e["kernel"], e["symbol"], round(e["ms_mean"], 5)] for e in pk],
               "roofline": roofline(pk[0], c.w)}
    elif "_raw_" in name:
        c = RawCall(W[name.replace("_raw_t", "_t")], torch, ccq, inputs)
        ms, ms_tr, pk = time_calls(torch, ccq, [c], max(5, steps // 2), 3, with_plain=True)
        dom = max(pk, key=lambda e: e["ms_mean"])
        res = {"tokens_per_s": round(c.w.tokens / (ms * 1e-3), 1), "ms": round(ms, 4),
               "ms_traced": round(ms_tr, 4),
               "kernels_ms": [[e["kernel"], e["symbol"], round(e["ms_mean"], 5)] for e in pk],
               "roofline": method_roofline(c.w, c.ms_call), "dominant_kernel": roofline(dom, c.w)}
    elif "_varlen_" in name:
        c = VarlenCall(W[name.replace("_varlen_t", "_t")], torch, ccq, inputs)
        ms, ms_tr, pk = time_calls(torch, ccq, [c], max(5, steps // 2), 3, with_plain=True)
        dom = max(pk, key=lambda e: e["ms_mean"])
        res = {"tokens_per_s": round(sum(c.lens) / (ms * 1e-3), 1), "ms": round(ms, 4),
               "ms_traced": round(ms_tr, 4), "sequences": len(c.lens),
               "packed_tokens": sum(c.lens), "padded_tokens": c.w.B * c.w.T,
               "kernels_ms": [[e["kernel"], e["symbol"], round(e["ms_mean"], 5)] for e in pk],
               "roofline": method_roofline(c.w, c.ms_call),
               "dominant_kernel": roofline(dom, c.w)}
    elif "_decode_" in name:
        c = DecodeCall(W[name.replace("_decode_t", "_t")], torch, ccq, inputs)
        ms, ms_tr, pk = time_calls(torch, ccq, [c], max(20, steps), 5, with_plain=True)
        res = {"tokens_per_s": round(c.w.B / (ms * 1e-3), 1), "ms": round(ms, 5),
               "ms_traced": round(ms_tr, 5), "position": c.t0 + 1,
               "kernels_ms": [[e["kernel"], e["symbol"], round(e["ms_mean"], 5)] for e in pk],
               "roofline": roofline(pk[0], c.w)}
    else:
        if "_decay_" in name:
            c = DecayCall(W[name.replace("_decay_t", "_t")], torch, ccq, inputs)
        else:
            c = existing.get(name) or Call(W[name], torch, ccq, inputs)
        ms, ms_tr, pk = time_calls(torch, ccq, [c], max(5, steps // 2), 3, with_plain=True)
        dom = max(pk, key=lambda e: e["ms_mean"])
        res = {"tokens_per_s": round(c.w.tokens / (ms * 1e-3), 1), "ms": round(ms, 4),
               "ms_traced": round(ms_tr, 4),
               "kernels_ms": [[e["kernel"], e["symbol"], round(e["ms_mean"], 5)] for e in pk],
               "roofline": method_roofline(c.w, c.ms_call,
                                           call_traffic(c.kernels, name if "_decay_" in name else c.w.name)),
               "dominant_kernel": roofline(dom, c.w, name)}
    if name not in existing:
        del c
        torch.cuda.empty_cache()
    return res


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(calls):
    """The fp64 oracle on the host cores (OpenMP over the (batch, head) sequences), run on
    the whole step: every sequence of every workload of the step, on the same inputs."""
    from oracle import ccq_oracle as O

    thr = O.threads()
    total = 0.0
    parts = []
    for c in calls:
        w = c.w
        d = {k: v.double().numpy() for k, v in c.cpu.items()}
        t0 = time.perf_counter()
        if w.backbone == 0:
            O.fwd(d["q"], d["k"], d["v"], d["g"], d["lam"], backbone=O.GLA)
        else:
            O.fwd(d["q"], d["k"], d["v"], d["logalpha"], d["lam"], beta=d["beta"], backbone=O.GDN)
        dt = time.perf_counter() - t0
        total += dt
        parts.append("%s: all %d sequences in %.2f s" % (w.name, w.B * w.H, dt))
    tokens = sum(c.w.tokens for c in calls)
    return {"value": round(tokens / total, 1), "unit": "tokens/s", "cores": thr,
            "kind": "oracle", "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "sample": "the whole step (no extrapolation): " + "; ".join(parts)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the per-workload figures")
    ap.add_argument("--only", metavar="WORKLOAD",
                    help="time only this per-workload entry (for profiling) and print its figures")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (HBM counter "
                         "calibration for rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    args = ap.parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the CCQ hot path here is single-GPU "
              "(heads are independent; multi-GPU sharding is a design note, not built). "
              "Run with --gpus 1.", file=sys.stderr)
        return 2

    import torch
    from paper_2606_01294_amd import ccq, inputs

    if args.copy_calibration:
        x = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": x.numel() * 4, "copy_bytes_written": y.numel() * 4,
                          "launches": 5}))
        return 0
    ccq.lib()  # fails loudly when libccq.so is missing
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    W = inputs.WORKLOADS
    if args.only:
        if args.only not in EXTRA:
            print("--only takes one of: " + ", ".join(EXTRA), file=sys.stderr)
            return 2
        res = {"workload": args.only}
        res.update(measure_extra(args.only, torch, ccq, inputs, args.steps, {}))
        print(json.dumps(res), flush=True)
        return 0
    step_calls = [Call(W["gla_500m_t2k"], torch, ccq, inputs), Call(W["gdn_1p3b_t4k"], torch, ccq, inputs)]
    ms_step, ms_traced, per_kernel = time_calls(torch, ccq, step_calls, args.steps, args.warmup,
                                                with_plain=True)
    tokens = sum(c.w.tokens for c in step_calls)
    value = tokens / (ms_step * 1e-3)

    wl = {c.w.name: c.w for c in step_calls}
    # the roofline of the call that dominates the step, on the method's own work
    dom_call = max(step_calls, key=lambda c: c.ms_call)
    roof = method_roofline(dom_call.w, dom_call.ms_call, call_traffic(dom_call.kernels, dom_call.w.name))
    roof = dict({"kernel": "ccq_%s_fwd" % ("gla" if dom_call.w.backbone == 0 else "gdn"),
                 "scope": "one whole forward call (%d launches: %s)" % (
                     len(dom_call.kernels), ", ".join(dom_call.kernels)),
                 "workload": dom_call.w.name}, **roof)
    dominant = max(per_kernel, key=lambda e: e["ms_mean"])
    step_roof_us = sum(method_roofline(c.w, c.ms_call)["roofline_us"] for c in step_calls)
    step_bytes = sum(method_cost(c.w)[0] for c in step_calls)
    step_flops = sum(method_cost(c.w)[1] for c in step_calls)
    kernels = []
    for e in per_kernel:
        by, fl = kernel_cost(e["kernel"], wl[e["workload"]])
        kernels.append({"workload": e["workload"], "kernel": e["symbol"],
                        "ms": round(e["ms_mean"], 5), "ms_std": round(e["ms_std"], 5),
                        "GB_s": round(by / (e["ms_mean"] * 1e-3) / 1e9, 1),
                        "TFLOP_s": round(fl / (e["ms_mean"] * 1e-3) / 1e12, 2)})

    extra = {}
    if not args.no_extra:
        for name in EXTRA:
            extra[name] = measure_extra(name, torch, ccq, inputs, args.steps,
                                        {c.w.name: c for c in step_calls})

    cpu = None if args.no_cpu_baseline else cpu_baseline(step_calls)

    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "ms_per_step_traced": round(ms_traced, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "ccq_fwd gla_500m_t2k+gdn_1p3b_t4k",
                   "gla": "B=8 T=2048 H=4 dk=128 dv=256 chunk=64 bf16 io, fp32 states",
                   "gdn": "B=4 T=4096 H=8 dk=256 dv=256 chunk=64 bf16 io, fp32 states",
                   "tokens_per_step": tokens},
        "mfma_frac": round(step_flops / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "hbm_frac": round(step_bytes / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "roofline": roof,
        "step_roofline": {"roofline_us": round(step_roof_us, 2),
                          "frac": round(step_roof_us * 1e-3 / ms_step, 4),
                          "calls_ms": {c.w.name: round(c.ms_call, 5) for c in step_calls}},
        "dominant_kernel": roofline(dominant, wl[dominant["workload"]]),
        "kernels": kernels,
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
