"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module draws random tensors and nothing else: it holds none of the CCQ
arithmetic, so the oracle and the HIP path can both be fed from it.  The
recipes stand in for the paper's layer activations (FineWeb-Edu at the 4K
training context, the 4K-20K extrapolation corpora): those datasets and the
trained weights are not available, so the shapes and distributions below are
synthetic.

Draw order (CPU torch.Generator, fp32, then a single cast to the io dtype):
q, k, v, gates, [auxiliary key directions], [random lambda], [dO].
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch
import torch.nn.functional as F

GLA, GDN = 0, 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    backbone: int
    B: int
    T: int
    H: int
    dk: int
    dv: int
    dtype: torch.dtype
    seed: int
    train: bool = False

    @property
    def tokens(self) -> int:
        return self.B * self.T


# The layer shapes the benchmark and the parity tests use.
WORKLOADS = {
    "gla_small_fp32": Workload("gla_small_fp32", GLA, 1, 256, 2, 64, 64, torch.float32, 0),
    "gla_500m_t2k": Workload("gla_500m_t2k", GLA, 8, 2048, 4, 128, 256, torch.bfloat16, 1),
    "gdn_1p3b_t4k": Workload("gdn_1p3b_t4k", GDN, 4, 4096, 8, 256, 256, torch.bfloat16, 2),
    "gla_500m_t20k": Workload("gla_500m_t20k", GLA, 1, 20480, 4, 128, 256, torch.bfloat16, 3),
    "gdn_1p3b_t20k": Workload("gdn_1p3b_t20k", GDN, 1, 20480, 8, 256, 256, torch.bfloat16, 3),
    "gla_train_t4k": Workload("gla_train_t4k", GLA, 4, 4096, 8, 128, 256, torch.bfloat16, 4,
                              train=True),
    "gdn_train_t4k": Workload("gdn_train_t4k", GDN, 4, 4096, 8, 256, 256, torch.bfloat16, 4,
                              train=True),
}


def _unit(x: torch.Tensor) -> torch.Tensor:
    return x / x.norm(dim=-1, keepdim=True).clamp_min(1e-12)


def make_inputs(backbone: int, B: int, T: int, H: int, dk: int, dv: int,
                dtype: torch.dtype = torch.bfloat16, gate_dtype: torch.dtype | None = None,
                seed: int = 0, keys: str = "iso", gates: str = "config", lam="const",
                lam_value: float = 0.5, with_dO: bool = False) -> dict:
    """Draw one batch.

    keys:  "iso"       k = unit(z)                         z ~ N(0, I)
           "aniso"     k = unit(z + 16 a u), a ~ N(0,1) per token, u a unit vector per head
           "meanshift" k = unit(z + 10 u)
    gates: GLA  "config": g = logsigmoid(N(0,1) + 4) / 16;  "strong": g = logsigmoid(N(0,1))
           GDN  beta = sigmoid(N(0,1)), logalpha = -softplus(N(0,1) - 3)
    lam:   "const" (lam_value everywhere) or "random" (sigmoid(N(0,1)) per token)
    q is N(0,1) for GLA and unit(N(0,1)) for GDN.
    """
    gen = torch.Generator().manual_seed(int(seed))
    q = torch.randn(B, T, H, dk, generator=gen)
    z = torch.randn(B, T, H, dk, generator=gen)
    v = torch.randn(B, T, H, dv, generator=gen)
    out = {}
    if backbone == GLA:
        x = torch.randn(B, T, H, dk, generator=gen)
        g = F.logsigmoid(x + 4.0) / 16.0 if gates == "config" else F.logsigmoid(x)
        out["g"] = g.to(gate_dtype or dtype)
    else:
        out["beta"] = torch.sigmoid(torch.randn(B, T, H, generator=gen))
        out["logalpha"] = -F.softplus(torch.randn(B, T, H, generator=gen) - 3.0)
        q = _unit(q)
    if keys == "iso":
        k = _unit(z)
    else:
        u = _unit(torch.randn(1, 1, H, dk, generator=gen))
        if keys == "aniso":
            a = torch.randn(B, T, H, 1, generator=gen)
            k = _unit(z + 16.0 * a * u)
        elif keys == "meanshift":
            k = _unit(z + 10.0 * u)
        else:
            raise ValueError(keys)
    if lam == "const":
        lam_t = torch.full((B, T, H), float(lam_value))
    elif lam == "random":
        lam_t = torch.sigmoid(torch.randn(B, T, H, generator=gen))
    else:
        raise ValueError(lam)
    out.update(q=q.to(dtype), k=k.to(dtype), v=v.to(dtype), lam=lam_t.float())
    if with_dO:
        out["dO"] = torch.randn(B, T, H, dv, generator=gen).to(dtype)
    return out


def workload_inputs(w: Workload, **kw) -> dict:
    kw.setdefault("with_dO", w.train)
    return make_inputs(w.backbone, w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=w.seed, **kw)


def varlen_lengths(w: Workload) -> list:
    """Sequence lengths of the packed-batch form of workload w: 2B sequences with
    lengths uniform in [T/4, 3T/4] (seeded), about as many tokens as w itself."""
    rng = np.random.default_rng(w.seed)
    return [int(x) for x in rng.integers(w.T // 4, 3 * w.T // 4 + 1, size=2 * w.B)]


def pack(inputs: dict, lens) -> dict:
    """Rows 0..lens[b]-1 of every sequence b of a [B, T, ...] input dict, packed."""
    return {k: torch.cat([t[b, :L] for b, L in enumerate(lens)], dim=0).contiguous()
            for k, t in inputs.items()}


def to_f64(inputs: dict) -> dict:
    """Exact fp64 copies (numpy) of the same values, for the oracle."""
    return {k: t.double().numpy() for k, t in inputs.items()}


def to_device(inputs: dict, device="cuda") -> dict:
    return {k: t.to(device).contiguous() for k, t in inputs.items()}


def slice_heads(inputs: dict, b: int, h: int) -> dict:
    """One (batch, head) pair of every token tensor, kept 4-D / 3-D ([1,T,1,...])."""
    res = {}
    for k, t in inputs.items():
        res[k] = t[b:b + 1, :, h:h + 1]
    return res


def rng_numpy(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)
