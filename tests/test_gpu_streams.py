"""The entry points on a stream that is not torch's current one.

The binding allocates the workspace (and the outputs) on the current stream and
hands the library the caller's stream; the results must equal those of the same
call on the current stream, bit for bit, also when the current stream allocates
and writes memory while the call's kernels may still run."""
import sys

import pytest
import torch

from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, GLA, make_inputs, to_device

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run(backbone, g, train, stream=None):
    if train:
        if backbone == GLA:
            return ccq.ccq_fwd_bwd(g["q"], g["k"], g["v"], g["g"], g["lam"], g["dO"], stream=stream)
        return ccq.ccq_fwd_bwd(g["q"], g["k"], g["v"], g["logalpha"], g["lam"], g["dO"],
                               backbone=ccq.CCQ_GDN, beta=g["beta"], stream=stream)
    if backbone == GLA:
        return ccq.ccq_gla_fwd(g["q"], g["k"], g["v"], g["g"], g["lam"], stream=stream)
    return ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                           stream=stream)


@pytest.mark.parametrize("train", [False, True])
@pytest.mark.parametrize("backbone", [GLA, GDN])
def test_non_current_stream(backbone, train):
    say("stream", backbone, train)
    d = make_inputs(backbone, 2, 700, 4, 128, 256, torch.bfloat16, seed=61, lam="random",
                    with_dO=train)
    g = to_device(d)
    ref = run(backbone, g, train)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    out = run(backbone, g, train, stream=side)
    # the current stream reuses freed memory at once: a workspace returned to the
    # current stream's pool would be overwritten here while `side` still uses it
    junk = [torch.full((1 << 22,), float("nan"), device="cuda") for _ in range(16)]
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    del junk
    for key in ref:
        assert torch.equal(ref[key], out[key]), key
