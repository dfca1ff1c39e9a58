"""The allocation-free Gated DeltaNet forward (ccq_gdn_fwd_noalloc) against the
workspace entry point ccq_gdn_fwd, through the C ABI.

Two calls in a row share the library's per-device scratch, the second with a
smaller input (so stale contents of the first call sit past the second call's
buffers and inside them).  Each must equal ccq_gdn_fwd on the same inputs bit for
bit (same kernels), and the oracle to the parity bar."""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, nerr, np64, oracle_fwd
from paper_2606_01294_amd import ccq
from paper_2606_01294_amd.inputs import GDN, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_against_workspace_call(d, dtype, **kw):
    g = to_device(d)
    shape = ccq.make_shape(*d["v"].shape[:3], d["q"].shape[-1], d["v"].shape[-1], dtype)
    assert ccq.ccq_workspace_size(shape, ccq.CCQ_GDN) <= ccq.NOALLOC_SCRATCH_BYTES
    a = ccq.ccq_gdn_fwd_noalloc(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                                want_qclean=True, **kw)
    torch.cuda.synchronize()
    b = ccq.ccq_gdn_fwd(g["q"], g["k"], g["v"], g["logalpha"], g["beta"], g["lam"],
                        want_qclean=True, **kw)
    torch.cuda.synchronize()
    for key in ("o", "ST", "CT", "muT", "qclean"):
        assert torch.equal(a[key], b[key]), key
    kw64 = {k: (np64(v) if isinstance(v, torch.Tensor) else v) for k, v in kw.items()}
    ref = oracle_fwd(GDN, d, **kw64)
    errs = {key: nerr(np64(a[key]), ref[key]) for key in ("o", "ST", "CT", "muT")}
    say("  errors", errs)
    assert all(v <= TOL[dtype] for v in errs.values()), errs
    return a


def test_noalloc_two_calls_second_smaller():
    bf = torch.bfloat16
    say("noalloc call 1: B=2 T=700 H=4 dk=dv=256")
    d1 = make_inputs(GDN, 2, 700, 4, 256, 256, bf, seed=71, keys="aniso", lam="random")
    check_against_workspace_call(d1, bf)
    say("noalloc call 2: B=1 T=150 H=2 dk=128 dv=256, initial states, t0=40")
    d2 = make_inputs(GDN, 1, 150, 2, 128, 256, bf, seed=72, keys="meanshift", lam="random")
    rng = np.random.default_rng(5)
    S0 = torch.from_numpy(rng.standard_normal((1, 2, 256, 128)) * 0.2).float().cuda()
    K = rng.standard_normal((40, 128))
    K /= np.linalg.norm(K, axis=-1, keepdims=True)
    C0 = torch.from_numpy(np.broadcast_to(K.T @ K / 40, (1, 2, 128, 128)).copy()).float().cuda()
    mu0 = torch.from_numpy(np.broadcast_to(K.mean(0), (1, 2, 128)).copy()).float().cuda()
    check_against_workspace_call(d2, bf, S0=S0, C0=C0, mu0=mu0, t0=40)


def test_noalloc_rejects_shapes_beyond_the_scratch():
    shape = ccq.make_shape(4, 4096, 8, 256, 256, torch.bfloat16)
    assert ccq.ccq_workspace_size(shape, ccq.CCQ_GDN) > ccq.NOALLOC_SCRATCH_BYTES
    q = torch.zeros(4, 4096, 8, 256, dtype=torch.bfloat16, device="cuda")
    s = torch.zeros(4, 4096, 8, device="cuda")
    with pytest.raises(ccq.CcqError) as e:
        ccq.ccq_gdn_fwd_noalloc(q, q, q, s, s, s)
    assert e.value.code == 3  # CCQ_ERR_WORKSPACE
