"""Host-side checks of the C ABI: the library loads, exports every function that
include/ccq.h declares, and rejects bad arguments before launching anything
(these paths touch no GPU, so they run on the CPU)."""
import ctypes
import os
import re

import pytest

from paper_2606_01294_amd import ccq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    txt = open(os.path.join(ROOT, "include", "ccq.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ccq_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    L = ccq.lib()
    names = declared_functions()
    assert set(names) == set(ccq.EXPORTS)
    for n in names:
        assert getattr(L, n) is not None


def test_version_and_status_strings():
    assert "gfx950" in ccq.ccq_version()
    for code in range(5):
        assert ccq.ccq_status_string(code)
    assert ccq.ccq_status_string(0) == "ok"


def shape(**kw):
    base = dict(B=2, T=100, H=3, dk=128, dv=256, io_dtype=__import__("torch").bfloat16)
    base.update(kw)
    return ccq.make_shape(**base)


def test_workspace_size():
    s = shape()
    ws = ccq.ccq_workspace_size(s, ccq.CCQ_GLA)
    assert ws >= 2 * 100 * 3 * 128 * 2
    wg = ccq.ccq_workspace_size(s, ccq.CCQ_GDN)
    assert wg > ws
    assert ccq.ccq_workspace_size(shape(dk=96), ccq.CCQ_GLA) == 0
    assert ccq.ccq_workspace_size(shape(chunk=32), ccq.CCQ_GLA) == 0


FAKE = 1 << 20  # an aligned address that is never dereferenced (validation fails first)


def call_gla(s, ws_bytes=1 << 30, ptr=FAKE, lam_ptr=FAKE, ws_ptr=FAKE):
    P = ctypes.c_void_p
    return ccq.lib().ccq_gla_fwd(ctypes.byref(s) if s is not None else None, P(ptr), P(ptr),
                                 P(ptr), P(ptr), P(lam_ptr), None, None, None, P(ptr), None, None,
                                 None, None, P(ws_ptr), ws_bytes, None)


def test_validation_errors_are_returned_before_launch():
    assert call_gla(None) == 1                            # no shape
    assert call_gla(shape(B=-1)) == 1                     # negative size
    assert call_gla(shape(dk=96)) == 2                    # unsupported head size
    assert call_gla(shape(dv=100)) == 2
    assert call_gla(shape(chunk=32)) == 2                 # unsupported chunk
    assert call_gla(shape(), lam_ptr=0) == 1              # missing tensor
    assert call_gla(shape(), lam_ptr=FAKE + 4) == 1       # misaligned tensor
    assert call_gla(shape(), ws_bytes=16) == 3            # workspace too small
    assert call_gla(shape(), ws_ptr=0) == 3               # no workspace
    s = shape()
    s.centered = 7
    assert call_gla(s) == 1
    s = shape()
    s.io_dtype = 9
    assert call_gla(s) == 1
    s = shape(io_dtype=__import__("torch").float32, dk=256)
    assert call_gla(s) == 2                               # fp32 path has dk <= 128
    assert call_gla(shape(dk=256)) == 2                   # GLA has dk <= 128


def test_empty_batch_is_a_no_op():
    assert call_gla(shape(B=0), ptr=0, lam_ptr=0, ws_ptr=0) == 0
    assert call_gla(shape(H=0), ptr=0, lam_ptr=0, ws_ptr=0) == 0


def test_gdn_requires_beta():
    P = ctypes.c_void_p
    s = shape(dk=256)
    rc = ccq.lib().ccq_gdn_fwd(ctypes.byref(s), P(FAKE), P(FAKE), P(FAKE), P(FAKE), None,
                               P(FAKE), None, None, None, P(FAKE), None, None, None, None,
                               P(FAKE), 1 << 30, None)
    assert rc == 1


def call_gdn_noalloc(s, ptr=FAKE, beta_ptr=FAKE):
    P = ctypes.c_void_p
    return ccq.lib().ccq_gdn_fwd_noalloc(ctypes.byref(s) if s is not None else None, P(ptr),
                                         P(ptr), P(ptr), P(ptr), P(beta_ptr), P(ptr), None, None,
                                         None, P(ptr), None, None, None, None, None)


def test_noalloc_validation_before_launch():
    """The allocation-free forward validates like ccq_gdn_fwd, and a shape whose workspace
    exceeds its scratch returns CCQ_ERR_WORKSPACE, all before any HIP call."""
    assert call_gdn_noalloc(None) == 1
    assert call_gdn_noalloc(shape(dk=96)) == 2
    assert call_gdn_noalloc(shape(dk=256), beta_ptr=0) == 1
    assert call_gdn_noalloc(shape(dk=256), ptr=FAKE + 4) == 1
    big = shape(B=4, T=4096, H=8, dk=256, dv=256)
    assert ccq.ccq_workspace_size(big, ccq.CCQ_GDN) > ccq.NOALLOC_SCRATCH_BYTES
    assert call_gdn_noalloc(big) == 3
    assert call_gdn_noalloc(shape(B=0, dk=256), ptr=0, beta_ptr=0) == 0


def test_forward_from_raw_validation():
    """ccq_fwd_raw: workspace = the forward's plus three floats per token and head; the
    pre-processing limits apply; errors before any launch."""
    P = ctypes.c_void_p
    s = shape(dk=128)
    ws = ccq.ccq_fwd_raw_workspace_size(s, ccq.CCQ_GLA)
    assert ws >= ccq.ccq_workspace_size(s, ccq.CCQ_GLA) + 3 * 2 * 100 * 3 * 4
    assert ccq.ccq_fwd_raw_workspace_size(shape(H=32, dk=64), ccq.CCQ_GLA) == 0  # W_lambda too large

    def call(s, bb=0, w=FAKE, beta=None, ws_bytes=1 << 30):
        return ccq.lib().ccq_fwd_raw(ctypes.byref(s), bb, P(FAKE), P(FAKE), P(w), P(FAKE), P(FAKE),
                                     P(FAKE), P(beta), None, None, None, P(FAKE), None, None, None,
                                     None, P(FAKE), ws_bytes, None)
    assert call(shape(), w=0) == 1                          # W_lambda required
    assert call(shape(dk=256), bb=1) == 1                   # Gated DeltaNet needs beta
    assert call(shape(H=32, dk=64)) == 2                    # W_lambda does not fit on chip
    assert call(shape(), ws_bytes=64) == 3


def test_binding_rejects_wrong_dtype_before_calling():
    import torch
    q = torch.zeros(1, 4, 1, 64)
    with pytest.raises(TypeError):
        ccq.ccq_gla_fwd(q, q, q, q, torch.zeros(1, 4, 1, dtype=torch.float64))


def call_bwd(s, bb=0, ws_bytes=1 << 34, ptr=FAKE):
    P = ctypes.c_void_p
    return ccq.lib().ccq_fwd_bwd(ctypes.byref(s), bb, P(ptr), P(ptr), P(ptr), P(ptr), None,
                                 P(ptr), P(ptr), P(ptr), P(ptr), P(ptr), P(ptr), P(ptr), None,
                                 P(ptr), P(ptr), ws_bytes, None)


def test_training_entry_point_validation():
    assert ccq.ccq_workspace_size(shape(), ccq.CCQ_GLA, True) > ccq.ccq_workspace_size(
        shape(), ccq.CCQ_GLA, False)
    # dk = 256: a Gated DeltaNet training step (the 1.3B layer's head size), no GLA one
    assert ccq.ccq_workspace_size(shape(dk=256), ccq.CCQ_GDN, True) > ccq.ccq_workspace_size(
        shape(dk=256), ccq.CCQ_GDN, False)
    assert ccq.ccq_workspace_size(shape(dk=256), ccq.CCQ_GLA, True) == 0
    assert ccq.ccq_workspace_size(shape(), ccq.CCQ_GDN, True) > ccq.ccq_workspace_size(
        shape(), ccq.CCQ_GDN, False)
    assert call_bwd(shape(dk=256), bb=0) == 2               # no GLA training step at dk = 256
    assert call_bwd(shape(dk=256), bb=1) == 1               # Gated DeltaNet needs beta, dbeta
    assert call_bwd(shape(), bb=1) == 1
    s = shape()
    s.t0 = 5
    assert call_bwd(s) == 1                                 # training starts from zero state
    assert call_bwd(shape(), ws_bytes=100) == 3             # workspace too small
    assert call_bwd(shape(io_dtype=__import__("torch").float32, dk=128)) == 2


def call_decode(s, bb=0, ws_bytes=1 << 30, ptr=FAKE, beta=None, ws_ptr=FAKE):
    P = ctypes.c_void_p
    return ccq.lib().ccq_decode(ctypes.byref(s), bb, P(ptr), P(ptr), P(ptr), P(ptr),
                                None if beta is None else P(beta), P(ptr), P(ptr), P(ptr),
                                P(ptr), P(ptr), None if ws_ptr is None else P(ws_ptr), ws_bytes,
                                None)


def test_decode_entry_point_validation():
    # six heads: the step is split into two launches that pass Cbar q through it
    s = shape(T=1, dk=256, dv=512)
    need = ccq.ccq_decode_workspace_size(s)
    assert need == 6 * 256 * 4
    # 256 heads have a workgroup each and need no workspace
    assert ccq.ccq_decode_workspace_size(shape(B=64, H=4, T=1)) == 0
    # the two decode workloads: 32 GLA heads (dk = 128, dv = 256) keep a workgroup per
    # head; 32 Gated DeltaNet heads of dk = dv = 256 take the two-launch split
    assert ccq.ccq_decode_workspace_size(shape(B=8, H=4, T=1, dk=128, dv=256)) == 0
    assert ccq.ccq_decode_workspace_size(shape(B=4, H=8, T=1, dk=256, dv=256)) == 32 * 256 * 4
    assert ccq.ccq_decode_workspace_size(shape(T=1, dk=96)) == 0
    assert call_decode(shape(T=2)) == 1                      # one token per call
    assert call_decode(shape(T=1, dk=96)) == 2               # unsupported head size
    assert call_decode(shape(T=1), bb=1) == 1                # Gated DeltaNet needs beta
    assert call_decode(shape(T=1), ptr=FAKE + 4) == 1        # misaligned tensor
    assert call_decode(s, ws_ptr=None) == 3                  # no workspace
    assert call_decode(s, ws_bytes=need - 4) == 3            # workspace too small
    assert call_decode(shape(B=0, T=1), ptr=0, ws_ptr=None) == 0


def test_prep_entry_point_validation():
    P = ctypes.c_void_p

    def call(s, ptr=FAKE):
        return ccq.lib().ccq_prep(ctypes.byref(s), P(ptr), P(ptr), P(ptr), P(ptr), P(ptr), P(ptr),
                                  P(ptr), None)
    assert call(shape(H=17, dk=64)) == 2                  # too many heads
    assert call(shape(H=16, dk=128)) == 2                 # W_lambda does not fit on chip
    assert call(shape(H=4, dk=96)) == 2
    assert call(shape(H=4, dk=64), ptr=FAKE + 4) == 1     # misaligned
    assert call(shape(B=0, H=4, dk=64), ptr=0) == 0


def test_varlen_entry_point_validation():
    P = ctypes.c_void_p
    s = shape(dk=128)
    # the forward reads the packed rows directly: the padded call's workspace
    assert ccq.ccq_varlen_workspace_size(s, ccq.CCQ_GLA) == ccq.ccq_workspace_size(s, ccq.CCQ_GLA)
    assert ccq.ccq_varlen_workspace_size(s, ccq.CCQ_GDN, True) > ccq.ccq_workspace_size(
        s, ccq.CCQ_GDN, True)
    assert ccq.ccq_varlen_workspace_size(shape(dk=96), ccq.CCQ_GLA) == 0

    def call(s, cu=FAKE, ptr=FAKE, ws_bytes=1 << 34):
        return ccq.lib().ccq_gla_fwd_varlen(ctypes.byref(s), None if cu is None else P(cu), P(ptr),
                                            P(ptr), P(ptr), P(ptr), P(ptr), None, None, None,
                                            P(ptr), None, None, None, P(FAKE), ws_bytes, None)
    assert call(shape(), cu=None) == 1                      # offsets required
    assert call(shape(), cu=FAKE + 2) == 1                  # misaligned offsets
    assert call(shape(B=70000)) == 2                        # one grid row per sequence
    assert call(shape(dk=96)) == 2
    assert call(shape(), ptr=FAKE + 4) == 1
    assert call(shape(), ws_bytes=64) == 3
    assert call(shape(B=0), cu=None, ptr=0) == 0

    def call_gdn(s, beta=FAKE):
        return ccq.lib().ccq_gdn_fwd_varlen(ctypes.byref(s), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                            P(FAKE), None if beta is None else P(beta), P(FAKE),
                                            None, None, None, P(FAKE), None, None, None, P(FAKE),
                                            1 << 34, None)
    assert call_gdn(shape(dk=256), beta=None) == 1

    def call_bwd(s, bb=0, t0=0):
        s.t0 = t0
        return ccq.lib().ccq_fwd_bwd_varlen(ctypes.byref(s), bb, P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                            P(FAKE), None, P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                            P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE),
                                            1 << 34, None)
    assert call_bwd(shape(), t0=3) == 1
    assert call_bwd(shape(), bb=1) == 1                     # Gated DeltaNet needs beta, dbeta
    assert call_bwd(shape(dk=256), bb=0) == 2                # no GLA training step at dk = 256
    assert call_bwd(shape(dk=256), bb=1) == 1                # Gated DeltaNet at dk = 256 needs beta


def test_decay_aligned_validation():
    """ccq_shape.decay_aligned: Gated DeltaNet forward only, from empty statistics; every
    other use is refused before any launch.  The field sits in the padding before t0, so
    the struct keeps its size and t0 its offset."""
    assert ctypes.sizeof(ccq.Shape) == 56 and ccq.Shape.t0.offset == 48
    P = ctypes.c_void_p

    def call_gdn(s, C0=None):
        return ccq.lib().ccq_gdn_fwd(ctypes.byref(s), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                     P(FAKE), P(FAKE), None, None if C0 is None else P(C0), None,
                                     P(FAKE), None, None, None, None, P(FAKE), 1 << 34, None)

    d = dict(dk=256, decay_aligned=True)
    assert call_gla(shape(decay_aligned=True)) == 2         # GLA: per-channel decay
    s = shape(**d)
    s.decay_aligned = 3
    assert call_gdn(s) == 1
    assert call_gdn(shape(t0=7, **d)) == 2                  # no cached decayed count
    assert call_gdn(shape(**d), C0=FAKE) == 2
    assert call_bwd(shape(**d), bb=1) == 2                  # forward only
    assert call_decode(shape(T=1, **d), bb=1, beta=FAKE) == 2
    # the flag does not change the workspace
    assert ccq.ccq_workspace_size(shape(**d), ccq.CCQ_GDN) == ccq.ccq_workspace_size(
        shape(dk=256), ccq.CCQ_GDN)
