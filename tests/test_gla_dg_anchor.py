"""The GLA decay gradient as the training kernels form it, checked on the CPU.

The chunk kernel does not sum db_t = qc_t * dqc_t - k_t * dk_t over the whole
rest of the sequence.  It anchors every chunk at the decay gradient of the
next chunk's first token, which is the state the gate multiplies times that
state's adjoint,
    dg_{(r+1)C}[c] = sum_v S_{r+1}[c, v] dS_{r+1}[c, v]
                   = e^{b_C[c]} sum_v S_r[c, v] dS_{r+1}[c, v] + sum_j k_j[c] dk_j^inter[c],
and sums only the chunk's own rows from there.  These tests form the chunk
quantities in fp64 (the GLA write of Eq. read in its chunk form, Alg. 1) and
check the identity against the oracle's token-level reverse pass, then show
that under bf16 rounding of the stored states and of the recurrences'
operands the anchored sum loses less accuracy than the sequence-long one.
"""
import numpy as np
import torch

from oracle import ccq_oracle as O

C = 64


def bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).double().numpy()


def chunk_terms(q, k, v, g, dO, scale, rnd=False):
    """Per-token db, the two forms of the anchor per chunk, for one head.
    rnd: round the stored states, their adjoints and the recurrences' operands to bf16."""
    R = bf16 if rnd else (lambda x: x)
    T, dk = k.shape
    dv = v.shape[1]
    N = (T + C - 1) // C
    sls = [slice(r * C, min(T, r * C + C)) for r in range(N)]
    bs = [np.cumsum(g[sl], axis=0) for sl in sls]
    S = np.zeros((dk, dv))
    states = []
    for r, sl in enumerate(sls):
        states.append(R(S))
        bC = bs[r][-1]
        S = np.exp(bC)[:, None] * S + R(k[sl] * np.exp(bC - bs[r])).T @ v[sl]
    states.append(R(S))
    D = np.zeros((dk, dv))
    adj = [None] * N  # adjoint of the state leaving chunk r
    for r in range(N - 1, -1, -1):
        adj[r] = R(D)
        bC = bs[r][-1]
        D = np.exp(bC)[:, None] * D + scale * R(q[sls[r]] * np.exp(bs[r])).T @ dO[sls[r]]
    db = np.zeros_like(k)
    anchor_in = np.zeros((N, dk))   # from the chunk's own operands
    anchor_out = np.zeros((N, dk))  # from the state leaving the chunk
    for r, sl in enumerate(sls):
        b, bC = bs[r], bs[r][-1]
        A = np.tril(dO[sl] @ v[sl].T)  # A[t, j] = dO_t . v_j, j <= t
        dqc = scale * (np.exp(b) * (dO[sl] @ states[r].T) + np.exp(b) * (A @ (k[sl] * np.exp(-b))))
        inter = np.exp(bC - b) * (v[sl] @ adj[r].T)
        dk_ = scale * np.exp(-b) * (A.T @ (q[sl] * np.exp(b))) + inter
        db[sl] = q[sl] * dqc - k[sl] * dk_
        anchor_in[r] = np.exp(bC) * (states[r] * adj[r]).sum(axis=1) + (k[sl] * inter).sum(axis=0)
        anchor_out[r] = (states[r + 1] * adj[r]).sum(axis=1)
    return sls, db, anchor_in, anchor_out


def anchored_dg(sls, db, anchor):
    dg = np.zeros_like(db)
    for r, sl in enumerate(sls):
        dg[sl] = np.cumsum(db[sl][::-1], axis=0)[::-1] + anchor[r]
    return dg


def inputs(T, dk, dv, seed):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, dk))
    k = rng.standard_normal((T, dk))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = rng.standard_normal((T, dv))
    g = -np.log1p(np.exp(-(rng.standard_normal((T, dk)) + 4.0))) / 16.0  # logsigmoid(x + 4) / 16
    dO = rng.standard_normal((T, dv))
    return q, k, v, g, dO


def oracle_dg(q, k, v, g, dO, scale):
    """The oracle's decay gradient with lam = 0 (q_clean = q), one head."""
    e = lambda x: x[None, :, None]
    lam = np.zeros((1, q.shape[0], 1))
    return O.gla_fwd_bwd(e(q), e(k), e(v), e(g), lam, e(dO), scale=scale)["dg"][0, :, 0]


def test_anchor_identity_fp64():
    """Both anchor forms equal the oracle's dg at the next chunk's first token, and the
    anchored sums give the oracle's dg at every token (ragged last chunk, scale != 1)."""
    q, k, v, g, dO = inputs(1000, 32, 48, seed=11)
    scale = 0.5
    ref = oracle_dg(q, k, v, g, dO, scale)
    sls, db, a_in, a_out = chunk_terms(q, k, v, g, dO, scale)
    den = np.abs(ref).max()
    # the sequence-long reverse sum of db is the oracle's dg
    assert np.abs(np.cumsum(db[::-1], axis=0)[::-1] - ref).max() / den < 1e-12
    for r in range(len(sls) - 1):
        t = sls[r + 1].start
        assert np.abs(a_in[r] - ref[t]).max() / den < 1e-12, r
        assert np.abs(a_out[r] - ref[t]).max() / den < 1e-12, r
    assert np.abs(a_in[-1]).max() < 1e-300 and np.abs(a_out[-1]).max() < 1e-300  # nothing after the end
    assert np.abs(anchored_dg(sls, db, a_in) - ref).max() / den < 1e-12


def test_anchor_limits_bf16_accumulation():
    """With the stored states, their adjoints and the recurrences' operands rounded to bf16,
    the anchored dg is closer to the exact one than the sequence-long sum of the same db."""
    q, k, v, g, dO = inputs(4096, 64, 128, seed=12)
    ref = oracle_dg(q, k, v, g, dO, 1.0)
    sls, db, a_in, _ = chunk_terms(q, k, v, g, dO, 1.0, rnd=True)
    den = np.abs(ref).max()
    err_sum = np.abs(np.cumsum(db[::-1], axis=0)[::-1] - ref).max() / den
    err_anchor = np.abs(anchored_dg(sls, db, a_in) - ref).max() / den
    print("bf16-rounded states: sequence-long sum %.2e, anchored %.2e" % (err_sum, err_anchor))
    assert err_anchor < 0.75 * err_sum
