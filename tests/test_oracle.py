"""Pins of the fp64 oracle against things other than itself.

Each test checks the oracle against a library routine, a closed form, an
invariant the paper states, a hand-worked example or finite differences, so
that a dropped term, a wrong sign or index or a transposed operand in the
oracle fails at least one of them.  All run on the CPU.
"""
import json
import os

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import ccq_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


def rnd_inputs(rng, B, T, H, dk, dv, backbone=O.GLA, unit_keys=True, lam="random"):
    q = rng.standard_normal((B, T, H, dk))
    k = rng.standard_normal((B, T, H, dk))
    if unit_keys:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, T, H, dv))
    if backbone == O.GLA:
        gate = -np.log1p(np.exp(-(rng.standard_normal((B, T, H, dk)) + 1.0)))  # logsigmoid
        beta = None
    else:
        gate = -np.log1p(np.exp(rng.standard_normal((B, T, H)) - 2.0))       # -softplus
        beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((B, T, H))))
    lam_t = (1.0 / (1.0 + np.exp(-rng.standard_normal((B, T, H))))) if lam == "random" \
        else np.full((B, T, H), float(lam))
    return dict(q=q, k=k, v=v, gate=gate, beta=beta, lam=lam_t)


def run(d, backbone=O.GLA, **kw):
    return O.fwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], beta=d["beta"], backbone=backbone,
                 **kw)


# ---------------------------------------------------------------- statistics


@pytest.mark.parametrize("centered", [True, False])
def test_correction_is_population_covariance_times_q(centered):
    """Sigma_t q_t against numpy's population covariance of the prefix keys (Sec. 3.2)."""
    rng = np.random.default_rng(1)
    d = rnd_inputs(rng, 1, 40, 2, 8, 5, unit_keys=False)
    r = run(d, centered=centered)
    for h in range(2):
        K = d["k"][0, :, h]
        for t in range(40):
            q = d["q"][0, t, h]
            lam = d["lam"][0, t, h]
            if centered:
                Sig = np.cov(K[: t + 1].T, bias=True) if t > 0 else np.zeros((8, 8))
            else:
                Sig = K[: t + 1].T @ K[: t + 1] / (t + 1)
            c = (q - r["qclean"][0, t, h]) / lam
            np.testing.assert_allclose(c, Sig @ q, rtol=0, atol=1e-12)


def test_final_statistics_are_hessian_of_log_partition():
    """Cbar_T - mu_T mu_T^T equals the finite-difference Hessian of A_T(q) = logsumexp(K q) at
    q = 0 (Eq. hess, App. A.2)."""
    rng = np.random.default_rng(2)
    d = rnd_inputs(rng, 1, 30, 1, 6, 3)
    r = run(d)
    K = d["k"][0, :, 0]
    Sig = r["CT"][0, 0] - np.outer(r["muT"][0, 0], r["muT"][0, 0])
    A = lambda x: logsumexp(K @ x)
    hstep = 1e-4
    Hfd = np.zeros((6, 6))
    E = np.eye(6) * hstep
    for i in range(6):
        for j in range(6):
            Hfd[i, j] = (A(E[i] + E[j]) - A(E[i] - E[j]) - A(-E[i] + E[j]) + A(-E[i] - E[j])) / (
                4 * hstep * hstep)
    np.testing.assert_allclose(Sig, Hfd, atol=1e-7)
    # the gradient at 0 is the mean (App. A.2)
    gfd = np.array([(A(E[i]) - A(-E[i])) / (2 * hstep) for i in range(6)])
    np.testing.assert_allclose(r["muT"][0, 0], gfd, atol=1e-8)


def test_first_token_is_not_cleaned():
    """t = 1: Sigma_1 = k k^T - k k^T = 0, so q_clean = q."""
    rng = np.random.default_rng(3)
    d = rnd_inputs(rng, 2, 1, 3, 16, 4)
    r = run(d)
    np.testing.assert_allclose(r["qclean"], d["q"], atol=1e-14)


def test_initial_statistics_are_continued():
    """Splitting a sequence and feeding (S_T, Cbar_T, mu_T) plus t0 back in reproduces the
    unsplit run (the inference cache of App. C)."""
    rng = np.random.default_rng(4)
    for bb in (O.GLA, O.GDN):
        d = rnd_inputs(rng, 1, 37, 2, 8, 6, backbone=bb)
        full = run(d, backbone=bb)
        t1 = 17
        a = {k: (None if v is None else v[:, :t1]) for k, v in d.items()}
        b = {k: (None if v is None else v[:, t1:]) for k, v in d.items()}
        ra = run(a, backbone=bb)
        rb = run(b, backbone=bb, S0=ra["ST"], C0=ra["CT"], mu0=ra["muT"], t0=t1)
        np.testing.assert_allclose(rb["o"], full["o"][:, t1:], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(rb["CT"], full["CT"], atol=1e-13)
        np.testing.assert_allclose(rb["ST"], full["ST"], atol=1e-12)


# ------------------------------------------------------------------ backbones


def test_gla_without_gate_is_linear_attention():
    """g = 0, lambda = 0: o = tril(Q K^T) V (Eq. prelim_linattn, write before read)."""
    rng = np.random.default_rng(5)
    d = rnd_inputs(rng, 1, 25, 1, 7, 4, lam=0.0)
    d["gate"] = np.zeros_like(d["gate"])
    r = run(d)
    Q, K, V = d["q"][0, :, 0], d["k"][0, :, 0], d["v"][0, :, 0]
    np.testing.assert_allclose(r["o"][0, :, 0], np.tril(Q @ K.T) @ V, atol=1e-12)


def test_gla_closed_form():
    """lambda = 0: o_t = sum_{j<=t} sum_c q_t[c] k_j[c] exp(sum_{s=j+1..t} g_s[c]) v_j."""
    rng = np.random.default_rng(6)
    T, dk, dv = 20, 5, 3
    d = rnd_inputs(rng, 1, T, 1, dk, dv, lam=0.0)
    r = run(d)
    Q, K, V, G = d["q"][0, :, 0], d["k"][0, :, 0], d["v"][0, :, 0], d["gate"][0, :, 0]
    for t in range(T):
        o = np.zeros(dv)
        for j in range(t + 1):
            decay = np.exp(G[j + 1: t + 1].sum(axis=0))
            o += np.sum(Q[t] * K[j] * decay) * V[j]
        np.testing.assert_allclose(r["o"][0, t, 0], o, atol=1e-12)


def test_gdn_delta_rule_acts_on_written_key():
    """Gated DeltaNet write: S_t k_t = (1 - beta_t) alpha_t S_{t-1} k_t + beta_t v_t for a unit
    key, and S_t x = alpha_t S_{t-1} x for x orthogonal to k_t.  These two actions fix S_t."""
    rng = np.random.default_rng(7)
    T, dk, dv = 9, 6, 4
    d = rnd_inputs(rng, 1, T, 1, dk, dv, backbone=O.GDN, lam=0.0)
    prev = np.zeros((dv, dk))
    for t in range(1, T + 1):
        sub = {k: (None if v is None else v[:, :t]) for k, v in d.items()}
        S = run(sub, backbone=O.GDN)["ST"][0, 0]
        kt = d["k"][0, t - 1, 0]
        al, be = np.exp(d["gate"][0, t - 1, 0]), d["beta"][0, t - 1, 0]
        np.testing.assert_allclose(S @ kt, (1 - be) * al * prev @ kt + be * d["v"][0, t - 1, 0],
                                   atol=1e-12)
        x = rng.standard_normal(dk)
        x -= (x @ kt) * kt
        np.testing.assert_allclose(S @ x, al * prev @ x, atol=1e-12)
        prev = S


def test_gdn_without_write_is_pure_decay():
    """beta = 0: S_t = (prod_{s<=t} alpha_s) S_0 and o_t = S_t q_t (lambda = 0)."""
    rng = np.random.default_rng(8)
    d = rnd_inputs(rng, 1, 12, 1, 5, 3, backbone=O.GDN, lam=0.0)
    d["beta"] = np.zeros_like(d["beta"])
    S0 = rng.standard_normal((1, 1, 3, 5))
    r = run(d, backbone=O.GDN, S0=S0)
    cum = np.exp(np.cumsum(d["gate"][0, :, 0]))
    for t in range(12):
        np.testing.assert_allclose(r["o"][0, t, 0], cum[t] * S0[0, 0] @ d["q"][0, t, 0],
                                   atol=1e-12)
    np.testing.assert_allclose(r["ST"][0, 0], cum[-1] * S0[0, 0], atol=1e-12)


# ------------------------------------------------------------- chunkwise form


@pytest.mark.parametrize("backbone", [O.GLA, O.GDN])
@pytest.mark.parametrize("chunk", [1, 16, 64, 1000])
@pytest.mark.parametrize("centered", [True, False])
def test_chunkwise_equals_recurrent(backbone, chunk, centered):
    """Alg. 1 (chunkwise, App. B) equals the token recurrence, including a ragged last
    chunk, t0 > 0 and nonzero initial states."""
    rng = np.random.default_rng(9 + chunk)
    B, T, H, dk, dv = 2, 83, 2, 8, 6
    d = rnd_inputs(rng, B, T, H, dk, dv, backbone=backbone)
    S0 = rng.standard_normal((B, H, dv, dk)) * 0.3
    Kp = rng.standard_normal((B, H, 11, dk))
    Kp /= np.linalg.norm(Kp, axis=-1, keepdims=True)
    C0 = np.einsum("bhnc,bhnd->bhcd", Kp, Kp) / 11
    mu0 = Kp.mean(axis=2)
    kw = dict(backbone=backbone, S0=S0, C0=C0, mu0=mu0, t0=11, centered=centered, scale=0.7)
    rec = O.fwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], beta=d["beta"], **kw)
    chk = O.chunk_fwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], beta=d["beta"], chunk=chunk,
                      **kw)
    for key in ("o", "ST", "CT", "muT", "qclean"):
        np.testing.assert_allclose(chk[key], rec[key], rtol=1e-11, atol=1e-11, err_msg=key)


@pytest.mark.parametrize("backbone", [O.GLA, O.GDN])
def test_running_mean_form_equals_sum_form(backbone):
    """Alg. 2's running-mean updates of Cbar and mu equal the raw-sum form."""
    rng = np.random.default_rng(10)
    d = rnd_inputs(rng, 1, 50, 2, 8, 5, backbone=backbone)
    a = run(d, backbone=backbone, form=0)
    b = run(d, backbone=backbone, form=1)
    for key in ("o", "ST", "CT", "muT", "qclean"):
        np.testing.assert_allclose(b[key], a[key], rtol=1e-11, atol=1e-12, err_msg=key)


# ------------------------------------------------------------ score-space form


def test_score_form_brute_force():
    """k_j . q_clean = k_j.q - (lam/t) sum_i (k_j.k_i)(k_i.q) + lam (k_j.mu)(mu.q)
    (Eq. score_form, App. A.4), for every stored key j <= t."""
    rng = np.random.default_rng(11)
    T, dk = 9, 4
    d = rnd_inputs(rng, 1, T, 1, dk, 2)
    r = run(d)
    K = d["k"][0, :, 0]
    for t in range(1, T + 1):
        q = d["q"][0, t - 1, 0]
        lam = d["lam"][0, t - 1, 0]
        mu = [sum(K[i, c] for i in range(t)) / t for c in range(dk)]
        qc = r["qclean"][0, t - 1, 0]
        for j in range(t):
            kq = sum(K[j, c] * q[c] for c in range(dk))
            second = sum(sum(K[j, c] * K[i, c] for c in range(dk)) *
                         sum(K[i, c] * q[c] for c in range(dk)) for i in range(t))
            mean = sum(K[j, c] * mu[c] for c in range(dk)) * sum(mu[c] * q[c] for c in range(dk))
            expect = kq - lam / t * second + lam * mean
            assert abs(float(K[j] @ qc) - expect) < 1e-12


def test_margin_shift_exact_for_rank_one_covariance():
    """At t = 2, Sigma_2 = (k1-k2)(k1-k2)^T / 4 is exactly rank one, so the CCQ margin between
    any target and distractor key shifts by lam rho (beta - alpha)(u.q) (Eq. margin_shift,
    App. H) with rho = |k1-k2|^2/4, u = (k1-k2)/|k1-k2|."""
    rng = np.random.default_rng(12)
    dk = 7
    d = rnd_inputs(rng, 1, 2, 1, dk, 3)
    r = run(d)
    k1, k2 = d["k"][0, 0, 0], d["k"][0, 1, 0]
    q, qc, lam = d["q"][0, 1, 0], r["qclean"][0, 1, 0], d["lam"][0, 1, 0]
    diff = k1 - k2
    rho = diff @ diff / 4
    u = diff / np.linalg.norm(diff)
    for _ in range(5):
        ks, kd = rng.standard_normal(dk), rng.standard_normal(dk)
        alpha, beta = ks @ u, kd @ u
        shift = (ks @ qc - kd @ qc) - (ks @ q - kd @ q)
        assert abs(shift - lam * rho * (beta - alpha) * (u @ q)) < 1e-12


def test_stability_bounds():
    """Unit keys, lam in (0,1): |Cbar|_2 <= 1, spec(I - lam Sigma) in [1-lam, 1],
    |q_clean| <= |q|, q^T Sigma q >= 0 (App. G)."""
    rng = np.random.default_rng(13)
    d = rnd_inputs(rng, 2, 64, 2, 16, 4)
    r = run(d)
    nq = np.linalg.norm(d["q"], axis=-1)
    nc = np.linalg.norm(r["qclean"], axis=-1)
    assert np.all(nc <= nq * (1 + 1e-12))
    assert np.all(np.einsum("bthc,bthc->bth", d["q"], d["q"] - r["qclean"]) >= -1e-12)
    for b in range(2):
        for h in range(2):
            C = r["CT"][b, h]
            mu = r["muT"][b, h]
            assert np.linalg.eigvalsh(C).max() <= 1 + 1e-12
            sig = np.linalg.eigvalsh(C - np.outer(mu, mu))
            assert sig.min() >= -1e-12 and sig.max() <= 1 + 1e-12
            np.testing.assert_allclose(np.trace(C), 1.0, atol=1e-12)  # trace Cbar = 1


def test_worked_example():
    """Hand-computed 3-token, 2-dim example (tests/golden/worked_2d.json)."""
    G = json.load(open(os.path.join(HERE, "golden", "worked_2d.json")))
    q = np.array(G["q"])[None, :, None]
    k = np.array(G["k"])[None, :, None]
    v = np.array(G["v"])[None, :, None]
    lam = np.array(G["lam"])[None, :, None]
    r = O.fwd(q, k, v, np.array(G["gla_g"])[None, :, None], lam)
    np.testing.assert_allclose(r["qclean"][0, :, 0], G["expected_qclean"], atol=1e-15)
    np.testing.assert_allclose(r["o"][0, :, 0, 0], G["expected_gla_o"], atol=1e-15)
    np.testing.assert_allclose(r["ST"][0, 0], G["expected_gla_ST"], atol=1e-15)
    np.testing.assert_allclose(r["CT"][0, 0], G["expected_CT"], atol=1e-15)
    np.testing.assert_allclose(r["muT"][0, 0], G["expected_muT"], atol=1e-15)
    r = O.fwd(q, k, v, np.array(G["gdn_logalpha"])[None, :, None], lam,
              beta=np.array(G["gdn_beta"])[None, :, None], backbone=O.GDN)
    np.testing.assert_allclose(r["o"][0, :, 0, 0], G["expected_gdn_o"], atol=1e-15)
    np.testing.assert_allclose(r["ST"][0, 0], G["expected_gdn_ST"], atol=1e-15)
    for bb, gate in ((O.GLA, np.array(G["gla_g"])[None, :, None]),
                     (O.GDN, np.array(G["gdn_logalpha"])[None, :, None])):
        beta = np.array(G["gdn_beta"])[None, :, None] if bb == O.GDN else None
        c = O.chunk_fwd(q, k, v, gate, lam, beta=beta, backbone=bb, chunk=2)
        e = G["expected_gla_o"] if bb == O.GLA else G["expected_gdn_o"]
        np.testing.assert_allclose(c["o"][0, :, 0, 0], e, atol=1e-15)


def test_empty_sequence_keeps_initial_state():
    rng = np.random.default_rng(14)
    d = rnd_inputs(rng, 1, 0, 2, 4, 3)
    S0 = rng.standard_normal((1, 2, 3, 4))
    C0 = np.tile(np.eye(4) / 4, (1, 2, 1, 1))
    mu0 = rng.standard_normal((1, 2, 4))
    for fn in (O.fwd, O.chunk_fwd):
        r = fn(d["q"], d["k"], d["v"], d["gate"], d["lam"], S0=S0, C0=C0, mu0=mu0, t0=5)
        np.testing.assert_array_equal(r["ST"], S0)
        # (t0 * C0) / t0 may differ from C0 in the last bit
        np.testing.assert_allclose(r["CT"], C0, rtol=1e-15, atol=0)
        np.testing.assert_allclose(r["muT"], mu0, rtol=1e-15, atol=0)


# ---------------------------------------------------------------- reverse pass


@pytest.mark.parametrize("centered,scale", [(True, 1.0), (False, 0.5)])
def test_reverse_pass_matches_finite_differences(centered, scale):
    """Gradients of L = sum <dO, o> from the oracle's reverse pass against central finite
    differences of the oracle forward, along random directions, at the size of the small
    fp32 workload (B=1, T=256, H=2, dk=dv=64)."""
    rng = np.random.default_rng(15)
    B, T, H, dk, dv = 1, 256, 2, 64, 64
    d = rnd_inputs(rng, B, T, H, dk, dv)
    d["gate"] = d["gate"] / 4
    dO = rng.standard_normal((B, T, H, dv))
    gr = O.gla_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], dO, scale=scale,
                       centered=centered, seg=64)
    base = O.fwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], scale=scale, centered=centered)
    np.testing.assert_allclose(gr["o"], base["o"], rtol=1e-12, atol=1e-12)

    def loss(dd):
        return float(np.sum(dO * O.fwd(dd["q"], dd["k"], dd["v"], dd["gate"], dd["lam"],
                                       scale=scale, centered=centered)["o"]))

    h = 1e-5
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("gate", "dg"), ("lam", "dlam")):
        e = rng.standard_normal(d[name].shape)
        dp = dict(d)
        dm = dict(d)
        dp[name] = d[name] + h * e
        dm[name] = d[name] - h * e
        fd = (loss(dp) - loss(dm)) / (2 * h)
        an = float(np.sum(gr[gname] * e))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_reverse_pass_segment_length_does_not_matter():
    rng = np.random.default_rng(16)
    d = rnd_inputs(rng, 1, 70, 2, 8, 5)
    dO = rng.standard_normal((1, 70, 2, 5))
    a = O.gla_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], dO, seg=64)
    b = O.gla_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], dO, seg=7)
    for key in a:
        np.testing.assert_allclose(a[key], b[key], rtol=1e-12, atol=1e-12, err_msg=key)


@pytest.mark.parametrize("centered,scale", [(True, 1.0), (False, 0.5)])
def test_gdn_reverse_pass_matches_finite_differences(centered, scale):
    """Gated DeltaNet + CCQ: gradients of L = sum <dO, o> from the oracle's reverse pass
    against central finite differences of the oracle forward, along random directions, at
    the size of the small fp32 workload (B=1, T=256, H=2, dk=dv=64)."""
    rng = np.random.default_rng(17)
    B, T, H, dk, dv = 1, 256, 2, 64, 64
    d = rnd_inputs(rng, B, T, H, dk, dv, backbone=O.GDN)
    dO = rng.standard_normal((B, T, H, dv))
    gr = O.gdn_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["beta"], d["lam"], dO, scale=scale,
                       centered=centered, seg=64)
    base = run(d, backbone=O.GDN, scale=scale, centered=centered)
    np.testing.assert_allclose(gr["o"], base["o"], rtol=1e-12, atol=1e-12)

    def loss(dd):
        return float(np.sum(dO * run(dd, backbone=O.GDN, scale=scale, centered=centered)["o"]))

    h = 1e-5
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("gate", "dlogalpha"),
                        ("beta", "dbeta"), ("lam", "dlam")):
        e = rng.standard_normal(d[name].shape)
        dp = dict(d)
        dm = dict(d)
        dp[name] = d[name] + h * e
        dm[name] = d[name] - h * e
        fd = (loss(dp) - loss(dm)) / (2 * h)
        an = float(np.sum(gr[gname] * e))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_gdn_reverse_pass_segment_length_does_not_matter():
    rng = np.random.default_rng(18)
    d = rnd_inputs(rng, 1, 70, 2, 8, 5, backbone=O.GDN)
    dO = rng.standard_normal((1, 70, 2, 5))
    a = O.gdn_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["beta"], d["lam"], dO, seg=64)
    b = O.gdn_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["beta"], d["lam"], dO, seg=7)
    for key in a:
        np.testing.assert_allclose(a[key], b[key], rtol=1e-12, atol=1e-12, err_msg=key)


def test_gdn_reverse_pass_without_contraction_or_decay():
    """With lam = 0, alpha = 1 and beta = 1 on one token the layer is o = (q . k) v, whose
    gradients are dq = (dO . v) k, dk = (dO . v) q, dv = (q . k) dO; dbeta = (dO . v)(q . k)
    (the write v k^T enters with weight beta), and dlogalpha = 0 (nothing to decay)."""
    rng = np.random.default_rng(19)
    q, k, v, dO = (rng.standard_normal((1, 1, 1, n)) for n in (4, 4, 3, 3))
    z = np.zeros((1, 1, 1))
    r = O.gdn_fwd_bwd(q, k, v, z, z + 1.0, z, dO)
    qk, dv_ = float(np.sum(q * k)), float(np.sum(dO * v))
    np.testing.assert_allclose(r["o"], qk * v, rtol=1e-14)
    np.testing.assert_allclose(r["dq"], dv_ * k, rtol=1e-14)
    np.testing.assert_allclose(r["dk"], dv_ * q, rtol=1e-14)
    np.testing.assert_allclose(r["dv"], qk * dO, rtol=1e-14)
    np.testing.assert_allclose(r["dbeta"], dv_ * qk, rtol=1e-14)
    np.testing.assert_allclose(r["dlogalpha"], 0.0, atol=1e-15)


# ---------------------------------------------------------------- pre-processing


def test_prep_normalises_each_head_and_is_scale_invariant():
    rng = np.random.default_rng(21)
    B, T, H, dk = 2, 5, 3, 8
    q = rng.standard_normal((B, T, H, dk)) * rng.uniform(0.1, 10, (B, T, H, 1))
    k = rng.standard_normal((B, T, H, dk))
    W = rng.standard_normal((H, H * dk))
    b = rng.standard_normal(H)
    r = O.prep(q, k, W, b)
    np.testing.assert_allclose(np.linalg.norm(r["q"], axis=-1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(np.linalg.norm(r["k"], axis=-1), 1.0, rtol=1e-14)
    s = O.prep(3.5 * q, 0.25 * k, W, b)
    np.testing.assert_allclose(s["q"], r["q"], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(s["k"], r["k"], rtol=1e-13, atol=1e-15)
    z = O.prep(np.zeros_like(q), k, W, b)
    assert np.all(z["q"] == 0.0)


def test_prep_gate_reads_the_raw_query_before_the_head_split():
    """W = 0 gives sigmoid(b); a single unit weight W[h][j] picks raw feature j of the whole
    token (head j // dk, channel j % dk) for gate h; flipping the sign of W and b gives
    1 - lambda; scaling q by c and W by 1/c leaves lambda unchanged (the gate uses the raw,
    unnormalised query)."""
    rng = np.random.default_rng(22)
    B, T, H, dk = 1, 4, 3, 4
    q = rng.standard_normal((B, T, H, dk))
    k = rng.standard_normal((B, T, H, dk))
    b = rng.standard_normal(H)
    r0 = O.prep(q, k, np.zeros((H, H * dk)), b)
    np.testing.assert_allclose(r0["lam"], np.broadcast_to(1 / (1 + np.exp(-b)), (B, T, H)), rtol=1e-14)
    W = np.zeros((H, H * dk))
    W[0, 2 * dk + 1] = 1.0       # gate 0 <- head 2, channel 1
    W[2, 3] = 1.0                # gate 2 <- head 0, channel 3
    r1 = O.prep(q, k, W, np.zeros(H))
    sig = lambda x: 1 / (1 + np.exp(-x))
    np.testing.assert_allclose(r1["lam"][..., 0], sig(q[:, :, 2, 1]), rtol=1e-14)
    np.testing.assert_allclose(r1["lam"][..., 1], 0.5, rtol=1e-14)
    np.testing.assert_allclose(r1["lam"][..., 2], sig(q[:, :, 0, 3]), rtol=1e-14)
    W = rng.standard_normal((H, H * dk))
    a = O.prep(q, k, W, b)
    f = O.prep(q, k, -W, -b)
    np.testing.assert_allclose(a["lam"] + f["lam"], 1.0, rtol=1e-14)
    c = O.prep(4.0 * q, k, W / 4.0, b)
    np.testing.assert_allclose(c["lam"], a["lam"], rtol=1e-13)


# ---------------------------------------------------------------- packed batches


def _pack(d, lens):
    """Rows of sequences b = 0.. (lengths lens) of a batched input dict, packed."""
    out = {}
    for n, x in d.items():
        if x is None:
            out[n] = None
            continue
        out[n] = np.concatenate([x[b, :L] for b, L in enumerate(lens)], axis=0)
    return out, np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


@pytest.mark.parametrize("backbone", [O.GLA, O.GDN])
def test_packed_batch_of_equal_lengths_is_the_batched_call(backbone):
    """With every length equal, the packed forward (one call per sequence) reproduces the
    batched C path, which walks the (batch, head) pairs itself."""
    rng = np.random.default_rng(40)
    B, T = 3, 23
    d = rnd_inputs(rng, B, T, 2, 6, 4, backbone=backbone)
    S0 = rng.standard_normal((B, 2, 4, 6))
    ref = run(d, backbone=backbone, S0=S0)
    p, cu = _pack(d, [T] * B)
    r = O.varlen_fwd(p["q"], p["k"], p["v"], p["gate"], p["lam"], cu, beta=p["beta"],
                     backbone=backbone, S0=S0)
    np.testing.assert_allclose(r["o"], ref["o"].reshape(B * T, 2, 4), rtol=0, atol=1e-12)
    for key in ("ST", "CT", "muT"):
        np.testing.assert_allclose(r[key], ref[key], rtol=0, atol=1e-12)


def test_packed_batch_sequences_are_independent():
    """Reordering the sequences of a packed batch reorders its outputs and nothing
    else; an empty sequence returns its initial cache."""
    rng = np.random.default_rng(41)
    lens = [11, 0, 30, 5]
    d = rnd_inputs(rng, 4, 30, 2, 5, 3)
    C0 = rng.standard_normal((4, 2, 5, 5))
    mu0 = rng.standard_normal((4, 2, 5))
    p, cu = _pack(d, lens)
    r = O.varlen_fwd(p["q"], p["k"], p["v"], p["gate"], p["lam"], cu, C0=C0, mu0=mu0, t0=7)
    perm = [2, 0, 3, 1]
    dp = {n: (None if x is None else x[perm]) for n, x in d.items()}
    pp, cup = _pack(dp, [lens[i] for i in perm])
    rp = O.varlen_fwd(pp["q"], pp["k"], pp["v"], pp["gate"], pp["lam"], cup, C0=C0[perm],
                      mu0=mu0[perm], t0=7)
    for j, b in enumerate(perm):
        np.testing.assert_array_equal(rp["o"][cup[j]:cup[j + 1]], r["o"][cu[b]:cu[b + 1]])
        for key in ("ST", "CT", "muT"):
            np.testing.assert_array_equal(rp[key][j], r[key][b])
    np.testing.assert_array_equal(r["CT"][1], C0[1])
    np.testing.assert_array_equal(r["muT"][1], mu0[1])


@pytest.mark.parametrize("backbone", [O.GLA, O.GDN])
def test_packed_reverse_pass_of_equal_lengths_is_the_batched_call(backbone):
    rng = np.random.default_rng(42)
    B, T = 2, 17
    d = rnd_inputs(rng, B, T, 1, 4, 3, backbone=backbone)
    dO = rng.standard_normal((B, T, 1, 3))
    if backbone == O.GLA:
        ref = O.gla_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["lam"], dO)
    else:
        ref = O.gdn_fwd_bwd(d["q"], d["k"], d["v"], d["gate"], d["beta"], d["lam"], dO)
        ref["dg"] = ref["dlogalpha"]
    d["dO"] = dO
    p, cu = _pack(d, [T] * B)
    r = O.varlen_fwd_bwd(p["q"], p["k"], p["v"], p["gate"], p["lam"], p["dO"], cu, beta=p["beta"],
                         backbone=backbone)
    for key in ("o", "dq", "dk", "dv", "dg", "dlam") + (("dbeta",) if backbone == O.GDN else ()):
        np.testing.assert_allclose(r[key], ref[key].reshape(r[key].shape), rtol=0, atol=1e-12)


# ---------------------------------------------- decay-aligned statistics (App. J)
# The reading: for Gated DeltaNet's scalar decay, key j enters token t's
# statistics with weight gamma_{j,t} = prod_{s=j+1..t} alpha_s, normalised by
# W_t = sum_j gamma_{j,t}.  These pins hold the oracle's decay=True path to
# numpy's weighted covariance, to the undecayed path at alpha = 1, to its own
# running-mean form, and to a restart where alpha vanishes.

def _gdn_decay_inputs(rng, T, dk, dv, H=1, B=1, logalpha=None):
    d = rnd_inputs(rng, B, T, H, dk, dv, backbone=O.GDN)
    if logalpha is not None:
        d["gate"] = logalpha
    return d


def test_decay_aligned_is_numpy_weighted_covariance():
    rng = np.random.default_rng(51)
    T, dk, dv = 14, 3, 2
    d = _gdn_decay_inputs(rng, T, dk, dv)
    d["gate"] = -rng.uniform(0.05, 1.5, size=(1, T, 1))      # strong forgetting
    d["k"] = d["k"] + 2.0                                     # a common key mean
    r = run(d, backbone=O.GDN, decay=True)
    L = np.cumsum(d["gate"][0, :, 0])
    k, q, lam = d["k"][0, :, 0], d["q"][0, :, 0], d["lam"][0, :, 0]
    for t in range(T):
        w = np.exp(L[t] - L[:t + 1])                          # gamma_{j,t}, j <= t
        if t == 0:
            sig = np.zeros((dk, dk))
        else:
            sig = np.cov(k[:t + 1].T, aweights=w, bias=True)
        qc = q[t] - lam[t] * sig @ q[t]
        np.testing.assert_allclose(r["qclean"][0, t, 0], qc, rtol=0, atol=1e-12)
    W = np.exp(L[-1] - L).sum()
    wT = np.exp(L[-1] - L)
    np.testing.assert_allclose(r["muT"][0, 0], (wT[:, None] * k).sum(0) / W, atol=1e-12)
    np.testing.assert_allclose(r["CT"][0, 0], np.einsum("j,ja,jb->ab", wT, k, k) / W, atol=1e-12)


def test_decay_aligned_without_decay_is_sigma():
    rng = np.random.default_rng(52)
    d = _gdn_decay_inputs(rng, 40, 5, 4, H=2)
    d["gate"] = np.zeros((1, 40, 2))                          # alpha = 1
    a = run(d, backbone=O.GDN, decay=True)
    b = run(d, backbone=O.GDN)
    for key in ("o", "qclean", "CT", "muT", "ST"):
        np.testing.assert_array_equal(a[key], b[key])


def test_decay_aligned_running_mean_form_agrees():
    rng = np.random.default_rng(53)
    d = _gdn_decay_inputs(rng, 50, 6, 5, H=2)
    a = run(d, backbone=O.GDN, decay=True, form=0)
    b = run(d, backbone=O.GDN, decay=True, form=1)
    for key in ("o", "qclean", "CT", "muT"):
        np.testing.assert_allclose(a[key], b[key], rtol=1e-10, atol=1e-12)


def test_decay_aligned_vanishing_alpha_restarts_the_statistics():
    """alpha_t = 0 at t* erases every earlier key from the statistics (and the Gated
    DeltaNet state), so from t* on the outputs are those of a fresh run on the suffix."""
    rng = np.random.default_rng(54)
    T, ts = 45, 17
    d = _gdn_decay_inputs(rng, T, 6, 4, H=2)
    d["gate"][:, ts] = -1e4                                   # exp(-1e4) == 0 in fp64
    full = run(d, backbone=O.GDN, decay=True)
    tail = {k_: (None if v is None else v[:, ts:]) for k_, v in d.items()}
    part = run(tail, backbone=O.GDN, decay=True)
    # Sigma^gamma = k k^T - k k^T = 0 there (up to the rounding of the two products)
    np.testing.assert_allclose(full["qclean"][:, ts], d["q"][:, ts], rtol=0, atol=1e-14)
    np.testing.assert_allclose(full["qclean"][:, ts:], part["qclean"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(full["o"][:, ts:], part["o"], rtol=1e-12, atol=1e-13)


def test_decay_aligned_rejected_where_not_defined():
    rng = np.random.default_rng(55)
    d = _gdn_decay_inputs(rng, 8, 4, 4)
    with pytest.raises(RuntimeError):
        run(rnd_inputs(rng, 1, 8, 1, 4, 4), backbone=O.GLA, decay=True)   # per-channel decay
    with pytest.raises(RuntimeError):
        run(d, backbone=O.GDN, decay=True, t0=5)                          # no decayed count cached
