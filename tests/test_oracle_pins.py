"""Pins for the oracle: checks against what the paper and the mathematics fix.

None of these re-types the oracle's formulas.  They use closed forms from
library routines (scipy's KL), finite differences of the oracle's own loss,
exact identities the paper states (the score-function identity, the exact
old-to-current importance-sampling identity, linearity over m samples), exact
enumeration on tiny vocabularies, and definitional special cases (k = V
equals dense, k = 1 is zero, KL = 0 when student equals teacher).  Each is
chosen so that a plausible mistake (a dropped term, a wrong sign or index, a
swapped direction, a sum instead of a mean) fails at least one of them.
"""
import itertools
import os

import numpy as np
import pytest
from scipy.special import log_softmax, logsumexp, softmax
from scipy.stats import entropy

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_logits(rng, V, scale=2.0):
    return rng.normal(0.0, scale, V)


def mc_inputs(rng, V, M, stale=0.7):
    """Behaviour samples and cached log-probs for a random student/teacher/behaviour triple."""
    z = rand_logits(rng, V)
    y = z + rng.normal(0, 1.0, V)
    b = z + rng.normal(0, stale, V)
    lq, lb = log_softmax(y), log_softmax(b)
    ids = rng.choice(V, size=M, replace=True, p=np.exp(lb))
    return z, y, b, ids, lq[ids], lb[ids]


# ---------------------------------------------------------------- dense KL


@pytest.mark.parametrize("seed", range(5))
def test_dense_kl_matches_scipy_entropy(seed):
    """D_F = KL(q||p) and D_R = KL(p||q) (Sec. 3, eq. dense-forward-kl / dense-reverse-kl)."""
    rng = np.random.default_rng(seed)
    V = 37
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    p, q = softmax(z), softmax(y)
    lf, _, lse, _ = oracle.row("fkl_dense", z, y=y)
    lr, _, _, _ = oracle.row("rkl_dense", z, y=y)
    assert lf == pytest.approx(entropy(q, p), rel=1e-12, abs=1e-14)
    assert lr == pytest.approx(entropy(p, q), rel=1e-12, abs=1e-14)
    assert lse == pytest.approx(logsumexp(z), rel=1e-14)


@pytest.mark.parametrize("est", ["fkl_dense", "rkl_dense"])
@pytest.mark.parametrize("seed", range(3))
def test_dense_kl_actions_at_minus_inf_in_both_rows_drop_out(est, seed):
    """A term of zero weight is zero (the KL divergence's 0 log(0/x) = 0): an
    action whose logit is -inf for both student and teacher contributes
    nothing, so the row equals the row with those actions removed, and their
    gradient entries are 0."""
    rng = np.random.default_rng(200 + seed)
    V = 29
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    gone = rng.choice(V, size=9, replace=False)
    keep = np.setdiff1d(np.arange(V), gone)
    z[gone] = -np.inf
    y[gone] = -np.inf
    loss, g, lse, _ = oracle.row(est, z, y=y, gamma=0.5)
    loss_r, g_r, lse_r, _ = oracle.row(est, z[keep], y=y[keep], gamma=0.5)
    assert np.isfinite(loss) and loss == pytest.approx(loss_r, rel=1e-13, abs=1e-15)
    assert lse == pytest.approx(lse_r, rel=1e-14)
    assert np.all(g[gone] == 0.0)
    np.testing.assert_allclose(g[keep], g_r, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", range(3))
def test_dense_kl_with_zero_weights_matches_scipy_entropy(seed):
    """Actions that only the weighting distribution excludes (student -inf
    where the teacher is finite, for D_R; the reverse for D_F): scipy's
    entropy applies the same 0 log(0/x) = 0 convention."""
    rng = np.random.default_rng(300 + seed)
    V = 31
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    zr = z.copy()
    zr[rng.choice(V, size=8, replace=False)] = -np.inf
    lr, gr, _, _ = oracle.row("rkl_dense", zr, y=y)
    assert lr == pytest.approx(entropy(softmax(zr), softmax(y)), rel=1e-12, abs=1e-14)
    assert np.all(gr[np.isneginf(zr)] == 0.0) and np.isfinite(gr).all()
    yf = y.copy()
    yf[rng.choice(V, size=8, replace=False)] = -np.inf
    lf, gf, _, _ = oracle.row("fkl_dense", z, y=yf)
    assert lf == pytest.approx(entropy(softmax(yf), softmax(z)), rel=1e-12, abs=1e-14)
    np.testing.assert_allclose(gf, softmax(z) - softmax(yf), rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------- finite differences


def fd_grad(f, z, h=1e-5):
    g = np.zeros_like(z)
    for j in range(z.size):
        e = np.zeros_like(z)
        e[j] = h
        g[j] = (f(z + e) - f(z - e)) / (2 * h)
    return g


@pytest.mark.parametrize("est", ["fkl_dense", "rkl_dense", "fkl_topk", "rkl_topk"])
@pytest.mark.parametrize("seed", range(3))
def test_gradient_matches_finite_differences(est, seed):
    rng = np.random.default_rng(100 + seed)
    V, k, gamma = 13, 5, 0.75
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    ids = rng.choice(V, size=k, replace=False)
    tau = log_softmax(y)[ids]
    kw = dict(y=y) if "dense" in est else dict(ids=ids, tau=tau)
    _, g, _, _ = oracle.row(est, z, gamma=gamma, **kw)
    fd = fd_grad(lambda zz: oracle.row(est, zz, want_grad=False, **kw)[0], z)
    np.testing.assert_allclose(g, gamma * fd, atol=1e-8, rtol=0)


@pytest.mark.parametrize("M", [1, 4, 9])
@pytest.mark.parametrize("seed", range(3))
def test_mc_gradient_is_fd_with_advantage_frozen(M, seed):
    """The MC surrogate is differentiated through rho only; A_theta is a
    stop-gradient weight (Sec. 5.1, "Exact importance-sampling identity").
    Finite differences hold A fixed by moving the cached teacher log-probs
    with the student log-probs, so tau - log p_theta stays constant."""
    rng = np.random.default_rng(200 + seed)
    V = 11
    z, _, _, ids, tau, beta = mc_inputs(rng, V, M)
    est = "rkl_mc1" if M == 1 else "rkl_mc"
    _, g, _, _ = oracle.row(est, z, ids=ids, tau=tau, beta=beta, gamma=1.0)
    lp0 = log_softmax(z)[ids]

    def frozen(zz):
        tau_shift = tau + (log_softmax(zz)[ids] - lp0)
        return oracle.row(est, zz, ids=ids, tau=tau_shift, beta=beta, want_grad=False)[0]

    np.testing.assert_allclose(g, fd_grad(frozen, z), atol=1e-8, rtol=0)
    # and it is NOT the derivative of the loss with A moving (the stop-gradient matters)
    naive = fd_grad(lambda zz: oracle.row(est, zz, ids=ids, tau=tau, beta=beta,
                                          want_grad=False)[0], z)
    assert np.max(np.abs(naive - g)) > 1e-4


# ---------------------------------------------------------------- definitional cases


@pytest.mark.parametrize("seed", range(4))
def test_topk_with_full_support_equals_dense(seed):
    """k = V: the renormalised restricted KL is the dense KL (App. A.1 with S = V)."""
    rng = np.random.default_rng(300 + seed)
    V = 17
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    ids = rng.permutation(V)
    tau = log_softmax(y)[ids]
    for sparse, dense in (("fkl_topk", "fkl_dense"), ("rkl_topk", "rkl_dense")):
        ls, gs, _, _ = oracle.row(sparse, z, ids=ids, tau=tau, gamma=1.3)
        ld, gd, _, _ = oracle.row(dense, z, y=y, gamma=1.3)
        assert ls == pytest.approx(ld, rel=1e-12, abs=1e-14)
        np.testing.assert_allclose(gs, gd, atol=1e-14, rtol=1e-11)


def test_topk_single_entry_support_is_zero():
    """k = 1: both renormalised distributions are the same point mass."""
    rng = np.random.default_rng(4)
    z = rand_logits(rng, 9)
    for est in ("fkl_topk", "rkl_topk"):
        loss, g, _, _ = oracle.row(est, z, ids=[3], tau=[-5.0])
        assert abs(loss) < 1e-15 and np.all(np.abs(g) < 1e-15)


@pytest.mark.parametrize("seed", range(6))
def test_kl_nonnegative(seed):
    rng = np.random.default_rng(500 + seed)
    V = 40
    z, y = rand_logits(rng, V, 3.0), rand_logits(rng, V, 3.0)
    ids = rng.choice(V, size=8, replace=False)
    tau = log_softmax(y)[ids]
    for est in ("fkl_topk", "rkl_topk"):
        assert oracle.row(est, z, ids=ids, tau=tau)[0] >= 0
    for est in ("fkl_dense", "rkl_dense"):
        assert oracle.row(est, z, y=y)[0] >= 0


def test_kl_zero_when_student_equals_teacher():
    rng = np.random.default_rng(6)
    V = 25
    z = rand_logits(rng, V)
    ids = rng.choice(V, size=6, replace=False)
    # the teacher log-probs equal the student's; shifting them by a constant
    # (an unnormalised teacher) changes nothing after renormalisation on S
    for shift in (0.0, 3.7):
        tau = log_softmax(z)[ids] + shift
        for est in ("fkl_topk", "rkl_topk"):
            loss, g, _, _ = oracle.row(est, z, ids=ids, tau=tau)
            assert abs(loss) < 1e-14 and np.max(np.abs(g)) < 1e-14
    for est in ("fkl_dense", "rkl_dense"):
        loss, g, _, _ = oracle.row(est, z, y=z + 1.25)
        assert abs(loss) < 1e-14 and np.max(np.abs(g)) < 1e-14
    # MC: teacher = student gives A = 0 for every sample, so surrogate and gradient vanish
    b = z + rng.normal(0, 0.5, V)
    ids = rng.choice(V, size=5)
    loss, g, _, _ = oracle.row("rkl_mc", z, ids=ids, tau=log_softmax(z)[ids],
                               beta=log_softmax(b)[ids])
    assert abs(loss) < 1e-14 and np.max(np.abs(g)) < 1e-14


@pytest.mark.parametrize("est", list(oracle.ESTIMATORS))
def test_gradient_rows_sum_to_zero_and_shift_invariance(est):
    """Softmax is invariant to z -> z + c, so every gradient row sums to zero
    and the loss and gradient do not move under a constant shift."""
    rng = np.random.default_rng(7)
    V = 30
    z, y, b, ids, tau, beta = mc_inputs(rng, V, 1 if est == "rkl_mc1" else 6)
    if est in oracle.DENSE:
        kw = dict(y=y)
    elif est in oracle.MC:
        kw = dict(ids=ids, tau=tau, beta=beta)
    else:
        ids = rng.choice(V, size=6, replace=False)
        kw = dict(ids=ids, tau=log_softmax(y)[ids])
    loss, g, _, _ = oracle.row(est, z, gamma=2.0, **kw)
    assert abs(g.sum()) < 1e-12
    loss2, g2, _, _ = oracle.row(est, z + 11.5, gamma=2.0, **kw)
    assert loss2 == pytest.approx(loss, rel=1e-10, abs=1e-12)
    np.testing.assert_allclose(g2, g, atol=1e-12, rtol=1e-9)


def test_gradient_scale_and_masked_rows():
    rng = np.random.default_rng(8)
    V = 12
    z, y, b, ids, tau, beta = mc_inputs(rng, V, 3)
    l1, g1, _, _ = oracle.row("rkl_mc", z, ids=ids, tau=tau, beta=beta, gamma=1.0)
    l2, g2, _, _ = oracle.row("rkl_mc", z, ids=ids, tau=tau, beta=beta, gamma=-0.25)
    assert l1 == l2
    np.testing.assert_allclose(g2, -0.25 * g1, rtol=1e-15, atol=0)
    l0, g0, lse0, gat0 = oracle.row("rkl_mc", z, ids=ids, tau=tau, beta=beta, valid=False)
    assert l0 == 0 and lse0 == 0 and not g0.any() and not gat0.any()


# ---------------------------------------------------------------- importance sampling


@pytest.mark.parametrize("seed", range(4))
def test_is_identity_by_enumeration_one_sample(seed):
    """D_R = -E_{p_old}[rho A_theta] exactly (Sec. 5.1), and the expected
    surrogate gradient is grad D_R (eq. reverse-kl-gradient via the score
    identity).  Exact enumeration over every action a of a tiny vocabulary."""
    rng = np.random.default_rng(900 + seed)
    V = 7
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    b = z + rng.normal(0, 1.0, V)
    lq, lb = log_softmax(y), log_softmax(b)
    pold = np.exp(lb)
    e_loss, e_grad = 0.0, np.zeros(V)
    for a in range(V):
        loss, g, _, _ = oracle.row("rkl_mc1", z, ids=[a], tau=[lq[a]], beta=[lb[a]])
        e_loss += pold[a] * loss
        e_grad += pold[a] * g
    d_loss, d_grad, _, _ = oracle.row("rkl_dense", z, y=y)
    assert e_loss == pytest.approx(d_loss, rel=1e-12, abs=1e-13)
    np.testing.assert_allclose(e_grad, d_grad, atol=1e-13, rtol=1e-11)


@pytest.mark.parametrize("M", [2, 3])
def test_is_identity_by_enumeration_m_samples_with_duplicates(M):
    """The m-sample average has the same expectation by linearity (Sec. 6.2);
    samples are iid with replacement, duplicates included (App. E).  Every
    ordered m-tuple is enumerated."""
    rng = np.random.default_rng(31 + M)
    V = 5
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    b = z + rng.normal(0, 0.8, V)
    lq, lb = log_softmax(y), log_softmax(b)
    pold = np.exp(lb)
    e_loss, e_grad = 0.0, np.zeros(V)
    for tup in itertools.product(range(V), repeat=M):
        ids = np.array(tup)
        w = np.prod(pold[ids])
        loss, g, _, _ = oracle.row("rkl_mc", z, ids=ids, tau=lq[ids], beta=lb[ids])
        e_loss += w * loss
        e_grad += w * g
    d_loss, d_grad, _, _ = oracle.row("rkl_dense", z, y=y)
    assert e_loss == pytest.approx(d_loss, rel=1e-12, abs=1e-13)
    np.testing.assert_allclose(e_grad, d_grad, atol=1e-13, rtol=1e-11)


def _exact_var(z, lq, lb, M):
    V = z.size
    pold = np.exp(lb)
    m1 = m2 = 0.0
    for tup in itertools.product(range(V), repeat=M):
        ids = np.array(tup)
        w = np.prod(pold[ids])
        est = "rkl_mc1" if M == 1 else "rkl_mc"
        loss = oracle.row(est, z, ids=ids, tau=lq[ids], beta=lb[ids], want_grad=False)[0]
        m1 += w * loss
        m2 += w * loss * loss
    return m2 - m1 * m1


def test_variance_of_m_sample_average_is_one_over_m():
    """Var(L_m | s) = Var(L_1 | s) / m for iid samples: the fixed-prefix ratio
    R_m^local of App. E is exactly 1/m.  The ratios the paper measured on a
    real student (Table 6) sit within 7% of that reference."""
    rng = np.random.default_rng(77)
    V = 5
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    b = z + rng.normal(0, 1.0, V)
    lq, lb = log_softmax(y), log_softmax(b)
    v1 = _exact_var(z, lq, lb, 1)
    assert v1 > 1e-3
    for M in (2, 3, 4):
        assert _exact_var(z, lq, lb, M) / v1 == pytest.approx(1.0 / M, rel=1e-10)
    table = np.loadtxt(os.path.join(GOLDEN, "table6_mc_variance_ratios.txt"))
    for m, r in table:
        assert abs(r - 1.0 / m) <= 0.07 / m


def test_mc_unbiased_by_sampling_and_biased_without_is():
    """Average of the one-sample estimator over many behaviour draws converges
    to D_R (within 5 standard errors).  Negative control (App. F): treating
    p_old samples as if they came from p_theta (rho forced to 1) is biased."""
    rng = np.random.default_rng(2024)
    V, S = 9, 100_000
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    b = z + rng.normal(0, 1.2, V)
    lq, lb, lp = log_softmax(y), log_softmax(b), log_softmax(z)
    ids = rng.choice(V, size=S, p=np.exp(lb))
    per_action = np.array([oracle.row("rkl_mc1", z, ids=[a], tau=[lq[a]], beta=[lb[a]],
                                      want_grad=False)[0] for a in range(V)])
    no_is = np.array([oracle.row("rkl_mc1", z, ids=[a], tau=[lq[a]], beta=[lp[a]],
                                 want_grad=False)[0] for a in range(V)])
    d_r = oracle.row("rkl_dense", z, y=y, want_grad=False)[0]
    samples = per_action[ids]
    se = samples.std() / np.sqrt(S)
    assert abs(samples.mean() - d_r) < 5 * se
    biased = no_is[ids]
    assert abs(biased.mean() - d_r) > 10 * biased.std() / np.sqrt(S)


def test_on_policy_case_is_the_plain_score_function_estimator():
    """With behaviour = current student, rho = 1 and the gradient is
    -A_theta(a) grad log p_theta(a) (App. A.2), whose logit gradient is
    -A (e_a - p)."""
    rng = np.random.default_rng(10)
    V = 15
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    lp, lq = log_softmax(z), log_softmax(y)
    for a in (0, 7, 14):
        _, g, _, _ = oracle.row("rkl_mc1", z, ids=[a], tau=[lq[a]], beta=[lp[a]])
        e_a = np.zeros(V)
        e_a[a] = 1.0
        np.testing.assert_allclose(g, -(lq[a] - lp[a]) * (e_a - softmax(z)), atol=1e-14, rtol=1e-12)


# ---------------------------------------------------------------- stored inputs


def f32_to_bf16_bits(x):
    """Truncating fp32 -> bf16 for values that are already bf16-exact."""
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_bf16_bits_are_widened_exactly():
    vals = np.array([1.0, -2.5, 0.0078125, -0.0, 3.140625, -65280.0, 1.5e-38], np.float32)
    bits = f32_to_bf16_bits(vals)
    # known encodings of bf16
    assert bits[0] == 0x3F80 and bits[1] == 0xC020
    V = vals.size
    exact = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ids = np.array([[0, 4, 2]], np.int32)
    tau = np.array([[-1.0, -2.0, -3.0]], np.float32)
    beta = np.array([[-1.5, -1.0, -2.0]], np.float32)
    out = oracle.rows("rkl_mc", oracle.BF16, bits[None, :], V, ids=ids, tau=tau, beta=beta)
    ref = oracle.row("rkl_mc", exact, ids=ids[0], tau=tau[0].astype(np.float64),
                     beta=beta[0].astype(np.float64))
    assert out["loss"][0] == ref[0]
    np.testing.assert_array_equal(out["grad"][0], ref[1])
    np.testing.assert_array_equal(out["gathered"][0], exact[[0, 4, 2]])


@pytest.mark.parametrize("est", list(oracle.ESTIMATORS))
def test_batch_driver_matches_single_rows_with_padding_stride(est):
    """oracle_rows walks rows of stride ld > V and per-row cache slices."""
    rng = np.random.default_rng(11)
    n, V, ld = 6, 23, 32
    K = 1 if est == "rkl_mc1" else 4
    logits = np.full((n, ld), np.nan, np.float32)
    logits[:, :V] = rng.normal(0, 2, (n, V))
    teacher = np.full((n, ld), np.nan, np.float32)
    teacher[:, :V] = logits[:, :V] + rng.normal(0, 1, (n, V))
    ids = np.stack([rng.choice(V, K, replace=False) for _ in range(n)]).astype(np.int32)
    tau = rng.normal(-3, 1, (n, K)).astype(np.float32)
    beta = rng.normal(-3, 1, (n, K)).astype(np.float32)
    mask = np.array([1, 1, 0, 1, 0, 1], np.uint8)
    kw = dict(teacher_logits=teacher) if est in oracle.DENSE else dict(ids=ids, tau=tau, beta=beta)
    out = oracle.rows(est, oracle.F32, logits, V, mask=mask, gamma=0.5, **kw)
    for r in range(n):
        rk = dict(y=teacher[r, :V]) if est in oracle.DENSE else dict(ids=ids[r], tau=tau[r],
                                                                       beta=beta[r])
        loss, g, lse, gat = oracle.row(est, logits[r, :V], gamma=0.5, valid=bool(mask[r]), **rk)
        assert out["loss"][r] == loss and out["lse"][r] == lse
        np.testing.assert_array_equal(out["grad"][r], g)
        if gat is not None:
            np.testing.assert_array_equal(out["gathered"][r], gat)


def test_rejects_bad_arguments():
    z = np.zeros(5)
    with pytest.raises(ValueError):
        oracle.row("rkl_mc", z, ids=[5], tau=[0.0], beta=[0.0])  # id out of range
    with pytest.raises(ValueError):
        oracle.row("rkl_mc1", z, ids=[0, 1], tau=[0.0, 0.0], beta=[0.0, 0.0])  # MC1 needs M = 1
    with pytest.raises(ValueError):
        oracle.row("rkl_mc", z, ids=[0], tau=[0.0])  # MC needs behaviour log-probs


# ---------------------------------------------------------------- surrogate family (Sec. 5.1) and App. F

THETA_ADV = ("rkl_mc", "rkl_mc_clip", "rkl_mc_nois")


def away_from_clip_kinks(z, ids, beta, eps, margin=1e-3):
    rho = np.exp(log_softmax(z)[ids] - beta)
    return np.all(np.abs(rho - (1 + eps)) > margin) and np.all(np.abs(rho - (1 - eps)) > margin)


@pytest.mark.parametrize("est", ["rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois"])
@pytest.mark.parametrize("seed", range(4))
def test_surrogate_family_gradients_match_finite_differences(est, seed):
    """Each surrogate is differentiated with its advantage held fixed.
    A_theta is frozen as before; A_old = log q - log p_old does not depend on
    the student, so plain finite differences apply.  Samples sit away from the
    clip boundaries, where the min is not differentiable."""
    rng = np.random.default_rng(600 + seed)
    V, M, eps = 12, 7, 0.2
    for _ in range(100):
        z, _, _, ids, tau, beta = mc_inputs(rng, V, M, stale=0.9)
        if away_from_clip_kinks(z, ids, beta, eps):
            break
    _, g, _, _ = oracle.row(est, z, ids=ids, tau=tau, beta=beta, eps=eps)
    lp0 = log_softmax(z)[ids]

    def f(zz):
        t = tau + (log_softmax(zz)[ids] - lp0) if est in THETA_ADV else tau
        return oracle.row(est, zz, ids=ids, tau=t, beta=beta, eps=eps, want_grad=False)[0]

    np.testing.assert_allclose(g, fd_grad(f, z), atol=1e-8, rtol=0)


@pytest.mark.parametrize("adv", ["theta", "old"])
def test_clip_is_inert_when_eps_is_huge_or_ratios_are_inside(adv):
    """The clipped surrogate equals the unclipped one when no ratio leaves
    [1 - eps, 1 + eps] (Sec. 3, eq. ppo-style-surrogate)."""
    clip, noclip = ("rkl_mc_clip", "rkl_mc") if adv == "theta" else ("rkl_mc_old_clip",
                                                                       "rkl_mc_old")
    rng = np.random.default_rng(13)
    V, M = 20, 9
    z, _, _, ids, tau, beta = mc_inputs(rng, V, M, stale=1.5)
    a = oracle.row(clip, z, ids=ids, tau=tau, beta=beta, eps=1e9)
    b = oracle.row(noclip, z, ids=ids, tau=tau, beta=beta)
    assert a[0] == pytest.approx(b[0], rel=1e-14, abs=1e-15)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-13, atol=1e-15)
    # behaviour log-probs within 0.05 of the student's: every rho within [0.95, 1.05]
    beta2 = log_softmax(z)[ids] + rng.uniform(-0.05, 0.05, M)
    rho = np.exp(log_softmax(z)[ids] - beta2)
    assert np.all(np.abs(rho - 1) < 0.2)
    a = oracle.row(clip, z, ids=ids, tau=tau, beta=beta2, eps=0.2)
    b = oracle.row(noclip, z, ids=ids, tau=tau, beta=beta2)
    assert a[0] == pytest.approx(b[0], rel=1e-14, abs=1e-15)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_ppo_clip_stops_the_gradient_outside_the_trust_region(sign):
    """One sample, advantage A: for A > 0 and rho > 1 + eps, or A < 0 and
    rho < 1 - eps, the min selects the constant clipped term, so the loss is
    -rho_bar A and the gradient is exactly zero; on the other side of the
    range the unclipped term is selected and the gradient is nonzero."""
    V, eps = 6, 0.2
    z = np.array([0.3, -1.0, 2.0, 0.5, -0.2, 1.1])
    lp = log_softmax(z)
    a = 2
    for est in ("rkl_mc_old_clip", "rkl_mc_clip"):
        # choose beta so rho = 1.5 (A > 0 case) or rho = 0.5 (A < 0 case)
        rho = 1.5 if sign > 0 else 0.5
        beta = lp[a] - np.log(rho)
        # choose tau so the advantage has the wanted sign, whichever advantage is used
        tau = (beta if est == "rkl_mc_old_clip" else lp[a]) + sign * 0.7
        loss, g, _, _ = oracle.row(est, z, ids=[a], tau=[tau], beta=[beta], eps=eps)
        A = tau - (beta if est == "rkl_mc_old_clip" else lp[a])
        rho_bar = min(max(rho, 1 - eps), 1 + eps)
        assert loss == pytest.approx(-rho_bar * A, rel=1e-12)
        assert not np.any(g)
        # mirrored ratio: the unclipped term is the smaller one, gradient flows
        rho2 = 0.5 if sign > 0 else 1.5
        beta2 = lp[a] - np.log(rho2)
        tau2 = (beta2 if est == "rkl_mc_old_clip" else lp[a]) + sign * 0.7
        loss2, g2, _, _ = oracle.row(est, z, ids=[a], tau=[tau2], beta=[beta2], eps=eps)
        A2 = tau2 - (beta2 if est == "rkl_mc_old_clip" else lp[a])
        assert loss2 == pytest.approx(-rho2 * A2, rel=1e-12)
        assert np.max(np.abs(g2)) > 0.1


def test_on_policy_samples_collapse_the_family():
    """With behaviour = current student (rho = 1, A_old = A_theta), every
    member of the family gives the same gradient, and the no-IS estimator
    (App. F) is the plain score-function estimator of App. A.2."""
    rng = np.random.default_rng(14)
    V, M = 16, 5
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    ids = rng.choice(V, M)
    lp, lq = log_softmax(z), log_softmax(y)
    base = oracle.row("rkl_mc", z, ids=ids, tau=lq[ids], beta=lp[ids])
    for est in ("rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois"):
        r = oracle.row(est, z, ids=ids, tau=lq[ids], beta=lp[ids])
        np.testing.assert_allclose(r[1], base[1], rtol=1e-12, atol=1e-14)
        if est != "rkl_mc_nois":
            assert r[0] == pytest.approx(base[0], rel=1e-12)
    # no-IS surrogate value: -(1/M) sum_i A_i log p(a_i), independent of beta
    A = lq[ids] - lp[ids]
    r = oracle.row("rkl_mc_nois", z, ids=ids, tau=lq[ids], beta=lp[ids] + 3.0)
    assert r[0] == pytest.approx(-(A * lp[ids]).mean(), rel=1e-12)


def test_only_the_current_advantage_gives_the_exact_identity():
    """Sec. 5.1: with A_theta the old-to-current IS surrogate averages to D_R
    exactly; the rollout-time advantage A_old does not (negative control),
    nor does dropping the ratio (App. F)."""
    rng = np.random.default_rng(15)
    V = 6
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    b = z + rng.normal(0, 1.0, V)
    lq, lb = log_softmax(y), log_softmax(b)
    pold = np.exp(lb)
    d_loss, d_grad, _, _ = oracle.row("rkl_dense", z, y=y)
    e = {}
    for est in ("rkl_mc1", "rkl_mc_old", "rkl_mc_nois"):
        gl, gg = 0.0, np.zeros(V)
        for a in range(V):
            l, g, _, _ = oracle.row(est, z, ids=[a], tau=[lq[a]], beta=[lb[a]])
            gl += pold[a] * l
            gg += pold[a] * g
        e[est] = (gl, gg)
    np.testing.assert_allclose(e["rkl_mc1"][1], d_grad, atol=1e-13)
    assert np.max(np.abs(e["rkl_mc_old"][1] - d_grad)) > 1e-3
    assert np.max(np.abs(e["rkl_mc_nois"][1] - d_grad)) > 1e-3


def test_clip_rejects_a_non_positive_eps():
    z = np.zeros(4)
    with pytest.raises(ValueError):
        oracle.row("rkl_mc_clip", z, ids=[1], tau=[0.0], beta=[0.0], eps=0.0)


# ---------------------------------------------------------------- truncated top-k


@pytest.mark.parametrize("est", ["fkl_topk_trunc", "rkl_topk_trunc"])
@pytest.mark.parametrize("seed", range(3))
def test_truncated_topk_gradient_matches_finite_differences(est, seed):
    rng = np.random.default_rng(700 + seed)
    V, k = 14, 5
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    ids = rng.choice(V, size=k, replace=False)
    tau = log_softmax(y)[ids]
    _, g, _, _ = oracle.row(est, z, ids=ids, tau=tau, gamma=0.5)
    fd = fd_grad(lambda zz: oracle.row(est, zz, ids=ids, tau=tau, want_grad=False)[0], z)
    np.testing.assert_allclose(g, 0.5 * fd, atol=1e-8, rtol=0)


def test_truncated_topk_with_full_support_is_dense():
    rng = np.random.default_rng(16)
    V = 19
    z, y = rand_logits(rng, V), rand_logits(rng, V)
    ids = rng.permutation(V)
    tau = log_softmax(y)[ids]
    for trunc, dense in (("fkl_topk_trunc", "fkl_dense"), ("rkl_topk_trunc", "rkl_dense")):
        a = oracle.row(trunc, z, ids=ids, tau=tau)
        b = oracle.row(dense, z, y=y)
        assert a[0] == pytest.approx(b[0], rel=1e-12, abs=1e-14)
        np.testing.assert_allclose(a[1], b[1], atol=1e-14, rtol=1e-11)


@pytest.mark.parametrize("seed", range(4))
def test_truncated_and_renormalised_topk_are_tied_by_the_support_masses(seed):
    """With Z_p = p(S) and Z_q = q(S), splitting each log-ratio into the
    renormalised one plus log(Z_q / Z_p) gives
      sum_S q (log q - log p) = Z_q KL(q~ || p~) + Z_q log(Z_q / Z_p),
      sum_S p (log p - log q) = Z_p KL(p~ || q~) + Z_p log(Z_p / Z_q)."""
    rng = np.random.default_rng(800 + seed)
    V, k = 40, 7
    z, y = rand_logits(rng, V, 2.5), rand_logits(rng, V, 2.5)
    ids = rng.choice(V, size=k, replace=False)
    lq = log_softmax(y)
    tau = lq[ids]
    Zp = softmax(z)[ids].sum()
    Zq = np.exp(lq[ids]).sum()
    f_t = oracle.row("fkl_topk_trunc", z, ids=ids, tau=tau, want_grad=False)[0]
    f_r = oracle.row("fkl_topk", z, ids=ids, tau=tau, want_grad=False)[0]
    r_t = oracle.row("rkl_topk_trunc", z, ids=ids, tau=tau, want_grad=False)[0]
    r_r = oracle.row("rkl_topk", z, ids=ids, tau=tau, want_grad=False)[0]
    assert f_t == pytest.approx(Zq * f_r + Zq * np.log(Zq / Zp), rel=1e-11, abs=1e-14)
    assert r_t == pytest.approx(Zp * r_r + Zp * np.log(Zp / Zq), rel=1e-11, abs=1e-14)


def test_truncated_forward_topk_can_be_negative():
    """Without renormalisation the restricted forward sum is not a KL: it is
    negative when the teacher puts less mass on S than the student does."""
    z = np.array([3.0, 0.0, 0.0, 0.0])
    y = np.array([0.0, 1.0, 1.0, 1.0])
    ids = np.array([0])
    loss = oracle.row("fkl_topk_trunc", z, ids=ids, tau=log_softmax(y)[ids], want_grad=False)[0]
    assert loss < 0
