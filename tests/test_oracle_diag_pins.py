"""Pins of the oracle's MC diagnostics (Sec. 5.2, Fig. 5: the p99 tail of
rho_theta; App. E, Table 6: variance of the m-sample estimator at a fixed
prefix and over a sequence).

Checked against a hand-computed two-sample row, numpy's inverted-CDF
quantile, exact expectations by enumeration over a small vocabulary
(unbiasedness of the per-token variance), the 1/m law for iid draws that
Table 6's fixed-prefix column follows, an exact identity between the two
ratios for one-token sequences, and the on-policy special case.
"""
import numpy as np
import pytest
from scipy.special import log_softmax

import oracle

EPS = oracle.CLIP_EPS


def test_two_sample_row_by_hand():
    # log p_theta = (log .5, log .25), beta = (log .25, log .5): rho = (2, .5);
    # tau = (log .3, log .1): A = (log .6, log .4); X = -rho A
    lse = np.array([0.0])
    g = np.log([[0.5, 0.25]])
    beta = np.log([[0.25, 0.5]]).astype(np.float32)
    tau = np.log([[0.3, 0.1]]).astype(np.float32)
    d = oracle.mc_diagnostics(lse, g, tau, beta, q=0.5)
    # tau and beta are stored as float32: recompute the expectation from them
    t, b = tau.astype(np.float64)[0], beta.astype(np.float64)[0]
    rho = np.exp(g[0] - b)
    X = -rho * (t - g[0])
    assert abs(rho[0] - 2.0) < 1e-6 and abs(rho[1] - 0.5) < 1e-6
    assert abs(d["mean"][0] - X.mean()) < 1e-12
    assert abs(d["var"][0] - (X[0] - X[1]) ** 2 / 2) < 1e-12
    assert abs(d["rho_max"][0] - rho[0]) < 1e-12
    assert d["rho_quantile"] == rho[1]                      # rank ceil(.5 * 2) = 1
    assert oracle.mc_diagnostics(lse, g, tau, beta, q=0.51)["rho_quantile"] == rho[0]
    assert d["clip_frac"] == 1.0                            # 2 and .5 both outside [.8, 1.2]


def _draws(rng, n_rows, V, M, spread=1.0):
    """Rows of one prefix: student z, teacher tau, behaviour p_old; M iid draws
    per row by inversion, with the loss call's lse and gathered logits."""
    z = rng.normal(0, spread, V)
    y = z + rng.normal(0, 1, V)
    b = z + rng.normal(0, 0.5, V)
    lz, ly, lb = log_softmax(z), log_softmax(y), log_softmax(b)
    ids = np.stack([oracle.sample_row(b, rng.random(M).astype(np.float32))[0]
                    for _ in range(n_rows)])
    lse = np.full(n_rows, np.logaddexp.reduce(z))
    return dict(lse=lse, gathered=z[ids], tau=ly[ids].astype(np.float32),
                beta=lb[ids].astype(np.float32), lz=lz, ly=ly, lb=lb)


def test_per_token_variance_is_unbiased_by_enumeration():
    rng = np.random.default_rng(1)
    V, M, rows = 7, 4, 6000
    d = _draws(rng, rows, V, M)
    # exact moments of X(a) = -rho(a) A(a) under a ~ p_old, from the same
    # float32-stored log-probs the draws carry
    lb32 = d["lb"].astype(np.float32).astype(np.float64)
    ly32 = d["ly"].astype(np.float32).astype(np.float64)
    rho = np.exp(d["lz"] - lb32)
    X = -rho * (ly32 - d["lz"])
    pold = np.exp(d["lb"])
    mean_x = np.sum(pold * X)
    var_x = np.sum(pold * X ** 2) - mean_x ** 2
    out = oracle.mc_diagnostics(d["lse"], d["gathered"], d["tau"], d["beta"])
    se_var = out["var"].std() / np.sqrt(rows)
    assert abs(out["var"].mean() - var_x) < 5 * se_var
    se_mean = out["mean"].std() / np.sqrt(rows)
    assert abs(out["mean"].mean() - mean_x) < 5 * se_mean
    # the IS identity: E_{p_old}[X] = -sum_a p_theta(a) A(a), up to float32 storage
    assert abs(mean_x + np.sum(np.exp(d["lz"]) * (ly32 - d["lz"]) * np.exp(d["lb"] - lb32))) < 1e-12


def test_fixed_prefix_ratio_follows_one_over_m():
    # iid draws: Var(mean of m) = Var(one) / m, the law Table 6's fixed-prefix
    # column follows (0.255 at m = 4, 0.0588 at m = 16)
    rng = np.random.default_rng(2)
    d = _draws(rng, 3000, 50, 16, spread=2.0)
    out = oracle.mc_diagnostics(d["lse"], d["gathered"], d["tau"], d["beta"],
                                group_sizes=[1, 2, 4, 8])
    r = out["ratio_local"]
    assert r[0] == 1.0
    for m, got in zip([2, 4, 8], r[1:]):
        assert abs(got * m - 1.0) < 0.08, (m, got)


def test_sequence_ratio_follows_one_over_m_and_equals_local_for_single_tokens():
    rng = np.random.default_rng(3)
    d = _draws(rng, 4096, 40, 16, spread=2.0)
    args = (d["lse"], d["gathered"], d["tau"], d["beta"])
    out = oracle.mc_diagnostics(*args, group_sizes=[1, 4, 8], seq_len=64)
    for m, got in zip([4, 8], out["ratio_seq"][1:]):
        assert abs(got * m - 1.0) < 0.25, (m, got)
    one = oracle.mc_diagnostics(*args, group_sizes=[2, 4, 8], seq_len=1)
    assert np.array_equal(one["ratio_seq"], one["ratio_local"])


def test_quantile_matches_numpy_inverted_cdf():
    rng = np.random.default_rng(4)
    N, M = 200, 8
    lse = rng.normal(10, 1, N)
    g = lse[:, None] + np.log(rng.random((N, M)))
    beta = (g - lse[:, None] + rng.normal(0, 1, (N, M))).astype(np.float32)
    tau = rng.normal(-5, 1, (N, M)).astype(np.float32)
    mask = (rng.random(N) < 0.8).astype(np.uint8)
    rho = np.exp(g - lse[:, None] - beta.astype(np.float64))[mask == 1].ravel()
    for q in (1e-9, 0.01, 0.5, 0.9, 0.99, 0.999, 1.0):
        got = oracle.mc_diagnostics(lse, g, tau, beta, mask=mask, q=q)["rho_quantile"]
        assert got == np.quantile(rho, q, method="inverted_cdf"), q
    clip = oracle.mc_diagnostics(lse, g, tau, beta, mask=mask)["clip_frac"]
    assert clip == np.mean(np.abs(rho - 1) > EPS)


def test_on_policy_ratios_are_one():
    # beta = log p_theta: rho = 1 everywhere (App. A.2), nothing clipped
    rng = np.random.default_rng(5)
    N, M = 50, 4
    lse = rng.normal(8, 1, N)
    lp = np.log(rng.random((N, M)))
    beta = lp.astype(np.float32)
    g = lp.astype(np.float32).astype(np.float64) + lse[:, None]
    tau = rng.normal(-4, 1, (N, M)).astype(np.float32)
    out = oracle.mc_diagnostics(lse, g, tau, beta)
    assert out["clip_frac"] == 0.0
    assert abs(out["rho_quantile"] - 1) < 1e-12 and np.all(np.abs(out["rho_max"] - 1) < 1e-12)
    A = tau.astype(np.float64) - (g - lse[:, None])
    assert np.allclose(out["mean"], -A.mean(1), atol=1e-12)


def test_masked_rows_are_excluded():
    rng = np.random.default_rng(6)
    d = _draws(rng, 300, 20, 8)
    mask = (rng.random(300) < 0.6).astype(np.uint8)
    args = (d["lse"], d["gathered"], d["tau"], d["beta"])
    full = oracle.mc_diagnostics(*args, mask=mask, group_sizes=[2, 4])
    keep = mask == 1
    sub = oracle.mc_diagnostics(*(a[keep] for a in args), group_sizes=[2, 4])
    assert np.array_equal(full["var"][keep], sub["var"]) and np.all(full["var"][~keep] == 0)
    for key in ("rho_quantile", "clip_frac"):
        assert full[key] == sub[key]
    assert np.allclose(full["ratio_local"], sub["ratio_local"], rtol=1e-12)


@pytest.mark.parametrize("kw", [dict(group_sizes=[3]), dict(group_sizes=[8]), dict(q=0.0),
                                dict(q=1.5), dict(group_sizes=[0])])
def test_bad_arguments(kw):
    g = np.zeros((2, 8))
    z = np.zeros((2, 8), np.float32)
    with pytest.raises(ValueError):
        oracle.mc_diagnostics(np.zeros(2), g, z, z, **kw)


def test_sequence_means_count_only_valid_tokens():
    # A sequence whose last two tokens are masked has the same token average
    # as one where those two tokens repeat its first two: the sequence ratio
    # must not change.  (Sequences differ in their own ratio, so a wrong
    # normaliser would move the pooled result.)
    rng = np.random.default_rng(7)
    d1 = _draws(rng, 4, 30, 8, spread=1.0)
    d2 = _draws(rng, 4, 30, 8, spread=3.0)
    cat = {k: np.concatenate([d1[k], d2[k]]) for k in ("lse", "gathered", "tau", "beta")}
    mask = np.array([1, 1, 1, 1, 1, 1, 0, 0], np.uint8)
    masked = oracle.mc_diagnostics(cat["lse"], cat["gathered"], cat["tau"], cat["beta"], mask=mask,
                                   group_sizes=[2, 4], seq_len=4)
    rep = {k: v.copy() for k, v in cat.items()}
    for k in rep:
        rep[k][6:8] = rep[k][4:6]
    full = oracle.mc_diagnostics(rep["lse"], rep["gathered"], rep["tau"], rep["beta"],
                                 group_sizes=[2, 4], seq_len=4)
    assert np.allclose(masked["ratio_seq"], full["ratio_seq"], rtol=1e-12)
