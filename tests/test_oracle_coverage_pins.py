"""Pins of the oracle's support coverage (App. A.1's restricted normalisers
Z_p^S and Z_q^S) to what the definitions fix, independently of its own code:

- the whole vocabulary as support holds all the mass (k = V gives 1 and 1);
- the exact identities that tie the normalisers to two other estimators of
  the oracle, computed without them: with KL~ the renormalised KL on S,
    sum_S q log(q/p) = Z_q KL(q~ || p~) + Z_q log(Z_q / Z_p)   (forward),
    sum_S p log(p/q) = Z_p KL(p~ || q~) + Z_p log(Z_p / Z_q)   (reverse);
- the truncated forward KL's gradient, summed over S, is gamma Z_q (Z_p - 1);
- additivity over a partition of the support, invariance to a shift of z,
  and a hand-computed row.
"""
import numpy as np
import pytest
from scipy.special import log_softmax

import oracle


def row(V=500, k=24, seed=0, sigma=2.0):
    rng = np.random.default_rng(seed)
    z = sigma * rng.standard_normal(V)
    y = z + rng.standard_normal(V)
    tau = log_softmax(y)
    ids = np.argsort(-y, kind="stable")[:k].astype(np.int32)
    return z, y, ids, tau[ids]


def test_hand_computed_row():
    # z = log(1, 2, 3, 4): p = (0.1, 0.2, 0.3, 0.4); S = {3, 1}: Z_p = 0.6
    z = np.log([1.0, 2.0, 3.0, 4.0])
    zp, zq = oracle.support_coverage(z, [3, 1], np.log([0.25, 0.5]))
    assert zp == pytest.approx(0.6, abs=1e-15)
    assert zq == pytest.approx(0.75, abs=1e-15)


def test_full_vocabulary_support_holds_all_mass():
    z, y, _, _ = row(V=300)
    ids = np.random.default_rng(1).permutation(300).astype(np.int32)
    zp, zq = oracle.support_coverage(z, ids, log_softmax(y)[ids])
    assert zp == pytest.approx(1.0, abs=1e-12)
    assert zq == pytest.approx(1.0, abs=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_truncated_equals_scaled_renormalised_plus_coverage_term(seed):
    z, y, ids, tau = row(seed=seed)
    zp, zq = oracle.support_coverage(z, ids, tau)
    assert 0 < zp < 1 and 0 < zq < 1
    one = lambda est: oracle.row(est, z, ids=ids, tau=tau, want_grad=False)[0]
    fwd_trunc, fwd = one("fkl_topk_trunc"), one("fkl_topk")
    rev_trunc, rev = one("rkl_topk_trunc"), one("rkl_topk")
    assert fwd_trunc == pytest.approx(zq * fwd + zq * np.log(zq / zp), rel=1e-10, abs=1e-13)
    assert rev_trunc == pytest.approx(zp * rev + zp * np.log(zp / zq), rel=1e-10, abs=1e-13)


def test_truncated_forward_gradient_mass_on_the_support():
    z, y, ids, tau = row(seed=7)
    zp, zq = oracle.support_coverage(z, ids, tau)
    gamma = 0.75
    _, grad, _, _ = oracle.row("fkl_topk_trunc", z, ids=ids, tau=tau, gamma=gamma)
    assert grad[ids].sum() == pytest.approx(gamma * zq * (zp - 1.0), rel=1e-10)


def test_additive_over_a_partition_and_shift_invariant():
    z, y, ids, tau = row(seed=3, k=30)
    a = oracle.support_coverage(z, ids[:11], tau[:11])
    b = oracle.support_coverage(z, ids[11:], tau[11:])
    whole = oracle.support_coverage(z, ids, tau)
    assert whole[0] == pytest.approx(a[0] + b[0], rel=1e-13)
    assert whole[1] == pytest.approx(a[1] + b[1], rel=1e-13)
    shifted = oracle.support_coverage(z + 17.5, ids, tau)
    assert shifted[0] == pytest.approx(whole[0], rel=1e-12)


def test_stale_support_covers_less_of_the_current_student():
    """Sec. 6: a support chosen by an older policy holds less of the current
    student's mass than the current student's own top-k."""
    rng = np.random.default_rng(5)
    z = 2.0 * rng.standard_normal(2000)
    z_old = z + 1.5 * rng.standard_normal(2000)
    k = 32
    cur = np.argsort(-z, kind="stable")[:k].astype(np.int32)
    old = np.argsort(-z_old, kind="stable")[:k].astype(np.int32)
    tau = np.full(k, -5.0)
    assert oracle.support_coverage(z, old, tau)[0] < oracle.support_coverage(z, cur, tau)[0]


def test_batch_driver_matches_rows_and_masks():
    import synth

    w = synth.TOPK32.replace(N=7, V=3000)
    d = synth.generate(w)
    mask = np.array([1, 0, 1, 1, 0, 1, 1], np.uint8)
    cov = oracle.coverage_rows(oracle.BF16, d["logits"], w.V, d["topk_idx"], d["topk_tau"],
                               mask=mask)
    z = synth.bf16_bits_to_f32(d["logits"]).astype(np.float64)
    for r in range(w.N):
        if mask[r] == 0:
            assert cov[r, 0] == 0 and cov[r, 1] == 0
        else:
            assert tuple(cov[r]) == oracle.support_coverage(z[r], d["topk_idx"][r],
                                                            d["topk_tau"][r].astype(np.float64))
