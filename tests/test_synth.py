"""The seeded input generator: determinism, row independence, and that the
cache it builds is what the rollout and teacher-scoring stages would record."""
import numpy as np
import pytest
from scipy.special import log_softmax

import synth

SMALL = synth.Workload("t", N=12, V=1001, dtype=synth.BF16, estimators=(), k=7, M=5,
                       sigma_student=3.0, boost_prob=0.05, boost_value=8.0, sigma_teacher=1.0,
                       sigma_behaviour=0.5, dense_teacher=True, seed=42)


def test_deterministic_and_rows_regenerate_independently():
    a = synth.generate(SMALL)
    b = synth.generate(SMALL, nthreads=1)
    c = synth.generate(SMALL, 5, 9)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
        np.testing.assert_array_equal(a[key][5:9], c[key])
    other = synth.generate(SMALL.replace(seed=43))
    assert not np.array_equal(a["logits"], other["logits"])


def test_row_stride_padding_is_left_untouched():
    a = synth.generate(SMALL, 0, 3, ld=1008)
    b = synth.generate(SMALL, 0, 3)
    np.testing.assert_array_equal(a["logits"][:, :1001], b["logits"])
    assert not a["logits"][:, 1001:].any()


def test_value_distributions():
    """Student logits: N(0, 3^2) plus +8 on a Bernoulli(0.01) share of entries."""
    from scipy.stats import norm
    w = SMALL.replace(V=200_000, N=2, boost_prob=0.01, k=0, M=0, dense_teacher=False)
    z = synth.as_f64(w, synth.generate(w)["logits"]).ravel()
    n = z.size
    assert z.mean() == pytest.approx(0.08, abs=5 * 3.1 / np.sqrt(n))
    assert z.var() == pytest.approx(9.0 + 0.01 * 0.99 * 64.0, rel=0.02)
    p_tail = 0.99 * norm.sf(8.0, 0, 3) + 0.01 * norm.sf(8.0, 8, 3)
    assert (z > 8.0).mean() == pytest.approx(p_tail, abs=5 * np.sqrt(p_tail / n))
    w2 = w.replace(boost_prob=0.0, dtype=synth.F32)
    z2 = synth.generate(w2)["logits"].astype(np.float64)
    assert z2.mean() == pytest.approx(0.0, abs=0.03) and z2.std() == pytest.approx(3.0, rel=0.01)


def test_topk_cache_is_teacher_topk_with_teacher_logprobs():
    d = synth.generate(SMALL)
    for r in range(SMALL.N):
        y = synth.teacher_row(SMALL, r)
        np.testing.assert_array_equal(synth.as_f64(SMALL, d["teacher_logits"][r]), y)
        order = np.lexsort((np.arange(y.size), -y))  # descending y, lower index first
        np.testing.assert_array_equal(d["topk_idx"][r], order[:SMALL.k])
        np.testing.assert_allclose(d["topk_tau"][r], log_softmax(y)[order[:SMALL.k]], rtol=1e-6)


def test_mc_cache_is_inverse_cdf_sampling_of_behaviour_policy():
    d = synth.generate(SMALL)
    for r in range(SMALL.N):
        b = synth.behaviour_row(SMALL, r)
        y = synth.teacher_row(SMALL, r)
        lb = log_softmax(b)
        ids = d["mc_ids"][r]
        assert ids.min() >= 0 and ids.max() < SMALL.V
        np.testing.assert_allclose(d["mc_beta"][r], lb[ids], rtol=1e-6)
        np.testing.assert_allclose(d["mc_tau"][r], log_softmax(y)[ids], rtol=1e-6)
        u = synth.uniforms(SMALL.seed, 5, r, SMALL.M)
        cum = np.cumsum(np.exp(lb))
        expect = np.searchsorted(cum, u * cum[-1], side="right")
        np.testing.assert_array_equal(ids, expect)


def test_mc_samples_follow_behaviour_distribution():
    w = SMALL.replace(V=4, N=1, M=20_000, k=0, dense_teacher=False, sigma_student=1.0)
    d = synth.generate(w)
    p = np.exp(log_softmax(synth.behaviour_row(w, 0)))
    freq = np.bincount(d["mc_ids"][0], minlength=4) / w.M
    np.testing.assert_allclose(freq, p, atol=5 * np.sqrt(p * (1 - p) / w.M).max())


def test_ragged_mask():
    w = synth.MC1_RAGGED
    m = synth.mask(w).reshape(-1, w.rollout_len)
    lengths = m.sum(1)
    assert lengths.min() >= w.len_lo and lengths.max() <= w.len_hi
    for r in range(m.shape[0]):
        assert m[r, : lengths[r]].all() and not m[r, lengths[r]:].any()
    assert synth.mask(synth.MC16).all()
