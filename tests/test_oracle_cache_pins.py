"""Pins of the oracle's cache-building functions (Sec. 4.1, Stages 1 and 2):
inverse-CDF draws from softmax(z), the top-k support, and scoring of cached
actions.

Each is checked against something other than itself: closed-form CDFs of
hand-built distributions, an exact count identity for a stratified grid of
uniforms, numpy's searchsorted / lexsort / scipy's log_softmax as independent
routines, and the special cases the definitions fix (zero-probability
actions never drawn, ties by lower index, undefined rows).
"""
import numpy as np
import pytest
from scipy.special import log_softmax

import oracle
import synth


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest even) and return the bit patterns."""
    b = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    return r


# ---------------------------------------------------------------- sampling

def test_sample_closed_form_cdf():
    # p = (0.1, 0.2, 0.3, 0.4): F = (0.1, 0.3, 0.6, 1.0)
    z = np.log([1.0, 2.0, 3.0, 4.0]) + 7.25
    u = np.array([0.0, 0.05, 0.0999, 0.1001, 0.2999, 0.3001, 0.5999, 0.6001, 0.9999], np.float32)
    ids, logp, lse = oracle.sample_row(z, u)
    assert ids.tolist() == [0, 0, 0, 1, 1, 2, 2, 3, 3]
    np.testing.assert_allclose(logp, np.log([0.1, 0.1, 0.1, 0.2, 0.2, 0.3, 0.3, 0.4, 0.4]),
                               rtol=0, atol=1e-13)
    assert abs(lse - (np.log(10.0) + 7.25)) < 1e-13


def test_sample_never_draws_zero_probability():
    # p = (0, 0.25, 0, 0.75, 0): the -inf entries must never be drawn, even at
    # u = 0 and at the largest float32 below 1.
    z = np.array([-np.inf, 0.0, -np.inf, np.log(3.0), -np.inf])
    u = np.array([0.0, 0.2499, 0.2501, 0.5, np.nextafter(np.float32(1), np.float32(0))],
                 np.float32)
    ids, logp, _ = oracle.sample_row(z, u)
    assert ids.tolist() == [1, 1, 3, 3, 3]
    np.testing.assert_allclose(logp, np.log([0.25, 0.25, 0.75, 0.75, 0.75]), atol=1e-13)


def test_sample_matches_searchsorted():
    rng = np.random.default_rng(3)
    for V in (2, 17, 1000, 32000):
        z = rng.normal(0.0, 3.0, V)
        u = rng.random(4096).astype(np.float32)
        ids, logp, lse = oracle.sample_row(z, u)
        F = np.cumsum(np.exp(log_softmax(z)))
        ref = np.searchsorted(F, u.astype(np.float64), side="right")
        # searchsorted and the oracle sum F in different orders; they may only
        # differ where u lies within rounding of a CDF boundary
        diff = ids != ref
        if diff.any():
            Fo = oracle.cdf(z)
            for i in np.flatnonzero(diff):
                assert min(abs(Fo[ref[i]] - u[i]), abs(Fo[ids[i]] - u[i])) < 1e-12
        assert diff.mean() < 1e-3
        np.testing.assert_allclose(logp, log_softmax(z)[ids], atol=1e-12)
        assert abs(lse - np.logaddexp.reduce(z)) < 1e-10


def test_sample_stratified_counts_are_exact():
    # A stratified grid u_i = (i + 1/2) / n puts exactly floor/ceil(n p_j)
    # points in each interval [F_{j-1}, F_j): |count_j - n p_j| <= 1.
    rng = np.random.default_rng(11)
    z = rng.normal(0.0, 1.5, 12)
    n = 1 << 17
    u = ((np.arange(n) + 0.5) / n).astype(np.float32)  # exact in float32
    ids, _, _ = oracle.sample_row(z, u)
    counts = np.bincount(ids, minlength=z.size)
    p = np.exp(log_softmax(z))
    assert np.all(np.abs(counts - n * p) <= 1.0 + 1e-9)


def test_sample_cdf_ends_above_every_float32_uniform():
    # In double the last cumulative value is within V * 2^-53 of 1, so it
    # exceeds the largest float32 below 1: the "no value exceeds u" fallback
    # of the definition is a guard for coarser arithmetic and is not reached
    # here (which is why it has no pin of its own).
    u_max = float(np.nextafter(np.float32(1), np.float32(0)))
    rng = np.random.default_rng(9)
    for V in (3, 1000, 151936):
        for scale in (0.1, 3.0, 30.0):
            F = oracle.cdf(rng.normal(0.0, scale, V))
            assert F[-1] > u_max and abs(F[-1] - 1.0) < V * 2.0 ** -50


def test_sample_is_monotone_in_u():
    rng = np.random.default_rng(5)
    z = rng.normal(0.0, 3.0, 5000)
    u = np.sort(rng.random(2000).astype(np.float32))
    ids, _, _ = oracle.sample_row(z, u)
    assert np.all(np.diff(ids) >= 0)


@pytest.mark.parametrize("bad", [-0.25, 1.0, 1.5, np.nan])
def test_sample_rejects_uniforms_outside_unit_interval(bad):
    ids, logp, _ = oracle.sample_row(np.zeros(8), np.array([0.55, bad], np.float32))
    assert ids[0] == 4 and ids[1] == -1 and np.isnan(logp[1])


@pytest.mark.parametrize("z", [np.array([0.0, np.nan, 1.0]), np.array([0.0, np.inf, 1.0]),
                               np.array([-np.inf, -np.inf, -np.inf])])
def test_sample_undefined_rows(z):
    ids, logp, _ = oracle.sample_row(z, np.array([0.0, 0.5], np.float32))
    assert ids.tolist() == [-1, -1] and np.all(np.isnan(logp))


def test_sample_agrees_with_generator_draws():
    # The generator draws its MC cache by inversion of softmax(b) with its own
    # double-precision code and uniforms; the oracle, given the same b and the
    # same uniforms, must draw the same ids (both are exact up to rounding at
    # boundaries, which these uniforms do not approach).
    w = synth.MC16.replace(N=3, V=4000)
    d = synth.generate(w)
    for r in range(w.N):
        b = synth.behaviour_row(w, r)
        u = synth.uniforms(w.seed, synth.STREAM_SAMPLE, r, w.M)
        ids, logp, _ = oracle.sample_row(b, u.astype(np.float32))
        F = oracle.cdf(b)
        checked = 0
        for i in range(w.M):
            # float32 rounding moves u by < 3e-8: the interval is kept when u
            # is farther than that from every boundary
            if np.min(np.abs(F - u[i])) > 1e-7:
                assert ids[i] == d["mc_ids"][r, i]
                assert abs(logp[i] - d["mc_beta"][r, i]) < 1e-5
                checked += 1
        assert checked >= w.M - 1


def test_sample_batch_driver_matches_rows():
    rng = np.random.default_rng(2)
    n, V, ld, M = 5, 300, 304, 7
    x = rng.normal(0, 2, (n, ld)).astype(np.float32)
    bits = _bf16_bits(x)
    u = rng.random((n, M)).astype(np.float32)
    mask = np.array([1, 0, 1, 1, 0], np.uint8)
    for dtype, stored in ((oracle.F32, x), (oracle.BF16, bits)):
        out = oracle.cache_rows("sample", dtype, stored, V, M, uniforms=u, mask=mask, nthreads=2)
        for r in range(n):
            if not mask[r]:
                assert np.all(out["ids"][r] == 0) and np.all(out["logp"][r] == 0)
                assert out["lse"][r] == 0
                continue
            z = (x[r, :V] if dtype == oracle.F32 else
                 (bits[r, :V].astype(np.uint32) << 16).view(np.float32)).astype(np.float64)
            ids, logp, lse = oracle.sample_row(z, u[r])
            assert np.array_equal(out["ids"][r], ids)
            assert np.array_equal(out["logp"][r], logp) and out["lse"][r] == lse


# ---------------------------------------------------------------- top-k support

def _lexsort_topk(values: np.ndarray, k: int) -> np.ndarray:
    order = np.lexsort((np.arange(values.size), -values.astype(np.float64)))
    return order[:k]


@pytest.mark.parametrize("V,k", [(10, 1), (10, 10), (1000, 16), (32000, 32), (151936, 256)])
def test_topk_matches_lexsort_float32(V, k):
    rng = np.random.default_rng(V + k)
    x = rng.normal(0, 3, V).astype(np.float32)
    x[rng.integers(0, V, V // 10)] = x[0]  # plant ties
    idx, logp, lse = oracle.topk_row(x, k)
    assert np.array_equal(idx, _lexsort_topk(x, k))
    np.testing.assert_allclose(logp, log_softmax(x.astype(np.float64))[idx], atol=1e-10)
    assert abs(lse - np.logaddexp.reduce(x.astype(np.float64))) < 1e-9


@pytest.mark.parametrize("k", [1, 32, 256])
def test_topk_matches_lexsort_bf16(k):
    # bf16 keeps 8 significant bits, so a 151,936-wide row has many ties.
    rng = np.random.default_rng(k)
    bits = _bf16_bits(rng.normal(0, 3, 151936).astype(np.float32))
    vals = (bits.astype(np.uint32) << 16).view(np.float32)
    idx, logp, _ = oracle.topk_row(bits, k, oracle.BF16)
    assert np.array_equal(idx, _lexsort_topk(vals, k))
    assert len(set(vals[idx].tolist())) < k or k == 1  # ties were exercised
    np.testing.assert_allclose(logp, log_softmax(vals.astype(np.float64))[idx], atol=1e-10)


def test_topk_constant_row_takes_lowest_indices():
    idx, _, _ = oracle.topk_row(np.full(500, 1.25, np.float32), 37)
    assert idx.tolist() == list(range(37))


def test_topk_special_values():
    nan_neg = np.array([0xFFC00000], np.uint32).view(np.float32)[0]
    x = np.array([-0.0, 0.0, -np.inf, np.inf, np.nan, 5.0, nan_neg, -3.0], np.float32)
    idx, _, _ = oracle.topk_row(x, 8)
    # +NaN above +inf; -0 ties +0 (lower index first); -NaN below -inf
    assert idx.tolist() == [4, 3, 5, 0, 1, 7, 2, 6]


def test_topk_batch_driver_matches_rows():
    rng = np.random.default_rng(8)
    n, V, ld, k = 4, 777, 784, 9
    x = rng.normal(0, 2, (n, ld)).astype(np.float32)
    mask = np.array([1, 1, 0, 1], np.uint8)
    out = oracle.cache_rows("topk", oracle.F32, x, V, k, mask=mask, nthreads=3)
    for r in range(n):
        if not mask[r]:
            assert np.all(out["ids"][r] == 0)
            continue
        idx, logp, lse = oracle.topk_row(x[r, :V], k)
        assert np.array_equal(out["ids"][r], idx) and np.array_equal(out["logp"][r], logp)


# ---------------------------------------------------------------- scoring

def test_score_matches_log_softmax():
    rng = np.random.default_rng(4)
    z = rng.normal(0, 3, 151936)
    ids = rng.integers(0, z.size, 256).astype(np.int32)
    ids[:4] = ids[4]  # repeats are scored independently
    logp, lse = oracle.score_row(z, ids)
    np.testing.assert_allclose(logp, log_softmax(z)[ids], atol=1e-10)
    assert abs(lse - np.logaddexp.reduce(z)) < 1e-9


def test_score_out_of_range_ids_are_nan():
    logp, _ = oracle.score_row(np.zeros(10), np.array([-1, 0, 10, 9], np.int32))
    assert np.isnan(logp[0]) and np.isnan(logp[2])
    np.testing.assert_allclose(logp[[1, 3]], np.log(0.1), atol=1e-14)


def test_score_batch_driver_keeps_ids_and_masks():
    rng = np.random.default_rng(6)
    n, V, K = 3, 64, 5
    x = rng.normal(0, 1, (n, V)).astype(np.float32)
    ids = rng.integers(0, V, (n, K)).astype(np.int32)
    mask = np.array([1, 0, 1], np.uint8)
    out = oracle.cache_rows("score", oracle.F32, x, V, K, ids=ids, mask=mask)
    assert np.array_equal(out["ids"], ids)
    for r in (0, 2):
        np.testing.assert_allclose(out["logp"][r], log_softmax(x[r].astype(np.float64))[ids[r]],
                                   atol=1e-12)
    assert np.all(out["logp"][1] == 0) and out["lse"][1] == 0


def test_cache_driver_rejects_bad_arguments():
    x = np.zeros((2, 8), np.float32)
    with pytest.raises(ValueError):
        oracle.cache_rows("sample", oracle.F32, x, 8, 2)  # no uniforms
    with pytest.raises(ValueError):
        oracle.cache_rows("topk", oracle.F32, x, 8, 9)  # k > V
    with pytest.raises(ValueError):
        oracle.cache_rows("topk", oracle.F32, x, 9, 2)  # ld < V
