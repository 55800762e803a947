"""GPU parity of the cache-building entry points (Sec. 4.1, Stages 1 and 2)
against the oracle, through the C ABI.

Draws (opd_sample_actions) must equal the oracle's, id for id.  Both
evaluate the index-order CDF in double precision (the device with a
table-driven exp and chunked sums, the oracle with libm's exp and a long double
running sum); they can disagree only where a uniform lies within about 1e-14
of a cumulative value, an event of probability about 2 V 1e-14 per draw
(3e-9 at V = 151,936), so no mismatch is admitted.  A mismatch is reported
with the uniform's distance to the drawn id's interval.
Top-k ids (opd_topk_support) are compared bit for bit.  Log-probabilities
and log-partitions: |gpu - ref| <= 1e-5 * (1 + |lse|) (fp32 evaluation of
L = m + log S, |L| up to ~40 here).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_24143_amd as opd
import synth
from gpu_common import DEV, say, to_dev

pytestmark = pytest.mark.gpu

LP_TOL = 1e-5

# (V, ld, dtype); the paths noted are those of the top-k kernel (scoring always
# streams; draws stream in 64-element chunks up to V = 262,144, and take the
# resident or chunked kernel beyond)
SHAPES = [
    (1000, 1000, synth.BF16),      # narrow resident row
    (3001, 3008, synth.BF16),      # V not a multiple of 4, padded stride
    (7, 8, synth.F32),             # a single partial vector
    (32000, 32000, synth.F32),     # fp32 resident
    (151936, 151936, synth.BF16),  # bf16 resident, 38 slots
    (151936, 151936, synth.F32),   # fp32 streamed (wider than the registers)
    (200000, 200000, synth.BF16),  # streamed
    (300000, 300000, synth.BF16),  # streamed; draws in two-vector CDF chunks
]
SHAPE_IDS = ["v%d_ld%d_%s" % (v, ld, "bf16" if dt == synth.BF16 else "f32") for v, ld, dt in SHAPES]


def make_logits(V, ld, dtype, N, seed=1):
    w = synth.MC16.replace(N=N, V=V, dtype=dtype, seed=seed, M=0, k=0)
    d = synth.generate(w, ld=ld)
    return d["logits"]


def as_device(stored: np.ndarray, V: int) -> torch.Tensor:
    t = to_dev(stored)
    return t[:, :V]


def f32_uniforms(seed, rows, M):
    """Uniforms on the float32 grid k / 2^24 (exact in float32, below 1)."""
    u = np.stack([synth.uniforms(seed, synth.STREAM_SAMPLE, r, M) for r in range(rows)])
    return (np.floor(u * 2.0 ** 24) / 2.0 ** 24).astype(np.float32)


def widen(stored: np.ndarray, dtype) -> np.ndarray:
    if dtype == synth.BF16:
        return synth.bf16_bits_to_f32(stored).astype(np.float64)
    return stored.astype(np.float64)


def check_draws(name, ids, logp, stored, V, dtype, u, ref):
    """GPU draws against the oracle's, id for id."""
    ids = np.asarray(ids)
    same = ids == ref["ids"]
    if not same.all():
        r, i = [int(x[0]) for x in np.nonzero(~same)]
        z = widen(stored[r, :V], dtype)
        F = oracle.cdf(z)
        j = int(ids[r, i])
        lo = F[j - 1] if 0 < j < V else 0.0
        hi = F[j] if 0 <= j < V else float("nan")
        raise AssertionError(
            "%s: %d of %d draws differ; first: row %d draw %d u=%r gpu id %d (interval [%r, %r], "
            "distance %.3g) oracle id %d" %
            (name, int((~same).sum()), same.size, r, i, u[r, i], j, lo, hi,
             min(abs(u[r, i] - lo), abs(u[r, i] - hi)), ref["ids"][r, i]))
    # log-probabilities at the GPU's ids
    z_at = np.take_along_axis(widen(stored[:, :V], dtype), ids.clip(0, V - 1).astype(np.int64), 1)
    want = z_at - ref["lse"][:, None]
    tol = LP_TOL * (1.0 + np.abs(ref["lse"]))[:, None]
    err = np.abs(np.asarray(logp, np.float64) - want)
    assert np.all(err <= tol), "%s: logp error %.3g" % (name, err.max())


@pytest.mark.parametrize("shape", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("M", [1, 16, 256])
def test_sample_parity(shape, M):
    V, ld, dtype = shape
    N = 6
    say("sample %s M=%d" % (shape, M))
    stored = make_logits(V, ld, dtype, N)
    u = f32_uniforms(7 + M, N, M)
    out = opd.sample_actions(as_device(stored, V), to_dev(u), want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("sample", dtype, stored, V, M, uniforms=u)
    check_draws("sample", out["ids"].cpu().numpy(), out["logp"].cpu().numpy(), stored, V, dtype,
                u, ref)
    lse = out["lse"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(lse - ref["lse"]) <= LP_TOL * (1 + np.abs(ref["lse"])))


def test_sample_wide_rows():
    # rows above 1,048,576 entries: more than one 128-vector step per chunk
    V, N, M = 1_200_000, 3, 64
    say("sample wide V=%d" % V)
    stored = make_logits(V, V, synth.BF16, N, seed=4)
    u = f32_uniforms(21, N, M)
    out = opd.sample_actions(as_device(stored, V), to_dev(u), want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("sample", synth.BF16, stored, V, M, uniforms=u)
    check_draws("wide", out["ids"].cpu().numpy(), out["logp"].cpu().numpy(), stored, V,
                synth.BF16, u, ref)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_sample_extreme_logit_ranges(dtype):
    """The double-precision terms across logit ranges: a large positive and a
    large negative row maximum, a row whose terms run through double's
    underflow range and below it (z - m down to -800), logits near zero, and
    a wide spread."""
    rng = np.random.default_rng(31)
    V, N, M = 20000, 5, 64
    x = rng.normal(0.0, 3.0, (N, V))
    x[0] += 5000.0
    x[1] -= 5000.0
    x[2] = -np.linspace(0.0, 800.0, V) + rng.normal(0.0, 0.5, V)
    x[3] *= 1e-7
    x[4] = rng.normal(0.0, 30.0, V)
    stored = to_stored(x.astype(np.float32), dtype)
    say("sample extreme ranges dtype=%d" % dtype)
    u = f32_uniforms(41, N, M)
    out = opd.sample_actions(as_device(stored, V), to_dev(u), want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("sample", dtype, stored, V, M, uniforms=u)
    check_draws("extreme", out["ids"].cpu().numpy(), out["logp"].cpu().numpy(), stored, V, dtype,
                u, ref)
    lse = out["lse"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(lse - ref["lse"]) <= LP_TOL * (1 + np.abs(ref["lse"])))


def test_sample_masked_rows_and_determinism():
    V, N, M = 4096, 8, 16
    stored = make_logits(V, V, synth.BF16, N)
    u = f32_uniforms(3, N, M)
    mask = np.array([1, 0, 1, 1, 0, 0, 1, 1], np.uint8)
    x = as_device(stored, V)
    a = opd.sample_actions(x, to_dev(u), mask=to_dev(mask), want_lse=True)
    b = opd.sample_actions(x, to_dev(u), mask=to_dev(mask), want_lse=True)
    torch.cuda.synchronize()
    for key in ("ids", "logp", "lse"):
        assert torch.equal(a[key], b[key]), key
    ids, logp, lse = (a[k].cpu().numpy() for k in ("ids", "logp", "lse"))
    assert np.all(ids[mask == 0] == 0) and np.all(logp[mask == 0] == 0) and np.all(lse[mask == 0] == 0)
    ref = oracle.cache_rows("sample", synth.BF16, stored, V, M, uniforms=u, mask=mask)
    keep = mask == 1
    check_draws("masked", ids[keep], logp[keep], stored[keep], V, synth.BF16, u[keep],
                {k: v[keep] for k, v in ref.items()})


def test_sample_zero_probability_ids_are_never_drawn():
    # most entries -inf (probability 0); uniforms everywhere in [0, 1),
    # including 0 and the largest float32 below 1
    V, N, M = 9000, 4, 256
    rng = np.random.default_rng(5)
    x = np.full((N, V), -np.inf, np.float32)
    for r in range(N):
        live = rng.choice(V, 40, replace=False)
        x[r, live] = rng.normal(0, 2, 40)
    u = f32_uniforms(11, N, M)
    u[:, 0] = 0.0
    u[:, 1] = np.nextafter(np.float32(1), np.float32(0))
    out = opd.sample_actions(to_dev(x), to_dev(u))
    torch.cuda.synchronize()
    ids = out["ids"].cpu().numpy()
    assert np.all(np.isfinite(np.take_along_axis(x, ids.astype(np.int64), 1)))
    ref = oracle.cache_rows("sample", synth.F32, x, V, M, uniforms=u)
    check_draws("sparse", ids, out["logp"].cpu().numpy(), x, V, synth.F32, u, ref)


def test_sample_bad_uniforms_and_undefined_rows():
    V = 64
    x = np.zeros((4, V), np.float32)
    x[1, 5] = np.nan
    x[2, 7] = np.inf
    x[3, :] = -np.inf
    u = np.tile(np.array([0.51, -0.25, 1.0, np.nan], np.float32), (4, 1))
    out = opd.sample_actions(to_dev(x), to_dev(u))
    torch.cuda.synchronize()
    ids, logp = out["ids"].cpu().numpy(), out["logp"].cpu().numpy()
    assert ids[0, 0] == 32 and abs(logp[0, 0] - np.log(1 / 64)) < 1e-5
    assert np.all(ids[0, 1:] == -1) and np.all(np.isnan(logp[0, 1:]))
    assert np.all(ids[1:] == -1) and np.all(np.isnan(logp[1:]))


def test_sample_stratified_uniforms_reproduce_the_distribution():
    # u_i = (i + 1/2) / n: each id receives n p_j draws up to 1 (exact CDF)
    V, n = 48, 1 << 16
    rng = np.random.default_rng(2)
    x = rng.normal(0, 1.5, (1, V)).astype(np.float32)
    per = 256
    u = ((np.arange(n) + 0.5) / n).astype(np.float32).reshape(-1, per)
    rows = u.shape[0]
    out = opd.sample_actions(to_dev(np.repeat(x, rows, 0)), to_dev(u))
    torch.cuda.synchronize()
    counts = np.bincount(out["ids"].cpu().numpy().ravel(), minlength=V)
    p = np.exp(x[0].astype(np.float64) - np.logaddexp.reduce(x[0].astype(np.float64)))
    assert np.all(np.abs(counts - n * p) <= 1)


@pytest.mark.slow
def test_sample_full_size_mc16():
    w = synth.MC16
    say("sample full size %s" % w.name)
    d = synth.generate(w)
    stored, V, M = d["logits"], w.V, w.M
    u = f32_uniforms(w.seed + 1, w.N, M)
    out = opd.sample_actions(as_device(stored, V), to_dev(u), want_lse=True)
    torch.cuda.synchronize()
    ids, logp = out["ids"].cpu().numpy(), out["logp"].cpu().numpy()
    assert ids.min() >= 0 and ids.max() < V and np.all(logp <= 1e-6) and np.all(np.isfinite(logp))
    # every draw of every row
    ref = oracle.cache_rows("sample", w.dtype, stored, V, M, uniforms=u)
    check_draws("full", ids, logp, stored, V, w.dtype, u, ref)


# ---------------------------------------------------------------- top-k

def check_topk(name, out, stored, V, k, dtype, ref):
    idx = out["idx"].cpu().numpy()
    bad = np.argwhere(idx != ref["ids"])
    assert bad.size == 0, "%s: first mismatch at %s: gpu %d oracle %d" % (
        name, bad[0], idx[tuple(bad[0])], ref["ids"][tuple(bad[0])])
    if "logp" in out:
        lp = out["logp"].cpu().numpy().astype(np.float64)
        tol = LP_TOL * (1.0 + np.abs(ref["lse"]))[:, None]
        fin = np.isfinite(ref["logp"])
        assert np.all(np.abs(lp - ref["logp"])[fin] <= np.broadcast_to(tol, lp.shape)[fin])


@pytest.mark.parametrize("shape", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("k", [1, 7, 32, 256])
def test_topk_parity(shape, k):
    V, ld, dtype = shape
    k = min(k, V)
    N = 6
    say("topk %s k=%d" % (shape, k))
    stored = make_logits(V, ld, dtype, N, seed=3)
    out = opd.topk_support(as_device(stored, V), k, want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("topk", dtype, stored, V, k)
    check_topk("topk", out, stored, V, k, dtype, ref)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("case", ["constant", "ties_2000", "ties_5000", "special", "k_eq_v"])
def test_topk_ties_and_special_values(dtype, case):
    # many equal maxima exercise the LDS sort (over 1024 candidates) and the
    # exact counting path (over 4096 candidates)
    rng = np.random.default_rng(17)
    V, N, k = 12000, 3, 256
    x = rng.normal(0, 1, (N, V)).astype(np.float32)
    if case == "constant":
        x[:] = 0.75
    elif case.startswith("ties_"):
        n = int(case[5:])
        for r in range(N):
            x[r, rng.choice(V, n, replace=False)] = 9.5
    elif case == "special":
        x[:, 10] = np.inf
        x[:, 20] = np.nan
        x[:, 30] = -0.0
        x[:, 31] = 0.0
        x[:, 40:100] = -np.inf
        x[1, :] = np.where(x[1] > 0, -0.0, 0.0)  # only signed zeros
    elif case == "k_eq_v":
        V, k = 200, 200
        x = x[:, :V].copy()
    if dtype == synth.BF16:
        b = x.view(np.uint32).astype(np.uint64)
        stored = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
        nan = np.isnan(x)
        stored[nan] = 0x7FC0
        ld = V
    else:
        stored, ld = x, V
    out = opd.topk_support(as_device(np.ascontiguousarray(stored), V), k, want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("topk", dtype, np.ascontiguousarray(stored), V, k)
    check_topk(case, out, stored, V, k, dtype, ref)


def to_stored(x, dtype):
    """float32 rows as stored logits (bf16 by round-to-nearest-even, NaN kept)."""
    if dtype != synth.BF16:
        return np.ascontiguousarray(x)
    b = x.view(np.uint32).astype(np.uint64)
    stored = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    stored[np.isnan(x)] = 0x7FC0
    return np.ascontiguousarray(stored)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("k", [16, 64])
@pytest.mark.parametrize("case", ["constant", "ties_100", "ties_300", "special", "ascending",
                                  "descending"])
def test_topk_streamed_ties_and_special_values(dtype, k, case):
    # rows wide enough for the streamed kernel (k <= 64): constant rows and
    # 300 equal maxima leave it too many candidates (the resident kernel
    # redoes those rows); 100 equal maxima are sorted in the streamed kernel
    rng = np.random.default_rng(23)
    V, N = 40000, 3
    x = rng.normal(0, 1, (N, V)).astype(np.float32)
    if case == "constant":
        x[:] = -1.25
    elif case.startswith("ties_"):
        n = int(case[5:])
        for r in range(N):
            x[r, rng.choice(V, n, replace=False)] = 9.5
    elif case == "special":
        x[:, 10] = np.inf
        x[:, 20] = np.nan
        x[:, 30] = -0.0
        x[:, 31] = 0.0
        x[:, 40:100] = -np.inf
        x[1, :] = np.where(x[1] > 0, -0.0, 0.0)  # only signed zeros
        x[2, 5000:6000] = np.nan
    elif case == "ascending":
        x = np.sort(x, axis=1)
    elif case == "descending":
        x = np.sort(x, axis=1)[:, ::-1].copy()
    stored = to_stored(x, dtype)
    say("topk streamed %s k=%d dtype=%d" % (case, k, dtype))
    out = opd.topk_support(as_device(stored, V), k, want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("topk", dtype, stored, V, k)
    check_topk(case, out, stored, V, k, dtype, ref)


@pytest.mark.parametrize("k", [16, 64])
@pytest.mark.parametrize("where", ["one_wave", "one_lane", "few_finite"])
def test_topk_streamed_concentrated_maxima(k, where):
    """The streamed kernel's bound is the smallest of the four waves'
    published values.  Rows whose largest values all lie in one wave's tiles
    (wave w reads tiles of 512 vectors numbered w mod 4; the other waves'
    bounds stay low), in one lane's elements (its slots overflow and the
    resident kernel redoes the row), or that hold only a few finite values
    among -inf (a lane that sees no finite value sends the row to the
    resident kernel when the log-partition is wanted)."""
    rng = np.random.default_rng(37)
    V, N = 65536, 3  # 16,384 vectors: 32 tiles, 8 per wave
    x = rng.normal(0.0, 1.0, (N, V)).astype(np.float32)
    vec = np.arange(V // 4)
    tile, lane = vec // 512, vec % 64
    if where == "one_wave":
        pos = np.flatnonzero(np.repeat(tile % 4 == 1, 4))
        for r in range(N):
            x[r, rng.choice(pos, 3 * k, replace=False)] = 6.0 + rng.random(3 * k)
    elif where == "one_lane":
        pos = np.flatnonzero(np.repeat((tile % 4 == 2) & (lane == 5), 4))
        for r in range(N):
            x[r, pos] = 6.0 + rng.random(pos.size)
    else:
        x[:] = -np.inf
        for r in range(N):
            x[r, rng.choice(V, k + 5, replace=False)] = rng.normal(0.0, 1.0, k + 5)
    stored = to_stored(x, synth.BF16)
    say("topk streamed concentrated %s k=%d" % (where, k))
    ref = oracle.cache_rows("topk", synth.BF16, stored, V, k)
    out = opd.topk_support(as_device(stored, V), k, want_lse=True)
    torch.cuda.synchronize()
    check_topk(where, out, stored, V, k, synth.BF16, ref)
    # without log-probs or the log-partition (the kernel variant without
    # the exponentials)
    out = opd.topk_support(as_device(stored, V), k, want_logp=False)
    torch.cuda.synchronize()
    check_topk(where + " ids only", out, stored, V, k, synth.BF16, ref)


def test_topk_streamed_masked_rows_and_no_logp():
    V, N, k = 20000, 6, 16
    stored = make_logits(V, V, synth.BF16, N, seed=9)
    mask = np.array([0, 1, 1, 0, 1, 1], np.uint8)
    out = opd.topk_support(as_device(stored, V), k, mask=to_dev(mask), want_logp=False)
    torch.cuda.synchronize()
    idx = out["idx"].cpu().numpy()
    assert np.all(idx[mask == 0] == 0)
    ref = oracle.cache_rows("topk", synth.BF16, stored, V, k, mask=mask)
    assert np.array_equal(idx, ref["ids"])


def test_topk_masked_rows_and_no_logp():
    V, N, k = 5000, 6, 16
    stored = make_logits(V, V, synth.BF16, N, seed=9)
    mask = np.array([0, 1, 1, 0, 1, 1], np.uint8)
    out = opd.topk_support(as_device(stored, V), k, mask=to_dev(mask), want_logp=False)
    torch.cuda.synchronize()
    idx = out["idx"].cpu().numpy()
    assert np.all(idx[mask == 0] == 0)
    ref = oracle.cache_rows("topk", synth.BF16, stored, V, k, mask=mask)
    assert np.array_equal(idx, ref["ids"])


@pytest.mark.slow
def test_topk_full_size():
    w = synth.TOPK32
    say("topk full size %s" % w.name)
    d = synth.generate(w)
    stored, V, k = d["logits"], w.V, w.k
    x = as_device(stored, V)
    out = opd.topk_support(x, k, want_lse=True)
    torch.cuda.synchronize()
    idx = out["idx"].long()
    # every row: the selected values are the k largest (torch.topk values)
    vals = torch.gather(x.float(), 1, idx)
    assert torch.equal(vals, torch.topk(x.float(), k, dim=1).values)
    rows = np.linspace(0, w.N - 1, 96).astype(np.int64)
    ref = oracle.cache_rows("topk", w.dtype, stored[rows], V, k)
    sub = {"idx": out["idx"][rows], "logp": out["logp"][rows]}
    check_topk("full", sub, stored[rows], V, k, w.dtype, ref)


# ---------------------------------------------------------------- scoring

@pytest.mark.parametrize("shape", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("K", [1, 16, 256])
def test_score_parity(shape, K):
    V, ld, dtype = shape
    N = 5
    stored = make_logits(V, ld, dtype, N, seed=4)
    rng = np.random.default_rng(V + K)
    ids = rng.integers(0, V, (N, K)).astype(np.int32)
    ids[:, 0] = ids[:, -1]  # a repeat
    if K > 2:
        ids[1, 1] = -3       # out of range below
        ids[2, 2] = V        # and above
    out = opd.score_actions(as_device(stored, V), to_dev(ids), want_lse=True)
    torch.cuda.synchronize()
    ref = oracle.cache_rows("score", dtype, stored, V, K, ids=ids)
    lp = out["logp"].cpu().numpy().astype(np.float64)
    nan_ref = np.isnan(ref["logp"])
    assert np.array_equal(np.isnan(lp), nan_ref)
    tol = LP_TOL * (1.0 + np.abs(ref["lse"]))[:, None]
    assert np.all(np.abs(lp - ref["logp"])[~nan_ref] <= np.broadcast_to(tol, lp.shape)[~nan_ref])
    lse = out["lse"].cpu().numpy()
    assert np.all(np.abs(lse - ref["lse"]) <= LP_TOL * (1 + np.abs(ref["lse"])))


def test_score_masked_rows():
    V, N, K = 3000, 4, 8
    stored = make_logits(V, V, synth.F32, N, seed=6)
    ids = np.tile(np.arange(K, dtype=np.int32), (N, 1))
    mask = np.array([1, 0, 0, 1], np.uint8)
    out = opd.score_actions(as_device(stored, V), to_dev(ids), mask=to_dev(mask), want_lse=True)
    torch.cuda.synchronize()
    lp = out["logp"].cpu().numpy()
    assert np.all(lp[mask == 0] == 0) and np.all(out["lse"].cpu().numpy()[mask == 0] == 0)
    ref = oracle.cache_rows("score", synth.F32, stored, V, K, ids=ids, mask=mask)
    assert np.all(np.abs(lp - ref["logp"]) <= LP_TOL * (1 + np.abs(ref["lse"]))[:, None])


@pytest.mark.slow
def test_score_full_size_matches_generator_cache():
    # the generator's MC cache stores the teacher log-probs of its draws in
    # double (rounded to fp32); scoring the teacher rows at those ids must
    # reproduce them
    w = synth.MC16.replace(N=4096, dense_teacher=True)
    say("score full size %s N=%d" % (w.name, w.N))
    d = synth.generate(w)
    out = opd.score_actions(as_device(d["teacher_logits"], w.V), to_dev(d["mc_ids"]), want_lse=True)
    torch.cuda.synchronize()
    lp = out["logp"].cpu().numpy().astype(np.float64)
    lse = out["lse"].cpu().numpy().astype(np.float64)
    tol = LP_TOL * (1 + np.abs(lse))[:, None] + 1e-6 * np.abs(d["mc_tau"])
    assert np.all(np.abs(lp - d["mc_tau"]) <= tol)
