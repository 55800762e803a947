"""GPU parity: the HIP path through the C ABI against the oracle, element by
element, on the same seeded inputs.

Small shapes cover every estimator, both input dtypes, both gradient dtypes,
every kernel path (register-resident rows, streaming rows, split
vocabulary), ragged tails (V not a multiple of the vector width), padded row
strides, masks, and the degenerate cases.  Full-size workloads run in the
configuration the benchmark times and compare every row's loss,
log-partition, gathered logits and coverage, and every gradient element."""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2606_24143_amd as opd
import synth
from gpu_common import (DENSE, DEV, MC, SUPPORT, TOPK, TRUNC, cache_arrays, check_grad, check_loss,
                        dlogits_f64, grad_mag, loss_scale, oracle_dtype, rtol_for, run_gpu, say,
                        to_dev, widen_dev)

pytestmark = pytest.mark.gpu

ALL = TOPK + TRUNC + MC + DENSE
SHAPES = {  # name: (N, V, ld)
    "v1000": (37, 1000, 1000),
    "v3001_tail": (19, 3001, 3008),
    "v32000": (24, 32000, 32000),
    "v151936": (6, 151936, 151936),
    "v7_tail": (5, 7, 8),
    "v200000_wide": (3, 200000, 200000),
    # an odd number of 4-element vectors (a trailing 8-byte bf16 vector), padded
    "v1004_odd": (9, 1004, 1008),
    # fp32 rows on the large register-resident dense variant
    "v50000": (4, 50000, 50000),
    # the shortest bf16 row the large dense variant takes (one slot past its LDS part)
    "v81920": (3, 81920, 81920),
}
PATHS = {"rowwise": opd.FLAG_FORCE_ROWWISE, "split": opd.FLAG_FORCE_SPLITV}


@functools.lru_cache(maxsize=8)
def small_inputs(shape: str, dtype: int):
    N, V, ld = SHAPES[shape]
    w = synth.Workload("t_" + shape, N=N, V=V, dtype=dtype, estimators=ALL, k=min(16, V), M=6,
                       sigma_student=2.5, sigma_teacher=1.0, sigma_behaviour=0.5,
                       dense_teacher=True, seed=7 + V + 3 * dtype)
    d = synth.generate(w, ld=ld)
    mask = np.ones(N, np.uint8)
    mask[1::4] = 0
    return w, d, mask


def compare(name, w, d, est, out, ref, mask=None, bf16_out=False, gamma=1.0, logits=None,
            teacher=None):
    """Loss, every gradient element, lse and gathered logits against the
    oracle.  logits / teacher: the stored rows (default d's)."""
    ids, tau, beta = cache_arrays(d, est)
    logits = d["logits"] if logits is None else logits
    if est in DENSE and teacher is None:
        teacher = d["teacher_logits"]
    check_loss(name, out["loss"].cpu().numpy(), ref["loss"],
               loss_scale(est, ids, tau, beta, ref), rtol_for(w.dtype), mask)
    mag = grad_mag(est, widen_dev(logits, w.V), ref, ids, tau, beta,
                   widen_dev(teacher, w.V) if est in DENSE else None, gamma, mask)
    worst = check_grad(name, out["dlogits"], ref["grad"], mag, bf16_out=bf16_out)
    say("%s: dlogits max err/bound %.3g" % (name, worst))
    if "lse" in out:
        lse = out["lse"].cpu().numpy().astype(np.float64)
        valid = ref["lse"] != 0
        np.testing.assert_allclose(lse[valid], ref["lse"][valid], rtol=2e-6, atol=0,
                                   err_msg=name + " lse")
    if "gathered" in out:
        g = out["gathered"].cpu().numpy().astype(np.float64)
        assert np.array_equal(g, ref["gathered"]), name + ": gathered logits not bit-exact"


def oracle_for(w, d, est, mask, gamma=1.0, eps=0.2):
    ids, tau, beta = cache_arrays(d, est)
    return oracle.rows(est, oracle_dtype(w.dtype), d["logits"], w.V, ids=ids, tau=tau, beta=beta,
                       teacher_logits=d.get("teacher_logits") if est in DENSE else None,
                       mask=mask, gamma=gamma, eps=eps)


@pytest.mark.parametrize("path", list(PATHS))
@pytest.mark.parametrize("est", ALL)
@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", list(SHAPES))
def test_parity_small(shape, dtype, est, path):
    w, d, mask = small_inputs(shape, dtype)
    N, V, ld = SHAPES[shape]
    say("parity %s %s %s %s" % (shape, "bf16" if dtype else "f32", est, path))
    logits = to_dev(d["logits"])[:, :V]
    teacher = to_dev(d["teacher_logits"])[:, :V] if est in DENSE else None
    ids, tau, beta = cache_arrays(d, est)
    out = run_gpu(logits, est, ids, tau, beta, teacher, mask=mask, grad_scale=0.75,
                  flags=PATHS[path], want_lse=True, want_gathered=est not in DENSE)
    ref = oracle_for(w, d, est, mask, gamma=0.75)
    compare("%s/%s/%s" % (shape, est, path), w, d, est, out, ref, mask, gamma=0.75)


@pytest.mark.parametrize("gamma", [-0.5, 0.0, 3.0])
@pytest.mark.parametrize("est", ALL)
@pytest.mark.parametrize("shape", ["v3001_tail", "v151936"])
def test_grad_scale_sign_and_zero(shape, est, gamma):
    """The gradient scale enters some kernels through the exponent (log2|gamma|)
    and its sign through the operand order: negative and zero scales, on every
    path, against the oracle's gamma * dloss/dz."""
    w, d, mask = small_inputs(shape, synth.BF16)
    N, V, ld = SHAPES[shape]
    say("grad-scale %s %s gamma=%g" % (shape, est, gamma))
    logits = to_dev(d["logits"])[:, :V]
    teacher = to_dev(d["teacher_logits"])[:, :V] if est in DENSE else None
    ids, tau, beta = cache_arrays(d, est)
    ref = oracle_for(w, d, est, mask, gamma=gamma)
    for path, flags in PATHS.items():
        out = run_gpu(logits, est, ids, tau, beta, teacher, mask=mask, grad_scale=gamma,
                      flags=flags)
        compare("%s/%s/%s/gamma=%g" % (shape, est, path, gamma), w, d, est, out, ref, mask,
                gamma=gamma)
        if gamma == 0.0:
            assert not out["dlogits"].any(), "a zero gradient scale leaves dlogits zero"


@pytest.mark.parametrize("est", ALL)
@pytest.mark.parametrize("shape", ["v1000", "v3001_tail", "v151936"])
def test_parity_bf16_gradient_output(shape, est):
    w, d, mask = small_inputs(shape, synth.BF16)
    N, V, ld = SHAPES[shape]
    say("bf16-out %s %s" % (shape, est))
    logits = to_dev(d["logits"])[:, :V]
    teacher = to_dev(d["teacher_logits"])[:, :V] if est in DENSE else None
    ids, tau, beta = cache_arrays(d, est)
    for flags in PATHS.values():
        out = run_gpu(logits, est, ids, tau, beta, teacher, mask=mask, flags=flags,
                      dlogits_dtype=torch.bfloat16)
        assert out["dlogits"].dtype == torch.bfloat16
        compare("%s/%s/bf16out" % (shape, est), w, d, est, out, oracle_for(w, d, est, mask), mask,
                bf16_out=True)


@pytest.mark.parametrize("K", [1, 2, 63, 64, 65, 100, 256])
@pytest.mark.parametrize("est", ["fkl_topk", "rkl_topk", "rkl_topk_trunc", "rkl_mc"])
def test_support_sizes(est, K):
    """k and M from 1 to the maximum, across the 64-entry wavefront boundary."""
    V = 4096
    w = synth.Workload("t_k", N=9, V=V, dtype=synth.BF16, estimators=(est,), k=K, M=K,
                       sigma_student=2.0, sigma_behaviour=0.4, seed=100 + K)
    d = synth.generate(w)
    say("support %s K=%d" % (est, K))
    ids, tau, beta = cache_arrays(d, est)
    logits = to_dev(d["logits"])
    for flags in PATHS.values():
        out = run_gpu(logits, est, ids, tau, beta, flags=flags, want_lse=True, want_gathered=True)
        compare("%s/K=%d" % (est, K), w, d, est, out, oracle_for(w, d, est, None))
        if est in TOPK and K == 1:
            assert not out["loss"].any() and not out["dlogits"].any()


COV_RTOL = 3e-5  # fp32 sums of at most 256 exponentials whose arguments carry L's error


def check_coverage(name, got, ref, mask=None):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref)
    assert np.all(err <= COV_RTOL * np.abs(ref) + 1e-30), (
        "%s: support coverage off by %.3g relative" % (name, np.max(err / np.maximum(ref, 1e-30))))
    if mask is not None:
        assert not got[mask == 0].any()


@pytest.mark.parametrize("est", SUPPORT)
@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", ["v1000", "v3001_tail", "v151936", "v200000_wide"])
def test_support_coverage(shape, dtype, est):
    """Z_p^S and Z_q^S (App. A.1) against the oracle on every path; for the
    renormalised estimators without lse_out the request alone makes the call
    read the rows.  The loss and gradient stay what they are without it."""
    w, d, mask = small_inputs(shape, dtype)
    N, V, ld = SHAPES[shape]
    say("coverage %s %s %s" % (shape, "bf16" if dtype else "f32", est))
    logits = to_dev(d["logits"])[:, :V]
    ids, tau, _ = cache_arrays(d, est)
    ref = oracle.coverage_rows(oracle_dtype(dtype), d["logits"], V, ids, tau, mask=mask)
    for path, flags in PATHS.items():
        out = run_gpu(logits, est, ids, tau, None, mask=mask, flags=flags, want_coverage=True)
        check_coverage("%s/%s/%s" % (shape, est, path), out["coverage"].cpu().numpy(), ref, mask)
        base = run_gpu(logits, est, ids, tau, None, mask=mask, flags=flags)
        assert torch.equal(out["loss"], base["loss"])
        assert torch.equal(out["dlogits"], base["dlogits"])


@pytest.mark.parametrize("eps", [0.02, 0.2, 1e9])
@pytest.mark.parametrize("est", ["rkl_mc_clip", "rkl_mc_old_clip"])
def test_clipped_surrogates_across_clip_ranges(est, eps):
    """A stale behaviour policy puts ratios on both sides of the clip range,
    so both branches of the min run; a huge eps reduces to the unclipped form."""
    V = 4096
    w = synth.Workload("t_clip", N=33, V=V, dtype=synth.BF16, estimators=(est,), M=24,
                       sigma_student=2.0, sigma_behaviour=1.2, seed=77)
    d = synth.generate(w)
    say("clip %s eps=%g" % (est, eps))
    ids, tau, beta = cache_arrays(d, est)
    for flags in PATHS.values():
        out = run_gpu(to_dev(d["logits"]), est, ids, tau, beta, flags=flags, clip_eps=eps,
                      want_gathered=True, want_lse=True)
        compare("%s/eps=%g" % (est, eps), w, d, est, out, oracle_for(w, d, est, None, eps=eps))


def test_no_is_estimator_needs_no_behaviour_logprobs():
    w, d, mask = small_inputs("v32000", synth.BF16)
    say("no-IS without behav_logp")
    ids, tau, _ = cache_arrays(d, "rkl_mc_nois")
    out = opd.loss_fwd_bwd(to_dev(d["logits"]), "rkl_mc_nois", sampled_ids=to_dev(ids),
                           teacher_logp=to_dev(tau), mask=to_dev(mask))
    torch.cuda.synchronize()
    compare("nois", w, d, "rkl_mc_nois", out, oracle_for(w, d, "rkl_mc_nois", mask), mask)


@pytest.mark.parametrize("rows", ["stream_f32", "resident_tail_bf16"])
@pytest.mark.parametrize("est", ["rkl_mc", "fkl_topk", "rkl_topk_trunc"])
def test_large_support_on_the_streaming_path(est, rows):
    """K = 256 on fp32 rows wider than the registers (the streaming kernel:
    spikes found through the entries sorted by vector) and on bf16 rows
    whose last vector is partial (the resident kernel's tail), each also on
    the split path; MC with repeated ids (40 distinct values over 256
    draws) adding in order."""
    dtype, V, ld = {"stream_f32": (synth.F32, 80000, 80000),
                    "resident_tail_bf16": (synth.BF16, 5001, 5008)}[rows]
    N, K = 5, 256
    w = synth.Workload("t_kstream", N=N, V=V, dtype=dtype, estimators=(est,), k=K, M=K,
                       sigma_student=2.0, sigma_behaviour=0.4, seed=77)
    d = synth.generate(w, ld=ld)
    if est == "rkl_mc":
        rng = np.random.default_rng(7)
        ids = d["mc_ids"].copy()
        for r in range(N):
            ids[r] = rng.choice(rng.choice(V, 40, replace=False), K)
        d = dict(d, mc_ids=ids)
    say("large support %s %s" % (rows, est))
    ids, tau, beta = cache_arrays(d, est)
    logits = to_dev(d["logits"])[:, :V]
    for flags in PATHS.values():
        out = run_gpu(logits, est, ids, tau, beta, flags=flags, want_lse=True, want_gathered=True)
        compare("%s/%s K=%d" % (est, rows, K), w, d, est, out, oracle_for(w, d, est, None))


def test_mc_duplicate_samples_accumulate():
    """Samples are iid with replacement (App. E): repeated ids are separate
    terms of the average, so their gradient spikes add."""
    V, N, M = 512, 8, 12
    w = synth.Workload("t_dup", N=N, V=V, dtype=synth.F32, estimators=("rkl_mc",), M=M, seed=5)
    d = synth.generate(w)
    rng = np.random.default_rng(0)
    ids = d["mc_ids"].copy()
    for r in range(N):  # force repeats: 3 distinct ids repeated over 12 slots
        ids[r] = rng.choice(rng.choice(V, 3, replace=False), M)
    d = dict(d, mc_ids=ids)
    say("mc duplicates")
    for flags in PATHS.values():
        out = run_gpu(to_dev(d["logits"]), "rkl_mc", *cache_arrays(d, "rkl_mc"), flags=flags,
                      want_gathered=True)
        compare("dup", w, d, "rkl_mc", out, oracle_for(w, d, "rkl_mc", None))


def test_topk_gradient_zero_pattern_is_exact():
    """Top-k gradients are exactly zero off the cached support (App. A.1)."""
    w, d, mask = small_inputs("v32000", synth.BF16)
    say("topk zero pattern")
    for est in TOPK:
        for flags in PATHS.values():
            out = run_gpu(to_dev(d["logits"]), est, *cache_arrays(d, est), flags=flags)
            g = out["dlogits"].cpu().numpy()
            support = np.zeros_like(g, dtype=bool)
            np.put_along_axis(support, d["topk_idx"].astype(np.int64), True, axis=1)
            assert not g[~support].any()
            assert np.count_nonzero(g[support]) > 0.9 * support.sum()


@pytest.mark.parametrize("out_dt", [torch.float32, torch.bfloat16], ids=["f32-grad", "bf16-grad"])
@pytest.mark.parametrize("N,V,ld", [(40, 32000, 32008), (600, 131071, 131072)],
                         ids=["one-launch", "fill-then-sparse"])
@pytest.mark.parametrize("est", ["fkl_topk", "rkl_topk"])
def test_write_only_topk_forms(N, V, ld, est, out_dt):
    """The renormalised top-k estimators without lse_out write only the
    gradient's zeros and the support entries: in one launch for small calls,
    as a zero fill and a sparse writer for large ones (over 128 MiB of
    gradient).  Both with masked rows, with and without SKIP_MASKED, rows
    with an out-of-range id (NaN over their V columns), padding columns and
    (for the large call) a partial last vector; a sample of the other rows
    against the oracle."""
    w = synth.Workload("t_wo", N=N, V=V, dtype=synth.BF16, estimators=(est,), k=16,
                       sigma_student=2.5, sigma_teacher=1.0, seed=N + V)
    d = synth.generate(w, ld=ld)
    ids, tau = d["topk_idx"].copy(), d["topk_tau"].copy()
    bad = [3, N - 2]
    ids[3, 5], ids[N - 2, 0] = V, -1
    mask = np.ones(N, np.uint8)
    mask[[0, 7, N - 1]] = 0
    good = np.array([r for r in range(N) if mask[r] and r not in bad])
    sel = good[::max(1, len(good) // 24)]
    ref = oracle.rows(est, oracle_dtype(synth.BF16), d["logits"][sel], V,
                      ids=np.ascontiguousarray(ids[sel]), tau=np.ascontiguousarray(tau[sel]),
                      mask=mask[sel])
    mag = grad_mag(est, widen_dev(d["logits"][sel], V), ref, ids[sel], tau[sel], None,
                   mask=mask[sel])
    for skip in (False, True):
        say("write-only top-k %s N=%d V=%d skip=%d" % (est, N, V, skip))
        sentinel = 5.0
        buf = torch.full((N, ld), sentinel, dtype=out_dt, device=DEV)
        loss = torch.full((N,), sentinel, dtype=torch.float32, device=DEV)
        run_gpu(to_dev(d["logits"])[:, :V], est, ids, tau, None, mask=mask,
                flags=opd.FLAG_SKIP_MASKED if skip else 0, dlogits_dtype=out_dt,
                out={"loss": loss, "dlogits": buf})
        b, lo = buf.float().cpu().numpy(), loss.cpu().numpy()
        m = mask == 0
        assert np.all(b[:, V:] == sentinel), "padding columns written"
        assert np.all(b[m, :V] == (sentinel if skip else 0.0)), "masked rows"
        assert np.all(lo[m] == 0.0)
        assert np.isnan(b[bad, :V]).all() and np.isnan(lo[bad]).all(), "bad rows not NaN"
        check_loss("wo/%s" % est, lo[sel], ref["loss"],
                   loss_scale(est, ids[sel], tau[sel], None, ref), rtol_for(synth.BF16),
                   mask[sel])
        check_grad("wo/%s" % est, torch.from_numpy(b[sel, :V].astype(np.float64)), ref["grad"],
                   mag, bf16_out=out_dt == torch.bfloat16)


def test_padding_columns_and_skip_masked_rows_untouched():
    N, V, ld = 11, 1001, 1008
    w = synth.Workload("t_pad", N=N, V=V, dtype=synth.BF16, estimators=("rkl_mc",), M=4, seed=9)
    d = synth.generate(w, ld=ld)
    mask = np.ones(N, np.uint8)
    mask[[0, 5, 10]] = 0
    say("padding / skip-masked")
    ids, tau, beta = cache_arrays(d, "rkl_mc")
    for flags in PATHS.values():
        buf = torch.full((N, ld), 7.0, dtype=torch.float32, device=DEV)
        loss = torch.empty(N, dtype=torch.float32, device=DEV)
        out = run_gpu(to_dev(d["logits"])[:, :V], "rkl_mc", ids, tau, beta, mask=mask,
                      flags=flags | opd.FLAG_SKIP_MASKED, out={"loss": loss, "dlogits": buf})
        b = buf.cpu().numpy()
        assert np.all(b[:, V:] == 7.0), "padding columns written"
        assert np.all(b[mask == 0] == 7.0), "masked rows written despite SKIP_MASKED"
        ref = oracle_for(w, d, "rkl_mc", mask)
        check_loss("pad", loss.cpu().numpy(), ref["loss"],
                   loss_scale("rkl_mc", ids, tau, beta, ref), rtol_for(w.dtype), mask)
        keep = mask != 0
        mag = grad_mag("rkl_mc", widen_dev(d["logits"], V), ref, ids, tau, beta, mask=mask)
        check_grad("pad", torch.from_numpy(b[keep, :V].astype(np.float64)), ref["grad"][keep],
                   mag[torch.from_numpy(keep).to(DEV)])


@pytest.mark.parametrize("dtype,V,ld,est,out_dt", [
    (synth.BF16, 5001, 5008, "rkl_mc", torch.float32),      # resident row, partial last vector
    (synth.BF16, 4096, 4104, "fkl_dense", torch.bfloat16),  # dense resident row, bf16 gradient
    (synth.F32, 80001, 80004, "rkl_mc", torch.float32),     # fp32 row wider than the registers
], ids=["mc-bf16-tail", "dense-bf16-out", "mc-f32-stream"])
def test_masked_rows_of_large_calls(dtype, V, ld, est, out_dt):
    """A mask on a call of over 4,096 rows (where the row kernels stagger
    their rows): every masked row exactly zero over its V columns, no padding
    column written, and the rows on either side of each masked run, and a
    random sample of the others, as the oracle's."""
    N = 4100
    w = synth.Workload("t_fillmask", N=N, V=V, dtype=dtype, estimators=(est,), M=4,
                       sigma_student=2.5, sigma_teacher=1.0, sigma_behaviour=0.5,
                       dense_teacher=est in DENSE, seed=V + N)
    d = synth.generate(w, ld=ld)
    rng = np.random.default_rng(V)
    mask = (rng.random(N) > 0.1).astype(np.uint8)
    for r0, r1 in [(0, 300), (1000, 1001), (2047, 2600), (N - 1, N)]:
        mask[r0:r1] = 0
    say("masked rows of a large call: %s V=%d %s" % ("bf16" if dtype else "f32", V, est))
    sentinel = -3.0
    buf = torch.full((N, ld), sentinel, dtype=out_dt, device=DEV)
    loss = torch.full((N,), sentinel, dtype=torch.float32, device=DEV)
    ids, tau, beta = cache_arrays(d, est)
    teacher = to_dev(d["teacher_logits"])[:, :V] if est in DENSE else None
    run_gpu(to_dev(d["logits"])[:, :V], est, ids, tau, beta, teacher, mask=mask,
            dlogits_dtype=out_dt, out={"loss": loss, "dlogits": buf})
    masked = torch.from_numpy(mask == 0).to(DEV)
    assert bool((buf[:, V:] == sentinel).all()), "padding columns written"
    assert bool((buf[masked, :V] == 0).all()), "masked rows not zero"
    assert bool((loss[masked] == 0).all()), "masked rows' loss not zero"
    sel = np.r_[0:4, 296:306, 996:1006, 2040:2052, 2596:2606, N - 12:N,
                rng.choice(N, 40, replace=False)]
    sub = lambda a: None if a is None else np.ascontiguousarray(a[sel])  # noqa: E731
    ref = oracle.rows(est, oracle_dtype(dtype), d["logits"][sel], V, ids=sub(ids), tau=sub(tau),
                      beta=sub(beta), mask=mask[sel],
                      teacher_logits=sub(d["teacher_logits"]) if est in DENSE else None)
    check_loss("fillmask", loss.cpu().numpy()[sel], ref["loss"],
               loss_scale(est, sub(ids), sub(tau), sub(beta), ref), rtol_for(dtype), mask[sel])
    mag = grad_mag(est, widen_dev(d["logits"][sel], V), ref, sub(ids), sub(tau), sub(beta),
                   widen_dev(d["teacher_logits"][sel], V) if est in DENSE else None,
                   mask=mask[sel])
    check_grad("fillmask", buf[torch.from_numpy(sel).to(DEV), :V], ref["grad"], mag,
               bf16_out=out_dt == torch.bfloat16)


def test_topk_full_support_matches_dense_on_gpu():
    """k = V: renormalised top-k equals the dense KL (App. A.1 with S = V)."""
    N, V = 6, 256
    w = synth.Workload("t_kv", N=N, V=V, dtype=synth.F32, estimators=(), k=V, dense_teacher=True,
                       seed=12)
    d = synth.generate(w)
    say("k = V vs dense")
    logits, teacher = to_dev(d["logits"]), to_dev(d["teacher_logits"])
    for sparse, dense in (("fkl_topk", "fkl_dense"), ("rkl_topk", "rkl_dense")):
        a = run_gpu(logits, sparse, d["topk_idx"], d["topk_tau"], None)
        b = run_gpu(logits, dense, None, None, None, teacher)
        np.testing.assert_allclose(a["loss"].cpu().numpy(), b["loss"].cpu().numpy(), rtol=1e-4,
                                   atol=1e-5)
        np.testing.assert_allclose(a["dlogits"].cpu().numpy(), b["dlogits"].cpu().numpy(),
                                   atol=1e-5)


def test_out_of_range_ids_give_nan_rows_and_are_flagged():
    V, N = 2048, 6
    w = synth.Workload("t_bad", N=N, V=V, dtype=synth.BF16, estimators=(), k=8, M=8, seed=3)
    d = synth.generate(w)
    bad_rows = [1, 4]
    say("out-of-range ids")
    for est in ("rkl_topk", "rkl_mc"):
        ids, tau, beta = [None if a is None else a.copy() for a in cache_arrays(d, est)]
        ids[1, 3] = V
        ids[4, 0] = -5
        for flags in PATHS.values():
            out = run_gpu(to_dev(d["logits"]), est, ids, tau, beta, flags=flags)
            loss = out["loss"].cpu().numpy()
            g = out["dlogits"].cpu().numpy()
            good = [r for r in range(N) if r not in bad_rows]
            assert np.isnan(loss[bad_rows]).all() and np.isfinite(loss[good]).all()
            assert np.isnan(g[bad_rows]).all() and np.isfinite(g[good]).all()
        kw = dict(idx=to_dev(ids), teacher_logp=to_dev(tau)) if est in SUPPORT else dict(
            sampled_ids=to_dev(ids), teacher_logp=to_dev(tau), behav_logp=to_dev(beta))
        assert opd.validate_cache(est, V, **kw) == 2


def test_validate_cache_counts_each_violation():
    V, N, k = 1000, 5, 6
    ids = np.tile(np.arange(k, dtype=np.int32), (N, 1))
    tau = np.full((N, k), -2.0, np.float32)
    beta = np.full((N, k), -2.0, np.float32)
    say("validate cache")
    assert opd.validate_cache("rkl_topk", V, idx=to_dev(ids), teacher_logp=to_dev(tau)) == 0
    ids[0, 1] = ids[0, 0]           # one repeated pair
    ids[2, :3] = 7                  # three equal ids: three pairs
    tau[3, 2] = np.inf
    ids[4, 5] = 1000                # out of range
    assert opd.validate_cache("fkl_topk", V, idx=to_dev(ids), teacher_logp=to_dev(tau)) == 6
    # MC: repeats are legal; NaN behaviour log-prob is not
    beta[1, 1] = np.nan
    assert opd.validate_cache("rkl_mc", V, sampled_ids=to_dev(ids), teacher_logp=to_dev(tau),
                              behav_logp=to_dev(beta)) == 3


def _store(a: np.ndarray, dtype: int) -> np.ndarray:
    """float32 rows in the stored format of dtype (bf16: RNE bits)."""
    if dtype == synth.F32:
        return np.ascontiguousarray(a, np.float32)
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _wide_range_rows(V: int, seed: int, est: str):
    """Dense-estimator rows whose maxima arrive late and far above the early
    values: rising and falling ramps over +-60, spikes of +40 to +50 near the
    end of the row, leading -inf blocks of different lengths (the one of the
    distribution that weights the KL's terms is the longer, so the KL stays
    finite), and a row that is -inf but for its last two entries."""
    rng = np.random.default_rng(seed)
    ramp = np.linspace(-60.0, 60.0, V)
    z = np.empty((5, V)); y = np.empty((5, V))
    z[0], y[0] = ramp, ramp[::-1] + 0.3 * rng.standard_normal(V)
    z[1], y[1] = ramp[::-1], ramp + 0.3 * rng.standard_normal(V)
    z[2], y[2] = rng.standard_normal(V), rng.standard_normal(V)
    z[2, [V - 7, V - 1000, V // 2 + 3]] = [45.0, 40.0, 41.0]
    y[2, [V - 5, V // 3]] = [50.0, 44.0]
    z[3], y[3] = 2.0 * rng.standard_normal(V), 2.0 * rng.standard_normal(V)
    long, short = (11 * V) // 20, (7 * V) // 20
    z[3, :long if est == "rkl_dense" else short] = -np.inf
    y[3, :short if est == "rkl_dense" else long] = -np.inf
    z[4], y[4] = -np.inf, -np.inf
    z[4, -2:], y[4, -2:] = [3.0, 1.0], [0.5, 2.5]
    return z, y


@pytest.mark.parametrize("est", DENSE)
@pytest.mark.parametrize("dtype,V", [(synth.BF16, 151936), (synth.BF16, 65536),
                                     (synth.F32, 50000), (synth.F32, 32768)],
                         ids=["bf16-large", "bf16-small", "f32-large", "f32-small"])
def test_dense_rows_with_late_and_far_maxima(dtype, V, est):
    """The register-resident dense kernel keeps per-lane offsets that it raises
    only when a value exceeds them by a wide margin; these rows force raises in
    late slots, whole waves that never see a finite value, and large gaps
    between the two rows' maxima."""
    z, y = _wide_range_rows(V, V + dtype, est)
    zs, ys = _store(z, dtype), _store(y, dtype)
    say("wide-range %s V=%d %s" % ("bf16" if dtype else "f32", V, est))
    ref = oracle.rows(est, oracle_dtype(dtype), zs, V, teacher_logits=ys, gamma=0.5)
    assert np.isfinite(ref["loss"]).all()
    w = synth.Workload("t_wide", N=5, V=V, dtype=dtype, estimators=(est,), dense_teacher=True)
    for path, flags in PATHS.items():
        out = run_gpu(to_dev(zs), est, None, None, None, to_dev(ys), flags=flags, grad_scale=0.5,
                      want_lse=True)
        compare("wide/%d/%s/%s" % (V, est, path), w, {}, est, out, ref, gamma=0.5, logits=zs,
                teacher=ys)


@pytest.mark.parametrize("est", DENSE)
def test_dense_rows_with_a_partial_last_vector(est):
    """bf16 rows of full width whose V is not a multiple of 4 (the dense
    kernel's TAIL variant): the last vector's missing elements, here NaN in
    the padding, must be neither read into the sums nor written."""
    V, ld, N = 151933, 151936, 5
    z, y = _wide_range_rows(V, V + 3, est)
    zs, ys = _store(z, synth.BF16), _store(y, synth.BF16)

    def padded(a):
        p = np.full((N, ld), 0x7FC0, np.uint16)  # bf16 NaN in the padding
        p[:, :V] = a
        return p

    say("dense partial last vector %s" % est)
    ref = oracle.rows(est, oracle_dtype(synth.BF16), zs, V, teacher_logits=ys, gamma=0.5)
    w = synth.Workload("t_dtail", N=N, V=V, dtype=synth.BF16, estimators=(est,),
                       dense_teacher=True)
    for path, flags in PATHS.items():
        sentinel = -12345.0
        out = {"loss": torch.empty(N, device=DEV),
               "dlogits": torch.full((N, ld), sentinel, device=DEV)}
        res = run_gpu(to_dev(padded(zs))[:, :V], est, None, None, None,
                      to_dev(padded(ys))[:, :V], flags=flags, grad_scale=0.5, want_lse=True,
                      out=out)
        compare("dtail/%s/%s" % (est, path), w, {}, est, res, ref, gamma=0.5, logits=zs,
                teacher=ys)
        assert bool((out["dlogits"][:, V:] == sentinel).all()), "padding columns written"


@pytest.mark.parametrize("est", ["rkl_mc", "fkl_topk", "rkl_dense"])
def test_prepared_call_repeats_the_call(est):
    """A prepared call re-issues the same C call on the same tensors: after
    new data is copied into the inputs it gives what a fresh call on that
    data gives, bit for bit, and it allocates no device memory."""
    w1, d1, mask = small_inputs("v32000", synth.BF16)
    w2 = synth.Workload("t_prep", N=w1.N, V=w1.V, dtype=synth.BF16, estimators=(est,),
                        k=w1.k, M=w1.M, dense_teacher=True, seed=77)
    d2 = synth.generate(w2)
    N, V = w1.N, w1.V
    say("prepared call %s" % est)

    def inputs(d):
        ids, tau, beta = cache_arrays(d, est)
        kw = {}
        if est in SUPPORT:
            kw = dict(idx=to_dev(ids), teacher_logp=to_dev(tau))
        elif est in MC:
            kw = dict(sampled_ids=to_dev(ids), teacher_logp=to_dev(tau), behav_logp=to_dev(beta))
        else:
            kw = dict(teacher_logits=to_dev(d["teacher_logits"]))
        return to_dev(d["logits"]), kw

    logits, kw = inputs(d1)
    m = to_dev(mask)
    out = {"loss": torch.empty(N, device=DEV), "dlogits": torch.empty(N, V, device=DEV)}
    call = opd.prepare_loss_fwd_bwd(logits, est, mask=m, out=out, want_lse=True, **kw)
    for d in (d1, d2, d1):
        new_logits, new_kw = inputs(d)
        logits.copy_(new_logits)
        for key, t in kw.items():
            t.copy_(new_kw[key])
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        res = call()
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before, "a prepared call allocated"
        ref = opd.loss_fwd_bwd(new_logits, est, mask=m, want_lse=True, **new_kw)
        torch.cuda.synchronize()
        for key in ("loss", "dlogits", "lse"):
            assert torch.equal(res[key], ref[key]), key


def test_nan_logits_propagate_to_their_row_only():
    w, d, _ = small_inputs("v1000", synth.F32)
    logits = d["logits"].copy()
    logits[2, 17] = np.nan
    say("nan logits")
    for est in ("rkl_mc", "fkl_dense"):
        for flags in PATHS.values():
            teacher = to_dev(d["teacher_logits"]) if est in DENSE else None
            out = run_gpu(to_dev(logits), est, *cache_arrays(d, est), teacher, flags=flags)
            loss = out["loss"].cpu().numpy()
            assert np.isnan(loss[2]) and np.isfinite(np.delete(loss, 2)).all()


def test_repeated_calls_are_bitwise_identical():
    w, d, mask = small_inputs("v151936", synth.BF16)
    say("determinism")
    for est in ("rkl_mc", "rkl_topk", "rkl_dense"):
        for flags in PATHS.values():
            teacher = to_dev(d["teacher_logits"]) if est in DENSE else None
            ids, tau, beta = cache_arrays(d, est)
            logits = to_dev(d["logits"])
            r = [run_gpu(logits, est, ids, tau, beta, teacher, mask=mask, flags=flags)
                 for _ in range(3)]
            for o in r[1:]:
                assert torch.equal(o["loss"], r[0]["loss"])
                assert torch.equal(o["dlogits"], r[0]["dlogits"])


def test_empty_batch_is_a_noop():
    say("empty batch")
    logits = torch.empty((0, 1000), dtype=torch.bfloat16, device=DEV)
    ids = torch.empty((0, 4), dtype=torch.int32, device=DEV)
    f = torch.empty((0, 4), dtype=torch.float32, device=DEV)
    out = opd.loss_fwd_bwd(logits, "rkl_mc", sampled_ids=ids, teacher_logp=f, behav_logp=f)
    assert out["loss"].numel() == 0


# ---------------------------------------------------------------- full-size workloads

FULL = ["n512_v32000_f32_topk16_mc4", "n8192_v151936_bf16_topk32_peaked",
        "n32768_v151936_bf16_mc1_ragged", "n32768_v151936_bf16_mc16",
        "n256_v151936_bf16_mc16_smallbatch", "n16384_v151936_bf16_dense"]


CHUNK = 1024


def full_runs(w):
    """(estimator, flags, with lse/gathered outputs) runs of a full-size
    workload.  Every estimator runs with lse_out and gathered_out (for the MC
    and dense estimators the kernel path the benchmark times, plus two small
    stores); the renormalised top-k estimators also run without them, which
    is their write-only path and the configuration the benchmark times.
    Small batches also run the split-vocabulary path."""
    runs = []
    for est in w.estimators:
        if est in TOPK:
            runs.append((est, 0, False))
        runs.append((est, 0, True))
    if w.N <= 1024:
        runs += [(est, opd.FLAG_FORCE_SPLITV, True) for est in w.estimators]
    return runs


@pytest.mark.parametrize("name", FULL)
def test_parity_full_size(name):
    """Every row of every output against the oracle: loss and log-partition
    per row, gathered logits bit for bit, and every gradient element at the
    per-element bound (oracle rows in chunks of CHUNK, compared on the GPU);
    plus the zero row-sum of every gradient row."""
    w = synth.WORKLOADS[name]
    say("full-size %s: generating" % name)
    d = synth.generate(w)
    mask = d["mask"]
    N, V = w.N, w.V
    logits = to_dev(d["logits"])
    teacher = to_dev(d["teacher_logits"]) if w.dense_teacher else None
    dense = w.dense_teacher
    for est, flags, aux in full_runs(w):
        say("full-size %s %s flags=%d aux=%d" % (name, est, flags, aux))
        ids, tau, beta = cache_arrays(d, est)
        out = run_gpu(logits, est, ids, tau, beta, teacher, mask=mask, want_lse=aux,
                      want_gathered=aux and est not in DENSE, flags=flags,
                      want_coverage=aux and est in SUPPORT)
        if aux and est in SUPPORT:
            check_coverage("%s/%s" % (name, est), out["coverage"].cpu().numpy(),
                           oracle.coverage_rows(oracle_dtype(w.dtype), d["logits"], V, ids, tau,
                                                mask=mask), mask)
        ref_loss, ref_lse = np.zeros(N), np.zeros(N)
        ref_gat = [] if est not in DENSE else None
        worst = 0.0
        for r0 in range(0, N, CHUNK):
            sl = slice(r0, min(N, r0 + CHUNK))
            c_ids, c_tau, c_beta = [None if a is None else a[sl] for a in (ids, tau, beta)]
            ref = oracle.rows(est, oracle_dtype(w.dtype), d["logits"][sl], V, ids=c_ids,
                              tau=c_tau, beta=c_beta,
                              teacher_logits=d["teacher_logits"][sl] if est in DENSE else None,
                              mask=mask[sl])
            ref_loss[sl], ref_lse[sl] = ref["loss"], ref["lse"]
            if ref_gat is not None:
                ref_gat.append(ref["gathered"])
            mag = grad_mag(est, logits[sl, :V].double(), ref, c_ids, c_tau, c_beta,
                           teacher[sl, :V].double() if est in DENSE else None, 1.0, mask[sl])
            worst = max(worst, check_grad("%s/%s" % (name, est), out["dlogits"][sl],
                                          ref["grad"], mag, row0=r0))
            del ref, mag
        say("%s/%s flags=%d: dlogits max err/bound %.3g over every element" %
            (name, est, flags, worst))
        gat_ref = {"lse": ref_lse, "gathered": None if ref_gat is None else np.concatenate(ref_gat)}
        check_loss("%s/%s" % (name, est), out["loss"].cpu().numpy(), ref_loss,
                   loss_scale(est, ids, tau, beta, gat_ref), rtol_for(w.dtype), mask)
        valid = mask != 0
        if aux:
            lse = out["lse"].cpu().numpy().astype(np.float64)
            np.testing.assert_allclose(lse[valid], ref_lse[valid], rtol=2e-6)
            assert np.all(lse[~valid] == 0.0)
            if est not in DENSE:
                assert np.array_equal(out["gathered"].cpu().numpy().astype(np.float64),
                                      gat_ref["gathered"]), "gathered logits not bit-exact"
        rs = out["dlogits"].sum(dim=1, dtype=torch.float64).cpu().numpy()
        assert np.all(np.abs(rs) < 1e-4), "gradient rows must sum to zero"
        del out
        torch.cuda.empty_cache()
