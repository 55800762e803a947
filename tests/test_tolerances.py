"""The parity bounds of tolerances.py bite, and are not tighter than fp32
arithmetic allows.  CPU only.

A float32 model of each estimator's arithmetic (the order the kernels use:
exp2 of z log2(e) minus L log2(e), fp32 sums, one row coefficient plus spikes)
must pass every bound against the oracle.  Plausible mistakes, planted in
copies of the oracle's outputs on the CPU, must each fail: a coefficient off
by 1e-3, a log-partition off by 1e-4, a dropped, flipped or misplaced spike,
a wrong advantage (A_old for A_theta), a missing importance ratio, a 0.1%
error confined to the entries below 1e-4 (the bulk of a wide row, which the
stated 1e-4 absolute bound alone cannot see), a dropped -D term, the
unrenormalised top-k probabilities, and a loss off by 5e-4 relative (inside
the stated 1e-3 relative tolerance for bf16 logits, outside the fp32 bound).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import tolerances as T

LOG2E = np.float32(1.4426950408889634)
CPU = torch.device("cpu")


def f32(x):
    return np.asarray(x, np.float32)


def widen(stored, dtype):
    return synth.bf16_bits_to_f32(stored) if dtype == synth.BF16 else stored.astype(np.float32)


def lse32(z):
    """fp32 log-sum-exp, max then sum of exp2."""
    m = z.max(axis=1, keepdims=True)
    s = np.exp2(z * LOG2E - m * LOG2E, dtype=np.float32).sum(axis=1, keepdims=True,
                                                                dtype=np.float32)
    return f32(m + np.log(s, dtype=np.float32))


def p32(z, L):
    return np.exp2(z * LOG2E - L * LOG2E, dtype=np.float32)


@pytest.fixture(scope="module")
def mc():
    w = synth.Workload("tol_mc", N=24, V=30000, dtype=synth.BF16, estimators=("rkl_mc",), M=16,
                       sigma_student=3.0, sigma_behaviour=0.5, seed=41)
    d = synth.generate(w)
    z = widen(d["logits"], w.dtype)
    ids, tau, beta = d["mc_ids"], d["mc_tau"], d["mc_beta"]
    ref = oracle.rows("rkl_mc", oracle.BF16, d["logits"], w.V, ids=ids, tau=tau, beta=beta)
    return w, z, ids, tau, beta, ref


def mc_model(z, ids, tau, beta, gamma=1.0, L_shift=0.0, coef=1.0, adv="theta", ratio=True):
    """fp32 model of the MC kernels: C p_j + spikes."""
    L = lse32(z) + f32(L_shift)
    gathered = np.take_along_axis(z, ids.astype(np.int64), 1)
    lp = f32(gathered - L)
    A = f32(tau - beta) if adv == "old" else f32(tau - lp)
    rho = np.exp(lp - beta, dtype=np.float32) if ratio else np.ones_like(lp)
    w = f32(rho * A)
    M = ids.shape[1]
    C = f32(w.sum(axis=1, keepdims=True, dtype=np.float32) / np.float32(M)) * f32(coef)
    g = f32(gamma) * C * p32(z, L)
    for r in range(z.shape[0]):
        for i in range(M):
            g[r, ids[r, i]] += f32(-gamma * w[r, i] / M)
    return g, f32(-C[:, 0] / coef)


def mag_mc(z, ids, tau, beta, ref, gamma=1.0):
    return T.grad_magnitude("rkl_mc", torch.from_numpy(z), ref["lse"], gathered=ref["gathered"],
                            ids=ids, tau=tau, beta=beta, gamma=gamma)


def n_bad(g, ref, mag):
    return T.grad_check(torch.from_numpy(np.asarray(g, np.float64)), ref["grad"], mag)[0]


def test_fp32_model_of_the_mc_kernels_passes(mc):
    w, z, ids, tau, beta, ref = mc
    g, loss = mc_model(z, ids, tau, beta)
    mag = mag_mc(z, ids, tau, beta, ref)
    bad, worst, _ = T.grad_check(torch.from_numpy(g.astype(np.float64)), ref["grad"], mag)
    assert bad == 0 and worst < 0.5, worst
    s = T.loss_scale("rkl_mc", ref["lse"], ref["gathered"], tau, beta)
    r = T.loss_check(loss, ref["loss"], s, 1e-3)
    assert r["scaled"] == r["plain"] == r["arith"] == 0, r


def test_most_gradient_entries_are_below_the_absolute_tolerance(mc):
    """Why the per-element bound is needed: at V = 30,000 and sigma 3 almost
    every entry is smaller than 1e-4, so the stated absolute tolerance alone
    constrains almost nothing."""
    ref = mc[5]
    assert np.mean(np.abs(ref["grad"]) < 1e-4) > 0.95


@pytest.mark.parametrize("mistake", ["coef_1e-3", "L_shift_1e-4", "adv_old", "no_ratio",
                                     "drop_spike", "flip_spike", "move_spike", "small_entries",
                                     "gamma_twice"])
def test_planted_mc_mistakes_fail(mc, mistake):
    w, z, ids, tau, beta, ref = mc
    kw = {"coef_1e-3": dict(coef=1.001), "L_shift_1e-4": dict(L_shift=1e-4),
          "adv_old": dict(adv="old"), "no_ratio": dict(ratio=False)}.get(mistake, {})
    g, _ = mc_model(z, ids, tau, beta, **kw)
    g = g.astype(np.float64)
    r = np.arange(z.shape[0])
    spike = -ref["grad"][r, ids[:, 0]] + np.exp(z[r, ids[:, 0]] - ref["lse"]) * -ref["loss"]
    if mistake == "drop_spike":
        g[r, ids[:, 0]] -= spike / np.maximum(1, (ids == ids[:, :1]).sum(1))
    elif mistake == "flip_spike":
        g[r, ids[:, 0]] -= 2 * spike / np.maximum(1, (ids == ids[:, :1]).sum(1))
    elif mistake == "move_spike":
        g[r, ids[:, 0]] -= spike
        g[r, (ids[:, 0] + 1) % z.shape[1]] += spike
    elif mistake == "small_entries":
        small = np.abs(ref["grad"]) < 1e-4
        g = np.where(small, ref["grad"] * 1.001, g)
    elif mistake == "gamma_twice":
        g = 2.0 * g
    assert n_bad(g, ref, mag_mc(z, ids, tau, beta, ref)) > 0, mistake


@pytest.fixture(scope="module")
def dense():
    w = synth.DENSE.replace(N=12, V=20000)
    d = synth.generate(w)
    z, y = widen(d["logits"], w.dtype), widen(d["teacher_logits"], w.dtype)
    return w, d, z, y


def dense_model(est, z, y, drop_D=False, fkl_form=False, shared_L=False):
    Lz, Ly = lse32(z), lse32(y)
    if shared_L:
        Ly = Lz
    p, q = p32(z, Lz), p32(y, Ly)
    if est == "fkl_dense" or fkl_form:
        return f32(p - q)
    ez = f32((p * (z - y)).sum(axis=1, keepdims=True, dtype=np.float32) /
             p.sum(axis=1, keepdims=True, dtype=np.float32))
    return f32(p * ((z - y) - (0.0 if drop_D else ez)))


@pytest.mark.parametrize("est", ["fkl_dense", "rkl_dense"])
def test_dense_fp32_model_passes_and_mistakes_fail(dense, est):
    w, d, z, y = dense
    ref = oracle.rows(est, oracle.BF16, d["logits"], w.V, teacher_logits=d["teacher_logits"])
    mag = T.grad_magnitude(est, torch.from_numpy(z), ref["lse"], y=torch.from_numpy(y),
                           loss=ref["loss"])
    bad, worst, _ = T.grad_check(torch.from_numpy(dense_model(est, z, y).astype(np.float64)),
                                 ref["grad"], mag)
    assert bad == 0 and worst < 0.5, worst
    # (the teacher's normaliser cancels from the reverse-KL gradient)
    planted = ([dict(drop_D=True), dict(fkl_form=True)] if est == "rkl_dense"
               else [dict(shared_L=True)])
    for kw in planted:
        g = dense_model(est, z, y, **kw).astype(np.float64)
        assert n_bad(g, ref, mag) > 0, kw


def test_topk_fp32_model_passes_and_unrenormalised_fails():
    w = synth.TOPK32.replace(N=16, V=20000)
    d = synth.generate(w)
    z = widen(d["logits"], w.dtype)
    ids, tau = d["topk_idx"], d["topk_tau"]
    ref = oracle.rows("fkl_topk", oracle.BF16, d["logits"], w.V, ids=ids, tau=tau)
    gz = np.take_along_axis(z, ids.astype(np.int64), 1)

    def model(renorm=True):
        ls = lse32(gz) if renorm else lse32(z)
        pt = np.exp(gz - ls, dtype=np.float32)
        qt = np.exp(tau - lse32(tau), dtype=np.float32)
        g = np.zeros_like(z)
        np.put_along_axis(g, ids.astype(np.int64), f32(pt - qt), 1)
        return g.astype(np.float64)

    mag = T.grad_magnitude("fkl_topk", torch.from_numpy(z), ref["lse"], gathered=ref["gathered"],
                           ids=ids, tau=tau)
    assert n_bad(model(), ref, mag) == 0
    assert n_bad(model(renorm=False), ref, mag) > 0
    # a nonzero entry off the support fails (the bound there is the fp32 underflow floor)
    g = model()
    off = np.setdiff1d(np.arange(w.V), ids[0])[0]
    g[0, off] = 1e-12
    assert n_bad(g, ref, mag) > 0


def test_loss_bounds_bite_inside_the_stated_bf16_tolerance(mc):
    """A loss 5e-4 off (relative) passes the stated 1e-3 tolerance for bf16
    logits but fails the fp32 evaluation's own bound."""
    w, z, ids, tau, beta, ref = mc
    s = T.loss_scale("rkl_mc", ref["lse"], ref["gathered"], tau, beta)
    got = ref["loss"] * (1 + 5e-4) + 5e-4 * s
    r = T.loss_check(got, ref["loss"], s, 1e-3)
    assert r["scaled"] == 0 and r["arith"] > 0
