"""Parity tolerances of the HIP path against the oracle, shared by the GPU
tests and the CPU test that shows they bite.  Plain torch, on whatever device
the tensors are on (the full-size GPU tests compare on the GPU, chunk by
chunk; the CPU test runs the same code on the host).

Gradient (fp32 output).  Every element must satisfy both
  |g - ref| <= 1e-4                      (the stated absolute tolerance), and
  |g - ref| <= GRAD_RTOL * mag + GRAD_FLOOR,
where mag is the element's natural magnitude: |gamma| times the sum of the
absolute values of the terms that make up dloss/dz_j, each term weighted as the
fp32 evaluation perturbs it.  For the gradients of Sec. 3 (dense), App. A.1
(top-k) and Sec. 5.1 / App. E (MC and the truncated KLs, all of the form
C p_j + spikes at the cached ids):
  MC family        p_j S_C + sum_{i: a_i = j} S_i, S_i = w_i (|A_i| + 1) / M,
                   w_i = rho_i (1 for the estimator without ratios), S_C = sum_i S_i
  truncated FKL    S_i = q_i,                       S_C = sum_i S_i
  truncated RKL    S_i = p_i (|log p_i - log q_i| + 2), S_C = sum_i S_i
  top-k FKL        p~_i + q~_i on S, 0 off S
  top-k RKL        p~_i (|log p~_i - log q~_i| + |D| + 1) on S, 0 off S
  dense FKL        p_j + q_j
  dense RKL        p_j (|z_j - y_j| + |E_p[z - y]| + 1), the two quantities
                   the kernel subtracts (E_p[z - y] = D_R + L_z - L_y)
GRAD_RTOL follows from the fp32 arithmetic of the kernels: p_j = exp2(z_j log2e
- L log2e) carries the error of L (an fp32 log-sum-exp: at most about 6e-6
absolute, from about 60 levels of fp32 sums, one log and one add), of the
rounded argument (at most about 3e-6 relative) and of exp2 (one ulp), about
1e-5 relative in all; the row coefficient C is an fp32 sum of M terms whose
weights carry the same errors, about 1e-5 of S_C.  The bound takes 3e-5.  A
wrong coefficient, a dropped term or a wrong normaliser moves an element by
1e-3 or more of its magnitude.  bf16 output adds one bf16 ulp (2^-7 |ref|;
round-to-nearest-even errs by up to half of that).  GRAD_FLOOR = 1e-30
covers underflow: an fp32 p_j below the normal range (1.2e-38) flushes, and
the weights that multiply it (|z - y| + |E_p[z - y]| on rows spanning +-60,
a ratio times an advantage) reach a few hundred; entries whose reference lies
below 1e-30 are held to that floor only.
Entries of magnitude 0 (masked rows, top-k entries off the support) must be
0 up to GRAD_FLOOR; the exact zero pattern has its own test.

Loss.  Per row, with s the natural magnitude of the row's terms (1 for the
KLs, whose weights sum to one; (1/M) sum_i w_i (|A_i| + 1) for the MC family):
  |l - ref| <= rtol (|ref| + s)        rtol = 1e-5 (fp32 logits) / 1e-3 (bf16)
  |l - ref| <= rtol |ref|              on rows with |ref| >= s / 2
  |l - ref| <= LOSS_ARITH_RTOL (|ref| + s)   (the fp32 evaluation's own
                                        bound; it binds for bf16 logits,
                                        whose widening is exact)
"""
from __future__ import annotations

import numpy as np
import torch

GRAD_ATOL = 1e-4
GRAD_RTOL = 3e-5
GRAD_FLOOR = 1e-30
BF16_ULP = 2.0 ** -7
LOSS_ARITH_RTOL = 2e-5

MC_IS = ("rkl_mc1", "rkl_mc", "rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip")
MC_OLD_ADV = ("rkl_mc_old", "rkl_mc_old_clip")


def as_t(a, device, dtype=torch.float64):
    if isinstance(a, torch.Tensor):
        return a.to(device=device, dtype=dtype)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


def mc_term_weights(est, lp, tau, beta):
    """S_i of the MC family and the truncated KLs (see the module docstring),
    before the 1/M or the gamma factor; lp = log p_theta at the cached ids."""
    if est == "fkl_topk_trunc":
        return torch.exp(tau)
    if est == "rkl_topk_trunc":
        return torch.exp(lp) * ((lp - tau).abs() + 2.0)
    A = tau - beta if est in MC_OLD_ADV else tau - lp
    w = torch.ones_like(lp) if est == "rkl_mc_nois" else torch.exp(lp - beta)
    return w * (A.abs() + 1.0)


def grad_magnitude(est, z, lse, *, gathered=None, ids=None, tau=None, beta=None, y=None,
                   loss=None, gamma=1.0, mask=None):
    """mag [n, V] (float64, on z's device) of every gradient element.

    z      [n, V] widened student logits (any float tensor)
    lse    [n] the oracle's log-partitions
    gathered, ids, tau, beta [n, K]  the oracle's gathered logits and the cache
    y      [n, V] widened teacher logits (dense estimators)
    loss   [n] the oracle's losses (the D of the reverse KLs)
    """
    dev = z.device
    z = z.to(torch.float64)
    lse = as_t(lse, dev)
    n, V = z.shape
    if est in ("fkl_dense", "rkl_dense"):
        y = as_t(y, dev)
        p = torch.exp(z - lse[:, None])
        ly = torch.logsumexp(y, dim=1, keepdim=True)
        if est == "fkl_dense":
            mag = p + torch.exp(y - ly)
        else:
            # the kernel forms (z - y) - E_p[z - y], E_p[z - y] = D_R + L_z - L_y
            ez = (as_t(loss, dev)[:, None] + lse[:, None] - ly).abs()
            mag = torch.where(p > 0, p * ((z - y).abs() + ez + 1.0), torch.zeros_like(p))
    else:
        g = as_t(gathered, dev)
        tau = as_t(tau, dev)
        ids = as_t(ids, dev, torch.int64).clamp(0, V - 1)
        mag = torch.zeros((n, V), dtype=torch.float64, device=dev)
        if est in ("fkl_topk", "rkl_topk"):
            lpt = g - torch.logsumexp(g, dim=1, keepdim=True)
            lqt = tau - torch.logsumexp(tau, dim=1, keepdim=True)
            pt, qt = torch.exp(lpt), torch.exp(lqt)
            if est == "fkl_topk":
                s = pt + qt
            else:
                D = (pt * (lpt - lqt)).sum(dim=1, keepdim=True).abs()
                s = pt * ((lpt - lqt).abs() + D + 1.0)
            mag.scatter_add_(1, ids, s)
        else:
            lp = g - lse[:, None]
            b = None if beta is None else as_t(beta, dev)
            M = g.shape[1]
            S = mc_term_weights(est, lp, tau, b)
            if est not in ("fkl_topk_trunc", "rkl_topk_trunc"):
                S = S / M
            SC = S.sum(dim=1, keepdim=True)
            mag = torch.exp(z - lse[:, None]) * SC
            mag.scatter_add_(1, ids, S)
    if mask is not None:
        keep = as_t(mask, dev) != 0
        mag = torch.where(keep[:, None], mag, torch.zeros_like(mag))
    return mag * abs(float(gamma))


def grad_check(got, ref, mag, bf16_out=False):
    """(number of violations, largest err / bound, index of the worst) of a
    gradient block against the oracle's.  All three on one device."""
    got = got.to(torch.float64)
    ref = as_t(ref, got.device)
    err = (got - ref).abs()
    extra = BF16_ULP * ref.abs() if bf16_out else 0.0
    tol = torch.minimum(torch.full_like(ref, GRAD_ATOL), GRAD_RTOL * mag + GRAD_FLOOR) + extra
    ratio = err / tol
    ratio = torch.where(torch.isnan(ratio), torch.full_like(ratio, float("inf")), ratio)
    bad = int((~(err <= tol)).sum())
    worst = int(torch.argmax(ratio))
    return bad, float(ratio.reshape(-1)[worst]), divmod(worst, ref.shape[1])


def loss_check(got, ref, scale, rtol, mask=None):
    """Violations of the three loss bounds; returns a dict with the counts and
    the largest relative errors (err / (|ref| + s) and, on the rows the plain
    relative check covers, err / |ref|)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.asarray(scale, np.float64)
    err = np.abs(got - ref)
    tol_s = rtol * (np.abs(ref) + scale)
    tol_a = LOSS_ARITH_RTOL * (np.abs(ref) + scale)
    plain = np.abs(ref) >= scale / 2
    res = {"scaled": int((~(err <= tol_s)).sum()),
           "arith": int((~(err <= tol_a)).sum()),
           "plain": int((~(err[plain] <= rtol * np.abs(ref[plain]))).sum()),
           "max_scaled_rel": float(np.max(err / np.maximum(np.abs(ref) + scale, 1e-300),
                                          initial=0.0)),
           "max_plain_rel": float(np.max(err[plain] / np.abs(ref[plain]), initial=0.0)),
           "plain_rows": int(plain.sum())}
    if mask is not None:
        res["masked_nonzero"] = int(np.count_nonzero(got[np.asarray(mask) == 0]))
    return res


def loss_scale(est, lse, gathered=None, tau=None, beta=None):
    """Per-row s of the loss bounds (see the module docstring).  The surrogate
    without ratios sums products A_i log p_i, so its s also counts |log p_i|."""
    lse = np.asarray(lse, np.float64)
    if est not in MC_IS + ("rkl_mc_nois",):
        return np.ones(lse.shape[0])
    lp = np.asarray(gathered, np.float64) - lse[:, None]
    tau = np.asarray(tau, np.float64)
    if est == "rkl_mc_nois":
        return (np.abs(tau - lp) + np.abs(lp) + 1.0).mean(axis=1)
    beta = np.asarray(beta, np.float64)
    A = tau - beta if est in MC_OLD_ADV else tau - lp
    return (np.exp(lp - beta) * (np.abs(A) + 1.0)).mean(axis=1)
