"""Shared helpers of the GPU parity tests: device copies of generated inputs,
one call through the C ABI, the oracle on the same inputs, and the
comparison at the stated tolerances.

Tolerances (per token loss): |gpu - ref| <= rtol * (|ref| + s), rtol = 1e-5
for fp32 logits and 1e-3 for bf16 logits (fp32 accumulation).  s is the
natural magnitude of the terms the loss sums: 1 for the top-k and dense KLs
(their weights sum to one), (1/M) sum_i rho_i (|A_i| + 1) for the MC
surrogates (A_theta or A_old), whose value can cancel to near zero while their
terms do not, and (1/M) sum_i (|A_i| + |log p_i| + 1) for the surrogate
without importance ratios, whose terms are products A_i log p_i.
Gradient: |gpu - ref| <= 1e-4 for fp32 output; bf16 output adds one bf16 ulp
(2^-8 relative).  Gathered logits are compared bit for bit.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2606_24143_amd as opd
import synth

DEV = torch.device("cuda:0")
TOPK = ("fkl_topk", "rkl_topk")             # renormalised on S
TRUNC = ("fkl_topk_trunc", "rkl_topk_trunc")  # truncated, full-vocabulary normalisers
SUPPORT = TOPK + TRUNC                        # every estimator reading the top-k cache
MC = ("rkl_mc1", "rkl_mc", "rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois")
MC_FAMILY = ("rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois")
DENSE = ("fkl_dense", "rkl_dense")


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype: int = None) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def cache_arrays(d: dict, est: str, M: int = None):
    """(ids, tau, beta) numpy arrays of the cache an estimator reads."""
    if est in SUPPORT:
        return d["topk_idx"], d["topk_tau"], None
    if est in MC:
        m = 1 if est == "rkl_mc1" else (M or d["mc_ids"].shape[1])
        return (np.ascontiguousarray(d["mc_ids"][:, :m]), np.ascontiguousarray(d["mc_tau"][:, :m]),
                np.ascontiguousarray(d["mc_beta"][:, :m]))
    return None, None, None


def run_gpu(logits_dev, est, ids, tau, beta, teacher_dev=None, mask=None, **kw):
    cache = {}
    if est in SUPPORT:
        cache = dict(idx=to_dev(ids), teacher_logp=to_dev(tau))
    elif est in MC:
        cache = dict(sampled_ids=to_dev(ids), teacher_logp=to_dev(tau), behav_logp=to_dev(beta))
    else:
        cache = dict(teacher_logits=teacher_dev)
    m = None if mask is None else to_dev(mask)
    out = opd.loss_fwd_bwd(logits_dev, est, mask=m, **cache, **kw)
    torch.cuda.synchronize()
    return out


def loss_scale(est, ids, tau, beta, ref):
    """Per-row s of the loss tolerance (see module docstring)."""
    n = ref["loss"].shape[0]
    if est not in MC:
        return np.ones(n)
    lp = ref["gathered"] - ref["lse"][:, None]
    tau = tau.astype(np.float64)
    if est == "rkl_mc_nois":
        return (np.abs(tau - lp) + np.abs(lp) + 1.0).mean(axis=1)
    beta = beta.astype(np.float64)
    A = tau - beta if est in ("rkl_mc_old", "rkl_mc_old_clip") else tau - lp
    rho = np.exp(lp - beta)
    return (rho * (np.abs(A) + 1.0)).mean(axis=1)


def check_loss(name, got, ref_loss, scale, rtol, mask=None):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref_loss)
    tol = rtol * (np.abs(ref_loss) + scale)
    bad = ~(err <= tol)
    if mask is not None:
        assert np.all(got[mask == 0] == 0.0), name + ": masked rows must have loss 0"
    if bad.any():
        i = int(np.argmax(np.where(bad, err / np.maximum(tol, 1e-30), 0)))
        raise AssertionError("%s: loss row %d got %.9g ref %.9g (tol %.3g); %d bad rows" %
                             (name, i, got[i], ref_loss[i], tol[i], int(bad.sum())))


def check_grad(name, got, ref_grad, bf16_out=False, atol=1e-4):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref_grad)
    tol = atol + (2.0 ** -8 * np.abs(ref_grad) if bf16_out else 0.0)
    bad = ~(err <= tol)
    if bad.any():
        idx = np.unravel_index(int(np.argmax(np.where(bad, err - tol, -np.inf))), err.shape)
        raise AssertionError("%s: dlogits %s got %.9g ref %.9g; %d bad entries" %
                             (name, idx, got[idx], ref_grad[idx], int(bad.sum())))


def dlogits_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def rtol_for(dtype: int) -> float:
    return 1e-5 if dtype == synth.F32 else 1e-3


def oracle_dtype(dtype: int) -> int:
    return oracle.BF16 if dtype == synth.BF16 else oracle.F32
