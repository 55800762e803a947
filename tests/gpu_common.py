"""Shared helpers of the GPU parity tests: device copies of generated inputs,
one call through the C ABI, the oracle on the same inputs, and the
comparison at the bounds of tolerances.py (per-token loss: the stated
relative tolerances plus the fp32 evaluation's own bound; gradient: every
element within 1e-4 and within GRAD_RTOL of its natural magnitude; gathered
logits bit for bit).  The gradient comparison runs on the GPU in torch,
chunk by chunk, against the oracle's values copied there.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2606_24143_amd as opd
import synth
import tolerances

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
    """Per-row s of the loss bounds (tolerances.loss_scale)."""
    return tolerances.loss_scale(est, ref["lse"], ref.get("gathered"), tau, beta)


def check_loss(name, got, ref_loss, scale, rtol, mask=None):
    r = tolerances.loss_check(got, ref_loss, scale, rtol, mask)
    say("%s: loss max err/(|ref|+s) %.3g, max plain relative err %.3g (%d rows)" %
        (name, r["max_scaled_rel"], r["max_plain_rel"], r["plain_rows"]))
    assert r.get("masked_nonzero", 0) == 0, name + ": masked rows must have loss 0"
    assert r["scaled"] == 0 and r["plain"] == 0 and r["arith"] == 0, (
        "%s: loss outside its bounds (%d scaled, %d plain-relative, %d fp32-arithmetic rows); "
        "max err/(|ref|+s) %.3g" % (name, r["scaled"], r["plain"], r["arith"],
                                    r["max_scaled_rel"]))


def widen_dev(stored, V: int) -> torch.Tensor:
    """Stored rows (uint16 bf16 bits or float32, [n, ld]) as float64 on the GPU."""
    return to_dev(stored)[:, :V].to(torch.float64)


def grad_mag(est, z_dev, ref, ids, tau, beta, y_dev=None, gamma=1.0, mask=None):
    """tolerances.grad_magnitude on the GPU from the oracle's outputs."""
    return tolerances.grad_magnitude(est, z_dev, ref["lse"], gathered=ref.get("gathered"),
                                     ids=ids, tau=tau, beta=beta, y=y_dev, loss=ref["loss"],
                                     gamma=gamma, mask=mask)


def check_grad(name, got, ref_grad, mag, bf16_out=False, row0=0):
    """Every element of a gradient block (got: GPU tensor) against the
    oracle's (numpy or tensor) at the per-element bound; returns the largest
    err / bound."""
    if not isinstance(got, torch.Tensor):
        got = torch.from_numpy(np.asarray(got, np.float64))
    got = got.to(DEV)
    ref = tolerances.as_t(ref_grad, DEV)
    bad, worst, (r, c) = tolerances.grad_check(got, ref, mag.to(DEV), bf16_out)
    if bad:
        raise AssertionError("%s: dlogits [%d, %d] got %.9g ref %.9g (bound %.3g); %d bad entries"
                             % (name, row0 + r, c, float(got[r, c]), float(ref[r, c]),
                                float(min(tolerances.GRAD_ATOL,
                                          tolerances.GRAD_RTOL * float(mag[r, c]) +
                                          tolerances.GRAD_FLOOR)), bad))
    return worst


def dlogits_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def rtol_for(dtype: int) -> float:
    return 1e-5 if dtype == synth.F32 else 1e-3


def oracle_dtype(dtype: int) -> int:
    return oracle.BF16 if dtype == synth.BF16 else oracle.F32
