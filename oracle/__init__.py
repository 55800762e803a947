"""The oracle: a plain double-precision CPU implementation of the OPD loss.

Test infrastructure.  Only tests/, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library (``paper_2606_24143_amd``) and never imports it.

The arithmetic lives in ``opd_oracle.c`` (one function per estimator, each
citing the passage of the paper it follows); this module only marshals numpy
arrays into it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "opd_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

ESTIMATORS = {"fkl_topk": 0, "rkl_topk": 1, "rkl_mc1": 2, "rkl_mc": 3, "fkl_dense": 4,
              "rkl_dense": 5, "rkl_mc_clip": 6, "rkl_mc_old": 7, "rkl_mc_old_clip": 8,
              "rkl_mc_nois": 9, "fkl_topk_trunc": 10, "rkl_topk_trunc": 11}
TOPK = ("fkl_topk", "rkl_topk", "fkl_topk_trunc", "rkl_topk_trunc")
DENSE = ("fkl_dense", "rkl_dense")
MC = ("rkl_mc1", "rkl_mc", "rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois")
CLIP_EPS = 0.2  # the paper's PPO clip range (App. B, Table 3)
F32, BF16 = 0, 1


def build(force: bool = False) -> str:
    """Compile liboracle.so in place with gcc."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp,
                        _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        L.oracle_row.argtypes = [ctypes.c_int, P, P, i64, P, P, P, ctypes.c_int, ctypes.c_double,
                                 ctypes.c_double, ctypes.c_int, P, P, P, P]
        L.oracle_row.restype = ctypes.c_int
        L.oracle_rows.argtypes = [ctypes.c_int, ctypes.c_int, P, P, i64, i64, i64, P, P, P,
                                  ctypes.c_int, P, ctypes.c_double, ctypes.c_double, P, P, P, P,
                                  ctypes.c_int]
        L.oracle_rows.restype = ctypes.c_int
        L.oracle_max_threads.restype = ctypes.c_int
        L.oracle_support_coverage.argtypes = [P, i64, P, P, ctypes.c_int, P, P]
        L.oracle_support_coverage.restype = ctypes.c_int
        L.oracle_coverage_rows.argtypes = [ctypes.c_int, P, i64, i64, i64, P, P, ctypes.c_int, P,
                                           P, ctypes.c_int]
        L.oracle_coverage_rows.restype = ctypes.c_int
        L.oracle_cdf.argtypes = [P, i64, P]
        L.oracle_cdf.restype = ctypes.c_int
        L.oracle_sample_row.argtypes = [P, i64, P, ctypes.c_int, P, P, P]
        L.oracle_sample_row.restype = ctypes.c_int
        L.oracle_topk_row.argtypes = [ctypes.c_int, P, i64, ctypes.c_int, P, P, P]
        L.oracle_topk_row.restype = ctypes.c_int
        L.oracle_score_row.argtypes = [P, i64, P, ctypes.c_int, P, P]
        L.oracle_score_row.restype = ctypes.c_int
        L.oracle_cache_rows.argtypes = [ctypes.c_int, ctypes.c_int, P, i64, i64, i64, ctypes.c_int,
                                        P, P, P, P, P, ctypes.c_int]
        L.oracle_cache_rows.restype = ctypes.c_int
        L.oracle_mc_diagnostics.argtypes = [P, P, P, P, i64, ctypes.c_int, P, ctypes.c_double,
                                            ctypes.c_double, P, ctypes.c_int, i64, P, P, P, P, P,
                                            P, P]
        L.oracle_mc_diagnostics.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def row(est: str, z, ids=None, tau=None, beta=None, y=None, gamma: float = 1.0,
        valid: bool = True, want_grad: bool = True, eps: float = CLIP_EPS):
    """One token row in double.  Returns (loss, grad or None, lse, gathered or None)."""
    z = np.ascontiguousarray(z, np.float64)
    V = z.size
    dense = est in DENSE
    y = None if y is None else np.ascontiguousarray(y, np.float64)
    if not dense:
        ids = np.ascontiguousarray(ids, np.int32)
        tau = np.ascontiguousarray(tau, np.float64)
        beta = None if beta is None else np.ascontiguousarray(beta, np.float64)
        K = ids.size
    else:
        K = 0
    loss = np.zeros(1, np.float64)
    lse = np.zeros(1, np.float64)
    grad = np.zeros(V, np.float64) if want_grad else None
    gathered = np.zeros(K, np.float64) if K else None
    rc = lib().oracle_row(ESTIMATORS[est], _p(z), _p(y), V, _p(ids), _p(tau), _p(beta), K, gamma,
                          eps, int(valid), _p(loss), _p(grad), _p(lse), _p(gathered))
    if rc != 0:
        raise ValueError("oracle_row rejected its arguments (%d)" % rc)
    return float(loss[0]), grad, float(lse[0]), gathered


def rows(est: str, dtype: int, logits: np.ndarray, V: int, *, ids=None, tau=None, beta=None,
         teacher_logits=None, mask=None, gamma: float = 1.0, want_grad: bool = True,
         nthreads: int = 0, eps: float = CLIP_EPS) -> dict:
    """Rows of stored inputs: logits [n, ld] (uint16 bf16 bits or float32)."""
    logits = np.ascontiguousarray(logits)
    n, ld = logits.shape
    dense = est in DENSE
    K = 0 if dense else ids.shape[1]
    if not dense:
        ids = np.ascontiguousarray(ids, np.int32)
        tau = np.ascontiguousarray(tau, np.float32)
        beta = None if beta is None else np.ascontiguousarray(beta, np.float32)
    if teacher_logits is not None:
        teacher_logits = np.ascontiguousarray(teacher_logits)
    mask = None if mask is None else np.ascontiguousarray(mask, np.uint8)
    out = {"loss": np.zeros(n, np.float64), "lse": np.zeros(n, np.float64)}
    out["grad"] = np.zeros((n, V), np.float64) if want_grad else None
    out["gathered"] = np.zeros((n, K), np.float64) if K else None
    rc = lib().oracle_rows(ESTIMATORS[est], dtype, _p(logits), _p(teacher_logits), n, V, ld,
                           _p(ids), _p(tau), _p(beta), K, _p(mask), gamma, eps, _p(out["loss"]),
                           _p(out["grad"]), _p(out["lse"]), _p(out["gathered"]), nthreads)
    if rc != 0:
        raise ValueError("oracle_rows rejected its arguments (%d)" % rc)
    return out


def support_coverage(z, ids, tau):
    """(Z_p^S, Z_q^S) of one row in double: the student's and the teacher's
    mass on the cached support (App. A.1's restricted normalisers)."""
    z = np.ascontiguousarray(z, np.float64)
    ids = np.ascontiguousarray(ids, np.int32)
    tau = np.ascontiguousarray(tau, np.float64)
    zp, zq = np.zeros(1), np.zeros(1)
    if lib().oracle_support_coverage(_p(z), z.size, _p(ids), _p(tau), ids.size, _p(zp),
                                     _p(zq)) != 0:
        raise ValueError("oracle_support_coverage rejected its arguments")
    return float(zp[0]), float(zq[0])


def coverage_rows(dtype: int, logits: np.ndarray, V: int, ids, tau, mask=None,
                  nthreads: int = 0) -> np.ndarray:
    """[n, 2] (Z_p^S, Z_q^S) of stored rows (zeros for masked rows)."""
    logits = np.ascontiguousarray(logits)
    n, ld = logits.shape
    ids = np.ascontiguousarray(ids, np.int32)
    tau = np.ascontiguousarray(tau, np.float32)
    mask = None if mask is None else np.ascontiguousarray(mask, np.uint8)
    cov = np.zeros((n, 2), np.float64)
    rc = lib().oracle_coverage_rows(dtype, _p(logits), n, V, ld, _p(ids), _p(tau), ids.shape[1],
                                    _p(mask), _p(cov), nthreads)
    if rc != 0:
        raise ValueError("oracle_coverage_rows rejected its arguments (%d)" % rc)
    return cov


def max_threads() -> int:
    return int(lib().oracle_max_threads())


# ---------------------------------------------------------------- cache building
# Stage 1 (rollout draws and their log-probs, or a top-k support) and Stage 2
# (teacher scoring) of Sec. 4.1.

CACHE_OPS = {"sample": 0, "topk": 1, "score": 2}


def cdf(z) -> np.ndarray:
    """F[j] = sum_{l <= j} softmax(z)_l, summed in index order, in double."""
    z = np.ascontiguousarray(z, np.float64)
    F = np.zeros(z.size, np.float64)
    if lib().oracle_cdf(_p(z), z.size, _p(F)) != 0:
        raise ValueError("oracle_cdf rejected its arguments")
    return F


def sample_row(z, u):
    """Draws by inversion at float32 uniforms u.  Returns (ids, logp, lse)."""
    z = np.ascontiguousarray(z, np.float64)
    u = np.ascontiguousarray(u, np.float32)
    ids = np.zeros(u.size, np.int32)
    logp = np.zeros(u.size, np.float64)
    lse = np.zeros(1, np.float64)
    if lib().oracle_sample_row(_p(z), z.size, _p(u), u.size, _p(ids), _p(logp), _p(lse)) != 0:
        raise ValueError("oracle_sample_row rejected its arguments")
    return ids, logp, float(lse[0])


def topk_row(row, k: int, dtype: int = F32):
    """Top-k of one stored row (float32 values, or uint16 bf16 bits with dtype=BF16).
    Returns (idx, logp, lse)."""
    row = np.ascontiguousarray(row, np.uint16 if dtype == BF16 else np.float32)
    idx = np.zeros(k, np.int32)
    logp = np.zeros(k, np.float64)
    lse = np.zeros(1, np.float64)
    if lib().oracle_topk_row(dtype, _p(row), row.size, k, _p(idx), _p(logp), _p(lse)) != 0:
        raise ValueError("oracle_topk_row rejected its arguments")
    return idx, logp, float(lse[0])


def score_row(z, ids):
    """log softmax(z) at ids.  Returns (logp, lse)."""
    z = np.ascontiguousarray(z, np.float64)
    ids = np.ascontiguousarray(ids, np.int32)
    logp = np.zeros(ids.size, np.float64)
    lse = np.zeros(1, np.float64)
    if lib().oracle_score_row(_p(z), z.size, _p(ids), ids.size, _p(logp), _p(lse)) != 0:
        raise ValueError("oracle_score_row rejected its arguments")
    return logp, float(lse[0])


def cache_rows(op: str, dtype: int, logits: np.ndarray, V: int, K: int, *, uniforms=None,
               ids=None, mask=None, nthreads: int = 0) -> dict:
    """Rows of stored inputs for op "sample" (uniforms [n, K]), "topk" (K = k) or
    "score" (ids [n, K]).  Returns {"ids", "logp", "lse"}."""
    logits = np.ascontiguousarray(logits)
    n, ld = logits.shape
    if op == "score":
        out_ids = np.ascontiguousarray(ids, np.int32).copy()
    else:
        out_ids = np.zeros((n, K), np.int32)
    u = None if uniforms is None else np.ascontiguousarray(uniforms, np.float32)
    mask = None if mask is None else np.ascontiguousarray(mask, np.uint8)
    logp = np.zeros((n, K), np.float64)
    lse = np.zeros(n, np.float64)
    rc = lib().oracle_cache_rows(CACHE_OPS[op], dtype, _p(logits), n, V, ld, K, _p(u), _p(mask),
                                 _p(out_ids), _p(logp), _p(lse), nthreads)
    if rc != 0:
        raise ValueError("oracle_cache_rows rejected its arguments (%d)" % rc)
    return {"ids": out_ids, "logp": logp, "lse": lse}


# ---------------------------------------------------------------- MC diagnostics

def mc_diagnostics(lse, gathered, tau, beta, *, mask=None, q: float = 0.99, eps: float = CLIP_EPS,
                   group_sizes=(), seq_len: int = 0) -> dict:
    """Diagnostics of the MC estimator in double from per-token lse [N],
    gathered student logits, tau and beta [N, M].  Returns per-token
    "mean", "var", "rho_max" and batch "rho_quantile", "clip_frac",
    "ratio_local", "ratio_seq" (one entry per group size)."""
    lse = np.ascontiguousarray(lse, np.float64)
    gathered = np.ascontiguousarray(gathered, np.float64)
    tau = np.ascontiguousarray(tau, np.float32)
    beta = np.ascontiguousarray(beta, np.float32)
    N, M = gathered.shape
    mask = None if mask is None else np.ascontiguousarray(mask, np.uint8)
    gs = np.ascontiguousarray(group_sizes, np.int32)
    out = {"mean": np.zeros(N), "var": np.zeros(N), "rho_max": np.zeros(N),
           "rho_quantile": np.zeros(1), "clip_frac": np.zeros(1),
           "ratio_local": np.zeros(max(len(gs), 1)), "ratio_seq": np.zeros(max(len(gs), 1))}
    rc = lib().oracle_mc_diagnostics(_p(lse), _p(gathered), _p(tau), _p(beta), N, M, _p(mask), q,
                                     eps, _p(gs) if len(gs) else None, len(gs), seq_len,
                                     _p(out["mean"]), _p(out["var"]), _p(out["rho_max"]),
                                     _p(out["rho_quantile"]), _p(out["clip_frac"]),
                                     _p(out["ratio_local"]), _p(out["ratio_seq"]))
    if rc != 0:
        raise ValueError("oracle_mc_diagnostics rejected its arguments (%d)" % rc)
    out["rho_quantile"] = float(out["rho_quantile"][0])
    out["clip_frac"] = float(out["clip_frac"][0])
    out["ratio_local"] = out["ratio_local"][:len(gs)]
    out["ratio_seq"] = out["ratio_seq"][:len(gs)]
    return out
