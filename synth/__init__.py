"""Seeded synthetic inputs for the learner-time OPD loss.

This package stands in for the two pipeline stages that run before the learner
(Sec. 4.1 of the paper: student rollout, then teacher scoring).  It draws
student logits, teacher logits and stale behaviour-policy logits from one seed
with a counter-based generator (so any row can be regenerated on its own), and
builds the finite teacher-score cache from them: the teacher top-k ids with
their teacher log-probs, or M behaviour-policy samples per token (iid, with
replacement, App. E) with their teacher and behaviour log-probs.

It holds none of the learner's loss arithmetic.  Both the oracle and the GPU
library consume its outputs; it imports neither.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "opd_synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")

F32 = 0
BF16 = 1
# counter-generator streams of opd_synth.c (one per kind of draw)
STREAM_STUDENT, STREAM_BOOST, STREAM_TEACHER, STREAM_BEHAVIOUR, STREAM_SAMPLE, STREAM_LENGTH = range(1, 7)


def build(force: bool = False) -> str:
    """Compile libsynth.so in place with gcc (host code only)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"],
                       check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class SynthCfg(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("V", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("pad_", ctypes.c_int32), ("sigma_student", ctypes.c_double),
                ("boost_prob", ctypes.c_double), ("boost_value", ctypes.c_double),
                ("sigma_teacher", ctypes.c_double), ("sigma_behaviour", ctypes.c_double)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        L.synth_rows.argtypes = [ctypes.POINTER(SynthCfg), i64, i64, P, i64, P, ctypes.c_int, P, P,
                                 ctypes.c_int, P, P, P, ctypes.c_int]
        L.synth_rows.restype = ctypes.c_int
        L.synth_behaviour_row.argtypes = [ctypes.POINTER(SynthCfg), i64, P]
        L.synth_teacher_row.argtypes = [ctypes.POINTER(SynthCfg), i64, P]
        L.synth_ragged_mask.argtypes = [ctypes.c_uint64, i64, i64, i64, i64, P, P]
        L.synth_uniforms.argtypes = [ctypes.c_uint64, ctypes.c_uint64, i64, i64, P]
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, dtypes and value distributions.

    Student logits ~ N(0, sigma_student^2) (plus `boost_value` on a
    `boost_prob` fraction of entries); teacher logits = student +
    N(0, sigma_teacher^2); behaviour logits = student + N(0, sigma_behaviour^2).
    `k` > 0 builds a teacher top-k cache, `M` > 0 a Monte-Carlo cache.
    `rollout_len` > 0 with `len_lo` < `rollout_len` gives ragged right-padded
    rollouts (lengths uniform on {len_lo..len_hi}).
    """
    name: str
    N: int
    V: int
    dtype: int
    estimators: tuple
    k: int = 0
    M: int = 0
    sigma_student: float = 3.0
    boost_prob: float = 0.0
    boost_value: float = 0.0
    sigma_teacher: float = 1.0
    sigma_behaviour: float = 0.5
    dense_teacher: bool = False
    rollout_len: int = 0
    len_lo: int = 0
    len_hi: int = 0
    seed: int = 0

    def cfg(self) -> SynthCfg:
        return SynthCfg(self.seed, self.V, self.dtype, 0, self.sigma_student, self.boost_prob,
                        self.boost_value, self.sigma_teacher, self.sigma_behaviour)

    @property
    def ragged(self) -> bool:
        return self.rollout_len > 0 and self.len_lo < self.rollout_len

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads of the measurement plan.  Shapes follow the paper's
# setting: Qwen3's vocabulary (151,936 entries), rollouts of 2,048 tokens
# (App. B, Table 3), learner micro-batches of a few rollouts.
SMALL_F32 = Workload("n512_v32000_f32_topk16_mc4", N=512, V=32000, dtype=F32,
                     estimators=("fkl_topk", "rkl_topk", "rkl_mc1", "rkl_mc"), k=16, M=4,
                     sigma_student=2.0, sigma_teacher=1.0, sigma_behaviour=0.3, seed=1001)
TOPK32 = Workload("n8192_v151936_bf16_topk32_peaked", N=8192, V=151936, dtype=BF16,
                  estimators=("fkl_topk", "rkl_topk", "fkl_topk_trunc", "rkl_topk_trunc"), k=32,
                  sigma_student=3.0, boost_prob=0.01, boost_value=8.0, sigma_teacher=1.0,
                  seed=1002)
MC1_RAGGED = Workload("n32768_v151936_bf16_mc1_ragged", N=32768, V=151936, dtype=BF16,
                      estimators=("rkl_mc1",), M=1, sigma_student=3.0, sigma_teacher=1.0,
                      sigma_behaviour=0.5, rollout_len=2048, len_lo=256, len_hi=2048, seed=1003)
MC16 = Workload("n32768_v151936_bf16_mc16", N=32768, V=151936, dtype=BF16,
                estimators=("rkl_mc", "rkl_mc_clip", "rkl_mc_old", "rkl_mc_old_clip", "rkl_mc_nois"),
                M=16, sigma_student=3.0, sigma_teacher=1.0, sigma_behaviour=0.5, seed=1004)
MC16_SMALLN = MC16.replace(name="n256_v151936_bf16_mc16_smallbatch", N=256, estimators=("rkl_mc",))
DENSE = Workload("n16384_v151936_bf16_dense", N=16384, V=151936, dtype=BF16,
                 estimators=("fkl_dense", "rkl_dense"), sigma_student=3.0, sigma_teacher=1.0,
                 dense_teacher=True, seed=1005)

WORKLOADS = {w.name: w for w in (SMALL_F32, TOPK32, MC1_RAGGED, MC16, MC16_SMALLN, DENSE)}


def generate(w: Workload, r0: int = 0, r1: Optional[int] = None, *, ld: Optional[int] = None,
             logits: bool = True, nthreads: int = 0) -> dict:
    """Rows [r0, r1) of workload `w` as numpy arrays.

    Keys: "logits" ([n, ld] uint16 bf16 bits or float32), "teacher_logits"
    (dense workloads), "topk_idx"/"topk_tau" (k > 0), "mc_ids"/"mc_tau"/
    "mc_beta" (M > 0), "mask" (uint8, all ones unless ragged).
    """
    if r1 is None:
        r1 = w.N
    n = r1 - r0
    ld = w.V if ld is None else ld
    et = np.uint16 if w.dtype == BF16 else np.float32
    out = {}
    lg = np.zeros((n, ld), et) if logits else None
    tl = np.zeros((n, ld), et) if w.dense_teacher else None
    ti = tt = mi = mt = mb = None
    if w.k > 0:
        ti = np.empty((n, w.k), np.int32)
        tt = np.empty((n, w.k), np.float32)
    if w.M > 0:
        mi = np.empty((n, w.M), np.int32)
        mt = np.empty((n, w.M), np.float32)
        mb = np.empty((n, w.M), np.float32)
    c = w.cfg()
    rc = lib().synth_rows(ctypes.byref(c), r0, r1, _ptr(lg), ld, _ptr(tl), w.k, _ptr(ti), _ptr(tt),
                          w.M, _ptr(mi), _ptr(mt), _ptr(mb), nthreads)
    if rc != 0:
        raise RuntimeError("synth_rows failed with code %d" % rc)
    if lg is not None:
        out["logits"] = lg
    if tl is not None:
        out["teacher_logits"] = tl
    if w.k > 0:
        out["topk_idx"], out["topk_tau"] = ti, tt
    if w.M > 0:
        out["mc_ids"], out["mc_tau"], out["mc_beta"] = mi, mt, mb
    out["mask"] = mask(w)[r0:r1]
    return out


def mask(w: Workload) -> np.ndarray:
    """The [N] uint8 padding mask of `w` (ones unless the workload is ragged)."""
    if not w.ragged:
        return np.ones(w.N, np.uint8)
    n_roll = w.N // w.rollout_len
    m = np.empty(n_roll * w.rollout_len, np.uint8)
    rc = lib().synth_ragged_mask(w.seed, n_roll, w.rollout_len, w.len_lo, w.len_hi, _ptr(m), None)
    if rc != 0:
        raise RuntimeError("synth_ragged_mask failed with code %d" % rc)
    out = np.zeros(w.N, np.uint8)
    out[: m.size] = m
    return out


def behaviour_row(w: Workload, row: int) -> np.ndarray:
    """Unrounded behaviour logits b of one row (float64), for tests."""
    b = np.empty(w.V, np.float64)
    c = w.cfg()
    if lib().synth_behaviour_row(ctypes.byref(c), row, _ptr(b)) != 0:
        raise RuntimeError("synth_behaviour_row failed")
    return b


def teacher_row(w: Workload, row: int) -> np.ndarray:
    """Teacher logits y of one row as stored (float64 holding dtype values)."""
    y = np.empty(w.V, np.float64)
    c = w.cfg()
    if lib().synth_teacher_row(ctypes.byref(c), row, _ptr(y)) != 0:
        raise RuntimeError("synth_teacher_row failed")
    return y


def uniforms(seed: int, stream: int, row: int, n: int) -> np.ndarray:
    u = np.empty(n, np.float64)
    lib().synth_uniforms(seed, stream, row, n, _ptr(u))
    return u


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


def as_f64(w: Workload, a: np.ndarray) -> np.ndarray:
    """Stored logits (either dtype) as exact float64 values."""
    if w.dtype == BF16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)
