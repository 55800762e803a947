"""The C ABI without a GPU: the library loads, exports every symbol the
header declares, and rejects every argument error before touching the device.

Each error case below has exactly one invalid argument and never reaches a
launch (the pointers are placeholders and are never dereferenced)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2606_24143_amd as opd
from paper_2606_24143_amd._binding import OpdCache, OpdOpts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "opd.h")

OK, NULL, SHAPE, SUPPORT, DTYPE, ALIGN, WORKSPACE, ESTIMATOR, FLAGS = 0, -1, -2, -3, -4, -5, -6, -7, -8
PARAM = -10
FAKE = 0x10000  # 16-byte aligned placeholder address, never dereferenced


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\**(opd_[a-z_]+)\(", text,
                                 re.M)))


def test_library_loads_and_exports_every_declared_symbol():
    L = opd.lib()
    declared = header_functions()
    assert declared == sorted(opd.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name
    dyn = subprocess.run(["nm", "-D", "--defined-only", opd.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (opd_[a-z_]+)$", dyn, re.M))
    assert set(declared) <= exported


def test_version_matches_header():
    m = re.search(r"#define OPD_VERSION (\d+)", open(HEADER).read())
    assert opd.version() == int(m.group(1))


def test_status_strings():
    for code in range(-11, 1):
        s = opd.status_string(code)
        assert s and s != "unknown status"
    assert opd.status_string(-100) == "unknown status"


def call(logits=FAKE, dtype=1, N=4, V=1024, ld=None, cache="mc", est=3, k=16, M=4, mask=None,
         opts=None, loss=FAKE, dlogits=FAKE, lse=None, gathered=None, coverage=None, ws=None,
         ws_bytes=0):
    ld = V if ld is None else ld
    if cache == "mc":
        c = OpdCache(None, FAKE, FAKE, FAKE, None)
    elif cache == "topk":
        c = OpdCache(FAKE, None, FAKE, None, None)
    elif cache == "dense":
        c = OpdCache(None, None, None, None, FAKE)
    else:
        c = cache
    cp = None if c is None else ctypes.byref(c)
    op = None if opts is None else ctypes.byref(opts)
    return opd.lib().opd_loss_fwd_bwd(logits, dtype, N, V, ld, cp, est, k, M, mask, op, loss,
                                      dlogits, lse, gathered, coverage, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(est=12), ESTIMATOR),
    (dict(est=10, cache="topk", k=0), SUPPORT),
    (dict(est=11, cache=OpdCache(None, FAKE, FAKE, FAKE, None)), NULL),
    (dict(est=-1), ESTIMATOR),
    (dict(dtype=2), DTYPE),
    (dict(opts=OpdOpts(1.0, 7, 0)), DTYPE),
    (dict(opts=OpdOpts(1.0, 0, 64)), FLAGS),
    (dict(opts=OpdOpts(1.0, 0, 2 | 4)), FLAGS),
    (dict(N=-1), SHAPE),
    (dict(N=2 ** 31), SHAPE),
    (dict(V=1), SHAPE),
    (dict(V=2 ** 31), SHAPE),
    (dict(ld=1000), SHAPE),
    (dict(est=3, M=0), SUPPORT),
    (dict(est=3, M=257), SUPPORT),
    (dict(est=2, M=2), SUPPORT),
    (dict(est=0, cache="topk", k=0), SUPPORT),
    (dict(est=1, cache="topk", k=257, V=4096), SUPPORT),
    (dict(est=0, cache="topk", k=9, V=8), SUPPORT),
    (dict(logits=None), NULL),
    (dict(loss=None), NULL),
    (dict(dlogits=None), NULL),
    (dict(cache=None), NULL),
    (dict(cache=OpdCache(None, None, FAKE, FAKE, None)), NULL),
    (dict(cache=OpdCache(None, FAKE, None, FAKE, None)), NULL),
    (dict(cache=OpdCache(None, FAKE, FAKE, None, None)), NULL),
    (dict(est=0, cache=OpdCache(None, FAKE, FAKE, FAKE, None)), NULL),
    (dict(est=1, cache=OpdCache(FAKE, None, None, None, None)), NULL),
    (dict(est=4, cache=OpdCache(FAKE, FAKE, FAKE, FAKE, None)), NULL),
    (dict(logits=FAKE + 2), ALIGN),
    (dict(dlogits=FAKE + 8), ALIGN),
    (dict(est=5, cache=OpdCache(None, None, None, None, FAKE + 4)), ALIGN),
    (dict(V=1020), ALIGN),                       # bf16 rows of 2040 bytes
    (dict(dtype=0, V=1022), ALIGN),              # fp32 rows of 4088 bytes
    (dict(dtype=0, V=1020, opts=OpdOpts(1.0, 1, 0)), ALIGN),  # bf16 gradient rows of 2040 bytes
    (dict(est=6, opts=OpdOpts(1.0, 0, 0, 0.0)), PARAM),     # clipped surrogate, eps = 0
    (dict(est=8, opts=OpdOpts(1.0, 0, 0, -0.2)), PARAM),
    (dict(est=6, opts=OpdOpts(1.0, 0, 0, float("inf"))), PARAM),
    (dict(est=7, cache=OpdCache(None, FAKE, FAKE, None, None)), NULL),  # A_old needs behav_logp
    (dict(est=9, M=0), SUPPORT),
    (dict(coverage=FAKE), PARAM),                # coverage needs a cached support (MC here)
    (dict(est=4, cache="dense", coverage=FAKE), PARAM),
    (dict(N=8, opts=OpdOpts(1.0, 0, 4)), WORKSPACE),  # split path forced, no workspace
    (dict(N=8, opts=OpdOpts(1.0, 0, 4), ws=FAKE, ws_bytes=16), WORKSPACE),
])
def test_argument_errors_are_reported_before_launch(kw, code):
    assert call(**kw) == code


def test_zero_rows_is_a_noop():
    assert call(N=0, logits=None, loss=None, dlogits=None, cache=None) == OK


def test_workspace_sizing():
    L = opd.lib()
    ws = L.opd_workspace_bytes
    # small N takes the split path: N * P * 8 floats
    b = ws(48, 151936, 1, 3, 0, 16, 0)
    assert b > 0 and b % (48 * 32) == 0
    P = b // (48 * 32)
    assert 1 <= P <= 64
    # from 64 rows, or forced row-wise: none
    assert ws(64, 151936, 1, 3, 0, 16, 0) == 0
    assert ws(256, 151936, 1, 3, 0, 16, 0) == 0
    assert ws(32768, 151936, 1, 3, 0, 16, 0) == 0
    assert ws(48, 151936, 1, 3, 0, 16, 2) == 0
    # forced split at large N
    assert ws(32768, 151936, 1, 3, 0, 16, 4) > 0
    # invalid arguments: 0
    assert ws(256, 1, 1, 3, 0, 16, 0) == 0
    assert ws(256, 151936, 1, 9, 0, 16, 0) == 0
    assert ws(0, 151936, 1, 3, 0, 16, 0) == 0


def test_validate_cache_argument_errors():
    L = opd.lib()
    c = OpdCache(FAKE, None, FAKE, None, None)
    assert L.opd_validate_cache(ctypes.byref(c), 12, 4, 100, 4, 0, FAKE, None) == ESTIMATOR
    assert L.opd_validate_cache(ctypes.byref(c), 0, 4, 1, 4, 0, FAKE, None) == SHAPE
    assert L.opd_validate_cache(ctypes.byref(c), 0, 4, 100, 0, 0, FAKE, None) == SUPPORT
    assert L.opd_validate_cache(ctypes.byref(c), 0, 4, 100, 4, 0, None, None) == NULL
    assert L.opd_validate_cache(None, 0, 4, 100, 4, 0, FAKE, None) == NULL
    assert L.opd_validate_cache(ctypes.byref(c), 3, 4, 100, 0, 4, FAKE, None) == NULL
    assert L.opd_validate_cache(ctypes.byref(c), 4, 4, 100, 0, 0, FAKE, None) == OK  # dense: no-op


# ---------------------------------------------------------------- cache building

def call_row(op, logits=FAKE, dtype=1, N=4, V=1024, ld=None, K=4, u=FAKE, ids=FAKE, mask=None,
             out=FAKE, logp=FAKE, lse=None):
    ld = V if ld is None else ld
    L = opd.lib()
    if op == "sample":
        return L.opd_sample_actions(logits, dtype, N, V, ld, K, u, mask, out, logp, lse, None)
    if op == "topk":
        return L.opd_topk_support(logits, dtype, N, V, ld, K, mask, out, logp, lse, None)
    return L.opd_score_actions(logits, dtype, N, V, ld, ids, K, mask, logp, lse, None)


@pytest.mark.parametrize("op", ["sample", "topk", "score"])
@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), DTYPE),
    (dict(dtype=-1), DTYPE),
    (dict(N=-1), SHAPE),
    (dict(N=2 ** 31), SHAPE),
    (dict(V=1), SHAPE),
    (dict(V=2 ** 31), SHAPE),
    (dict(ld=1000), SHAPE),
    (dict(K=0), SUPPORT),
    (dict(K=257), SUPPORT),
    (dict(logits=None), NULL),
    (dict(logits=FAKE + 2), ALIGN),
    (dict(V=1020), ALIGN),                  # bf16 rows of 2040 bytes
    (dict(dtype=0, V=1022), ALIGN),         # fp32 rows of 4088 bytes
])
def test_cache_argument_errors_are_reported_before_launch(op, kw, code):
    assert call_row(op, **kw) == code


@pytest.mark.parametrize("op,kw,code", [
    ("sample", dict(u=None), NULL),
    ("sample", dict(out=None), NULL),
    ("sample", dict(K=300, V=100000), SUPPORT),   # M is limited to 256 draws
    ("topk", dict(out=None), NULL),
    ("topk", dict(K=9, V=8), SUPPORT),            # k > V
    ("score", dict(ids=None), NULL),
    ("score", dict(logp=None), NULL),
])
def test_cache_required_pointers_and_sizes(op, kw, code):
    assert call_row(op, **kw) == code


@pytest.mark.parametrize("op", ["sample", "topk", "score"])
def test_cache_zero_rows_is_a_noop(op):
    assert call_row(op, N=0, logits=None, u=None, ids=None, out=None, logp=None) == OK


# ---------------------------------------------------------------- MC diagnostics

def call_diag(N=4, M=8, q=0.99, eps=0.2, groups=(2, 4), seq=0, out=True, ws=FAKE,
              ws_bytes=1 << 30, ptrs=(FAKE, FAKE, FAKE, FAKE)):
    gs = (ctypes.c_int32 * max(len(groups), 1))(*groups)
    st = opd.OpdMcDiag(FAKE, None, None, None, None, None, None) if out else None
    L = opd.lib()
    return L.opd_mc_diagnostics(*ptrs, N, M, None, q, eps, gs, len(groups), seq,
                                ctypes.byref(st) if st else None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(N=-1), SHAPE),
    (dict(M=0), SUPPORT),
    (dict(M=257), SUPPORT),
    (dict(q=0.0), PARAM),
    (dict(q=1.5), PARAM),
    (dict(q=float("nan")), PARAM),
    (dict(eps=-0.1), PARAM),
    (dict(eps=float("inf")), PARAM),
    (dict(groups=(3,)), PARAM),           # 3 does not divide 8
    (dict(groups=(8,)), PARAM),           # a single group has no variance
    (dict(groups=(0,)), PARAM),
    (dict(groups=(1,) * 9), PARAM),       # at most 8 group sizes
    (dict(seq=-1), PARAM),
    (dict(out=False), NULL),
    (dict(ptrs=(None, FAKE, FAKE, FAKE)), NULL),
    (dict(ptrs=(FAKE, FAKE, FAKE, None)), NULL),
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=16), WORKSPACE),
    (dict(ws=FAKE + 4), WORKSPACE),
])
def test_diag_argument_errors_are_reported_before_launch(kw, code):
    assert call_diag(**kw) == code


def test_diag_ratio_seq_needs_seq_len():
    gs = (ctypes.c_int32 * 1)(2)
    st = opd.OpdMcDiag(None, None, None, None, None, None, FAKE)
    L = opd.lib()
    assert L.opd_mc_diagnostics(FAKE, FAKE, FAKE, FAKE, 4, 8, None, 0.99, 0.2, gs, 1, 0,
                                ctypes.byref(st), FAKE, 1 << 30, None) == PARAM


def test_diag_workspace_sizing():
    L = opd.lib()
    gs = (ctypes.c_int32 * 3)(2, 4, 8)
    a = L.opd_mc_diag_workspace_bytes(32768, 16, gs, 3, 0)
    b = L.opd_mc_diag_workspace_bytes(32768, 16, gs, 3, 2048)
    assert 32768 * 16 * 4 < a < b          # the sequence ratios add replicate columns
    assert L.opd_mc_diag_workspace_bytes(32768, 16, gs, 3, -1) == 0
    assert L.opd_mc_diag_workspace_bytes(4, 0, gs, 0, 0) == 0
    assert call_diag(N=0, ptrs=(None, None, None, None), ws=None) == OK
