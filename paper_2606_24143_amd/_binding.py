"""ctypes binding over libopd.so (the C ABI declared in include/opd.h).

Argument marshalling only: this module turns torch tensors into device
pointers, sizes and a HIP stream, allocates the output buffers, and raises on
a non-zero status.  Every step of the computation runs in the library's HIP
kernels.  There is no fallback: if libopd.so is missing or a GPU is absent,
calls fail loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libopd.so")

# opd_estimator, opd_dtype, flags (include/opd.h)
ESTIMATORS = {"fkl_topk": 0, "rkl_topk": 1, "rkl_mc1": 2, "rkl_mc": 3, "fkl_dense": 4,
              "rkl_dense": 5, "rkl_mc_clip": 6, "rkl_mc_old": 7, "rkl_mc_old_clip": 8,
              "rkl_mc_nois": 9, "fkl_topk_trunc": 10, "rkl_topk_trunc": 11}
# estimators that read the top-k cache (idx, k)
TOPK = ("fkl_topk", "rkl_topk", "fkl_topk_trunc", "rkl_topk_trunc")
DENSE = ("fkl_dense", "rkl_dense")
F32, BF16 = 0, 1
FLAG_SKIP_MASKED = 1
FLAG_FORCE_ROWWISE = 2
FLAG_FORCE_SPLITV = 4
K_MAX = 256

STATUS = {0: "OPD_OK", -1: "OPD_ERR_NULL", -2: "OPD_ERR_SHAPE", -3: "OPD_ERR_SUPPORT",
          -4: "OPD_ERR_DTYPE", -5: "OPD_ERR_ALIGN", -6: "OPD_ERR_WORKSPACE",
          -7: "OPD_ERR_ESTIMATOR", -8: "OPD_ERR_FLAGS", -9: "OPD_ERR_HIP", -10: "OPD_ERR_PARAM",
          -11: "OPD_ERR_SCRATCH"}

# every symbol include/opd.h declares
EXPORTS = ("opd_loss_fwd_bwd", "opd_loss_fwd_bwd_noalloc", "opd_noalloc_scratch_bytes",
           "opd_workspace_bytes", "opd_validate_cache", "opd_sample_actions",
           "opd_topk_support", "opd_score_actions", "opd_mc_diag_workspace_bytes",
           "opd_mc_diagnostics", "opd_status_string", "opd_version")


class OpdError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.status = STATUS.get(code, str(code))
        super().__init__("%s failed: %s (%s)" % (where, self.status, status_string(code)))


class OpdCache(ctypes.Structure):
    _fields_ = [("idx", ctypes.c_void_p), ("sampled_ids", ctypes.c_void_p),
                ("teacher_logp", ctypes.c_void_p), ("behav_logp", ctypes.c_void_p),
                ("teacher_logits", ctypes.c_void_p)]


class OpdOpts(ctypes.Structure):
    _fields_ = [("grad_scale", ctypes.c_float), ("dlogits_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("clip_eps", ctypes.c_float)]


class OpdMcDiag(ctypes.Structure):
    _fields_ = [("row_mean", ctypes.c_void_p), ("row_var", ctypes.c_void_p),
                ("row_rho_max", ctypes.c_void_p), ("rho_quantile", ctypes.c_void_p),
                ("clip_frac", ctypes.c_void_p), ("ratio_local", ctypes.c_void_p),
                ("ratio_seq", ctypes.c_void_p)]


_lib = None


def lib():
    """Load libopd.so (built by __graft_entry__.build() or paper_2606_24143_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libopd.so is not built at %s; run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.opd_loss_fwd_bwd.argtypes = [P, i32, i64, i64, i64, ctypes.POINTER(OpdCache), i32, i32,
                                       i32, P, ctypes.POINTER(OpdOpts), P, P, P, P, P, P,
                                       ctypes.c_size_t, P]
        L.opd_loss_fwd_bwd.restype = ctypes.c_int
        L.opd_loss_fwd_bwd_noalloc.argtypes = [P, i32, i64, i64, i64, ctypes.POINTER(OpdCache),
                                               i32, i32, i32, P, ctypes.POINTER(OpdOpts), P, P,
                                               P, P, P, P]
        L.opd_loss_fwd_bwd_noalloc.restype = ctypes.c_int
        L.opd_noalloc_scratch_bytes.argtypes = []
        L.opd_noalloc_scratch_bytes.restype = ctypes.c_size_t
        L.opd_workspace_bytes.argtypes = [i64, i64, i32, i32, i32, i32, ctypes.c_uint32]
        L.opd_workspace_bytes.restype = ctypes.c_size_t
        L.opd_validate_cache.argtypes = [ctypes.POINTER(OpdCache), i32, i64, i64, i32, i32, P, P]
        L.opd_validate_cache.restype = ctypes.c_int
        L.opd_sample_actions.argtypes = [P, i32, i64, i64, i64, i32, P, P, P, P, P, P]
        L.opd_sample_actions.restype = ctypes.c_int
        L.opd_topk_support.argtypes = [P, i32, i64, i64, i64, i32, P, P, P, P, P]
        L.opd_topk_support.restype = ctypes.c_int
        L.opd_score_actions.argtypes = [P, i32, i64, i64, i64, P, i32, P, P, P, P]
        L.opd_score_actions.restype = ctypes.c_int
        L.opd_mc_diag_workspace_bytes.argtypes = [i64, i32, P, i32, i64]
        L.opd_mc_diag_workspace_bytes.restype = ctypes.c_size_t
        L.opd_mc_diagnostics.argtypes = [P, P, P, P, i64, i32, P, ctypes.c_float, ctypes.c_float,
                                         P, i32, i64, ctypes.POINTER(OpdMcDiag), P,
                                         ctypes.c_size_t, P]
        L.opd_mc_diagnostics.restype = ctypes.c_int
        L.opd_status_string.argtypes = [ctypes.c_int]
        L.opd_status_string.restype = ctypes.c_char_p
        L.opd_version.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().opd_status_string(code).decode()


def version() -> int:
    return int(lib().opd_version())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError("logits must be float32 or bfloat16, got %s" % t.dtype)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _rowmajor(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor) or t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("%s must be a 2-D tensor with unit column stride" % name)


def _need(t, name: str, dtypes, shape, device=None):
    """t must be a contiguous tensor of one of `dtypes` with exactly `shape`
    (and, when given, on `device`): the library reads and writes it as a dense
    row-major array of that element type."""
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if t.dtype not in dtypes:
        raise ValueError("%s must have dtype %s, got %s" %
                         (name, " or ".join(str(d) for d in dtypes), t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the logits on %s" % (name, t.device, device))


def _need_rows(t, name: str, dtype, N: int, V: int, ld: int, device=None):
    """t must be an [N, >= V] tensor of `dtype` whose rows lie `ld` elements
    apart with unit column stride: the library addresses row r at r * ld."""
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must have dtype %s, got %s" % (name, dtype, t.dtype))
    if t.dim() != 2 or t.shape[0] != N or t.shape[1] < V:
        raise ValueError("%s must have shape [%d, >= %d], got %s" % (name, N, V, tuple(t.shape)))
    if N > 0 and (t.stride(1) != 1 or (N > 1 and t.stride(0) != ld)):
        raise ValueError("%s must have row stride %d and unit column stride, got strides %s" %
                         (name, ld, tuple(t.stride())))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the logits on %s" % (name, t.device, device))


_MASK_DTYPES = (torch.uint8, torch.bool)


def _need_gpu(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor (the library runs HIP kernels only)" % name)


def workspace_bytes(N: int, V: int, dtype: int, estimator: str, k: int = 0, M: int = 0,
                    flags: int = 0) -> int:
    return int(lib().opd_workspace_bytes(N, V, dtype, ESTIMATORS[estimator], k, M, flags))


class PreparedCall:
    """A library call whose arguments were checked and marshalled once.

    Calling it issues the same C call again: the same tensors, options and
    stream (the one given, or the current one, at preparation).  It checks
    nothing and allocates nothing, so a loop that repeats one call on the
    same buffers pays only for the foreign call.  `outputs` holds the result
    tensors the call writes; the prepared object keeps every tensor it was
    prepared with alive.
    """
    __slots__ = ("_fn", "_args", "_name", "_keep", "outputs")

    def __init__(self, fn, args, name, keep, outputs):
        self._fn, self._args, self._name, self._keep = fn, args, name, keep
        self.outputs = outputs

    def __call__(self):
        rc = self._fn(*self._args)
        if rc != 0:
            raise OpdError(rc, self._name)
        return self.outputs


def loss_fwd_bwd(logits: torch.Tensor, estimator: str, **kw):
    """One fused forward+backward call of opd_loss_fwd_bwd.

    logits: [N, V] device tensor (a row-strided view of an [N, ld] buffer is
    fine).  Cache tensors are [N, k] / [N, M] device tensors.  Returns a dict
    with "loss" [N], "dlogits" [N, V] (a view of the [N, ld] buffer), and
    "lse" / "gathered" / "coverage" ([N, 2]: Z_p^S, Z_q^S; estimators with a
    cached support only) when requested.  The keyword arguments are those of
    prepare_loss_fwd_bwd.
    """
    return prepare_loss_fwd_bwd(logits, estimator, **kw)()


def prepare_loss_fwd_bwd(logits: torch.Tensor, estimator: str, *, idx=None, sampled_ids=None,
                         teacher_logp=None, behav_logp=None, teacher_logits=None, mask=None,
                         grad_scale: float = 1.0, dlogits_dtype=torch.float32, flags: int = 0,
                         clip_eps: float = 0.2, want_lse: bool = False,
                         want_gathered: bool = False, want_coverage: bool = False,
                         workspace=None, out=None, stream=None,
                         no_alloc: bool = False) -> PreparedCall:
    """The checks, output allocation and marshalling of one opd_loss_fwd_bwd
    call, returned as a PreparedCall (nothing is launched until it is
    called; its `outputs` are loss_fwd_bwd's result dict).

    The arguments are loss_fwd_bwd's.  `workspace=None` allocates what the
    split path needs; pass a tensor to supply your own (or an empty one to
    force the row-per-workgroup path).  `out` may hold preallocated "loss"
    and "dlogits" ([N, ld]) tensors.  `no_alloc=True` calls
    opd_loss_fwd_bwd_noalloc instead, whose split path uses the library's
    static scratch (no workspace is allocated or passed).
    """
    if estimator not in ESTIMATORS:
        raise ValueError("unknown estimator %r" % (estimator,))
    est = ESTIMATORS[estimator]
    _rowmajor(logits, "logits")
    N, V = logits.shape
    ld = logits.stride(0) if N > 1 else V
    dev = logits.device
    dt = _dt(logits)
    if dlogits_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("dlogits_dtype must be torch.float32 or torch.bfloat16")
    odt = {torch.float32: F32, torch.bfloat16: BF16}[dlogits_dtype]
    ids = idx if estimator in TOPK else sampled_ids
    if estimator in DENSE:
        if teacher_logits is None:
            raise ValueError("%s needs teacher_logits" % estimator)
        _need_rows(teacher_logits, "teacher_logits", logits.dtype, N, V, ld, dev)
    else:
        if ids is None or teacher_logp is None:
            raise ValueError("%s needs %s and teacher_logp" %
                             (estimator, "idx" if estimator in TOPK else "sampled_ids"))
        if ids.dim() != 2:
            raise ValueError("%s must be a 2-D [N, K] tensor" %
                             ("idx" if estimator in TOPK else "sampled_ids"))
        K = int(ids.shape[1])
        _need(ids, "idx" if estimator in TOPK else "sampled_ids", (torch.int32,), (N, K), dev)
        _need(teacher_logp, "teacher_logp", (torch.float32,), (N, K), dev)
        if behav_logp is not None:
            _need(behav_logp, "behav_logp", (torch.float32,), (N, K), dev)
    k = int(idx.shape[1]) if estimator in TOPK else 0
    M = int(sampled_ids.shape[1]) if ids is not None and estimator not in TOPK else 0
    if mask is not None:
        _need(mask, "mask", _MASK_DTYPES, (N,), dev)
    if workspace is not None:
        _need(workspace, "workspace", (torch.uint8,), (workspace.numel(),), dev)
    if out is not None:
        loss, dbuf = out["loss"], out["dlogits"]
        _need(loss, "out['loss']", (torch.float32,), (N,), dev)
        _need_rows(dbuf, "out['dlogits']", dlogits_dtype, N, V, ld, dev)
    else:
        loss = dbuf = None
    _need_gpu(logits, "logits")
    cache = OpdCache(_ptr(idx) if estimator in TOPK else None,
                     _ptr(sampled_ids) if estimator not in TOPK and estimator not in DENSE else None,
                     _ptr(teacher_logp), _ptr(behav_logp), _ptr(teacher_logits))
    opts = OpdOpts(grad_scale, odt, flags, clip_eps)
    if out is None:
        loss = torch.empty(N, dtype=torch.float32, device=dev)
        dbuf = torch.empty((N, ld), dtype=dlogits_dtype, device=dev)
    lse = torch.empty(N, dtype=torch.float32, device=dev) if want_lse else None
    K = k if estimator in TOPK else M
    gathered = (torch.empty((N, max(K, 1)), dtype=torch.float32, device=dev)
                if want_gathered and estimator not in DENSE else None)
    if want_coverage and estimator not in TOPK:
        raise ValueError("support coverage exists for the estimators with a cached support only")
    coverage = torch.empty((N, 2), dtype=torch.float32, device=dev) if want_coverage else None
    keep = (logits, idx, sampled_ids, teacher_logp, behav_logp, teacher_logits, mask, loss, dbuf,
            lse, gathered, coverage, cache, opts)
    if no_alloc:
        fn, name = lib().opd_loss_fwd_bwd_noalloc, "opd_loss_fwd_bwd_noalloc"
        args = (_ptr(logits), dt, N, V, ld, ctypes.byref(cache), est, k, M, _ptr(mask),
                ctypes.byref(opts), _ptr(loss), _ptr(dbuf), _ptr(lse), _ptr(gathered),
                _ptr(coverage), _stream(stream))
    else:
        if workspace is None:
            nbytes = workspace_bytes(N, V, dt, estimator, k, M, flags)
            workspace = (torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
                         if nbytes else None)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        fn, name = lib().opd_loss_fwd_bwd, "opd_loss_fwd_bwd"
        args = (_ptr(logits), dt, N, V, ld, ctypes.byref(cache), est, k, M, _ptr(mask),
                ctypes.byref(opts), _ptr(loss), _ptr(dbuf), _ptr(lse), _ptr(gathered),
                _ptr(coverage), _ptr(workspace) if ws_bytes else None, ws_bytes, _stream(stream))
        keep = keep + (workspace,)
    res = {"loss": loss, "dlogits": dbuf[:, :V]}
    if lse is not None:
        res["lse"] = lse
    if gathered is not None:
        res["gathered"] = gathered[:, :K]
    if coverage is not None:
        res["coverage"] = coverage
    return PreparedCall(fn, args, name, keep, res)


def validate_cache(estimator: str, V: int, *, idx=None, sampled_ids=None, teacher_logp=None,
                   behav_logp=None, stream=None) -> int:
    """Number of cache entries violating the estimator's preconditions (synchronises)."""
    ids = idx if idx is not None else sampled_ids
    if not isinstance(ids, torch.Tensor) or ids.dim() != 2:
        raise ValueError("validate_cache needs idx or sampled_ids as an [N, K] int32 tensor")
    N, K = ids.shape
    dev = ids.device
    _need(ids, "idx" if idx is not None else "sampled_ids", (torch.int32,), (N, K), dev)
    if teacher_logp is not None:
        _need(teacher_logp, "teacher_logp", (torch.float32,), (N, K), dev)
    if behav_logp is not None:
        _need(behav_logp, "behav_logp", (torch.float32,), (N, K), dev)
    _need_gpu(ids, "ids")
    counter = torch.zeros(1, dtype=torch.int32, device=dev)
    cache = OpdCache(_ptr(idx), _ptr(sampled_ids), _ptr(teacher_logp), _ptr(behav_logp), None)
    k = K if estimator in TOPK else 0
    M = K if estimator not in TOPK and estimator not in DENSE else 0
    rc = lib().opd_validate_cache(ctypes.byref(cache), ESTIMATORS[estimator], N, V, k, M,
                                  _ptr(counter), _stream(stream))
    if rc != 0:
        raise OpdError(rc, "opd_validate_cache")
    return int(counter.item())


# ---------------------------------------------------------------- building the cache

def _row_call(logits: torch.Tensor, mask=None):
    _rowmajor(logits, "logits")
    N, V = logits.shape
    ld = logits.stride(0) if N > 1 else V
    dt = _dt(logits)
    if mask is not None:
        _need(mask, "mask", _MASK_DTYPES, (N,), logits.device)
    return N, V, ld, dt


def sample_actions(logits: torch.Tensor, uniforms: torch.Tensor, *, mask=None,
                   want_logp: bool = True, want_lse: bool = False, stream=None) -> dict:
    """M draws per row from softmax(logits) by inversion at the given uniforms
    ([N, M] float32 in [0, 1)).  Returns {"ids" [N, M] int32, "logp" [N, M]
    (log-probs at the draws), "lse" [N] when requested}."""
    N, V, ld, dt = _row_call(logits, mask)
    if not isinstance(uniforms, torch.Tensor) or uniforms.dim() != 2:
        raise ValueError("uniforms must be a contiguous [N, M] float32 tensor")
    M = int(uniforms.shape[1])
    _need(uniforms, "uniforms", (torch.float32,), (N, M), logits.device)
    _need_gpu(logits, "logits")
    dev = logits.device
    ids = torch.empty((N, M), dtype=torch.int32, device=dev)
    logp = torch.empty((N, M), dtype=torch.float32, device=dev) if want_logp else None
    lse = torch.empty(N, dtype=torch.float32, device=dev) if want_lse else None
    rc = lib().opd_sample_actions(_ptr(logits), dt, N, V, ld, M, _ptr(uniforms), _ptr(mask),
                                  _ptr(ids), _ptr(logp), _ptr(lse), _stream(stream))
    if rc != 0:
        raise OpdError(rc, "opd_sample_actions")
    out = {"ids": ids}
    if logp is not None:
        out["logp"] = logp
    if lse is not None:
        out["lse"] = lse
    return out


def topk_support(logits: torch.Tensor, k: int, *, mask=None, want_logp: bool = True,
                 want_lse: bool = False, stream=None) -> dict:
    """The k largest logits per row (descending, ties by lower index).  Returns
    {"idx" [N, k] int32, "logp" [N, k], "lse" [N] when requested}."""
    N, V, ld, dt = _row_call(logits, mask)
    _need_gpu(logits, "logits")
    dev = logits.device
    idx = torch.empty((N, k), dtype=torch.int32, device=dev)
    logp = torch.empty((N, k), dtype=torch.float32, device=dev) if want_logp else None
    lse = torch.empty(N, dtype=torch.float32, device=dev) if want_lse else None
    rc = lib().opd_topk_support(_ptr(logits), dt, N, V, ld, k, _ptr(mask), _ptr(idx), _ptr(logp),
                                _ptr(lse), _stream(stream))
    if rc != 0:
        raise OpdError(rc, "opd_topk_support")
    out = {"idx": idx}
    if logp is not None:
        out["logp"] = logp
    if lse is not None:
        out["lse"] = lse
    return out


def score_actions(logits: torch.Tensor, ids: torch.Tensor, *, mask=None, want_lse: bool = False,
                  stream=None) -> dict:
    """log softmax(logits) at ids ([N, K] int32).  Returns {"logp" [N, K], "lse"}."""
    N, V, ld, dt = _row_call(logits, mask)
    if not isinstance(ids, torch.Tensor) or ids.dim() != 2:
        raise ValueError("ids must be a contiguous [N, K] int32 tensor")
    K = int(ids.shape[1])
    _need(ids, "ids", (torch.int32,), (N, K), logits.device)
    _need_gpu(logits, "logits")
    dev = logits.device
    logp = torch.empty((N, K), dtype=torch.float32, device=dev)
    lse = torch.empty(N, dtype=torch.float32, device=dev) if want_lse else None
    rc = lib().opd_score_actions(_ptr(logits), dt, N, V, ld, _ptr(ids), K, _ptr(mask), _ptr(logp),
                                 _ptr(lse), _stream(stream))
    if rc != 0:
        raise OpdError(rc, "opd_score_actions")
    out = {"logp": logp}
    if lse is not None:
        out["lse"] = lse
    return out


# ---------------------------------------------------------------- MC diagnostics

DIAG_OUTPUTS = ("row_mean", "row_var", "row_rho_max", "rho_quantile", "clip_frac", "ratio_local",
                "ratio_seq")


def mc_diagnostics(lse: torch.Tensor, gathered: torch.Tensor, teacher_logp: torch.Tensor,
                   behav_logp: torch.Tensor, *, mask=None, quantile: float = 0.99,
                   clip_eps: float = 0.2, group_sizes=(), seq_len: int = 0, want=None,
                   stream=None) -> dict:
    """Diagnostics of the MC estimator from an MC loss call's lse_out and
    gathered_out and the cache's teacher and behaviour log-probs (see
    opd_mc_diagnostics).  Returns the requested outputs as device tensors."""
    if not isinstance(gathered, torch.Tensor) or gathered.dim() != 2:
        raise ValueError("gathered must be a contiguous [N, M] float32 tensor")
    N, M = gathered.shape
    dev = gathered.device
    _need(lse, "lse", (torch.float32,), (N,), dev)
    for t, name in ((gathered, "gathered"), (teacher_logp, "teacher_logp"),
                    (behav_logp, "behav_logp")):
        _need(t, name, (torch.float32,), (N, M), dev)
    if mask is not None:
        _need(mask, "mask", _MASK_DTYPES, (N,), dev)
    _need_gpu(gathered, "gathered")
    if want is None:
        want = DIAG_OUTPUTS if seq_len and len(group_sizes) else DIAG_OUTPUTS[:-1]
    gs = (ctypes.c_int32 * max(len(group_sizes), 1))(*group_sizes)
    dev = gathered.device
    sizes = {"row_mean": N, "row_var": N, "row_rho_max": N, "rho_quantile": 1, "clip_frac": 1,
             "ratio_local": max(len(group_sizes), 1), "ratio_seq": max(len(group_sizes), 1)}
    out = {k: torch.empty(sizes[k], dtype=torch.float32, device=dev) for k in want}
    st = OpdMcDiag(*[_ptr(out.get(k)) for k in DIAG_OUTPUTS])
    nbytes = int(lib().opd_mc_diag_workspace_bytes(N, M, gs, len(group_sizes), seq_len))
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    rc = lib().opd_mc_diagnostics(_ptr(lse), _ptr(gathered), _ptr(teacher_logp), _ptr(behav_logp),
                                  N, M, _ptr(mask), quantile, clip_eps, gs, len(group_sizes),
                                  seq_len, ctypes.byref(st), _ptr(ws), nbytes, _stream(stream))
    if rc != 0:
        raise OpdError(rc, "opd_mc_diagnostics")
    for k in ("ratio_local", "ratio_seq"):
        if k in out:
            out[k] = out[k][:len(group_sizes)]
    return out
