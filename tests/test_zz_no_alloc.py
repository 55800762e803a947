"""opd_loss_fwd_bwd_noalloc: the loss entry point that allocates nothing.

Through the C ABI it must return, bitwise, what opd_loss_fwd_bwd returns for
the same arguments (the same kernels; only the split path's workspace moves
to the library's static scratch array), on consecutive calls that reuse the
scratch, the second with a smaller input; and it must refuse, before touching
the device, a forced split call that needs more scratch than the array holds.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2606_24143_amd as opd
import synth
from paper_2606_24143_amd._binding import OpdCache, OpdOpts

FAKE = 0x10000  # 16-byte aligned placeholder address, never dereferenced
SCRATCH = -11


def test_scratch_size_and_oversized_forced_split_is_refused_before_launch():
    L = opd.lib()
    cap = int(L.opd_noalloc_scratch_bytes())
    assert cap == 1 << 20
    V, M = 151936, 16
    # forced split: P = 1 chunk per row at this N, 8 floats per record
    N = cap // 32 + 1
    assert L.opd_workspace_bytes(N, V, 1, 3, 0, M, 4) > cap
    c = OpdCache(None, FAKE, FAKE, FAKE, None)
    rc = L.opd_loss_fwd_bwd_noalloc(FAKE, 1, N, V, V, ctypes.byref(c), 3, 0, M, None,
                                    ctypes.byref(OpdOpts(1.0, 0, 4, 0.2)), FAKE, FAKE, None, None,
                                    None, None)
    assert rc == SCRATCH
    assert opd.status_string(rc) != "unknown status"
    # argument errors come first, as for the allocating entry point
    rc = L.opd_loss_fwd_bwd_noalloc(FAKE + 2, 1, 8, V, V, ctypes.byref(c), 3, 0, M, None, None,
                                    FAKE, FAKE, None, None, None, None)
    assert rc == -5  # OPD_ERR_ALIGN
    rc = L.opd_loss_fwd_bwd_noalloc(FAKE, 1, 8, V, V, ctypes.byref(c), 3, 0, 0, None, None,
                                    FAKE, FAKE, None, None, None, None)
    assert rc == -3  # OPD_ERR_SUPPORT


def _inputs(N, V, seed):
    w = synth.Workload("noalloc", N=N, V=V, dtype=synth.BF16,
                       estimators=("rkl_mc", "fkl_topk", "fkl_dense"), k=16, M=8,
                       sigma_student=3.0, sigma_behaviour=0.5, dense_teacher=True, seed=seed)
    d = synth.generate(w)
    mask = np.ones(N, np.uint8)
    mask[2::5] = 0
    return w, d, mask


def _dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _call(d, est, mask, flags, no_alloc):
    kw = {}
    if est == "fkl_topk":
        kw = dict(idx=_dev(d["topk_idx"]), teacher_logp=_dev(d["topk_tau"]))
    elif est == "fkl_dense":
        kw = dict(teacher_logits=_dev(d["teacher_logits"]))
    else:
        kw = dict(sampled_ids=_dev(d["mc_ids"]), teacher_logp=_dev(d["mc_tau"]),
                  behav_logp=_dev(d["mc_beta"]))
    out = opd.loss_fwd_bwd(_dev(d["logits"]), est, mask=_dev(mask), flags=flags, grad_scale=0.5,
                           want_lse=True, want_gathered=est != "fkl_dense", no_alloc=no_alloc,
                           **kw)
    torch.cuda.synchronize()
    return out


# (rows of the first call, rows of the second, flags): the split path chosen
# for small N, the split path forced at a larger N, and the row-wise path
CASES = [(48, 24, 0), (700, 130, opd.FLAG_FORCE_SPLITV), (300, 200, 0)]


@pytest.mark.gpu
@pytest.mark.parametrize("est", ["rkl_mc", "fkl_topk", "fkl_dense"])
@pytest.mark.parametrize("case", CASES, ids=["split", "forced-split", "rowwise"])
def test_noalloc_matches_the_allocating_entry_point(est, case):
    n1, n2, flags = case
    V = 32000
    print("noalloc %s N=%d then N=%d flags=%d" % (est, n1, n2, flags), flush=True)
    for step, N in enumerate((n1, n2)):
        w, d, mask = _inputs(N, V, seed=11 + step)
        want = opd.workspace_bytes(N, V, w.dtype, est, 16, 8, flags)
        assert (want > 0) == (flags != 0 or N < 64)
        assert want <= opd.lib().opd_noalloc_scratch_bytes()
        a = _call(d, est, mask, flags, no_alloc=False)
        b = _call(d, est, mask, flags, no_alloc=True)
        for key in a:
            assert torch.equal(a[key], b[key]), "%s N=%d: %s differs" % (est, N, key)
        # and both against the oracle's loss (the allocating path's full parity
        # is the subject of the parity tests)
        ids, tau, beta = ((d["topk_idx"], d["topk_tau"], None) if est == "fkl_topk" else
                          (d["mc_ids"], d["mc_tau"], d["mc_beta"]) if est == "rkl_mc" else
                          (None, None, None))
        ref = oracle.rows(est, oracle.BF16, d["logits"], V, ids=ids, tau=tau, beta=beta,
                          teacher_logits=d["teacher_logits"] if est == "fkl_dense" else None,
                          mask=mask, gamma=0.5, want_grad=False)
        got = b["loss"].cpu().numpy().astype(np.float64)
        s = np.ones(N) if est != "rkl_mc" else 10.0
        assert np.all(np.abs(got - ref["loss"]) <= 2e-5 * (np.abs(ref["loss"]) + s))
