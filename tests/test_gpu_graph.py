"""The library's calls captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed: every replay must equal the eager call bit for bit.  Between
replays the test runs eager library work on other buffers and synchronizes,
so a node that kept state from the capture, or one that only the first
replay ran correctly, shows up.  The calls launch kernels only (no memset,
allocation or host synchronization inside), which is what makes them
capturable.
"""
import numpy as np
import pytest
import torch

import paper_2606_24143_amd as opd
import synth
from gpu_common import DEV, cache_arrays, say, to_dev

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _inputs(est, N, V, dtype, seed):
    w = synth.Workload("t_graph", N=N, V=V, dtype=dtype, estimators=(est,), k=16, M=8,
                       sigma_student=2.0, sigma_behaviour=0.4, seed=seed)
    d = synth.generate(w)
    ids, tau, beta = cache_arrays(d, est)
    cache = {}
    if ids is not None:
        key = "idx" if est.startswith(("fkl_topk", "rkl_topk")) else "sampled_ids"
        cache = {key: to_dev(ids), "teacher_logp": to_dev(tau)}
        if beta is not None:
            cache["behav_logp"] = to_dev(beta)
    return to_dev(d["logits"]), cache


def _replays_match(name, capture_call, eager_call, outputs, other_work):
    eager_call()
    torch.cuda.synchronize()
    want = [t.clone() for t in outputs]
    for t in outputs:
        t.fill_(float("nan")) if t.is_floating_point() else t.fill_(-7)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        capture_call()  # warm-up on the capture stream, outside the graph
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        capture_call()
    for r in range(REPLAYS):
        for t in outputs:
            t.fill_(float("nan")) if t.is_floating_point() else t.fill_(-7)
        other_work()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outputs, want)):
            assert torch.equal(a, b), "%s: replay %d, output %d differs from the eager call" % (
                name, r, i)
    say("%s: %d replays equal the eager call" % (name, REPLAYS))


@pytest.mark.parametrize("est,flags,want_lse", [
    ("rkl_mc", opd.FLAG_FORCE_ROWWISE, True),     # register-resident row kernel
    ("rkl_mc", opd.FLAG_FORCE_SPLITV, True),      # split path, workspace allocated before
    ("fkl_topk", 0, False),                       # zero fill + sparse writer
    ("rkl_topk_trunc", opd.FLAG_FORCE_ROWWISE, True),
])
def test_loss_call_in_a_graph(est, flags, want_lse):
    N, V = 64, 32768
    logits, cache = _inputs(est, N, V, synth.BF16, 11)
    other_logits, other_cache = _inputs(est, N, V, synth.BF16, 12)
    out = {"loss": torch.empty(N, device=DEV), "dlogits": torch.empty(N, V, device=DEV)}
    ws = None
    if flags == opd.FLAG_FORCE_SPLITV:
        nb = opd.workspace_bytes(N, V, synth.BF16, est, 0, 8, flags)
        ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=DEV)
    lse = {}

    def call(lg=logits, c=cache, o=out):
        r = opd.loss_fwd_bwd(lg, est, flags=flags, want_lse=want_lse, out=o, workspace=ws, **c)
        if want_lse:
            lse.setdefault("t", r["lse"])
            lse["t"].copy_(r["lse"])

    other_out = {"loss": torch.empty(N, device=DEV), "dlogits": torch.empty(N, V, device=DEV)}
    call()
    torch.cuda.synchronize()
    outputs = [out["loss"], out["dlogits"]] + ([lse["t"]] if want_lse else [])
    _replays_match("loss %s flags %d" % (est, flags), call, call, outputs,
                   lambda: opd.loss_fwd_bwd(other_logits, est, flags=flags, out=other_out,
                                            workspace=ws, **other_cache))


def test_noalloc_call_in_a_graph():
    """The entry point that allocates nothing, on the split path it serves."""
    N, V = 16, 32768
    logits, cache = _inputs("rkl_mc", N, V, synth.BF16, 21)
    out = {"loss": torch.empty(N, device=DEV), "dlogits": torch.empty(N, V, device=DEV)}

    def call():
        opd.loss_fwd_bwd(logits, "rkl_mc", flags=opd.FLAG_FORCE_SPLITV, out=out, no_alloc=True,
                         **cache)

    other_logits, other_cache = _inputs("rkl_mc", N, V, synth.BF16, 22)
    other_out = {"loss": torch.empty(N, device=DEV), "dlogits": torch.empty(N, V, device=DEV)}
    _replays_match("noalloc split", call, call, [out["loss"], out["dlogits"]],
                   lambda: opd.loss_fwd_bwd(other_logits, "rkl_mc", flags=opd.FLAG_FORCE_SPLITV,
                                            out=other_out, no_alloc=True, **other_cache))


@pytest.mark.parametrize("op", ["sample", "topk", "score"])
def test_cache_calls_in_a_graph(op):
    N, V, M = 32, 151936, 16
    logits, _ = _inputs("rkl_mc", N, V, synth.BF16, 31)
    other_logits, _ = _inputs("rkl_mc", N, V, synth.BF16, 32)
    rng = np.random.default_rng(5)
    u = to_dev((np.floor(rng.random((N, M)) * 2.0 ** 24) / 2.0 ** 24).astype(np.float32))
    ids = to_dev(rng.integers(0, V, (N, M)).astype(np.int32))
    res = {}

    def call(lg=logits, keep=True):
        if op == "sample":
            r = opd.sample_actions(lg, u, want_lse=True)
        elif op == "topk":
            r = opd.topk_support(lg, 32, want_logp=True, want_lse=True)
        else:
            r = opd.score_actions(lg, ids, want_lse=True)
        if keep:
            for k, v in r.items():
                res.setdefault(k, torch.empty_like(v))
                res[k].copy_(v)

    call()
    torch.cuda.synchronize()
    _replays_match("%s" % op, call, call, list(res.values()),
                   lambda: call(other_logits, keep=False))
