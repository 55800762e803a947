"""Benchmark of the learner-time OPD loss forward+backward on one MI355X.

A step is one fused forward+backward call over a batch of N token rows
(student log-softmax over V, gather at the cached support, estimator,
gradient write).  The default workload is 16-sample Monte-Carlo reverse KL
over N = 32,768 tokens of a V = 151,936 vocabulary with bf16 logits and fp32
gradients.  Inputs are synthetic (seeded generator), resident in HBM before
the timed region.

Prints one JSON line on stdout:
  value       tokens per second over the timed steps (valid tokens)
  roofline    HBM roofline of the loss kernel: algorithmic bytes per launch
              (one read of the logits, one write of the gradient, the cache)
              over the mean launch time measured with HIP events on the
              launch stream, against the 8 TB/s MI355X peak; also the same
              rate as a fraction of a plain device copy measured in the same
              process (frac_of_copy), and a plain read's rate (read_GBps, from
              bench_probe.so; for the cache-building calls also frac_of_read)
  accounting_model  the launch priced with a second read of each row for the
              estimators whose gradient is dense (MC, truncated top-k,
              dense), as a two-read/one-write accounting counts it.  The
              kernels hold the row on chip and do not move those bytes, so
              this is bookkeeping, not a bandwidth figure
  cpu_baseline  the oracle on a bounded sample of the same workload, on the
              host cores, plus a one-thread figure on 1,024 rows
Working sets under 1 GiB (which the 256 MB Infinity Cache could partly hold
between steps) are rotated over several copies of the inputs and outputs, so
consecutive steps read and write different memory; config.buffer_sets says how
many.

The loss calls are prepared once per buffer set (the binding's checks and
marshalling; prepare_loss_fwd_bwd), so a timed step costs the host one
foreign call.  --graph captures each call in a HIP graph and times the
replays instead (config.launch says which was timed).

--op sample|topk|score times one of the cache-building calls instead (Stage
1 draws with their log-probs, the top-k support, or scoring at cached ids)
on the same kind of rows; each reads every valid row once.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
_CSRC = os.path.join(ROOT, "paper_2606_24143_amd", "csrc")
_COMMON_SOURCES = ("opd_api.cpp", "opd_internal.h", "opd_device.h")
# the sources each op's kernels are built from
KERNEL_SOURCES = {"loss": ("opd_kernels.hip",) + _COMMON_SOURCES,
                  "sample": ("opd_cache_kernels.hip",) + _COMMON_SOURCES,
                  "topk": ("opd_cache_kernels.hip",) + _COMMON_SOURCES,
                  "score": ("opd_cache_kernels.hip",) + _COMMON_SOURCES,
                  "diag": ("opd_diag_kernels.hip",) + _COMMON_SOURCES}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# estimators that read the top-k cache (renormalised and truncated)
SUPPORT = ("fkl_topk", "rkl_topk", "fkl_topk_trunc", "rkl_topk_trunc")


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def kernel_hash(op: str = "loss") -> str:
    """Hash of the sources the op's kernels are built from."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[op]:
        with open(os.path.join(_CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(w, est: str, n_valid: int, n_masked: int) -> int:
    """Bytes the method must move per launch: each valid row's logits read
    once, every gradient row written once (masked rows are written as zeros),
    the cache entries read once, and the per-token loss written."""
    in_b = 2 if w.dtype == 1 else 4
    out_b = 4
    V = w.V
    K = w.k if est in SUPPORT else (1 if est == "rkl_mc1" else w.M)
    # the MC family reads ids and teacher log-probs, and behaviour log-probs
    # except the no-IS ablation
    if est in ("fkl_topk", "rkl_topk"):
        row_read = K * in_b                 # only the cached logits are needed
        cache = K * (4 + 4)
    elif est in SUPPORT:                    # truncated top-k: dense gradient, row read
        row_read = V * in_b
        cache = K * (4 + 4)
    elif est in ("fkl_dense", "rkl_dense"):
        row_read = 2 * V * in_b             # student and teacher rows
        cache = 0
    else:
        row_read = V * in_b
        cache = K * (4 + 4 + (0 if est == "rkl_mc_nois" else 4))
    return n_valid * (row_read + cache) + (n_valid + n_masked) * (V * out_b + 4)


def second_read_bytes(w, est: str, n_valid: int) -> int:
    """Extra bytes of the two-read accounting model: estimators whose dense
    gradient depends on every logit (MC, truncated top-k, dense) are charged
    a second read of each valid row (both rows for the dense estimators), as
    a kernel that does not hold the row on chip would move.  The renormalised
    top-k estimators read only the cached entries and are charged nothing."""
    in_b = 2 if w.dtype == 1 else 4
    if est in ("fkl_topk", "rkl_topk"):
        return 0
    rows = 2 if est in ("fkl_dense", "rkl_dense") else 1
    return n_valid * rows * w.V * in_b


def cache_op_bytes(w, op: str, n_valid: int, K: int) -> int:
    """Bytes a cache-building call must move: each valid row read once, plus
    its per-token inputs and outputs (uniforms in, ids and log-probs out for
    sampling; ids and log-probs out for top-k; ids in and log-probs out for
    scoring)."""
    in_b = 2 if w.dtype == 1 else 4
    if op == "diag":
        # reads lse, gathered logits, tau and beta; writes three per-token values
        return n_valid * (4 + K * 12 + 12)
    per_tok = {"sample": K * (4 + 4 + 4), "topk": K * (4 + 4), "score": K * (4 + 4)}[op]
    return n_valid * (w.V * in_b + per_tok)


def cpu_cache_baseline(w, op, d, u, rows: int, threads: int):
    """The oracle's cache-building function over the first `rows` rows."""
    import oracle

    n = min(rows, w.N) if rows > 0 else w.N
    dt = oracle.BF16 if w.dtype == 1 else oracle.F32
    K = w.k if op == "topk" else w.M
    t0 = time.perf_counter()
    oracle.cache_rows(op, dt, d["logits"][:n], w.V, K, uniforms=None if u is None else u[:n],
                      ids=d["mc_ids"][:n] if op == "score" else None, mask=d["mask"][:n],
                      nthreads=threads)
    el = time.perf_counter() - t0
    used = threads if threads > 0 else oracle.max_threads()
    return {"value": n / el, "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": "first %d of the %d token rows of the timed workload, fp64 oracle %s, "
                      "%.1f s wall on %d threads" % (n, w.N, op, el, used)}


def cpu_diag_baseline(w, d, lse, gathered, seq):
    """The oracle's MC diagnostics over the whole batch (single-threaded)."""
    import oracle

    t0 = time.perf_counter()
    oracle.mc_diagnostics(lse, gathered, d["mc_tau"], d["mc_beta"], mask=d["mask"],
                          group_sizes=(2, 4, 8), seq_len=seq)
    el = time.perf_counter() - t0
    return {"value": w.N / el, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": "all %d token rows of the timed workload, fp64 oracle diagnostics, "
                      "%.2f s wall on 1 thread" % (w.N, el)}


FUSED_TOPK_MAX_BYTES = 128 << 20  # fp32 gradient bytes below which top-k takes one launch


def dominant_kernels(op: str, est: str, w, split: bool):
    """Names of the kernels a launch runs (as rocprofv3 lists them)."""
    if op == "loss":
        if split:
            return ["k_split_stats", "k_split_write"]
        if est in ("fkl_topk", "rkl_topk"):
            # (the library writes gradients of at most 128 MiB in one launch)
            if w.N * ((w.V + 3) // 4) * 16 <= FUSED_TOPK_MAX_BYTES:
                return ["k_topk_fused"]
            return ["k_fill_zero", "k_topk_sparse"]
        if est in ("fkl_dense", "rkl_dense"):
            return ["k_row_dense_resident"]
        return ["k_row_resident"]
    return {"sample": ["k_sample"], "topk": ["k_topk_stream", "k_topk"],
            "score": ["k_score"], "diag": ["k_diag_*"]}[op]


def read_traffic(est_key: str, op: str):
    """Measured HBM bytes per launch from the committed counter summary, if it
    was taken on the current sources of the op's kernels."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    e = t.get("workloads", {}).get(est_key)
    if e is None or e.get("kernel_hash") != kernel_hash(op):
        return None
    return e.get("bytes_per_launch")


def single_thread_baseline(w, est, d, rows: int = 1024):
    """The oracle on one thread over the first `rows` rows."""
    r = cpu_baseline(w, est, d, rows, 1)
    return {"value": r["value"], "unit": "tokens/s", "rows": min(rows, w.N), "threads": 1}


def copy_peak(dev, stream, mib: int = 2048):
    """GB/s (bytes read + written) of plain device copies of `mib` MiB of
    output: fp32 to fp32 (the runtime's copy) and bf16 to fp32 (torch's
    elementwise conversion, the loss kernels' own 2 + 4 bytes per element).
    Returns {pattern: GB/s}."""
    import torch

    n = mib * (1 << 20) // 4
    out = torch.empty(n, dtype=torch.float32, device=dev)
    res = {}
    for name, src in (("f32_to_f32", torch.ones(n, dtype=torch.float32, device=dev)),
                      ("bf16_to_f32", torch.ones(n, dtype=torch.bfloat16, device=dev))):
        for _ in range(3):
            out.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(10):
            out.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        res[name] = (src.element_size() + 4) * n * 10 / (e0.elapsed_time(e1) / 1e3) / 1e9
        del src
    del out
    torch.cuda.empty_cache()
    return res


def read_peak(dev, stream, mib: int = 2048):
    """GB/s of one plain read of `mib` MiB by bench_probe.so (8,192
    workgroups of 256 lanes, each streaming its own share with non-temporal
    16-byte loads); None when the probe is not built."""
    import ctypes

    import torch

    path = os.path.join(ROOT, "bench_probe.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.bench_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                                     ctypes.c_int, ctypes.c_void_p]
    lib.bench_read_probe.restype = ctypes.c_int
    nbytes, groups = mib << 20, 8192
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    out = torch.empty(groups, dtype=torch.int32, device=dev)

    def once():
        rc = lib.bench_read_probe(ctypes.c_void_p(buf.data_ptr()), nbytes,
                                  ctypes.c_void_p(out.data_ptr()), groups,
                                  ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError("bench_read_probe failed: hipError_t %d" % rc)

    for _ in range(3):
        once()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        once()
    e1.record(stream)
    torch.cuda.synchronize()
    gbs = nbytes * 10 / (e0.elapsed_time(e1) / 1e3) / 1e9
    del buf, out
    torch.cuda.empty_cache()
    return gbs


def cpu_baseline(w, est, d, rows: int, threads: int, chunk: int = 512):
    """The oracle as it stands, over the first `rows` token rows of the timed
    workload, in chunks (so its fp64 gradient buffer stays small); only the
    oracle calls are timed."""
    import numpy as np

    import oracle

    n = min(rows, w.N) if rows > 0 else w.N
    dt = 0.0
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        ids = tau = beta = None
        if est in SUPPORT:
            ids, tau = d["topk_idx"][r0:r1], d["topk_tau"][r0:r1]
        elif est.startswith("rkl_mc"):
            m = 1 if est == "rkl_mc1" else w.M
            ids = np.ascontiguousarray(d["mc_ids"][r0:r1, :m])
            tau = np.ascontiguousarray(d["mc_tau"][r0:r1, :m])
            beta = np.ascontiguousarray(d["mc_beta"][r0:r1, :m])
        teacher = d["teacher_logits"][r0:r1] if "teacher_logits" in d else None
        t0 = time.perf_counter()
        oracle.rows(est, oracle.BF16 if w.dtype == 1 else oracle.F32, d["logits"][r0:r1], w.V,
                    ids=ids, tau=tau, beta=beta, teacher_logits=teacher, mask=d["mask"][r0:r1],
                    nthreads=threads)
        dt += time.perf_counter() - t0
    used = threads if threads > 0 else oracle.max_threads()
    return {"value": n / dt, "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": "first %d of the %d token rows of the timed workload, fp64 oracle "
                      "forward+backward, %.1f s wall on %d threads" % (n, w.N, dt, used)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="n32768_v151936_bf16_mc16")
    ap.add_argument("--estimator", default=None)
    ap.add_argument("--op", default="loss", choices=("loss", "sample", "topk", "score", "diag"),
                    help="time the loss (default), one cache-building call, or the MC "
                         "diagnostics")
    ap.add_argument("--cpu-rows", type=int, default=0, help="0 = every row")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=2048,
                    help="size of the plain device copy timed for frac_of_copy (0: skip)")
    ap.add_argument("--rows", type=int, default=0,
                    help="time only the first ROWS rows of the workload (0 = all)")
    ap.add_argument("--path", default="auto", choices=("auto", "rowwise", "split"),
                    help="force the loss call's path (the split path gets its workspace)")
    ap.add_argument("--graph", action="store_true",
                    help="capture each call in a HIP graph and time its replays (no host "
                         "launch overhead in the timed steps)")
    ap.add_argument("--min-set-gib", type=float, default=1.0,
                    help="rotate input/output copies until the timed steps span this many GiB")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (rows are independent; "
              "each GPU would run the same kernel on its own share of rows). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_24143_amd as opd
    import synth

    opd.lib()  # fails loudly when the HIP library is not built
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    w = synth.WORKLOADS[args.workload]
    if args.rows:
        # rows are generated independently from the seed: the first ROWS rows
        w = w.replace(N=min(args.rows, w.N))
    path_flags = {"auto": 0, "rowwise": opd.FLAG_FORCE_ROWWISE, "split": opd.FLAG_FORCE_SPLITV}[
        args.path]
    est = args.estimator or w.estimators[0]
    op = args.op
    if op == "topk" and w.k == 0 or op in ("sample", "score", "diag") and w.M == 0:
        print("--op %s needs a workload with %s" % (op, "k > 0" if op == "topk" else "M > 0"),
              file=sys.stderr)
        sys.exit(2)

    log("generating %s ..." % w.name)
    t0 = time.perf_counter()
    d = synth.generate(w)
    log("generated in %.1f s" % (time.perf_counter() - t0))

    def dev_t(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    mask_np = d["mask"]
    mask = dev_t(mask_np) if w.ragged else None
    n_valid = int(mask_np.sum())
    N = w.N
    in_b = 2 if w.dtype == 1 else 4
    stream = torch.cuda.current_stream()
    copies = copy_peak(dev, stream, args.copy_mib) if args.copy_mib else None
    copy_gbs = max(copies.values()) if copies else None
    read_gbs = read_peak(dev, stream, args.copy_mib) if args.copy_mib else None

    def loss_inputs():
        kw = {}
        if est in SUPPORT:
            kw = dict(idx=dev_t(d["topk_idx"]), teacher_logp=dev_t(d["topk_tau"]))
        elif est.startswith("rkl_mc"):
            m = 1 if est == "rkl_mc1" else w.M
            kw = dict(sampled_ids=dev_t(d["mc_ids"][:, :m]),
                      teacher_logp=dev_t(d["mc_tau"][:, :m]),
                      behav_logp=dev_t(d["mc_beta"][:, :m]))
        else:
            kw = dict(teacher_logits=dev_t(d["teacher_logits"]))
        return kw

    logits = dev_t(d["logits"])
    kw = loss_inputs()
    u_np = None
    sets = 1
    if op == "loss":
        # one buffer set: logits (and teacher logits), cache, loss and gradient
        set_bytes = N * w.V * (in_b * (2 if "teacher_logits" in kw else 1) + 4)
        sets = max(1, -(-int(args.min_set_gib * (1 << 30)) // set_bytes))
        bufs = []
        for i in range(sets):
            bufs.append({"logits": logits if i == 0 else logits.clone(),
                         "kw": kw if i == 0 else {k: v.clone() for k, v in kw.items()},
                         "out": {"loss": torch.empty(N, dtype=torch.float32, device=dev),
                                 "dlogits": torch.empty((N, w.V), dtype=torch.float32,
                                                        device=dev)}})
        nbytes = opd.workspace_bytes(N, w.V, w.dtype, est, w.k, w.M, path_flags)
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev) if nbytes else None
        counter = [0]
        # each buffer set's call is checked and marshalled once per stream
        # (a prepared call); a step then costs the host one foreign call
        prepared = {}

        def prepare(i, s):
            b = bufs[i]
            return opd.prepare_loss_fwd_bwd(b["logits"], est, mask=mask, out=b["out"],
                                            workspace=ws, stream=s, flags=path_flags, **b["kw"])

        for i in range(sets):
            prepared[(i, stream.cuda_stream)] = prepare(i, stream)

        def step(s=stream):
            i = counter[0] % sets
            counter[0] += 1
            call = prepared.get((i, s.cuda_stream))
            if call is None:
                call = prepared[(i, s.cuda_stream)] = prepare(i, s)
            call()
    else:
        if op == "sample":
            u_np = np.stack([synth.uniforms(w.seed + 1, synth.STREAM_SAMPLE, r, w.M)
                             for r in range(N)])
            u_np = (np.floor(u_np * 2.0 ** 24) / 2.0 ** 24).astype(np.float32)
            u_dev = dev_t(u_np)

            def step(s=stream):
                opd.sample_actions(logits, u_dev, mask=mask, stream=s)
        elif op == "topk":
            def step(s=stream):
                opd.topk_support(logits, w.k, mask=mask, stream=s)
        elif op == "diag":
            # the inputs are what an MC loss call returns (lse_out, gathered_out)
            aux = opd.loss_fwd_bwd(logits, est, mask=mask, want_lse=True, want_gathered=True, **kw)
            lse_dev, gat_dev = aux["lse"], aux["gathered"].contiguous()
            del aux
            tau_dev, beta_dev = kw["teacher_logp"], kw["behav_logp"]
            seq = w.rollout_len if w.ragged else 2048

            def step(s=stream):
                opd.mc_diagnostics(lse_dev, gat_dev, tau_dev, beta_dev, mask=mask,
                                   group_sizes=(2, 4, 8), seq_len=seq, stream=s)
        else:
            ids_dev = dev_t(d["mc_ids"])

            def step(s=stream):
                opd.score_actions(logits, ids_dev, mask=mask, stream=s)
        nbytes = 0

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.graph and op == "diag":
        print("--graph covers the loss and cache-building calls", file=sys.stderr)
        sys.exit(2)
    if args.graph:
        # one HIP graph per buffer set, each holding one call; the timed steps
        # replay them in turn on the launch stream
        graphs = []
        for _ in range(sets):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(torch.cuda.current_stream())
            graphs.append(g)
        torch.cuda.synchronize()
        turn = [0]

        def step(s=stream):
            graphs[turn[0] % len(graphs)].replay()
            turn[0] += 1

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    mean_launch_s = sum(launch_ms) / len(launch_ms) / 1e3
    ms_per_step = wall / args.steps * 1e3

    if op == "loss":
        alg = algorithmic_bytes(w, est, n_valid, N - n_valid)
        key = w.name + "/" + est
        metric = "OPD loss fwd+bwd tokens/sec at V=151,936 bf16; achieved HBM GB/s vs peak"
    else:
        K = w.k if op == "topk" else w.M
        alg = cache_op_bytes(w, op, n_valid, K)
        key = w.name + "/" + op
        metric = ("OPD MC diagnostics tokens/sec; achieved HBM GB/s vs peak" if op == "diag" else
                  "OPD cache build (%s) tokens/sec at V=151,936 bf16; achieved HBM GB/s vs peak" % op)
    achieved = alg / mean_launch_s / 1e9
    traffic = read_traffic(key, op)
    res = {
        "metric": metric,
        "value": n_valid / (ms_per_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "op": op, "estimator": est if op == "loss" else None,
                   "tokens": N, "valid_tokens": n_valid,
                   "vocab": w.V, "logits_dtype": "bf16" if w.dtype == 1 else "f32",
                   "dlogits_dtype": "f32", "k": w.k, "M": w.M,
                   "path": "split" if nbytes and op == "loss" else "rowwise",
                   "first_rows_of": synth.WORKLOADS[args.workload].N if args.rows else None,
                   "buffer_sets": sets, "launch": ("hip_graph" if args.graph else
                                                      "eager, prepared" if op == "loss" else "eager")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS,
                     "traffic": traffic,
                     "algorithmic_bytes_per_launch": alg,
                     "mean_launch_ms": mean_launch_s * 1e3,
                     "min_launch_ms": min(launch_ms)},
    }
    res["roofline"]["median_launch_ms"] = sorted(launch_ms)[len(launch_ms) // 2]
    res["roofline"]["kernels"] = dominant_kernels(op, est, w, nbytes > 0)
    if copy_gbs:
        res["roofline"]["copy_GBps"] = copy_gbs
        res["roofline"]["copy_patterns_GBps"] = copies
        res["roofline"]["frac_of_copy"] = achieved / copy_gbs
    if read_gbs:
        res["roofline"]["read_GBps"] = read_gbs
        if op != "loss":  # the cache-building calls read each row once and write little
            res["roofline"]["frac_of_read"] = achieved / read_gbs
    if op == "loss":
        model = alg + second_read_bytes(w, est, n_valid)
        res["accounting_model"] = {
            "bytes_per_launch": model, "GBps": model / mean_launch_s / 1e9,
            "frac": model / mean_launch_s / 1e9 / PEAK_HBM_GBS,
            "note": "prices a second read of each row that the kernel does not perform "
                    "(the row is held in registers); bookkeeping, not achieved bandwidth"}
    if not args.no_cpu_baseline:
        del logits
        torch.cuda.empty_cache()
        log("timing the oracle ...")
        if op == "loss":
            res["cpu_baseline"] = cpu_baseline(w, est, d, args.cpu_rows, args.cpu_threads)
            res["cpu_baseline"]["single_thread"] = single_thread_baseline(w, est, d)
        elif op == "diag":
            res["cpu_baseline"] = cpu_diag_baseline(w, d, lse_dev.cpu().numpy(),
                                                    gat_dev.cpu().numpy(), seq)
        else:
            res["cpu_baseline"] = cpu_cache_baseline(w, op, d, u_np, args.cpu_rows,
                                                     args.cpu_threads)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
